// Routing-table construction (Section 3.2, Eq. 11-14): per-id scores from a
// routing corpus and the table of the calibrated threshold.
//
// Per-id sums of a corpus split, in two launches without global atomics:
//   route_part_kernel<DAMAGE>
//       a chunk of kRouteChunk occurrences per workgroup: the excess damage
//       d = max(0, l_sparse - l_base) (Eq. 11) of each, in float32, as an
//       integer number of 2^-32 units (rounded half to even); the chunk's
//       occurrences are gathered per id in an LDS hash table (open
//       addressing, twice as many slots as occurrences, so every probe
//       sequence ends) and written out as one (id, count, sum) entry per
//       distinct id, grouped by id range (2^rbits ids a range, at most
//       kRouteRanges ranges), with the start of each range's entries.
//       DAMAGE false: counts only (the held-out split).
//   route_merge_kernel<DAMAGE>
//       workgroup (r, p) adds the entries of range r of the chunks of group p
//       into an LDS table of the range's ids and writes it to totals part p
//       (every id of the range, zeros included).  Integer sums are exact in
//       any order, so neither the order of a chunk's entries nor the split
//       into groups changes a total.
//   route_accum_kernel<DAMAGE>
//       vocabularies past kRoutePartMaxVocab: the chunk's LDS table adds
//       each id's sum and count into totals copy w % kRouteCopies with one
//       global integer atomic each.
//   route_score_kernel
//       the parts added (integers), s(x) = 2^-32 (double(S_x) / double(C_x))
//       (the empirical mean of Eq. 12), +inf for ids without occurrences;
//       the held-out counts' parts likewise; and F, the held-out
//       occurrences whose id has a finite score.
//   route_select_pass_kernel, route_select_final_kernel
//       Eq. 14 on the device: T, the least count c <= F with c / n_heldout
//       >= r_tar; the T-th smallest held-out occurrence score o by a radix
//       select on the bits of the scores (eight passes of 8 bits, each a
//       histogram weighted by the held-out counts; the first is made by the
//       score launch, and each launch takes the bits chosen so far from the
//       previous one and the previous histogram); then the smallest score
//       above o and the counts at or below and below o, and the last
//       workgroup picks of o and that next score the one whose R is nearer
//       r_tar, o on ties.
//   route_table_kernel
//       table[x] = 0 (sparse path) if s(x) < tau, else 1 (Eq. 13).
#pragma once

#include "kernels.hpp"

namespace sats {

constexpr int kRouteThreads = 1024;
constexpr int kRouteChunk = 4096;  // occurrences per workgroup (4 per thread)
constexpr uint32_t kRouteNoId = 0xffffffffu;
constexpr int kRouteCopies = 32;  // copies of the per-id totals (atomic form)
constexpr int kRouteRanges = kRouteThreads;  // id ranges of the partitioned form (one per thread in a scan)
constexpr int kRouteMaxRangeBits = 12;       // ids per range at most 4096 (the merge's LDS table)
constexpr int64_t kRoutePartMaxVocab = (int64_t)kRouteRanges << kRouteMaxRangeBits;
constexpr int kRouteParts = 8;               // chunk groups of the merge: parts of the totals

struct RouteAccumArgs {
  const int32_t *ids;
  const float *lb, *ls;           // DAMAGE: per-occurrence losses of the base and sparse paths
  int64_t n;
  int vocab;
  unsigned long long *sum;        // [kRouteCopies][vocab] sums of d in 2^-32 units (DAMAGE)
  unsigned *count;                // [kRouteCopies][vocab]
  unsigned *err;                  // 1: an id out of [0, vocab); 2: a loss difference NaN or >= 2^31 (skipped);
                                  // 3: the chunk's table had no free slot (cannot happen: twice the slots)
};

constexpr int kRouteSlots = 2 * kRouteChunk;
static_assert(kRouteSlots == 1 << 13, "the slot hash takes the top 13 bits");

// The chunk's occurrences [base, base + kRouteChunk) gathered per id into
// the LDS table skey / scnt / ssum (every slot initialised here); ends with
// a barrier.
template <bool DAMAGE>
__device__ __forceinline__ void route_chunk_table(const int32_t *ids, const float *lb, const float *ls, int64_t n,
                                                  int vocab, unsigned *err, int64_t base, uint32_t *skey,
                                                  uint32_t *scnt, unsigned long long *ssum) {
  const int tid = threadIdx.x;
  constexpr int PER = kRouteChunk / kRouteThreads, SPER = kRouteSlots / kRouteThreads;
  uint32_t k[PER];
  unsigned long long q[PER];
  // the chunk's loads first, then the table's initialisation
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int64_t i = base + tid + m * kRouteThreads;
    k[m] = kRouteNoId;
    q[m] = 0ull;
    if (i < n) {
      const int32_t x = ids[i];
      if (x >= 0 && x < vocab) {
        k[m] = (uint32_t)x;
        if constexpr (DAMAGE) {
          const float diff = ls[i] - lb[i];  // float32, as in Eq. 11
          if (diff < 2147483648.0f) {         // also false for NaN
            // d 2^32 is exact in float32 and rintf rounds half to even: an
            // integer-valued float below 2^63, converted exactly
            q[m] = (unsigned long long)rintf(fmaxf(diff, 0.0f) * 4294967296.0f);
          } else {
            k[m] = kRouteNoId;
            __hip_atomic_store(err, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
        }
      } else {
        __hip_atomic_store(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
#pragma unroll
  for (int m = 0; m < SPER; ++m) {
    const int sl = tid + m * kRouteThreads;
    skey[sl] = kRouteNoId;
    scnt[sl] = 0u;
    if constexpr (DAMAGE) ssum[sl] = 0ull;
  }
  __syncthreads();
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    if (k[m] == kRouteNoId) continue;
    uint32_t h = (k[m] * 2654435761u) >> (32 - 13);  // multiplicative hash into 2^13 slots
    // at most kRouteChunk ids share kRouteSlots slots, so a free slot is met
    // within kRouteSlots probes; the bound only guards that argument
    int probe = 0;
    for (; probe < kRouteSlots; ++probe) {
      const uint32_t prev = atomicCAS(&skey[h], kRouteNoId, k[m]);
      if (prev == kRouteNoId || prev == k[m]) {
        atomicAdd(&scnt[h], 1u);
        if constexpr (DAMAGE) atomicAdd(&ssum[h], q[m]);
        break;
      }
      h = (h + 1) & (kRouteSlots - 1);
    }
    if (probe == kRouteSlots) __hip_atomic_store(err, 3u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
}

template <bool DAMAGE>
__global__ __launch_bounds__(kRouteThreads) void route_accum_kernel(RouteAccumArgs a) {
  __shared__ uint32_t skey[kRouteSlots];
  __shared__ uint32_t scnt[kRouteSlots];
  __shared__ unsigned long long ssum[DAMAGE ? kRouteSlots : 1];
  constexpr int SPER = kRouteSlots / kRouteThreads;
  const int tid = threadIdx.x;
  route_chunk_table<DAMAGE>(a.ids, a.lb, a.ls, a.n, a.vocab, a.err, (int64_t)blockIdx.x * kRouteChunk, skey, scnt,
                            ssum);
  const size_t cp = (size_t)(blockIdx.x % kRouteCopies) * (size_t)a.vocab;
#pragma unroll
  for (int m = 0; m < SPER; ++m) {
    const int sl = tid + m * kRouteThreads;
    const uint32_t key = skey[sl];
    if (key == kRouteNoId) continue;
    atomicAdd(&a.count[cp + key], scnt[sl]);
    if constexpr (DAMAGE) atomicAdd(&a.sum[cp + key], ssum[sl]);
  }
}

struct RoutePartArgs {
  const int32_t *ids;
  const float *lb, *ls;  // DAMAGE: per-occurrence losses of the base and sparse paths
  int64_t n;
  int vocab;
  int rbits, nr;         // 2^rbits ids a range, nr ranges (<= kRouteRanges)
  int nchunks;
  u32x4 *ent;            // [nchunks][kRouteChunk] (id, count, sum lo, sum hi), grouped by range
  uint32_t *off;         // [nr + 1][nchunks] start of range r in chunk c's entries (row nr: their number)
  unsigned *err;
};

template <bool DAMAGE>
__global__ __launch_bounds__(kRouteThreads) void route_part_kernel(RoutePartArgs a) {
  __shared__ uint32_t skey[kRouteSlots];
  __shared__ uint32_t scnt[kRouteSlots];
  __shared__ unsigned long long ssum[DAMAGE ? kRouteSlots : 1];
  __shared__ uint32_t hist[kRouteRanges];
  __shared__ uint32_t wtot[kRouteThreads / 64];
  static_assert(kRouteRanges == kRouteThreads, "one range per thread in the scan");
  constexpr int SPER = kRouteSlots / kRouteThreads;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c = blockIdx.x;
  hist[tid] = 0u;
  route_chunk_table<DAMAGE>(a.ids, a.lb, a.ls, a.n, a.vocab, a.err, (int64_t)c * kRouteChunk, skey, scnt, ssum);
#pragma unroll
  for (int m = 0; m < SPER; ++m) {
    const uint32_t key = skey[tid + m * kRouteThreads];
    if (key != kRouteNoId) atomicAdd(&hist[key >> a.rbits], 1u);
  }
  __syncthreads();
  // exclusive scan of the ranges' entry counts: within the wavefront, then
  // the wavefronts' totals
  const uint32_t hv = hist[tid];
  uint32_t incl = hv;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  if (lane == 63) wtot[wv] = incl;
  __syncthreads();
  uint32_t excl = incl - hv;
  for (int q = 0; q < wv; ++q) excl += wtot[q];
  if (tid < a.nr) a.off[(size_t)tid * a.nchunks + c] = excl;
  if (tid == kRouteThreads - 1) a.off[(size_t)a.nr * a.nchunks + c] = excl + hv;  // ranges past nr are empty
  hist[tid] = excl;  // the range's next free entry (every thread read its count above)
  __syncthreads();
  u32x4 *ce = a.ent + (size_t)c * kRouteChunk;
#pragma unroll
  for (int m = 0; m < SPER; ++m) {
    const int sl = tid + m * kRouteThreads;
    const uint32_t key = skey[sl];
    if (key == kRouteNoId) continue;
    const uint32_t pos = atomicAdd(&hist[key >> a.rbits], 1u);
    const unsigned long long sm = DAMAGE ? ssum[sl] : 0ull;
    ce[pos] = u32x4{key, scnt[sl], (uint32_t)sm, (uint32_t)(sm >> 32)};
  }
}

struct RouteMergeArgs {
  const u32x4 *ent;
  const uint32_t *off;
  int nchunks, rbits, nr, vocab, parts;
  unsigned *count;           // [parts][vocab]
  unsigned long long *sum;   // [parts][vocab] (DAMAGE)
};

template <bool DAMAGE>
__global__ __launch_bounds__(kRouteThreads) void route_merge_kernel(RouteMergeArgs a) {
  constexpr int WMAX = 1 << kRouteMaxRangeBits, U = 4;
  __shared__ uint32_t lc[WMAX];
  __shared__ unsigned long long lsum[DAMAGE ? WMAX : 1];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int r = blockIdx.x, p = blockIdx.y, W = 1 << a.rbits;
  for (int i = tid; i < W; i += kRouteThreads) {
    lc[i] = 0u;
    if constexpr (DAMAGE) lsum[i] = 0ull;
  }
  __syncthreads();
  const int c0 = (int)((int64_t)p * a.nchunks / a.parts), c1 = (int)((int64_t)(p + 1) * a.nchunks / a.parts);
  for (int c = c0 + wv; c < c1; c += kRouteThreads / 64) {
    const uint32_t b = a.off[(size_t)r * a.nchunks + c], e = a.off[(size_t)(r + 1) * a.nchunks + c];
    const u32x4 *ce = a.ent + (size_t)c * kRouteChunk;
    for (uint32_t j = b + lane; j < e; j += 64 * U) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = (j + 64 * u < e) ? ce[j + 64 * u] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (j + 64 * u >= e) continue;
        const uint32_t k = v[u][0] & (uint32_t)(W - 1);
        atomicAdd(&lc[k], v[u][1]);
        if constexpr (DAMAGE) atomicAdd(&lsum[k], (unsigned long long)v[u][2] | ((unsigned long long)v[u][3] << 32));
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < W; i += kRouteThreads) {
    const int64_t id = (int64_t)r * W + i;
    if (id < a.vocab) {
      a.count[(size_t)p * a.vocab + id] = lc[i];
      if constexpr (DAMAGE) a.sum[(size_t)p * a.vocab + id] = lsum[i];
    }
  }
}

// Device-side words of the Eq. 14 selection (zeroed before the score launch).
enum : int {
  kSelF = 0,                         // held-out occurrences with a finite score
  kSelDone = 1,                      // workgroups of the final pass finished (the last one decides)
  kSelHist = 8,                      // [8][256] weighted byte histograms of the radix passes
  kSelNext = kSelHist + 8 * 256,     // ~bits of the smallest score above o (atomic max; 0: none)
  kSelAtOrBelow = kSelNext + 1,      // held-out occurrences scoring <= o
  kSelBelow = kSelNext + 2,          // ... < o
  kSelState = kSelNext + 3,          // [9][2] bits chosen and rank left after k radix passes
  kSelT = kSelState + 18,            // T (written by the first radix launch)
  kSelWords = kSelT + 1
};

// Candidate ids of Eq. 14: held out (weight h > 0) with a finite score.
// Scores are >= 0, so their bit patterns order like the doubles.
__device__ __forceinline__ bool route_candidate(unsigned w, double s) { return w && s != __builtin_huge_val(); }

// Radix pass k's histogram: the weights of the candidates whose score bits
// match `prefix` above byte k (from the top), by their byte k.
__device__ __forceinline__ void route_hist_add(unsigned long long *lh, unsigned long long bits, unsigned w, int k,
                                               unsigned long long prefix) {
  if (k == 0 || (bits >> (64 - 8 * k)) == (prefix >> (64 - 8 * k)))
    atomicAdd(&lh[(bits >> (56 - 8 * k)) & 255ull], (unsigned long long)w);
}

// Totals of the parts, the scores (Eq. 12), the held-out totals, F, and the
// first radix pass's histogram (which does not depend on the rank).
__global__ __launch_bounds__(256) void route_score_kernel(const unsigned long long *sum, const unsigned *count,
                                                          const unsigned *hcount, int parts, int vocab,
                                                          double *score, unsigned *hcount_total,
                                                          unsigned long long *sel) {
  __shared__ unsigned long long wsum[4];
  __shared__ unsigned long long lh[256];
  const int x = blockIdx.x * 256 + threadIdx.x;
  lh[threadIdx.x] = 0ull;
  __syncthreads();
  unsigned long long f = 0ull;
  if (x < vocab) {
    unsigned long long sx = 0ull;
    unsigned c = 0u, h = 0u;
    for (int k = 0; k < parts; ++k) {
      sx += sum[(size_t)k * vocab + x];
      c += count[(size_t)k * vocab + x];
      h += hcount[(size_t)k * vocab + x];
    }
    const double sc = c ? ldexp((double)sx / (double)c, -32) : __builtin_huge_val();
    score[x] = sc;
    hcount_total[x] = h;
    if (route_candidate(h, sc)) {
      f = h;
      route_hist_add(lh, __builtin_bit_cast(unsigned long long, sc), h, 0, 0ull);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) f += __shfl_xor(f, o, 64);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = f;
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned long long t = wsum[0] + wsum[1] + wsum[2] + wsum[3];
    if (t) atomicAdd(sel + kSelF, t);
  }
  if (lh[threadIdx.x]) atomicAdd(sel + kSelHist + threadIdx.x, lh[threadIdx.x]);
}

// R(c) = c / n_heldout, and T = the least c in [0, F] with R(c) >= r_tar
// (F + 1 when there is none).
__device__ __forceinline__ double route_r(unsigned long long c, long long nh) {
  return nh ? (double)c / (double)nh : 0.0;
}
__device__ __forceinline__ unsigned long long route_target(unsigned long long F, long long nh, double r_tar) {
  unsigned long long lo = 0ull, hi = F + 1ull;
  while (lo < hi) {
    const unsigned long long mid = lo + (hi - lo) / 2ull;
    if (route_r(mid, nh) >= r_tar) hi = mid;
    else lo = mid + 1ull;
  }
  return lo;
}

struct RouteSelArgs {
  const double *score;
  const unsigned *h;       // held-out occurrences per id
  int vocab;
  long long nh;
  double r_tar;
  unsigned long long *sel; // kSelWords
  double *out;             // [2] tau*, R(tau*)
  const unsigned *err;
};

// The state after k radix passes (k >= 1) in st[0] (bits chosen) and st[1]
// (rank left), from the state after k - 1 (state 0: nothing chosen, rank T)
// and pass k - 1's histogram hb: byte b is the first bin whose running total
// reaches the rank (bin 255 at the latest), the rank less the bins before
// it.  Workgroup 0 records the state for the next launch.  Also st[2]:
// whether a radix select runs at all (0 < T <= F), st[3]: T, st[4]: F.
// Every workgroup computes the same values.
__device__ __forceinline__ void route_state(const RouteSelArgs &a, int k, unsigned long long *hb,
                                            unsigned long long *st) {
  __shared__ unsigned long long wt[4];
  const int tid = threadIdx.x, lane = tid & 63;
  if (tid < 256) hb[tid] = a.sel[kSelHist + 256 * (k - 1) + tid];
  if (tid == 0) {
    const unsigned long long F = a.sel[kSelF], T = k == 1 ? route_target(F, a.nh, a.r_tar) : a.sel[kSelT];
    if (k == 1 && blockIdx.x == 0) a.sel[kSelT] = T;
    st[2] = (T > 0ull && T <= F) ? 1ull : 0ull;
    st[3] = T;
    st[4] = F;
    st[0] = k == 1 ? 0ull : a.sel[kSelState + 2 * (k - 1)];
    st[1] = k == 1 ? T : a.sel[kSelState + 2 * (k - 1) + 1];
  }
  __syncthreads();
  // every thread takes the state before the one thread that picks the bin
  // rewrites it (after the next barrier)
  const unsigned long long pfx = st[0], rank = st[1];
  const bool on = st[2] != 0ull;
  // running totals of the 256 bins: within each wavefront, then the
  // wavefronts before
  unsigned long long cum = 0ull;
  if (tid < 256) {
    cum = hb[tid];
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const unsigned long long t = __shfl_up(cum, o, 64);
      if (lane >= o) cum += t;
    }
    if (lane == 63) wt[tid >> 6] = cum;
  }
  __syncthreads();
  if (tid < 256 && on) {
    for (int q = 0; q < (tid >> 6); ++q) cum += wt[q];
    const unsigned long long excl = cum - hb[tid];
    if (excl < rank && (cum >= rank || tid == 255)) {  // exactly one bin
      st[0] = pfx | ((unsigned long long)tid << (56 - 8 * (k - 1)));
      st[1] = rank - excl;
      if (blockIdx.x == 0) {
        a.sel[kSelState + 2 * k] = pfx | ((unsigned long long)tid << (56 - 8 * (k - 1)));
        a.sel[kSelState + 2 * k + 1] = rank - excl;
      }
    }
  }
  __syncthreads();
}

// Radix pass k (1..7): the histogram of byte k of the candidates matching
// the bytes chosen so far.
__global__ __launch_bounds__(1024) void route_select_pass_kernel(RouteSelArgs a, int k) {
  __shared__ unsigned long long lh[256], hb[256], st[5];
  const int tid = threadIdx.x;
  const int x = blockIdx.x * 1024 + tid;
  // this thread's id first: its loads overlap those of the state
  const unsigned w = x < a.vocab ? a.h[x] : 0u;
  const double s = x < a.vocab ? a.score[x] : 0.0;
  if (tid < 256) lh[tid] = 0ull;
  route_state(a, k, hb, st);
  if (!st[2]) return;  // no radix select (uniform)
  if (route_candidate(w, s)) route_hist_add(lh, __builtin_bit_cast(unsigned long long, s), w, k, st[0]);
  __syncthreads();
  if (tid < 256 && lh[tid]) atomicAdd(a.sel + kSelHist + 256 * k + tid, lh[tid]);
}

// After the eight passes, o = the T-th smallest held-out occurrence score:
// the smallest candidate score above o (every candidate when T = 0) and the
// weights at or below and below o; the last workgroup to finish then picks
// tau* and R(tau*): of o and the next score the one whose R is nearer
// r_tar (o on ties); +inf when even every candidate falls short of r_tar.
__global__ __launch_bounds__(1024) void route_select_final_kernel(RouteSelArgs a) {
  __shared__ unsigned long long lw[3], hb[256], st[5];
  __shared__ int last;
  const int tid = threadIdx.x;
  const int x = blockIdx.x * 1024 + tid;
  const unsigned w = x < a.vocab ? a.h[x] : 0u;
  const double s = x < a.vocab ? a.score[x] : 0.0;
  if (tid < 3) lw[tid] = 0ull;
  route_state(a, 8, hb, st);
  const unsigned long long F = st[4], T = st[3], o = st[0];
  const int mode = T > F ? 0 : (T == 0ull ? 1 : 2);  // 0: +inf; 1: the smallest candidate; 2: around o
  if (mode) {
    if (route_candidate(w, s)) {
      const unsigned long long bits = __builtin_bit_cast(unsigned long long, s);
      if (mode == 1 || bits > o) atomicMax(&lw[0], ~bits);
      if (mode == 2 && bits <= o) atomicAdd(&lw[1], (unsigned long long)w);
      if (mode == 2 && bits < o) atomicAdd(&lw[2], (unsigned long long)w);
    }
  }
  __syncthreads();
  if (tid == 0 && lw[0]) __hip_atomic_fetch_max(a.sel + kSelNext, lw[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (tid == 1 && lw[1]) __hip_atomic_fetch_add(a.sel + kSelAtOrBelow, lw[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (tid == 2 && lw[2]) __hip_atomic_fetch_add(a.sel + kSelBelow, lw[2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // the last workgroup to arrive sees every other one's totals
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0) {
    const unsigned long long prev = __hip_atomic_fetch_add(a.sel + kSelDone, 1ull, __ATOMIC_RELAXED,
                                                           __HIP_MEMORY_SCOPE_AGENT);
    last = prev == gridDim.x - 1ull;
  }
  __syncthreads();
  if (!last || tid != 0) return;
  const double inf = __builtin_huge_val();
  if (mode == 0) {  // every candidate falls short of r_tar: the largest, +inf
    a.out[0] = inf;
    a.out[1] = route_r(F, a.nh);
    return;
  }
  const unsigned long long nx = __hip_atomic_load(a.sel + kSelNext, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const double vstar = nx ? __builtin_bit_cast(double, ~nx) : inf;
  if (mode == 1) {  // no occurrence below: the smallest candidate
    a.out[0] = vstar;
    a.out[1] = route_r(0ull, a.nh);
    return;
  }
  const unsigned long long wle = __hip_atomic_load(a.sel + kSelAtOrBelow, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const unsigned long long wpred = __hip_atomic_load(a.sel + kSelBelow, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const unsigned long long wstar = nx ? wle : F;
  if (fabs(route_r(wpred, a.nh) - a.r_tar) <= fabs(route_r(wstar, a.nh) - a.r_tar)) {
    a.out[0] = __builtin_bit_cast(double, o);
    a.out[1] = route_r(wpred, a.nh);
  } else {
    a.out[0] = vstar;
    a.out[1] = route_r(wstar, a.nh);
  }
}

__global__ __launch_bounds__(256) void route_table_kernel(const double *score, int vocab, const double *tau,
                                                          const unsigned *err, uint8_t *table) {
  const int x = blockIdx.x * 256 + threadIdx.x;
  if (x < vocab && !*err) table[x] = score[x] < *tau ? 0 : 1;
}

// Zeroes n words (a kernel, not a memset, so that it can sit in a captured graph).
__global__ __launch_bounds__(256) void route_clear_kernel(unsigned long long *w, int n, unsigned *err) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) w[i] = 0ull;
  if (blockIdx.x == 0 && threadIdx.x == 0) *err = 0u;
}

}  // namespace sats
