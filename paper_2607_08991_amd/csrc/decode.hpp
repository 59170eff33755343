// Persistent single-token kernel: every layer of one call in one cooperative
// launch (decode batch 1).
//
// Each of the G co-resident workgroups owns a contiguous strip of the d_ff
// columns made of whole 128-byte row segments (neighbouring strips sit on the
// same XCD).
// Per layer:
//   1. layer input h in LDS: the call input for layer 0, otherwise
//      rho(y / sqrt(mean(y^2) + 1e-6)) from the previous layer's y;
//   2. gate: a = h . W_gate for the strip's columns over all d rows (no
//      cross-workgroup partials), SiLU (Eq. 2), the keep rule (Eq. 4-5, or
//      every column on the base path, Eq. 13), ballot compaction of the kept
//      columns, published with their g values;
//   3. grid barrier; the kept rows of all strips are split evenly over the
//      workgroups (a prefix over the published counts); the workgroup forms
//      u_j = W_up_T[j].h and p_j = g_j u_j (Eq. 1) for its rows, then
//      accumulates p_j W_down[j] over them, each wavefront owning a slice of
//      the columns, and writes one partial y;
//   4. grid barrier; workgroup w sums every partial for its own slice of
//      columns in workgroup order, giving y (or the rounded output on the last
//      layer) and the slice's sum of squares;
//   5. grid barrier before the next layer.
// The assignment of work depends only on the data, never on timing, so every
// sum has a fixed order and results are bitwise reproducible.  Waits are
// grid barriers of a cooperative launch, bounded so that a launch always ends.
#pragma once

#include "kernels.hpp"

namespace sats {

// Optional phase timestamps (build with -DSATS_TRACE): per workgroup, wall
// clock at fixed points of the first layer, read back with sats_trace_read().
#ifdef SATS_TRACE
__device__ unsigned long long sats_trace_buf[4096 * 8];
#define SATS_TRACE_POINT(i)                                                               \
  do {                                                                                    \
    if (threadIdx.x == 0 && blockIdx.x < 4096) sats_trace_buf[blockIdx.x * 8 + (i)] = wall_clock64(); \
  } while (0)
#else
#define SATS_TRACE_POINT(i) \
  do {                      \
  } while (0)
#endif

constexpr int kDecodeThreads = 512;
constexpr int kDecodeMaxD = 4096;        // h lives in LDS
constexpr int kStripMax = 256;           // columns one workgroup may own
constexpr int kDecodeMaxG = 1024;        // workgroups of one launch
constexpr unsigned kSpinLimit = 1u << 20;  // about a second of polling

struct DecodeArgs {
  const void *x;          // [d] call input (storage type)
  void *out;              // [d]
  const void *Wg, *Wu, *Wd;  // stacked weights
  const float *thr;       // [L] (unused on the base path)
  const int32_t *ids;
  const uint8_t *lut;
  int route_mode;
  int L, d, d_ff;
  int *kcount;            // [G]             kept columns of each strip
  int *kidx;              // [G][kStripMax]  the kept columns
  float *kg;              // [G][kStripMax]  their SiLU values
  float *ypart;           // [G][d]          per-workgroup partial y
  float *ybuf;            // [d]
  float *sspart;          // [G]
  unsigned *bar;          // [2] barrier count, generation
  unsigned *err;          // [1] set when a bounded wait gives up
  uint8_t *route_out;     // optional [1]
  uint8_t *keep_out;      // optional [L][d_ff]
  void *layer_in;         // optional [L][d]
};

__device__ __forceinline__ void store_coherent_i(int *p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int load_coherent_i(const int *p) {
  return __hip_atomic_load(const_cast<int *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Four consecutive floats (16-byte aligned) written through to the
// device-coherent level in one 16-byte store.
__device__ __forceinline__ void store_coherent4(float *p, float x0, float x1, float x2, float x3) {
  const f32x4 v = {x0, x1, x2, x3};
  asm volatile("global_store_dwordx4 %0, %1, off sc1" : : "v"(p), "v"(v) : "memory");
}

// True once a bounded wait of this launch has given up: later waits return at
// once, so a failed launch still ends quickly.
__device__ __forceinline__ bool wait_failed(unsigned *err) {
  return __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u;
}

// Barrier over all G workgroups (co-resident by the cooperative launch).
// Device-coherent stores issued before it are visible to device-coherent
// loads after it.  Two levels keep atomic contention low: workgroups count in
// at one counter per XCD (workgroup w runs on XCD w % 8), the last of each
// XCD counts in globally, and the last of those bumps the generation that
// every workgroup polls.  Counters sit 128 bytes apart.
constexpr int kBarGen = 1, kBarGroup = 32;  // word offsets: [0] global count, [1] generation

__device__ __forceinline__ bool spin_until_changed(unsigned *word, unsigned old, unsigned *err) {
  unsigned spins = 0;
  while (__hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == old) {
    __builtin_amdgcn_s_sleep(1);
    if ((++spins & 255u) == 0u && (spins > kSpinLimit || wait_failed(err))) {
      __hip_atomic_store(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return false;
    }
  }
  return true;
}

__device__ __forceinline__ void grid_barrier(unsigned *bar, unsigned G, unsigned *err) {
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned gen = __hip_atomic_load(bar + kBarGen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    const unsigned ngroups = G < 8u ? G : 8u;
    const unsigned grp = blockIdx.x % 8u;
    const unsigned gsize = (G - grp + 7u) / 8u;
    unsigned *gc = bar + kBarGroup * (1u + grp);
    bool last = false;
    if (__hip_atomic_fetch_add(gc, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == gsize - 1u) {
      __hip_atomic_store(gc, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_s_waitcnt(0);
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      if (__hip_atomic_fetch_add(bar, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == ngroups - 1u) {
        __hip_atomic_store(bar, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __builtin_amdgcn_s_waitcnt(0);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __hip_atomic_fetch_add(bar + kBarGen, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        last = true;
      }
    }
    if (!last) spin_until_changed(bar + kBarGen, gen, err);
  }
  __syncthreads();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

template <typename T>
__global__ __launch_bounds__(kDecodeThreads) void decode_kernel(DecodeArgs a) {
  constexpr int THREADS = kDecodeThreads;
  constexpr int VEC = Elem<T>::kVec;      // elements per 16-byte load
  constexpr int NW = THREADS / 64;        // wavefronts per workgroup
  constexpr int CH = 64 * VEC;            // elements per wavefront-wide 16-byte load
  constexpr int DMAX = kDecodeMaxD / CH;  // wavefront loads per row

  __shared__ float hs[kDecodeMaxD];       // layer input
  __shared__ float red[kDecodeMaxD];      // gate reduction / workgroup partial y
  __shared__ int pref[kDecodeMaxG + 1];   // prefix of the strips' kept counts
  __shared__ int mj[THREADS];             // this workgroup's kept rows ...
  __shared__ float mg[THREADS];           // ... their g values ...
  __shared__ float mp[THREADS];           // ... and p_j = g_j u_j
  __shared__ int wcnt[NW];
  __shared__ float scal[NW];

  const int G = gridDim.x, w = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d = a.d, d_ff = a.d_ff;
  const size_t wl = (size_t)d * d_ff;
  const int base = token_is_base(a.route_mode, a.ids, a.lut, 0);
  if (a.route_out && w == 0 && tid == 0) a.route_out[0] = (uint8_t)base;

  // this workgroup's strip of columns: whole 128-byte units (one cache line
  // of a W_gate row), split as evenly as possible over the 8 XCDs and then
  // over the workgroups of each XCD (workgroups are dealt to the XCDs
  // round-robin), so each XCD streams one contiguous block of every row
  constexpr int UNIT = 128 / (VEC * (int)sizeof(T));  // 16-byte vectors per unit
  const int nvec = d_ff / VEC;
  const int nunits = (nvec + UNIT - 1) / UNIT;
  int u0, nu;
  if (G % 8 == 0) {
    const int x = w % 8, ix = w / 8, per = G / 8;
    const int ux = nunits / 8 + (x < nunits % 8 ? 1 : 0);
    const int ub = x * (nunits / 8) + min(x, nunits % 8);
    nu = ux / per + (ix < ux % per ? 1 : 0);
    u0 = ub + ix * (ux / per) + min(ix, ux % per);
  } else {
    nu = nunits / G + (w < nunits % G ? 1 : 0);
    u0 = w * (nunits / G) + min(w, nunits % G);
  }
  const int v0 = u0 * UNIT;
  const int LC = max(0, min(nu * UNIT, nvec - v0));  // lanes across the strip (one vector each)
  const int c0 = v0 * VEC, ncols = LC * VEC;
  const int RG = LC > 0 ? THREADS / LC : 0;  // row groups
  const int lc = LC > 0 ? tid % LC : 0, rg = LC > 0 ? tid / LC : THREADS;

  SATS_TRACE_POINT(0);
  // gate rows of this thread: k = rg + RG * r, r < nrows, loaded GB at a time
  // (GB 16-byte loads in flight per thread; a tail batch re-reads the last
  // row and gives it weight 0)
  constexpr int GB = 32;
  const int nrows = (rg < RG) ? (d - rg + RG - 1) / RG : 0;
  const int nb = (nrows + GB - 1) / GB;
  for (int l = 0; l < a.L; ++l) {
    const T *__restrict__ Wg = static_cast<const T *>(a.Wg) + (size_t)l * wl + c0 + lc * VEC;
    // ------------------------------------------------ 1. layer input
    if (l == 0) {
      for (int k0 = tid * VEC; k0 < d; k0 += THREADS * VEC) {  // one 16-byte load per thread
        const u32x4 xv = *reinterpret_cast<const u32x4 *>(static_cast<const T *>(a.x) + k0);
#pragma unroll
        for (int v = 0; v < VEC; ++v) hs[k0 + v] = unpack<T>(xv, v);
        if (a.layer_in && w == 0) *reinterpret_cast<u32x4 *>(static_cast<T *>(a.layer_in) + k0) = xv;
      }
    } else {
      float s = 0.0f;  // total sum of squares of y, in a fixed order
      if (tid < G) s = sum_coherent(a.sspart + tid, THREADS, (G - tid + THREADS - 1) / THREADS);
      s = wave_sum(s);
      if (lane == 0) scal[wv] = s;
      __syncthreads();
      float tot = 0.0f;
      for (int i = 0; i < NW; ++i) tot += scal[i];
      const float scale = sqrtf(tot / (float)d + kGlueEps);
      for (int k0 = 0; k0 < d; k0 += THREADS * 8) {
        float yv[8];  // all loads in flight before the first use
#pragma unroll
        for (int i = 0; i < 8; ++i) yv[i] = load_coherent(a.ybuf + min(k0 + i * THREADS + tid, d - 1));
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int k = k0 + i * THREADS + tid;
          if (k < d) {
            const T hv = Elem<T>::round(yv[i] / scale);
            hs[k] = Elem<T>::value(hv);
            if (a.layer_in && w == 0) static_cast<T *>(a.layer_in)[(size_t)l * d + k] = hv;
          }
        }
      }
    }
    __syncthreads();
    if (l == 0) SATS_TRACE_POINT(1);

    // ------------------------------------------------ 2. gate over the strip
    {
      float acc[VEC];
#pragma unroll
      for (int v = 0; v < VEC; ++v) acc[v] = 0.0f;
      if (rg < RG) {  // every row group writes its partial, zero when it has no rows
        for (int b = 0; b < nb; ++b) {
          u32x4 gbuf[GB];
#pragma unroll
          for (int u = 0; u < GB; ++u)
            gbuf[u] = load_raw<T>(Wg + (size_t)(rg + min(b * GB + u, nrows - 1) * RG) * d_ff);
#pragma unroll
          for (int u = 0; u < GB; ++u) {
            const int r = b * GB + u;
            const float hv = (r < nrows) ? hs[rg + r * RG] : 0.0f;
#pragma unroll
            for (int v = 0; v < VEC; ++v) acc[v] = fmaf(hv, unpack<T>(gbuf[u], v), acc[v]);
          }
        }
#pragma unroll
        for (int v = 0; v < VEC; ++v) red[rg * ncols + lc * VEC + v] = acc[v];
      }
      __syncthreads();
      const float thr = base ? 0.0f : a.thr[l];
      bool keep = false;
      float g = 0.0f;
      if (tid < ncols) {
        float s = 0.0f;
        for (int r = 0; r < RG; ++r) s += red[r * ncols + tid];
        g = silu(s);
        keep = base || (fabsf(g) >= thr);
        if (a.keep_out) a.keep_out[(size_t)l * d_ff + c0 + tid] = (uint8_t)keep;
      }
      const uint64_t bal = __ballot(keep);
      const int rank = __popcll(bal & ((1ull << lane) - 1ull));
      if (lane == 0) wcnt[wv] = __popcll(bal);
      __syncthreads();
      int off = 0, tot = 0;
      for (int i = 0; i < NW; ++i) {
        off += (i < wv) ? wcnt[i] : 0;
        tot += wcnt[i];
      }
      if (keep) {
        store_coherent_i(a.kidx + (size_t)w * kStripMax + off + rank, c0 + tid);
        store_coherent(a.kg + (size_t)w * kStripMax + off + rank, g);
      }
      if (tid == 0) store_coherent_i(a.kcount + w, tot);
    }
    if (l == 0) SATS_TRACE_POINT(2);
    grid_barrier(a.bar, (unsigned)G, a.err);
    if (l == 0) SATS_TRACE_POINT(3);

    // ------------------------------------------------ 3. kept rows, split evenly
    // Up pass: the workgroup's kept rows are dealt to its wavefronts, four at
    // a time, for u_j = W_up_T[j] . h and p_j = g_j u_j (kept in LDS).  Down
    // pass: wavefront v owns columns chunks v, v + NW, ... of y and streams
    // its slice of every kept row of W_down, so y's partial needs no
    // cross-wavefront reduction and each lane holds only VEC accumulators per
    // chunk.
    {
      // exclusive prefix of the strips' counts, in workgroup order
      for (int g0 = 0; g0 < G; g0 += THREADS)
        if (g0 + tid < G) pref[g0 + tid + 1] = load_coherent_i(a.kcount + g0 + tid);
      if (tid == 0) pref[0] = 0;
      __syncthreads();
      if (wv == 0) {
        int carry = 0;
        for (int b0 = 1; b0 <= G; b0 += 64) {
          const int b = b0 + lane;
          int incl = (b <= G) ? pref[b] : 0;
#pragma unroll
          for (int o = 1; o < 64; o <<= 1) {
            const int u = __shfl_up(incl, o, 64);
            if (lane >= o) incl += u;
          }
          if (b <= G) pref[b] = carry + incl;
          carry += __shfl(incl, 63, 64);
        }
      }
      __syncthreads();
      const int U = pref[G];
      const int R = U / G, Rr = U - R * G;
      const int p0 = w * R + min(w, Rr);
      const int nR = R + (w < Rr ? 1 : 0);

      constexpr int NCH = (DMAX + NW - 1) / NW;  // column chunks per wavefront
      float yacc[NCH][VEC];
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int v = 0; v < VEC; ++v) yacc[c][v] = 0.0f;

      const T *__restrict__ Wu = static_cast<const T *>(a.Wu) + (size_t)l * wl;
      const T *__restrict__ Wd = static_cast<const T *>(a.Wd) + (size_t)l * wl;
      for (int m0 = 0; m0 < nR; m0 += THREADS) {
        const int mn = min(THREADS, nR - m0);
        __syncthreads();
        if (tid < mn) {  // row metadata of the chunk, all loads at once
          const int p = p0 + m0 + tid;
          int lo = 0, hi = G - 1;  // strip holding position p: largest o with pref[o] <= p
          while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (pref[mid] <= p) lo = mid; else hi = mid - 1;
          }
          const size_t e = (size_t)lo * kStripMax + (p - pref[lo]);
          mj[tid] = load_coherent_i(a.kidx + e);
          mg[tid] = load_coherent(a.kg + e);
        }
        __syncthreads();
        if (l == 0 && m0 == 0) SATS_TRACE_POINT(4);

        // up pass
        constexpr int RU = (sizeof(T) == 2) ? 4 : 2;  // rows in flight per wavefront
        for (int i0 = wv * RU; i0 < mn; i0 += NW * RU) {
          u32x4 wr[RU][DMAX];
#pragma unroll
          for (int r = 0; r < RU; ++r) {
            const int jr = __builtin_amdgcn_readfirstlane(mj[min(i0 + r, mn - 1)]);
            const T *__restrict__ ur = Wu + (size_t)jr * d;
#pragma unroll
            for (int t = 0; t < DMAX; ++t) {
              const int k = t * CH + lane * VEC;
              wr[r][t] = (k < d && i0 + r < mn) ? load_raw<T>(ur + k) : u32x4{0u, 0u, 0u, 0u};
            }
          }
          float u[RU];
#pragma unroll
          for (int r = 0; r < RU; ++r) u[r] = 0.0f;
#pragma unroll
          for (int t = 0; t < DMAX; ++t) {
            const int k = t * CH + lane * VEC;
            if (k < d) {
#pragma unroll
              for (int v = 0; v < VEC; ++v) {
                const float hv = hs[k + v];
#pragma unroll
                for (int r = 0; r < RU; ++r) u[r] = fmaf(hv, unpack<T>(wr[r][t], v), u[r]);
              }
            }
          }
#pragma unroll
          for (int r = 0; r < RU; ++r) {
            const float ur = wave_sum(u[r]);
            if (lane == 0 && i0 + r < mn) mp[i0 + r] = mg[i0 + r] * ur;
          }
        }
        __syncthreads();

        // down pass: this wavefront's column chunks of every row, RD rows in flight
        constexpr int RD = (sizeof(T) == 2) ? 32 : 16;
        for (int i0 = 0; i0 < mn; i0 += RD) {
          u32x4 wr[RD][NCH];
#pragma unroll
          for (int r = 0; r < RD; ++r) {
            const int jr = __builtin_amdgcn_readfirstlane(mj[min(i0 + r, mn - 1)]);
            const T *__restrict__ dr = Wd + (size_t)jr * d;
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
              const int k = (wv + c * NW) * CH + lane * VEC;
              wr[r][c] = (k < d && i0 + r < mn) ? load_raw<T>(dr + k) : u32x4{0u, 0u, 0u, 0u};
            }
          }
#pragma unroll
          for (int r = 0; r < RD; ++r) {
            const float pr = (i0 + r < mn) ? mp[i0 + r] : 0.0f;
#pragma unroll
            for (int c = 0; c < NCH; ++c)
#pragma unroll
              for (int v = 0; v < VEC; ++v) yacc[c][v] = fmaf(pr, unpack<T>(wr[r][c], v), yacc[c][v]);
          }
        }
      }
      if (l == 0) SATS_TRACE_POINT(5);
      // this workgroup's partial y, written by column owner
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const int k = (wv + c * NW) * CH + lane * VEC;
        if (k < d) {
#pragma unroll
          for (int v = 0; v < VEC; v += 4)
            store_coherent4(a.ypart + (size_t)w * d + k + v, yacc[c][v], yacc[c][v + 1], yacc[c][v + 2],
                            yacc[c][v + 3]);
        }
      }
    }
    grid_barrier(a.bar, (unsigned)G, a.err);
    if (l == 0) SATS_TRACE_POINT(6);

    // ------------------------------------------------ 4. reduction over workgroups
    {
      const int cpw = (d + G - 1) / G;          // columns of this workgroup (<= THREADS)
      const int cw0 = w * cpw;
      const int nc = max(0, min(cpw, d - cw0));
      const int ngr = THREADS / cpw;            // partial groups
      const int c = tid % cpw, gr = tid / cpw;
      float s = 0.0f;
      if (c < nc && gr < ngr && gr < G)
        s = sum_coherent(a.ypart + (size_t)gr * d + cw0 + c, (size_t)ngr * d, (G - gr + ngr - 1) / ngr);
      red[tid] = s;
      __syncthreads();
      float y = 0.0f;
      if (tid < nc) {
        for (int qg = 0; qg < ngr && qg < G; ++qg) y += red[qg * cpw + tid];
        if (l == a.L - 1) static_cast<T *>(a.out)[cw0 + tid] = Elem<T>::round(y);
        else store_coherent(a.ybuf + cw0 + tid, y);
      }
      float sq = (tid < nc) ? y * y : 0.0f;  // slice sum of squares, fixed order
      sq = wave_sum(sq);
      __syncthreads();
      if (lane == 0) scal[wv] = sq;
      __syncthreads();
      if (tid == 0 && l < a.L - 1) {
        float tot = 0.0f;
        for (int i = 0; i < NW; ++i) tot += scal[i];
        store_coherent(a.sspart + w, tot);
      }
    }
    if (l == 0) SATS_TRACE_POINT(7);
    if (l < a.L - 1) grid_barrier(a.bar, (unsigned)G, a.err);
  }
}

}  // namespace sats
