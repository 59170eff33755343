// Routing-table construction (Section 3.2, Eq. 11-14): per-id scores from a
// routing corpus and the table of the calibrated threshold.
//
//   route_accum_kernel<DAMAGE>
//       a chunk of kRouteChunk occurrences per workgroup: the excess damage
//       d = max(0, l_sparse - l_base) (Eq. 11) of each, in float32, as an
//       integer number of 2^-32 units (rounded half to even); the chunk's
//       occurrences are gathered per id in an LDS hash table (open
//       addressing, twice as many slots as occurrences, so every probe
//       sequence ends) with LDS integer atomics, and each id of the chunk
//       then adds its sum and count to the id's totals with one global
//       integer atomic each (a frequent id costs one atomic per chunk, not
//       per occurrence; integer sums are exact in any order).  The totals
//       are held in kRouteCopies copies, workgroup w adding into copy
//       w % kRouteCopies: a frequent id's atomics, which serialise per
//       address, are spread over the copies.  DAMAGE false: counts only
//       (the held-out split).
//   route_score_kernel
//       the copies added (integers), s(x) = 2^-32 (double(S_x) / double(C_x))
//       (the empirical mean of Eq. 12), +inf for ids without occurrences;
//       the held-out counts' copies added likewise.
//   route_table_kernel
//       table[x] = 0 (sparse path) if s(x) < tau, else 1 (Eq. 13).
#pragma once

#include "kernels.hpp"

namespace sats {

constexpr int kRouteThreads = 1024;
constexpr int kRouteChunk = 4096;  // occurrences per workgroup (4 per thread)
constexpr uint32_t kRouteNoId = 0xffffffffu;
constexpr int kRouteCopies = 32;  // copies of the per-id totals

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

template <bool DAMAGE>
__global__ __launch_bounds__(kRouteThreads) void route_accum_kernel(RouteAccumArgs a) {
  __shared__ uint32_t skey[kRouteSlots];
  __shared__ uint32_t scnt[kRouteSlots];
  __shared__ unsigned long long ssum[DAMAGE ? kRouteSlots : 1];
  const int tid = threadIdx.x;
  const int64_t base = (int64_t)blockIdx.x * kRouteChunk;
  constexpr int PER = kRouteChunk / kRouteThreads, SPER = kRouteSlots / kRouteThreads;
  uint32_t k[PER];
  unsigned long long q[PER];
  // the chunk's loads first, then the table's initialisation
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int64_t i = base + tid + m * kRouteThreads;
    k[m] = kRouteNoId;
    q[m] = 0ull;
    if (i < a.n) {
      const int32_t x = a.ids[i];
      if (x >= 0 && x < a.vocab) {
        k[m] = (uint32_t)x;
        if constexpr (DAMAGE) {
          const float diff = a.ls[i] - a.lb[i];  // float32, as in Eq. 11
          if (diff < 2147483648.0f) {             // also false for NaN
            // d 2^32 is exact in float32 and rintf rounds half to even: an
            // integer-valued float below 2^63, converted exactly
            q[m] = (unsigned long long)rintf(fmaxf(diff, 0.0f) * 4294967296.0f);
          } else {
            k[m] = kRouteNoId;
            __hip_atomic_store(a.err, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
        }
      } else {
        __hip_atomic_store(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
    if (probe == kRouteSlots) __hip_atomic_store(a.err, 3u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
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

__global__ __launch_bounds__(256) void route_score_kernel(const unsigned long long *sum, const unsigned *count,
                                                          const unsigned *hcount, int vocab, double *score,
                                                          unsigned *hcount_total) {
  const int x = blockIdx.x * 256 + threadIdx.x;
  if (x >= vocab) return;
  unsigned long long sx = 0ull;
  unsigned c = 0u, h = 0u;
#pragma unroll
  for (int k = 0; k < kRouteCopies; ++k) {
    sx += sum[(size_t)k * vocab + x];
    c += count[(size_t)k * vocab + x];
    h += hcount[(size_t)k * vocab + x];
  }
  score[x] = c ? ldexp((double)sx / (double)c, -32) : __builtin_huge_val();
  hcount_total[x] = h;
}

__global__ __launch_bounds__(256) void route_table_kernel(const double *score, int vocab, double tau,
                                                          uint8_t *table) {
  const int x = blockIdx.x * 256 + threadIdx.x;
  if (x < vocab) table[x] = score[x] < tau ? 0 : 1;
}

}  // namespace sats
