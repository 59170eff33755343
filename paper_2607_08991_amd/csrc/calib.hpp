// SATS calibration (Section 3.1, Eq. 6-10): the kernels around the error
// product of dense.hpp (cal_err_kernel).
//
//   cal_hist0_kernel / cal_histk_kernel / cal_select_kernel
//       exact order statistics of the post-gate magnitudes |g| over all
//       n x d_ff calibration values (the Eq. 3 percentiles that make up the
//       candidate set): a radix select on the float bits of |g| (for
//       non-negative floats the bit pattern orders like the value), 12 + 12 +
//       8 bits in three counting passes; every level is resolved at once.
//   cal_bucket_kernel
//       c = #{r : t_r <= |g|} per calibration value (the removed test of the
//       error product), and the histogram of c, which gives the sparsity
//       sp(t_r) = #{|g| < t_r} / (n d_ff) = #{c <= r} / (n d_ff).
//   cal_reduce_kernel
//       finishes Eq. 6 from the column-tile sums of squares: per row
//       e_r = ||y - y_t_r|| / (||y|| + eps), and Err(t_r) = mean of e_r.
//
// Counting uses integer atomics (exact in any order); every float sum has a
// fixed order.
#pragma once

#include "kernels.hpp"

namespace sats {

constexpr int kCalThreads = 256;
constexpr int kCalMaxLevels = 64;     // levels of one quantile call
constexpr int kCalCand = 15;          // candidates of one error product (row 15 is y)
constexpr float kCalEps = 1e-6f;      // eps of Eq. 6

__device__ __forceinline__ uint32_t abs_bits(float v) { return __float_as_uint(v) & 0x7fffffffu; }

// Pass 0: histogram of bits 31..20 of |g| (4096 bins, the top one never set)
// over all values, in LDS per workgroup, then added to the global one.
__global__ __launch_bounds__(kCalThreads) void cal_hist0_kernel(const float *G, size_t N, uint32_t *hist) {
  __shared__ uint32_t h[4096];
  for (int i = threadIdx.x; i < 4096; i += kCalThreads) h[i] = 0u;
  __syncthreads();
  for (size_t i = blockIdx.x * (size_t)kCalThreads + threadIdx.x; i < N; i += (size_t)gridDim.x * kCalThreads)
    atomicAdd(&h[abs_bits(G[i]) >> 20], 1u);
  __syncthreads();
  for (int i = threadIdx.x; i < 4096; i += kCalThreads)
    if (h[i]) atomicAdd(&hist[i], h[i]);
}

// Pass 1 (shift 8, 4096 bins) or 2 (shift 0, 256 bins): for each level k,
// the histogram of the next bits of the values whose higher bits equal the
// level's prefix so far.
__global__ __launch_bounds__(kCalThreads) void cal_histk_kernel(const float *G, size_t N, const uint32_t *prefix,
                                                                int K, int shift, int bins, uint32_t *hist) {
  __shared__ uint32_t pf[kCalMaxLevels];
  for (int k = threadIdx.x; k < K; k += kCalThreads) pf[k] = prefix[k];
  __syncthreads();
  const int hs = shift + (bins == 4096 ? 12 : 8);
  for (size_t i = blockIdx.x * (size_t)kCalThreads + threadIdx.x; i < N; i += (size_t)gridDim.x * kCalThreads) {
    const uint32_t b = abs_bits(G[i]);
    const uint32_t hi = b >> hs, key = (b >> shift) & (uint32_t)(bins - 1);
    for (int k = 0; k < K; ++k)
      if (pf[k] == hi) atomicAdd(&hist[(size_t)k * bins + key], 1u);
  }
}

// Level k (thread k): the bin holding its remaining rank (1-based) in its
// histogram (hist0 is shared by all levels: stride 0), the prefix extended
// by that bin and the rank within it.  On the last pass the prefix is the
// whole bit pattern of the order statistic.  A level of rank 0 stays at 0
// (threshold 0, below every value).
__global__ void cal_select_kernel(const uint32_t *hist, size_t stride, int bins, int bits, uint32_t *prefix,
                                  uint32_t *rank, int K, float *t_out) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= K) return;
  uint32_t r = rank[k];
  if (r == 0u) {
    prefix[k] = 0u;
    if (t_out) t_out[k] = 0.0f;
    return;
  }
  const uint32_t *h = hist + stride * (size_t)k;
  uint32_t cum = 0u;
  int b = 0;
  for (; b < bins; ++b) {
    if (cum + h[b] >= r) break;
    cum += h[b];
  }
  b = min(b, bins - 1);
  prefix[k] = (prefix[k] << bits) | (uint32_t)b;
  rank[k] = r - cum;
  if (t_out) t_out[k] = __uint_as_float(prefix[k]);
}

// c = #{r < 15 : t_r <= |g|} as a byte, and the histogram of c over the
// launch (16 counters).
__global__ __launch_bounds__(kCalThreads) void cal_bucket_kernel(const float *G, size_t N, const float *thr15,
                                                                 uint8_t *cnt, unsigned long long *hist16) {
  __shared__ float t[kCalCand];
  __shared__ unsigned int h[16];
  if (threadIdx.x < kCalCand) t[threadIdx.x] = thr15[threadIdx.x];
  if (threadIdx.x < 16) h[threadIdx.x] = 0u;
  __syncthreads();
  for (size_t i = blockIdx.x * (size_t)kCalThreads + threadIdx.x; i < N; i += (size_t)gridDim.x * kCalThreads) {
    const float v = fabsf(G[i]);
    int c = 0;
#pragma unroll
    for (int r = 0; r < kCalCand; ++r) c += (t[r] <= v) ? 1 : 0;
    cnt[i] = (uint8_t)c;
    atomicAdd(&h[c], 1u);
  }
  __syncthreads();
  if (threadIdx.x < 16 && h[threadIdx.x]) atomicAdd(&hist16[threadIdx.x], (unsigned long long)h[threadIdx.x]);
}

// Eq. 6 from part[tile][m][16] (sums of squares over column tile `tile`):
// one workgroup; thread i takes rows i, i + 1024, ... in order, and the
// per-thread sums of e_r are added over threads by a fixed tree.  Row 15 of
// every calibration row holds ||y||^2.
constexpr int kCalReduceThreads = 1024;
__global__ __launch_bounds__(kCalReduceThreads) void cal_reduce_kernel(const float *part, int ntiles, int n, int K,
                                                                        float *err_rows, int rows_ld,
                                                                        double *err_sum) {
  __shared__ double red[kCalReduceThreads];
  double s[kCalCand];
#pragma unroll
  for (int r = 0; r < kCalCand; ++r) s[r] = 0.0;
  for (int m = threadIdx.x; m < n; m += kCalReduceThreads) {
    float e2[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) e2[r] = 0.0f;
    for (int tl = 0; tl < ntiles; ++tl) {
      const float *p = part + ((size_t)tl * n + m) * 16;
#pragma unroll
      for (int r = 0; r < 16; ++r) e2[r] += p[r];
    }
    const float ny = sqrtf(e2[15]);
#pragma unroll
    for (int r = 0; r < kCalCand; ++r) {
      const float e = sqrtf(e2[r]) / (ny + kCalEps);
      if (r < K) {
        s[r] += (double)e;
        if (err_rows) err_rows[(size_t)m * rows_ld + r] = e;
      }
    }
  }
  for (int r = 0; r < K; ++r) {
    red[threadIdx.x] = s[r];
    __syncthreads();
    for (int o = kCalReduceThreads / 2; o > 0; o >>= 1) {
      if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
      __syncthreads();
    }
    if (threadIdx.x == 0) err_sum[r] = red[0];
    __syncthreads();
  }
}

}  // namespace sats
