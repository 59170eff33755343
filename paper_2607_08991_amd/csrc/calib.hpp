// SATS calibration (Section 3.1, Eq. 6-10): the kernels around the error
// product of dense.hpp (cal_err_kernel).
//
//   cal_hist_kernel / cal_hist_reduce_kernel / cal_select_kernel
//       exact order statistics of the post-gate magnitudes |g| over all
//       n x d_ff calibration values (the Eq. 3 percentiles that make up the
//       candidate set): a radix select on the float bits of |g| (for
//       non-negative floats the bit pattern orders like the value), 12 + 8 +
//       8 + 4 bits in four counting passes; every level is resolved at once.
//   cal_bucket_kernel
//       c = #{r : t_r <= |g|} per calibration value (the removed test of the
//       error product), and the histogram of c, which gives the sparsity
//       sp(t_r) = #{|g| < t_r} / (n d_ff) = #{c <= r} / (n d_ff).
//   cal_transpose_kernel
//       W_down^T for the error product (its B operands are k-contiguous).
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

// Radix pass of the select: for each level k of [0, K), the histogram of
// the `bits` bits at `shift` of the values whose higher bits (from shift +
// bits up) equal the level's prefix so far (pass 0: every value, one
// histogram).  Levels ascend, so their prefixes do too: the levels a value
// counts for are the run of equal prefixes found by binary search.  Counted
// in LDS per workgroup (K x 2^bits counters, at most kCalHistLds) and
// written whole to part[workgroup] (no global atomics); cal_hist_reduce_kernel
// adds the workgroups' histograms in workgroup order.
constexpr int kCalHistLds = 16384;
constexpr int kCalHistThreads = 1024;
__global__ __launch_bounds__(kCalHistThreads) void cal_hist_kernel(const float *G, size_t N, const uint32_t *prefix,
                                                                   int K, int shift, int bits, uint32_t *part) {
  __shared__ uint32_t pf[kCalMaxLevels];
  __shared__ uint32_t h[kCalHistLds];
  const int bins = 1 << bits, nh = K * bins;
  const int hs = shift + bits;  // 32 on pass 0: no prefix
  for (int k = threadIdx.x; k < K; k += kCalHistThreads) pf[k] = hs >= 32 ? 0u : prefix[k];
  for (int i = threadIdx.x; i < nh; i += kCalHistThreads) h[i] = 0u;
  __syncthreads();
  for (size_t i = blockIdx.x * (size_t)kCalHistThreads + threadIdx.x; i < N;
       i += (size_t)gridDim.x * kCalHistThreads) {
    const uint32_t b = abs_bits(G[i]);
    const uint32_t hi = hs >= 32 ? 0u : b >> hs, key = (b >> shift) & (uint32_t)(bins - 1);
    int lo = 0, up = K;  // first level whose prefix is >= hi
    while (lo < up) {
      const int mid = (lo + up) >> 1;
      if (pf[mid] < hi) lo = mid + 1;
      else up = mid;
    }
    for (int k = lo; k < K && pf[k] == hi; ++k) atomicAdd(&h[k * bins + key], 1u);
  }
  __syncthreads();
  uint32_t *o = part + (size_t)blockIdx.x * nh;
  for (int i = threadIdx.x; i < nh; i += kCalHistThreads) o[i] = h[i];
}

// hist[i] = sum over the `parts` workgroup histograms of entry i, in order.
__global__ __launch_bounds__(kCalThreads) void cal_hist_reduce_kernel(const uint32_t *part, int parts, int nh,
                                                                      uint32_t *hist) {
  const int i = blockIdx.x * kCalThreads + threadIdx.x;
  if (i >= nh) return;
  uint32_t s = 0u;
#pragma unroll 8
  for (int q = 0; q < parts; ++q) s += part[(size_t)q * nh + i];
  hist[i] = s;
}

// Level k (workgroup k): the bin holding its remaining rank (1-based) in its
// histogram (the pass-0 one is shared by all levels: stride 0), found by a prefix sum
// over the bins; the prefix is extended by that bin and the rank becomes the
// rank within it.  On the last pass the prefix is the whole bit pattern of
// the order statistic.  A level of rank 0 stays at 0 (threshold 0, below
// every value).
constexpr int kCalSelThreads = 256;
__global__ __launch_bounds__(kCalSelThreads) void cal_select_kernel(const uint32_t *hist, size_t stride, int bins,
                                                                    int bits, uint32_t *prefix, uint32_t *rank,
                                                                    float *t_out) {
  __shared__ uint32_t part[kCalSelThreads];
  const int k = blockIdx.x, tid = threadIdx.x;
  const uint32_t r = rank[k];
  if (r == 0u) {
    if (tid == 0) {
      prefix[k] = 0u;
      if (t_out) t_out[k] = 0.0f;
    }
    return;
  }
  const uint32_t *h = hist + stride * (size_t)k;
  const int per = (bins + kCalSelThreads - 1) / kCalSelThreads;  // bins per thread (the last ones may hold none)
  const int b0 = min(tid * per, bins), b1 = min(b0 + per, bins);
  uint32_t s = 0u;
  for (int i = b0; i < b1; ++i) s += h[i];
  part[tid] = s;
  __syncthreads();
  // inclusive prefix over threads (Hillis-Steele)
  for (int o = 1; o < kCalSelThreads; o <<= 1) {
    const uint32_t v = tid >= o ? part[tid - o] : 0u;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  const uint32_t before = tid ? part[tid - 1] : 0u;
  if (before < r && r <= part[tid]) {  // the bin is in this thread's run (not empty)
    uint32_t cum = before;
    int b = b0;
    for (; b < b1 - 1; ++b) {
      if (cum + h[b] >= r) break;
      cum += h[b];
    }
    rank[k] = r - cum;
    prefix[k] = (prefix[k] << bits) | (uint32_t)b;
    if (t_out) t_out[k] = __uint_as_float(prefix[k]);
  }
}

// W_down^T [d][d_ff] from W_down [d_ff][d] (bf16), 64 x 64 tiles through
// LDS; grid (d / 64, d_ff / 64).
__global__ __launch_bounds__(kCalThreads) void cal_transpose_kernel(const uint16_t *W, int d_ff, int d,
                                                                    uint16_t *WT) {
  __shared__ uint16_t tile[64][66];
  const int c0 = blockIdx.x * 64, k0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 2 elements per thread and row
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = ty + 8 * i;
    const uint32_t v = *reinterpret_cast<const uint32_t *>(W + (size_t)(k0 + r) * d + c0 + 2 * tx);
    tile[r][2 * tx] = (uint16_t)(v & 0xffffu);
    tile[r][2 * tx + 1] = (uint16_t)(v >> 16);
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int c = ty + 8 * i;
    const uint32_t v = (uint32_t)tile[2 * tx][c] | ((uint32_t)tile[2 * tx + 1][c] << 16);
    *reinterpret_cast<uint32_t *>(WT + (size_t)(c0 + c) * d_ff + k0 + 2 * tx) = v;
  }
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
