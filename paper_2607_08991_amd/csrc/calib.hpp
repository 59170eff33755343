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
//       error product), and ge_r = #{|g| >= t_r}, which gives the sparsity
//       sp(t_r) = #{|g| < t_r} / (n d_ff) = 1 - ge_r / (n d_ff).
//   cal_transpose_kernel
//       W_down^T for the error product (its B operands are k-contiguous).
//   cal_reduce_kernel / cal_reduce_sum_kernel
//       finish Eq. 6 from the column-tile sums of squares: per row
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
// histogram).  Levels ascend, so their prefixes do too, and the levels of
// one prefix are a run.  A value finds its run in a hash table in LDS
// (slot = low kCalTabBits bits of the prefix, entry = prefix << 16 | run
// length << 8 | first level; 0 = empty): one read rejects a value that
// matches no level.  A slot that two prefixes share holds kCalTabMixed, and
// its values find their run by binary search over the prefixes.  Counted in
// LDS per workgroup (K x 2^bits counters, at most kCalHistLds) and written
// whole to part[workgroup] (no global atomics); cal_hist_reduce_kernel adds
// the workgroups' histograms.  A thread reads four values per 16-byte load
// and has kCalLoads loads in flight; workgroup 0 takes the N % 4 tail.
constexpr int kCalHistLds = 16384;
constexpr int kCalHistThreads = 1024;
constexpr int kCalLoads = 4;
constexpr int kCalTabBits = 12;
constexpr unsigned long long kCalTabMixed = 0xff00ull;  // run length 255: more than kCalMaxLevels
__device__ __forceinline__ void hist_add(uint32_t b, unsigned long long e, const uint32_t *pf, int K, int hs,
                                         int shift, int bins, uint32_t *h) {
  const uint32_t key = (b >> shift) & (uint32_t)(bins - 1);
  if (hs >= 32) {  // pass 0: one histogram
    atomicAdd(&h[key], 1u);
    return;
  }
  const uint32_t hi = b >> hs;
  int k = 0, k1 = 0;
  if (e == kCalTabMixed) {
    int up = K;  // first level whose prefix is >= hi
    while (k < up) {
      const int mid = (k + up) >> 1;
      if (pf[mid] < hi) k = mid + 1;
      else up = mid;
    }
    for (k1 = k; k1 < K && pf[k1] == hi; ++k1) {
    }
  } else if (e != 0ull && (uint32_t)(e >> 16) == hi) {
    k = (int)(e & 0xffu);
    k1 = k + (int)((e >> 8) & 0xffu);
  }
  for (; k < k1; ++k) atomicAdd(&h[k * bins + key], 1u);
}

__global__ __launch_bounds__(kCalHistThreads) void cal_hist_kernel(const float *G, size_t N, const uint32_t *prefix,
                                                                   int K, int shift, int bits, uint32_t *part) {
  __shared__ uint32_t pf[kCalMaxLevels];
  __shared__ uint32_t nslot[1 << kCalTabBits];
  __shared__ unsigned long long tab[1 << kCalTabBits];
  __shared__ uint32_t h[kCalHistLds];
  constexpr uint32_t kMask = (1u << kCalTabBits) - 1;
  const int bins = 1 << bits, nh = K * bins;
  const int hs = shift + bits;  // 32 on pass 0: no prefix
  for (int k = threadIdx.x; k < K; k += kCalHistThreads) pf[k] = hs >= 32 ? 0u : prefix[k];
  for (int i = threadIdx.x; i < nh; i += kCalHistThreads) h[i] = 0u;
  for (int i = threadIdx.x; i < (1 << kCalTabBits); i += kCalHistThreads) {
    tab[i] = 0ull;
    nslot[i] = 0u;
  }
  __syncthreads();
  // the level that starts a run enters it (K <= kCalMaxLevels <= the threads)
  const int k = threadIdx.x;
  const bool start = hs < 32 && k < K && (k == 0 || pf[k - 1] != pf[k]);
  if (start) {
    int n = 1;
    while (k + n < K && pf[k + n] == pf[k]) ++n;
    atomicAdd(&nslot[pf[k] & kMask], 1u);
    tab[pf[k] & kMask] = (unsigned long long)pf[k] << 16 | (unsigned long long)n << 8 | (unsigned long long)k;
  }
  __syncthreads();
  if (start && nslot[pf[k] & kMask] > 1u) tab[pf[k] & kMask] = kCalTabMixed;
  __syncthreads();
  const size_t N4 = N / 4, stride = (size_t)gridDim.x * kCalHistThreads;
  const float4 *G4 = reinterpret_cast<const float4 *>(G);
  for (size_t i = blockIdx.x * (size_t)kCalHistThreads + threadIdx.x; i < N4; i += kCalLoads * stride) {
    float4 v[kCalLoads];
#pragma unroll
    for (int j = 0; j < kCalLoads; ++j) v[j] = G4[min(i + j * stride, N4 - 1)];  // clamped: loads stay unconditional
    uint32_t b[4 * kCalLoads];
    unsigned long long e[4 * kCalLoads];
#pragma unroll
    for (int j = 0; j < kCalLoads; ++j) {
      b[4 * j] = abs_bits(v[j].x);
      b[4 * j + 1] = abs_bits(v[j].y);
      b[4 * j + 2] = abs_bits(v[j].z);
      b[4 * j + 3] = abs_bits(v[j].w);
    }
#pragma unroll
    for (int q = 0; q < 4 * kCalLoads; ++q) e[q] = hs >= 32 ? 0ull : tab[(b[q] >> hs) & kMask];
#pragma unroll
    for (int q = 0; q < 4 * kCalLoads; ++q)
      if (i + (q / 4) * stride < N4) hist_add(b[q], e[q], pf, K, hs, shift, bins, h);
  }
  if (blockIdx.x == 0 && threadIdx.x < N - 4 * N4) {
    const uint32_t b = abs_bits(G[4 * N4 + threadIdx.x]);
    hist_add(b, hs >= 32 ? 0ull : tab[(b >> hs) & kMask], pf, K, hs, shift, bins, h);
  }
  __syncthreads();
  uint32_t *o = part + (size_t)blockIdx.x * nh;
  for (int i = threadIdx.x; i < nh; i += kCalHistThreads) o[i] = h[i];
}

// hist[i] = sum over the `parts` workgroup histograms of entry i: a
// workgroup takes 64 entries, its 16 wavefronts one sixteenth of the parts
// each (integer sums: exact in any order).
constexpr int kCalHRBins = 64, kCalHRChunks = kCalHistThreads / kCalHRBins;
__global__ __launch_bounds__(kCalHistThreads) void cal_hist_reduce_kernel(const uint32_t *part, int parts, int nh,
                                                                          uint32_t *hist) {
  __shared__ uint32_t acc[kCalHRChunks][kCalHRBins];
  const int b = threadIdx.x % kCalHRBins, c = threadIdx.x / kCalHRBins, i = blockIdx.x * kCalHRBins + b;
  uint32_t s = 0u;
  if (i < nh)
#pragma unroll 8
    for (int q = c; q < parts; q += kCalHRChunks) s += part[(size_t)q * nh + i];
  acc[c][b] = s;
  __syncthreads();
  if (c == 0 && i < nh) {
    uint32_t t = 0u;
#pragma unroll
    for (int j = 0; j < kCalHRChunks; ++j) t += acc[j][b];
    hist[i] = t;
  }
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

// c = #{r < 15 : t_r <= |g|} per value, as a byte (the error product
// removes a neuron at candidate r when c <= r), and ge[r] = #{|g| >= t_r},
// the values kept at t_r, over the launch (integer counts: exact in any
// order; ge must be zero on entry).  A thread reads four values per 16-byte
// load and has kCalLoads loads in flight; workgroup 0 takes the N % 4 tail.
__global__ __launch_bounds__(kCalThreads) void cal_bucket_kernel(const float *G, size_t N, const float *thr15,
                                                                 uint8_t *cnt, unsigned long long *ge) {
  __shared__ unsigned int h[kCalCand];
  if (threadIdx.x < kCalCand) h[threadIdx.x] = 0u;
  float t[kCalCand];
  uint32_t n_ge[kCalCand];
#pragma unroll
  for (int r = 0; r < kCalCand; ++r) {
    t[r] = thr15[r];
    n_ge[r] = 0u;
  }
  auto bucket = [&](float g) -> uint32_t {
    const float v = fabsf(g);
    uint32_t c = 0u;
#pragma unroll
    for (int r = 0; r < kCalCand; ++r) {
      const uint32_t f = t[r] <= v ? 1u : 0u;
      c += f;
      n_ge[r] += f;
    }
    return c;
  };
  const size_t N4 = N / 4, stride = (size_t)gridDim.x * kCalThreads;
  const float4 *G4 = reinterpret_cast<const float4 *>(G);
  uint32_t *C4 = reinterpret_cast<uint32_t *>(cnt);
  for (size_t i = blockIdx.x * (size_t)kCalThreads + threadIdx.x; i < N4; i += kCalLoads * stride) {
    float4 v[kCalLoads];
#pragma unroll
    for (int j = 0; j < kCalLoads; ++j) v[j] = G4[min(i + j * stride, N4 - 1)];  // clamped: loads stay unconditional
#pragma unroll
    for (int j = 0; j < kCalLoads; ++j)
      if (i + j * stride < N4)
        C4[i + j * stride] = bucket(v[j].x) | bucket(v[j].y) << 8 | bucket(v[j].z) << 16 | bucket(v[j].w) << 24;
  }
  if (blockIdx.x == 0 && threadIdx.x < N - 4 * N4) cnt[4 * N4 + threadIdx.x] = (uint8_t)bucket(G[4 * N4 + threadIdx.x]);
#pragma unroll
  for (int r = 0; r < kCalCand; ++r)
    for (int o = 32; o > 0; o >>= 1) n_ge[r] += __shfl_xor(n_ge[r], o);
  __syncthreads();
  if ((threadIdx.x & 63) == 0)
#pragma unroll
    for (int r = 0; r < kCalCand; ++r)
      if (n_ge[r]) atomicAdd(&h[r], n_ge[r]);
  __syncthreads();
  if (threadIdx.x < kCalCand && h[threadIdx.x]) atomicAdd(&ge[threadIdx.x], (unsigned long long)h[threadIdx.x]);
}

// Eq. 6 from part[tile][m][16] (sums of squares over column tile `tile`;
// entry 15 of every calibration row holds ||y||^2): workgroup b takes rows
// 64 b .. 64 b + 63 (a lane per row), its wavefront w the tiles w, w + 8,
// ...; wavefront 0 adds the eight sums in order and forms per row
// e_r = ||y - y_t_r|| / (||y|| + eps), and the sums of e_r over the rows
// (a fixed tree over the lanes) go to rsum[b][r], which
// cal_reduce_sum_kernel adds over workgroups in order.  ny2_out (or null)
// keeps ||y||^2 of each row for later products; a product without a y row
// takes it from ny2_in.
constexpr int kCalRedWaves = 8;
__global__ __launch_bounds__(64 * kCalRedWaves) void cal_reduce_kernel(const float *part, int ntiles, int n, int K,
                                                                       float *err_rows, int rows_ld, double *rsum,
                                                                       const float *ny2_in, float *ny2_out) {
  __shared__ float acc[kCalRedWaves][16][65];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, m = blockIdx.x * 64 + lane;
  float e2[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) e2[r] = 0.0f;
  if (m < n) {
#pragma unroll 4
    for (int tl = w; tl < ntiles; tl += kCalRedWaves) {
      const float4 *p = reinterpret_cast<const float4 *>(part + ((size_t)tl * n + m) * 16);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 v = p[q];
        e2[4 * q] += v.x;
        e2[4 * q + 1] += v.y;
        e2[4 * q + 2] += v.z;
        e2[4 * q + 3] += v.w;
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[w][r][lane] = e2[r];
  __syncthreads();
  if (w != 0) return;
#pragma unroll
  for (int r = 0; r < 16; ++r)
    for (int j = 1; j < kCalRedWaves; ++j) e2[r] += acc[j][r][lane];
  if (ny2_out && m < n) ny2_out[m] = e2[15];
  const float ny = sqrtf((ny2_in && m < n) ? ny2_in[m] : e2[15]);
#pragma unroll
  for (int r = 0; r < kCalCand; ++r) {
    double s = 0.0;
    if (m < n && r < K) {
      const float e = sqrtf(e2[r]) / (ny + kCalEps);
      if (err_rows) err_rows[(size_t)m * rows_ld + r] = e;
      s = (double)e;
    }
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) rsum[(size_t)blockIdx.x * 16 + r] = s;
  }
}

// err_sum[r] = sum over the `blocks` workgroup sums rsum[b][r], in order.
__global__ __launch_bounds__(64) void cal_reduce_sum_kernel(const double *rsum, int blocks, int K, double *err_sum) {
  const int r = threadIdx.x;
  if (r >= K) return;
  double s = 0.0;
  for (int b = 0; b < blocks; ++b) s += rsum[(size_t)b * 16 + r];
  err_sum[r] = s;
}

// err_rows[m][k] = 0 for k < ncols: candidates at or below 0 remove no
// neuron (no |g| is below them), so their Eq. 6 terms are 0 exactly.
__global__ __launch_bounds__(kCalThreads) void cal_zero_cols_kernel(float *rows, size_t n, int ld, int ncols) {
  const size_t tot = n * (size_t)ncols;
  for (size_t i = blockIdx.x * (size_t)kCalThreads + threadIdx.x; i < tot; i += (size_t)gridDim.x * kCalThreads)
    rows[(i / ncols) * ld + i % ncols] = 0.0f;
}

}  // namespace sats
