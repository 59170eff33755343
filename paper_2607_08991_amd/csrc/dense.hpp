// Batched calls: token routing with a stable partition, and the base-path
// (dense) group on MFMA matrix cores.
//
// route_kernel   per token r = table[id] (Eq. 13); a stable partition puts
//                the base-path tokens first (perm), counts them (n_dense) and
//                gathers their inputs into a packed [n_dense][d] buffer.  When
//                n_dense reaches the MFMA threshold the dense group is done
//                by the kernels below and the compacted sparse path skips
//                those tokens (flag per token); otherwise the sparse path
//                also takes the base-path tokens, keeping every column.
// dense_gateup   [rows x d] . W_gate and . W_up for 64 columns of d_ff per
//                workgroup with v_mfma_f32_16x16x32_bf16; epilogue
//                p = SiLU(a) * u (Eq. 1, 2) where the row keeps the column
//                (every column on the base path, |SiLU(a)| >= t otherwise,
//                Eq. 4-5) and 0 where it does not, rounded to bf16 for the
//                next product.  For batches the group can be the whole batch:
//                once any token takes the base path every row of the weights
//                is read anyway, so one MFMA stream serves every token.
// dense_down     [n_dense x d_ff] . W_down, split over d_ff chunks (partials).
// dense_glue     sums the partials in chunk order and writes the output row
//                of each dense token (scattered back through perm) or the
//                next layer's input rho(y / sqrt(mean(y^2) + 1e-6)).
//
// MFMA operand layout of v_mfma_f32_16x16x32_bf16 (wavefront of 64 lanes):
// lane l supplies A[l % 16][8 (l / 16) + e] and B[8 (l / 16) + e][l % 16],
// e = 0..7, and receives C[4 (l / 16) + r][l % 16], r = 0..3.  W_gate and
// W_down are stored with the output dimension contiguous, so their tiles are
// staged through LDS and read back k-major; W_up_T rows are already k-major.
#pragma once

#include "kernels.hpp"

namespace sats {

constexpr int kMfmaMinTokens = 8;   // dense group size from which MFMA is used
constexpr int kDenseMaxTokens = 64; // tokens of one pass (four 16-row MFMA tiles)
constexpr int kDenseNT = 64;        // output columns per workgroup
constexpr int kDenseKT = 32;        // k per MFMA step
constexpr int kLdsPitch = 66;       // bf16 per staged row (132 bytes: conflict-free k-major reads)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

struct RouteArgs {
  const int32_t *ids;
  const uint8_t *lut;
  int route_mode;
  int n, d;
  const uint16_t *x;      // [n][d] bf16 (this pass)
  int *perm;              // [n] base-path tokens first, then the others, each in order
  int *ctl;               // [0] n_dense, [1] dense group on MFMA (0/1)
  uint8_t *skip;          // [n] 1: token handled by the dense MFMA path
  uint8_t *route_out;     // optional [n]
  uint16_t *xd;           // [n][d] packed inputs of the dense group
  uint16_t *layer_in0;    // optional: inspection copy of the call input, [n][d]
  uint8_t *gbase;         // [n] base-path flag of each group row (group order)
  int mfma;               // the call may use the MFMA path
  int whole;              // the MFMA group is the whole batch (keep rule applied per row)
};

__global__ __launch_bounds__(kThreads) void route_kernel(RouteArgs a) {
  __shared__ int s_perm[kDenseMaxTokens];
  __shared__ int s_nd, s_on;
  const int tid = threadIdx.x, lane = tid & 63;
  if (tid < 64) {
    const bool valid = tid < a.n;
    const int base = valid ? token_is_base(a.route_mode, a.ids, a.lut, tid) : 0;
    const uint64_t bal = __ballot(valid && base);
    const int nd = __popcll(bal);
    const int rank_d = __popcll(bal & ((1ull << lane) - 1ull));
    // group on MFMA: the base-path tokens once there are enough of them, or the
    // whole batch (every row then applies its own keep rule)
    const int ng = a.whole ? a.n : nd;
    const int on = (a.mfma && ng >= kMfmaMinTokens) ? 1 : 0;
    if (valid) {
      const int pos = base ? rank_d : nd + (tid - rank_d);
      s_perm[pos] = tid;
      a.perm[pos] = tid;
      a.gbase[pos] = (uint8_t)base;
      a.skip[tid] = (uint8_t)(on && (base || a.whole));
      if (a.route_out) a.route_out[tid] = (uint8_t)base;
    }
    if (tid == 0) {
      a.ctl[0] = ng;
      a.ctl[1] = on;
      s_nd = ng;
      s_on = on;
    }
  }
  __syncthreads();
  if (!s_on) return;
  // gather the dense group's inputs, 16 bytes per thread and step
  const int vpr = a.d / 8;  // 16-byte vectors per row (d % 32 == 0 on this path)
  for (int i = tid; i < s_nd * vpr; i += kThreads) {
    const int m = i / vpr, v = i - m * vpr;
    const u32x4 q = *reinterpret_cast<const u32x4 *>(a.x + (size_t)s_perm[m] * a.d + v * 8);
    *reinterpret_cast<u32x4 *>(a.xd + (size_t)m * a.d + v * 8) = q;
    if (a.layer_in0) *reinterpret_cast<u32x4 *>(a.layer_in0 + (size_t)s_perm[m] * a.d + v * 8) = q;
  }
}

struct DenseArgs {
  const int *ctl;         // [0] rows of the MFMA group, [1] MFMA path on
  const uint8_t *gbase;   // [rows] base-path flag per group row
  const int *perm;        // group row -> token of the pass
  const float *thr;       // threshold of this layer (gate/up)
  uint8_t *keep_out;      // optional inspection: [n][N] keep flags, rows through perm
  const uint16_t *H;      // [n_dense][K] bf16 layer input (gate/up) or p (down)
  const uint16_t *Wb;     // W_gate [K][N] or W_down [K][N] (output dim contiguous)
  const uint16_t *Wt;     // W_up_T [N][K] (gate/up only)
  uint16_t *P;            // gate/up output p, [n_dense][N] bf16
  float *part;            // down output partials, [KSPLIT][n_dense][N]
  int K, N, kchunk;       // reduction length, output columns, k per split (down)
};

// One 32 x 64 tile of a row-major [K][N] bf16 matrix, staged into LDS with a
// 132-byte row pitch.  Thread t copies row t / 8, columns 8 (t % 8) .. + 8.
__device__ __forceinline__ u32x4 tile_load(const uint16_t *W, int N, int k0, int n0) {
  const int t = threadIdx.x;
  return __builtin_nontemporal_load(
      reinterpret_cast<const u32x4 *>(W + (size_t)(k0 + t / 8) * N + n0 + 8 * (t % 8)));
}
__device__ __forceinline__ void tile_store(uint32_t *lds, const u32x4 &v) {
  const int t = threadIdx.x;
  uint32_t *p = lds + (t / 8) * (kLdsPitch / 2) + 4 * (t % 8);
  p[0] = v.x;
  p[1] = v.y;
  p[2] = v.z;
  p[3] = v.w;
}
// k-major operand of column c (0..63) of the staged tile: rows 8 g .. 8 g + 7
__device__ __forceinline__ bf16x8 tile_operand(const uint32_t *lds, int c, int g) {
  const uint16_t *p = reinterpret_cast<const uint16_t *>(lds);
  bf16x8 b;
#pragma unroll
  for (int e = 0; e < 8; ++e) b[e] = __builtin_bit_cast(__bf16, p[(8 * g + e) * kLdsPitch + c]);
  return b;
}
__device__ __forceinline__ bf16x8 load_k8(const uint16_t *p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

// p = SiLU(h W_gate) * (h W_up) for 64 columns (blockIdx.x) and every dense token
__global__ __launch_bounds__(kThreads) void dense_gateup_kernel(DenseArgs a) {
  if (!a.ctl[1]) return;
  __shared__ uint32_t lds[kDenseKT * kLdsPitch / 2];
  const int nd = a.ctl[0];
  const int mtiles = (nd + 15) / 16;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, g = lane / 16;
  const int n0 = blockIdx.x * kDenseNT;
  const int ncol = n0 + 16 * wv + (lane % 16);
  typedef float f4 __attribute__((ext_vector_type(4)));
  f4 accg[4], accu[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) accg[mt] = accu[mt] = f4{0.f, 0.f, 0.f, 0.f};
  u32x4 next = tile_load(a.Wb, a.N, 0, n0);
  for (int k0 = 0; k0 < a.K; k0 += kDenseKT) {
    __syncthreads();
    tile_store(lds, next);
    __syncthreads();
    if (k0 + kDenseKT < a.K) next = tile_load(a.Wb, a.N, k0 + kDenseKT, n0);
    const bf16x8 bg = tile_operand(lds, 16 * wv + (lane % 16), g);
    const bf16x8 bu = load_k8(a.Wt + (size_t)ncol * a.K + k0 + 8 * g);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      if (mt < mtiles) {
        const int m = 16 * mt + (lane % 16);
        bf16x8 av = load_k8(a.H + (size_t)min(m, nd - 1) * a.K + k0 + 8 * g);
        if (m >= nd) av = bf16x8{};
        accg[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bg, accg[mt], 0, 0, 0);
        accu[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bu, accu[mt], 0, 0, 0);
      }
    }
  }
  const float thr = a.thr ? *a.thr : 0.0f;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = 16 * mt + 4 * g + r;
      if (mt < mtiles && m < nd) {
        const float gv = silu(accg[mt][r]);
        const bool keep = a.gbase[m] || fabsf(gv) >= thr;  // Eq. 4-5; every column on the base path
        a.P[(size_t)m * a.N + ncol] = keep ? f32_to_bf16(gv * accu[mt][r]) : (uint16_t)0;
        if (a.keep_out) a.keep_out[(size_t)a.perm[m] * a.N + ncol] = (uint8_t)keep;
      }
    }
  }
}

// partial y over k chunk blockIdx.y for 64 output columns (blockIdx.x)
__global__ __launch_bounds__(kThreads) void dense_down_kernel(DenseArgs a) {
  if (!a.ctl[1]) return;
  __shared__ uint32_t lds[kDenseKT * kLdsPitch / 2];
  const int nd = a.ctl[0];
  const int mtiles = (nd + 15) / 16;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, g = lane / 16;
  const int n0 = blockIdx.x * kDenseNT;
  const int ncol = n0 + 16 * wv + (lane % 16);
  const int kb = blockIdx.y * a.kchunk, ke = min(a.K, kb + a.kchunk);
  typedef float f4 __attribute__((ext_vector_type(4)));
  f4 acc[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) acc[mt] = f4{0.f, 0.f, 0.f, 0.f};
  u32x4 next = u32x4{0u, 0u, 0u, 0u};
  if (kb < ke) next = tile_load(a.Wb, a.N, kb, n0);
  for (int k0 = kb; k0 < ke; k0 += kDenseKT) {
    __syncthreads();
    tile_store(lds, next);
    __syncthreads();
    if (k0 + kDenseKT < ke) next = tile_load(a.Wb, a.N, k0 + kDenseKT, n0);
    const bf16x8 b = tile_operand(lds, 16 * wv + (lane % 16), g);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      if (mt < mtiles) {
        const int m = 16 * mt + (lane % 16);
        bf16x8 av = load_k8(a.H + (size_t)min(m, nd - 1) * a.K + k0 + 8 * g);
        if (m >= nd) av = bf16x8{};
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, b, acc[mt], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = 16 * mt + 4 * g + r;
      if (mt < mtiles && m < nd) a.part[((size_t)blockIdx.y * nd + m) * a.N + ncol] = acc[mt][r];
    }
}

struct GlueArgs {
  const int *ctl;
  const int *perm;
  const float *part;      // [KSPLIT][n_dense][d]
  int ksplit, d;
  uint16_t *out;          // last layer: [n][d] of the pass, rows through perm; else null
  uint16_t *hnext;        // otherwise: next layer input of the dense group, [n_dense][d]
  uint16_t *layer_in;     // optional: inspection copy of the next layer input, rows through perm
};

// one workgroup per dense token (blockIdx.x)
__global__ __launch_bounds__(kThreads) void dense_glue_kernel(GlueArgs a) {
  if (!a.ctl[1]) return;
  const int m = blockIdx.x;
  if (m >= a.ctl[0]) return;
  const int nd = a.ctl[0];
  __shared__ float ssw[kThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  constexpr int PT = 16;  // columns per thread (d <= 4096)
  float y[PT];
  float sq = 0.0f;
#pragma unroll
  for (int i = 0; i < PT; ++i) {
    const int c = tid + i * kThreads;
    float s = 0.0f;
    if (c < a.d)
      for (int q = 0; q < a.ksplit; ++q) s += a.part[((size_t)q * nd + m) * a.d + c];
    y[i] = s;
    sq = fmaf(s, s, sq);
  }
  const int row = a.perm[m];
  if (a.out) {
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int c = tid + i * kThreads;
      if (c < a.d) a.out[(size_t)row * a.d + c] = f32_to_bf16(y[i]);
    }
    return;
  }
  sq = wave_sum(sq);
  if (lane == 0) ssw[wv] = sq;
  __syncthreads();
  float tot = 0.0f;
  for (int i = 0; i < kThreads / 64; ++i) tot += ssw[i];
  const float scale = sqrtf(tot / (float)a.d + kGlueEps);
#pragma unroll
  for (int i = 0; i < PT; ++i) {
    const int c = tid + i * kThreads;
    if (c < a.d) {
      const uint16_t hv = f32_to_bf16(y[i] / scale);
      a.hnext[(size_t)m * a.d + c] = hv;
      if (a.layer_in) a.layer_in[(size_t)row * a.d + c] = hv;
    }
  }
}

}  // namespace sats
