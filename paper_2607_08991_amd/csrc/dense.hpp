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
// e = 0..7, and receives C[4 (l / 16) + r][l % 16], r = 0..3.  W_gate_T,
// W_up_T and H rows are k-major (one row per output column or input row);
// W_down is stored with the output dimension contiguous, so its operand is
// read from LDS transposed.
#pragma once

#include "kernels.hpp"

namespace sats {

constexpr int kMfmaMinTokens = 2;   // group size from which MFMA is used
constexpr int kDenseMaxTokens = 64; // tokens of one pass (four 16-row MFMA tiles)
constexpr int kDenseNT = 64;        // output columns per workgroup (gate/up)
constexpr int kDenseDownNT = 128;   // output columns per workgroup (down)
constexpr int kDenseMaxKsplit = 16; // d_ff chunks of the down-projection, at most

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
  int min_group;          // smallest group the MFMA path takes (kMfmaMinTokens; 1 for LoRA passes)
};

// One workgroup per token of the pass: every workgroup forms the same
// partition (64 table reads), workgroup 0 publishes it, and workgroup b
// gathers row b of the dense group's inputs.
__global__ __launch_bounds__(kThreads) void route_kernel(RouteArgs a) {
  __shared__ int s_perm[kDenseMaxTokens];
  __shared__ int s_nd, s_on;
  const int tid = threadIdx.x, lane = tid & 63;
  const bool pub = blockIdx.x == 0;
  if (tid < 64) {
    const bool valid = tid < a.n;
    const int base = valid ? token_is_base(a.route_mode, a.ids, a.lut, tid) : 0;
    const uint64_t bal = __ballot(valid && base);
    const int nd = __popcll(bal);
    const int rank_d = __popcll(bal & ((1ull << lane) - 1ull));
    // group on MFMA: the base-path tokens once there are enough of them, or the
    // whole batch (every row then applies its own keep rule)
    const int ng = a.whole ? a.n : nd;
    const int on = (a.mfma && ng >= a.min_group) ? 1 : 0;
    if (valid) {
      const int pos = base ? rank_d : nd + (tid - rank_d);
      s_perm[pos] = tid;
      if (pub) {
        a.perm[pos] = tid;
        a.gbase[pos] = (uint8_t)base;
        a.skip[tid] = (uint8_t)(on && (base || a.whole));
        if (a.route_out) a.route_out[tid] = (uint8_t)base;
      }
    }
    if (tid == 0) {
      if (pub) {
        a.ctl[0] = ng;
        a.ctl[1] = on;
      }
      s_nd = ng;
      s_on = on;
    }
  }
  __syncthreads();
  const int m = blockIdx.x;
  if (!s_on || m >= s_nd) return;
  // row m of the dense group, 16 bytes per thread and step
  const int vpr = a.d / 8;  // 16-byte vectors per row (d % 32 == 0 on this path)
  const int src = s_perm[m];
  for (int v = tid; v < vpr; v += kThreads) {
    const u32x4 q = *reinterpret_cast<const u32x4 *>(a.x + (size_t)src * a.d + v * 8);
    *reinterpret_cast<u32x4 *>(a.xd + (size_t)m * a.d + v * 8) = q;
    if (a.layer_in0) *reinterpret_cast<u32x4 *>(a.layer_in0 + (size_t)src * a.d + v * 8) = q;
  }
}

struct DenseArgs {
  const int *ctl;         // [0] rows of the MFMA group, [1] MFMA path on
  const uint8_t *gbase;   // [rows] base-path flag per group row
  const int *perm;        // group row -> token of the pass
  const float *thr;       // threshold of this layer (gate/up)
  uint8_t *keep_out;      // optional inspection: [n][N] keep flags, rows through perm
  const uint16_t *H;      // [n_dense][K] bf16 layer input (gate/up) or p (down)
  const uint16_t *Wb;     // down: W_down [K][N] (output dim contiguous)
  const uint16_t *Wg;     // gate/up: W_gate_T [N][K]
  const uint16_t *Wt;     // gate/up: W_up_T [N][K]
  uint16_t *P;            // gate/up output p, [n_dense][N] bf16
  uint8_t *uflag;         // gate/up: [N] 1 where some row keeps the column (the union of the
                          // keep sets; every column once a base-path row is in the group);
                          // down: the same flags of its K rows, rows without one are not read
  float *part;            // down output partials, [KSPLIT][n_dense][N]
  int K, N, kchunk;       // reduction length, output columns, k per split (down)
  int nt;                 // gate/up: output columns per workgroup (a multiple of 8, at most 64)
  int hcap;               // rows of H allocated (the first stages read them all, before the group's size is known)
  float *cal_g;           // calibration (gate/up): g = SiLU(a) in float32, [rows][N] (P unused) ...
  uint16_t *cal_ph, *cal_pl;  // ... and p = g u as two bf16 terms, hi = rne(p), lo = rne(p - hi)
  // calibration in one launch (the CAL instance): workgroup b takes column tile
  // (b / 8 / cal_passes) * 8 + b % 8 and pass (b / 8) % cal_passes (rows
  // 64 pass ..; ctl, H, hcap and the cal outputs above are those of pass 0):
  // the passes of a tile run at once on one XCD (workgroup b on XCD b mod 8)
  // and read its weights through that XCD's L2; tiles past cal_tiles return
  int cal_passes, cal_tiles;
  // LoRA adapters of the sparse path (gate/up with LORA): lv [2][kDenseMaxTokens][rank]
  // = s (h A_gate), s (h A_up) per group row; B_gate [rank][N], B_up_T [N][rank] and
  // A_down [N][rank] of the layer; zpart [tiles][kDenseMaxTokens][rank]: per column
  // tile, sum of p_j A_down[j] over its columns (zero for base-path rows)
  const float *lv;
  const uint16_t *Bg, *BuT, *Ad;
  float *zpart;
  int rank;
};

// ---------------------------------------------------------------- MFMA GEMMs
//
// Both products stream a weight matrix once and reuse each weight over the
// rows of the group, so they are bound by HBM, not by the matrix cores: what
// matters is how many bytes stay in flight and how little work each byte
// costs on its way to the MFMA.  A workgroup of 512 threads owns a tile of
// output columns and walks its k range in stages of 64 rows.  Each stage
// (24 KB) is loaded straight into LDS with buffer loads that write LDS
// (no register staging, no LDS store instructions) into a ring of six stage
// buffers: five stages are in flight while the wavefronts read the MFMA
// operands of the sixth.  One barrier per stage; before it every wavefront
// waits until its own loads of that stage have landed.
//
// A buffer load into LDS writes 16 bytes per lane at consecutive addresses,
// so the tile layout is chosen through the global address each lane reads.
// LDS tiles:
//   k-row tile  W_down rows (256 bytes each) of the stage; chunk q (16
//               bytes) of row r sits at position q ^ (2 ((r >> 3) & 3)), so
//               that the transposed operand reads of a wavefront touch
//               distinct banks
//   row tile    W_gate_T or W_up_T rows n0..n0+63, or H rows, 128 bytes
//               (64 k) each; chunk q of row r sits at q ^ ((r >> 1) & 7)

constexpr int kDenseThreads = 512;             // 8 wavefronts
constexpr int kDenseKC = 64;                   // k rows per stage
constexpr int kDenseStageBytes = 24 * 1024;    // one stage buffer
constexpr int kDenseXP = 68;                   // floats per row of the gate/up exchange tile

typedef float f32x4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t dense_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
constexpr uint32_t kDenseOffNone = 0x80000000u;  // past every buffer: the load returns zeros
// offset of a load that is skipped when !v; the skipped loads of one stage
// get distinct offsets so that they stay separate loads
__device__ __forceinline__ uint32_t dense_off(bool v, uint32_t off, int tag) {
  return v ? off : kDenseOffNone + 16u * (uint32_t)tag;
}
// 16 bytes per lane from the buffer into LDS at dst + 16 * lane (dst is the
// same for the whole wavefront); aux 2 streams past the caches
template <int AUX>
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint8_t *dst, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)dst, 16, (int)off, 0, 0, AUX);
}
// wait until at most `vm` buffer loads of this wavefront are outstanding and
// its LDS reads are done, then meet the other wavefronts
template <int VM>
__device__ __forceinline__ void dense_stage_barrier() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((VM & 15) | (7 << 4) | (0 << 8) | ((VM >> 4) << 14));
  __builtin_amdgcn_s_barrier();
}

__device__ __forceinline__ int krow_pos(int r, int q) { return q ^ (2 * ((r >> 3) & 3)); }
__device__ __forceinline__ int row_pos(int r, int q) { return q ^ ((r >> 1) & 7); }

// MFMA operand from a row tile: row r, k = 32 j + 8 g .. + 7 of the stage
__device__ __forceinline__ bf16x8 row_operand(const uint8_t *tile, int r, int j, int g) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(tile + r * 128 + row_pos(r, 4 * j + g) * 16));
}
// transposed MFMA operand from a k-row tile of `pitch` bytes per row:
// column c, rows 32 j + 8 g .. + 7
__device__ __forceinline__ bf16x8 krow_operand(const uint8_t *tile, int pitch, int c, int j, int g) {
  const uint16_t *p = reinterpret_cast<const uint16_t *>(tile);
  bf16x8 b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int r = 32 * j + 8 * g + e;
    b[e] = __builtin_bit_cast(__bf16, p[r * (pitch / 2) + krow_pos(r, c >> 3) * 8 + (c & 7)]);
  }
  return b;
}
__device__ __forceinline__ f32x4v mfma16(const bf16x8 &a, const bf16x8 &b, const f32x4v &c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// The stage loop shared by both products: stage s lives in ring buffer
// s % 6; `issue(buf, s)` starts three buffer loads per lane for stage s
// (loads past the k range read zeros) and `compute(buf)` consumes a stage.
// SATS_DENSE_RING_H runs HOOK after the first two stages are issued.
#define SATS_DENSE_RING(S, ISSUE, COMPUTE) SATS_DENSE_RING_H(S, ISSUE, COMPUTE, (void)0)
#define SATS_DENSE_RING_H(S, ISSUE, COMPUTE, HOOK)                                           \
  {                                                                                          \
    uint8_t *const rb_[6] = {rg0, rg1, rg2, rg3, rg4, rg5};                                  \
    (void)rb_;                                                                               \
    ISSUE(rg0, 0);                                                                           \
    ISSUE(rg1, 1);                                                                           \
    HOOK;                                                                                    \
    ISSUE(rg2, 2);                                                                           \
    ISSUE(rg3, 3);                                                                           \
    ISSUE(rg4, 4);                                                                           \
    for (int s0 = 0; s0 < (S); s0 += 6) {                                                    \
      SATS_DENSE_STEP(S, ISSUE, COMPUTE, rg0, rg5, 0)                                        \
      SATS_DENSE_STEP(S, ISSUE, COMPUTE, rg1, rg0, 1)                                        \
      SATS_DENSE_STEP(S, ISSUE, COMPUTE, rg2, rg1, 2)                                        \
      SATS_DENSE_STEP(S, ISSUE, COMPUTE, rg3, rg2, 3)                                        \
      SATS_DENSE_STEP(S, ISSUE, COMPUTE, rg4, rg3, 4)                                        \
      SATS_DENSE_STEP(S, ISSUE, COMPUTE, rg5, rg4, 5)                                        \
    }                                                                                        \
    __builtin_amdgcn_s_waitcnt(0); /* the zero-filling loads past the range land too */     \
  }
// stage s: its loads are the oldest of the five stages in flight (three
// loads each), so at most 12 may still be outstanding.  After the barrier
// every wavefront is done with stage s - 1, whose buffer takes stage s + 5.
#define SATS_DENSE_STEP(S, ISSUE, COMPUTE, CUR, NXT, P)                                      \
  {                                                                                          \
    const int s_ = s0 + (P);                                                                 \
    dense_stage_barrier<12>();                                                               \
    ISSUE(NXT, s_ + 5);                                                                      \
    if (s_ < (S)) COMPUTE(CUR);                                                              \
  }

// The ring of groups of at most 16 rows: eight 18 KB stages (W_gate_T and
// W_up_T 8 KB each, H 2 KB), seven in flight.  Wavefronts 0-1 also load the
// 16 H rows (three loads per stage, the others two), so their wait allows
// 18 outstanding loads and the others' 12.
#define SATS_DENSE_RING8(S, ISSUE, COMPUTE) SATS_DENSE_RING8_H(S, ISSUE, COMPUTE, (void)0)
#define SATS_DENSE_RING8_H(S, ISSUE, COMPUTE, HOOK)                                          \
  {                                                                                          \
    ISSUE(rg0, 0);                                                                           \
    ISSUE(rg1, 1);                                                                           \
    HOOK;                                                                                    \
    ISSUE(rg2, 2);                                                                           \
    ISSUE(rg3, 3);                                                                           \
    ISSUE(rg4, 4);                                                                           \
    ISSUE(rg5, 5);                                                                           \
    ISSUE(rg6, 6);                                                                           \
    for (int s0 = 0; s0 < (S); s0 += 8) {                                                    \
      SATS_DENSE_STEP8(S, ISSUE, COMPUTE, rg0, rg7, 0)                                       \
      SATS_DENSE_STEP8(S, ISSUE, COMPUTE, rg1, rg0, 1)                                       \
      SATS_DENSE_STEP8(S, ISSUE, COMPUTE, rg2, rg1, 2)                                       \
      SATS_DENSE_STEP8(S, ISSUE, COMPUTE, rg3, rg2, 3)                                       \
      SATS_DENSE_STEP8(S, ISSUE, COMPUTE, rg4, rg3, 4)                                       \
      SATS_DENSE_STEP8(S, ISSUE, COMPUTE, rg5, rg4, 5)                                       \
      SATS_DENSE_STEP8(S, ISSUE, COMPUTE, rg6, rg5, 6)                                       \
      SATS_DENSE_STEP8(S, ISSUE, COMPUTE, rg7, rg6, 7)                                       \
    }                                                                                        \
    __builtin_amdgcn_s_waitcnt(0);                                                           \
  }
#define SATS_DENSE_STEP8(S, ISSUE, COMPUTE, CUR, NXT, P)                                     \
  {                                                                                          \
    const int s_ = s0 + (P);                                                                 \
    if (w < 2)                                                                               \
      dense_stage_barrier<18>();                                                             \
    else                                                                                     \
      dense_stage_barrier<12>();                                                             \
    ISSUE(NXT, s_ + 7);                                                                      \
    if (s_ < (S)) COMPUTE(CUR);                                                              \
  }

// p = SiLU(h W_gate) * (h W_up) for the nt columns [nt b, nt b + nt) of
// workgroup b and every row of the group (MT 16-row tiles; rows past the group
// are read as zeros).  The MFMA tiles always span 64 columns: rows of W_gate_T
// and W_up_T past the workgroup's columns are read as zeros without a memory
// access (nt = d_ff / 256 fills every compute unit at the Llama and Qwen3
// shapes).  Wavefronts 0-3 accumulate h W_gate, 4-7 h W_up, 16 columns each.
// Groups of one row tile use the eight-stage ring of 18 KB stages, larger ones
// six stages of 24 KB.
template <int MT, bool LORA = false, bool CAL = false>
__global__ __launch_bounds__(kDenseThreads) void dense_gateup_kernel(DenseArgs a) {
  constexpr int NB = MT == 1 ? 8 : 6, SB = MT == 1 ? 18 * 1024 : kDenseStageBytes;  // ring stages and their bytes
  __shared__ __attribute__((aligned(1024))) uint8_t ring[NB * SB];
  uint8_t *const rg0 = ring, *const rg1 = ring + SB, *const rg2 = ring + 2 * SB, *const rg3 = ring + 3 * SB,
                 *const rg4 = ring + 4 * SB, *const rg5 = ring + 5 * SB;
  uint8_t *const rg6 = ring + (NB > 6 ? 6 : 0) * SB, *const rg7 = ring + (NB > 7 ? 7 : 0) * SB;
  (void)rg6;
  (void)rg7;
  int tile = blockIdx.x;
  if (CAL) {  // calibration passes in one launch (see DenseArgs)
    const int j = blockIdx.x >> 3, pass = j % a.cal_passes;
    tile = (j / a.cal_passes) * 8 + (blockIdx.x & 7);
    if (tile >= a.cal_tiles) return;
    const size_t rows = (size_t)pass * kDenseMaxTokens;
    a.ctl += 2 * pass;
    a.H += rows * a.K;
    a.hcap -= (int)rows;
    a.cal_g += rows * a.N;
    a.cal_ph += rows * a.N;
    a.cal_pl += rows * a.N;
  }
  // the group's control words are read while the first two stages load
  // (every allocated row of H: rows past the group feed only results that
  // are not stored); a workgroup of an empty group then waits for its loads
  // and returns
  const int ctl_on = a.ctl[1], ctl_n = a.ctl[0];
  int nd = 16 * MT;
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int mat = w >> 2, g = lane >> 4, l16 = lane & 15, c = 16 * (w & 3) + l16;
  const int n0 = tile * a.nt;
  const int K = a.K, N = a.N;
  const int ncol = min(a.nt, N - n0);  // this workgroup's columns (a multiple of 8)
  const int S = K / kDenseKC;
  const __amdgpu_buffer_rsrc_t rsg = dense_rsrc(a.Wg, (uint32_t)((size_t)K * N * 2));
  const __amdgpu_buffer_rsrc_t rsu = dense_rsrc(a.Wt, (uint32_t)((size_t)K * N * 2));
  const __amdgpu_buffer_rsrc_t rsh = dense_rsrc(a.H, (uint32_t)((size_t)min(a.hcap, 16 * MT) * K * 2));
  // wavefront w loads rows 8 w .. 8 w + 7 of each tile (1 KB); lane: row dr, slot dp
  const int dr = 8 * w + (lane >> 3), dp = lane & 7;
  const bool wv_ = dr < ncol;  // a weight row of this workgroup (else zeros, no memory access)
  const uint32_t ou = (uint32_t)(((size_t)(n0 + min(dr, ncol - 1)) * K + 8 * row_pos(dr, dp)) * 2);
  const uint32_t oh = (uint32_t)(((size_t)dr * K + 8 * row_pos(dr, dp)) * 2);
  bool hv = true;  // rows of the group (all rows until the group's size is known)
  const uint32_t sk = kDenseKC * 2;  // per stage
  f32x4v acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4v{0.f, 0.f, 0.f, 0.f};
#define SATS_GU_ISSUE(BUF, SN)                                                               \
  {                                                                                          \
    const bool v_ = (SN) < S;                                                                \
    const uint32_t ss_ = (uint32_t)(SN);                                                     \
    dma16<2>(rsg, (BUF) + w * 1024, dense_off(v_ && wv_, ou + ss_ * sk, 0));                 \
    dma16<2>(rsu, (BUF) + 8192 + w * 1024, dense_off(v_ && wv_, ou + ss_ * sk, 1));          \
    if (MT > 1 || w < 2) dma16<0>(rsh, (BUF) + 16384 + w * 1024, dense_off(v_ && hv, oh + ss_ * sk, 2)); \
  }
#define SATS_GU_COMPUTE(BUF)                                                                 \
  {                                                                                          \
    _Pragma("unroll") for (int j = 0; j < 2; ++j) {                                          \
      const bf16x8 b_ = row_operand((BUF) + 8192 * mat, c, j, g);                            \
      _Pragma("unroll") for (int mt = 0; mt < MT; ++mt)                                      \
        acc[mt] = mfma16(row_operand((BUF) + 16384, 16 * mt + l16, j, g), b_, acc[mt]);      \
    }                                                                                        \
  }
  // LoRA: this tile's adapter operands are loaded before the stream (16 bytes
  // per load: one each of B_gate[:, tile], B_up_T[tile] and A_down[tile] for
  // the first 8 R threads, up to four of s (h A)) and written to LDS after it
  const int R = LORA ? a.rank : 0;
  u32x4 pbg = {0u, 0u, 0u, 0u}, pbu = {0u, 0u, 0u, 0u}, pad = {0u, 0u, 0u, 0u}, plv[4];
  if (LORA) {
    const int t = threadIdx.x;
    if (t < 8 * R) {  // columns of the tile only (zeros past them)
      if (8 * (t & 7) < ncol) pbg = *reinterpret_cast<const u32x4 *>(a.Bg + (size_t)(t >> 3) * N + n0 + 8 * (t & 7));
      if (8 * t < ncol * R) {  // rows n0 .. n0 + ncol - 1: contiguous
        pbu = *reinterpret_cast<const u32x4 *>(a.BuT + (size_t)n0 * R + 8 * t);
        pad = *reinterpret_cast<const u32x4 *>(a.Ad + (size_t)n0 * R + 8 * t);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = t + kDenseThreads * j;  // 4 floats of lv [2][kDenseMaxTokens][R]
      plv[j] = (e < 32 * R) ? *reinterpret_cast<const u32x4 *>(a.lv + 4 * e) : u32x4{0u, 0u, 0u, 0u};
    }
  }
#define SATS_GU_GROUP                                                                        \
  if (!ctl_on) {                                                                             \
    __builtin_amdgcn_s_waitcnt(0);                                                           \
    return;                                                                                  \
  }                                                                                          \
  nd = min(ctl_n, 16 * MT);                                                                  \
  hv = dr < nd
  if constexpr (MT == 1) {
    SATS_DENSE_RING8_H(S, SATS_GU_ISSUE, SATS_GU_COMPUTE, SATS_GU_GROUP)
  } else {
    SATS_DENSE_RING_H(S, SATS_GU_ISSUE, SATS_GU_COMPUTE, SATS_GU_GROUP)
  }
#undef SATS_GU_GROUP
#undef SATS_GU_ISSUE
#undef SATS_GU_COMPUTE
  // epilogue: SiLU(a) through LDS to the W_up wavefronts, p through LDS to
  // 16-byte row stores
  __syncthreads();
  float *xs = reinterpret_cast<float *>(rg0);
  uint16_t *pt = reinterpret_cast<uint16_t *>(rg1);
  // LoRA: the adapter terms are small products on the same MFMA tiles.  The
  // gate term s (h A_gate) B_gate is added into the gate accumulators as a
  // product with K = 2 R: s (h A_gate) enters as two bf16 terms (hi, then the
  // rounded remainder lo) against B_gate twice, so it keeps about 16 bits;
  // the up term likewise with B_up_T.  K is padded to a whole MFMA step (32)
  // with zeros.  LDS (bf16):
  //   lvh [rows][KP]  hi | lo of s (h A) per group row (zero rows past the group)
  //   lbt [64][R]     B_gate^T / B_up_T of the tile's columns, ranks contiguous
  //   ladT [R][64]    A_down^T of the tile's columns, columns contiguous
  const int KP = R >= 16 ? 2 * R : 32;
  uint16_t *lvhg = reinterpret_cast<uint16_t *>(rg2), *lvhu = reinterpret_cast<uint16_t *>(rg3);
  uint16_t *lbgt = reinterpret_cast<uint16_t *>(rg4), *lbut = reinterpret_cast<uint16_t *>(rg5);
  uint16_t *ladt = reinterpret_cast<uint16_t *>(rg1 + 8192);
  if (LORA) {
    const int t = threadIdx.x;
    if (t < 8 * R) {
      const int i = t >> 3, q = t & 7;  // B_gate[i][n0 + 8 q .. + 7]
#pragma unroll
      for (int k = 0; k < 8; ++k)
        lbgt[(8 * q + k) * R + i] = (uint16_t)((k & 1) ? (pbg[k >> 1] >> 16) : (pbg[k >> 1] & 0xffffu));
      *reinterpret_cast<u32x4 *>(lbut + 8 * t) = pbu;  // B_up_T rows n0 .. n0 + 63 as they are
#pragma unroll
      for (int k = 0; k < 8; ++k) {  // element 8 t + k of A_down rows n0 ..: column (8 t + k) / R, rank (8 t + k) % R
        const int e = 8 * t + k;
        ladt[(e % R) * 64 + e / R] = (uint16_t)((k & 1) ? (pad[k >> 1] >> 16) : (pad[k >> 1] & 0xffffu));
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = t + kDenseThreads * j;
      if (e < 32 * R)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int fi = 4 * e + u, half = fi / (kDenseMaxTokens * R), rem = fi % (kDenseMaxTokens * R);
          const int m = rem / R, i = rem % R;
          const float v = m < nd ? __uint_as_float(plv[j][u]) : 0.0f;
          const uint16_t hi = f32_to_bf16(v);
          uint16_t *row = (half ? lvhu : lvhg) + m * KP;
          row[i] = hi;
          row[R + i] = f32_to_bf16(v - bf16_to_f32(hi));
        }
    }
    if (R < 16)  // K padding (columns 2 R .. 31 of every row)
      for (int e = t; e < 2 * kDenseMaxTokens * (KP - 2 * R); e += kDenseThreads) {
        const int half = e / (kDenseMaxTokens * (KP - 2 * R)), rem = e % (kDenseMaxTokens * (KP - 2 * R));
        (half ? lvhu : lvhg)[(rem / (KP - 2 * R)) * KP + 2 * R + rem % (KP - 2 * R)] = 0;
      }
    __syncthreads();
    // += [hi | lo] (rows of the tile) x [B; B] (columns c): lane operands as in the main loop
    const uint16_t *lvh = mat ? lvhu : lvhg, *lbt = mat ? lbut : lbgt;
    for (int j = 0; j < KP / 32; ++j) {
      const int k0 = 32 * j + 8 * g;
      const bf16x8 b_ = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(lbt + c * R + (k0 % R)));
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        acc[mt] = mfma16(__builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(lvh + (16 * mt + l16) * KP + k0)),
                         b_, acc[mt]);
    }
  }
  if (mat == 0) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) xs[(16 * mt + 4 * g + r) * kDenseXP + c] = silu(acc[mt][r]);
  }
  __syncthreads();
  if (a.cal_g) {  // calibration: g and p = g u (float32, no keep rule), p split into bf16 hi + lo
    if (mat == 1) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = 16 * mt + 4 * g + r;
          if (m < nd && c < ncol) {
            const float gv = xs[m * kDenseXP + c];
            const float pv = gv * acc[mt][r];
            const uint16_t hi = f32_to_bf16(pv);
            const size_t o = (size_t)m * N + n0 + c;
            a.cal_g[o] = gv;
            a.cal_ph[o] = hi;
            a.cal_pl[o] = f32_to_bf16(pv - bf16_to_f32(hi));
          }
        }
    }
    return;
  }
  if (mat == 1) {
    const float thr = a.thr ? *a.thr : 0.0f;
    bool any = false;  // some row of the group keeps column c
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = 16 * mt + 4 * g + r;
        if (m < nd) {
          const float gv = xs[m * kDenseXP + c];
          const bool keep = a.gbase[m] || fabsf(gv) >= thr;  // Eq. 4-5; every column on the base path
          pt[m * 64 + c] = keep ? f32_to_bf16(gv * acc[mt][r]) : (uint16_t)0;
          any = any || keep;
          if (a.keep_out && c < ncol) a.keep_out[(size_t)a.perm[m] * N + n0 + c] = (uint8_t)keep;
        }
      }
    // the four lanes of column c (g = 0..3) hold its rows; lane g = 0 publishes the union flag
    int u = any ? 1 : 0;
    u |= __shfl_xor(u, 16, 64);
    u |= __shfl_xor(u, 32, 64);
    if (a.uflag && g == 0 && c < ncol) a.uflag[n0 + c] = (uint8_t)u;
  }
  __syncthreads();
  const int lr = threadIdx.x >> 3, lq = threadIdx.x & 7;
  if (lr < nd && 8 * lq < ncol)
    *reinterpret_cast<u32x4 *>(a.P + (size_t)lr * N + n0 + 8 * lq) = *reinterpret_cast<const u32x4 *>(pt + lr * 64 + 8 * lq);
  if (LORA) {  // z partial of this column tile: p (as rounded for the down product) x A_down[tile], on MFMA
    const int nct = (R + 15) / 16;
    for (int tt = w; tt < MT * nct; tt += kDenseThreads / 64) {
      const int mt = tt / nct, ct = tt % nct, i = 16 * ct + l16;
      f32x4v z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int k0 = 32 * j + 8 * g;
        const u32x4 bw = i < R ? *reinterpret_cast<const u32x4 *>(ladt + i * 64 + k0) : u32x4{0u, 0u, 0u, 0u};
        z = mfma16(__builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(pt + (16 * mt + l16) * 64 + k0)),
                   __builtin_bit_cast(bf16x8, bw), z);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = 16 * mt + 4 * g + r;
        if (m < nd && i < R) a.zpart[((size_t)tile * kDenseMaxTokens + m) * R + i] = a.gbase[m] ? 0.0f : z[r];
      }
    }
  }
}

// partial y over one k chunk for 128 output columns; workgroup b takes
// column tile b / ks and k chunk b % ks, so that consecutive workgroups (which
// the dispatcher spreads over the 8 XCDs in turn) take different k chunks and
// each XCD's L2 fetches only its chunks of p, not all of it;
// wavefront w takes columns 16 w .. 16 w + 15.  A stage holds 64 W_down
// rows of 256 bytes (16 KB) and the matching 64 entries of p rows (8 KB).
//
// Rows of W_down that no row of the group keeps (their p column is zero for
// every row: the union of the keep sets excludes them) are not read: their
// loads take the offset past the buffer, which writes zeros to LDS without a
// memory access.  Each lane holds the union flags of its two rows in every
// stage of the chunk as a bit mask (up to kDownFlagStages stages; longer
// chunks read every row), formed while the first two stages, which read
// every row, are in flight.  With a base-path row in the group every flag is
// set and every row is read.
constexpr int kDownFlagStages = 32;

template <int MT>
__global__ __launch_bounds__(kDenseThreads) void dense_down_kernel(DenseArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t rg0[kDenseStageBytes], rg1[kDenseStageBytes],
      rg2[kDenseStageBytes], rg3[kDenseStageBytes], rg4[kDenseStageBytes], rg5[kDenseStageBytes];
  // the group's control words are read while the first two stages load (as
  // in the gate/up kernel)
  const int ctl_on = a.ctl[1], ctl_n = a.ctl[0];
  int nd = 16 * MT;
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4, l16 = lane & 15, c = 16 * w + l16;
  const int ks = gridDim.x / (a.N / kDenseDownNT), kc = blockIdx.x % ks;
  const int n0 = (blockIdx.x / ks) * kDenseDownNT;
  const int K = a.K, N = a.N;
  const int kb = kc * a.kchunk, ke = min(K, kb + a.kchunk);
  const int S = ke > kb ? (ke - kb) / kDenseKC : 0;
  const __amdgpu_buffer_rsrc_t rsw = dense_rsrc(a.Wb, (uint32_t)((size_t)K * N * 2));
  const __amdgpu_buffer_rsrc_t rsh = dense_rsrc(a.H, (uint32_t)((size_t)min(a.hcap, 16 * MT) * K * 2));
  // wavefront w loads W_down rows 8 w .. 8 w + 7 (two loads of 4 rows) and
  // p rows 8 w .. 8 w + 7
  const int wr = 8 * w + (lane >> 4), wp = lane & 15;
  const uint32_t ow0 = (uint32_t)(((size_t)(kb + wr) * N + n0 + 8 * krow_pos(wr, wp)) * 2);
  const uint32_t ow1 = (uint32_t)(((size_t)(kb + wr + 4) * N + n0 + 8 * krow_pos(wr + 4, wp)) * 2);
  const int hr = 8 * w + (lane >> 3), hp = lane & 7;
  const uint32_t oh = (uint32_t)(((size_t)hr * K + kb + 8 * row_pos(hr, hp)) * 2);
  bool hv = true;  // rows of the group (all rows until the group's size is known)
  const uint32_t sw = (uint32_t)kDenseKC * N * 2, sk = kDenseKC * 2;
  // bit 2 s (2 s + 1): row wr (wr + 4) of stage s is in the union of the keep
  // sets.  Lane t < S loads the flags of this wavefront's rows 8 w .. 8 w + 7
  // in stage t (8 bytes); one ballot per row gathers that row's flags over
  // the stages, and each lane interleaves the two rows it loads.  The flags'
  // load goes out first and the first two stages read every row, so the mask
  // is formed while they are in flight.
  const bool use_fl = a.uflag && S <= kDownFlagStages;
  const uint64_t f8 =
      (use_fl && lane < S) ? *reinterpret_cast<const uint64_t *>(a.uflag + kb + kDenseKC * lane + 8 * w) : 0ull;
  uint64_t fl = ~0ull;
  auto row_flags = [&]() -> uint64_t {
    if (!use_fl) return ~0ull;
    const int r0 = lane >> 4;  // wr = 8 w + r0
    uint64_t b0 = 0ull, b4 = 0ull;
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const uint64_t x0 = __ballot(((f8 >> (8 * rr)) & 0xffull) != 0ull);
      const uint64_t x4 = __ballot(((f8 >> (8 * (rr + 4))) & 0xffull) != 0ull);
      if (rr == r0) {
        b0 = x0;
        b4 = x4;
      }
    }
    auto spread = [](uint64_t v) {  // bit i to bit 2 i (i < 32)
      v &= 0xffffffffull;
      v = (v | (v << 16)) & 0x0000ffff0000ffffull;
      v = (v | (v << 8)) & 0x00ff00ff00ff00ffull;
      v = (v | (v << 4)) & 0x0f0f0f0f0f0f0f0full;
      v = (v | (v << 2)) & 0x3333333333333333ull;
      v = (v | (v << 1)) & 0x5555555555555555ull;
      return v;
    };
    return spread(b0) | (spread(b4) << 1);
  };
  f32x4v acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4v{0.f, 0.f, 0.f, 0.f};
#define SATS_DN_ISSUE(BUF, SN)                                                               \
  {                                                                                          \
    const bool v_ = (SN) < S;                                                                \
    const uint32_t ss_ = (uint32_t)(SN);                                                     \
    const bool f0_ = v_ && ((fl >> (2 * ((SN) & 31))) & 1ull);                              \
    const bool f1_ = v_ && ((fl >> (2 * ((SN) & 31) + 1)) & 1ull);                          \
    dma16<2>(rsw, (BUF) + w * 2048, dense_off(f0_, ow0 + ss_ * sw, 0));                      \
    dma16<2>(rsw, (BUF) + w * 2048 + 1024, dense_off(f1_, ow1 + ss_ * sw, 1));               \
    dma16<0>(rsh, (BUF) + 16384 + w * 1024, dense_off(v_ && hv, oh + ss_ * sk, 2));          \
  }
#define SATS_DN_COMPUTE(BUF)                                                                 \
  {                                                                                          \
    _Pragma("unroll") for (int j = 0; j < 2; ++j) {                                          \
      const bf16x8 b_ = krow_operand((BUF), 256, c, j, g);                                   \
      _Pragma("unroll") for (int mt = 0; mt < MT; ++mt)                                      \
        acc[mt] = mfma16(row_operand((BUF) + 16384, 16 * mt + l16, j, g), b_, acc[mt]);      \
    }                                                                                        \
  }
#define SATS_DN_GROUP                                                                        \
  if (!ctl_on) {                                                                             \
    __builtin_amdgcn_s_waitcnt(0);                                                           \
    return;                                                                                  \
  }                                                                                          \
  nd = min(ctl_n, 16 * MT);                                                                  \
  hv = hr < nd;                                                                              \
  fl = row_flags()
  SATS_DENSE_RING_H(S, SATS_DN_ISSUE, SATS_DN_COMPUTE, SATS_DN_GROUP)
#undef SATS_DN_GROUP
#undef SATS_DN_ISSUE
#undef SATS_DN_COMPUTE
  // through LDS to 16-byte row stores: rows 0-31 in one stage buffer, 32-63 in the next
  __syncthreads();
  constexpr int XP = 132;
  float *x0 = reinterpret_cast<float *>(rg0), *x1 = reinterpret_cast<float *>(rg1);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) (mt < 2 ? x0 : x1)[(16 * (mt & 1) + 4 * g + r) * XP + c] = acc[mt][r];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int e = threadIdx.x + i * kDenseThreads, m = e >> 5, q = e & 31;
    if (m < nd)
      *reinterpret_cast<f32x4v *>(a.part + ((size_t)kc * nd + m) * N + n0 + 4 * q) =
          *reinterpret_cast<const f32x4v *>((m < 32 ? x0 : x1) + (m & 31) * XP + 4 * q);
  }
}
// ---------------------------------------------------------------- SATS error curves
//
// Eq. 6 for one layer and up to 15 candidate thresholds t_0 <= ... <= t_14
// (missing ones +inf).  For calibration row m, y - y_t = sum over the
// neurons removed at t (|g_j| < t) of p_j W_down[j]; every candidate is one
// row of a product with W_down: row (m, r) of A is p_m masked to the
// neurons removed at t_r, and row (m, 15) is p_m itself (y).  The removed
// test is an integer compare: c[m][j] = #{r : t_r <= |g_mj|} counts the
// candidates at or below the neuron's magnitude, and neuron j is removed at
// t_r exactly when c <= r.  p enters as two bf16 terms (p = hi + lo, lo the
// rounded remainder), so that hi W + lo W carries about 16 bits of p into
// float32 accumulation.
//
// Each workgroup takes 16 calibration rows and 128 output columns and walks
// all of d_ff in stages of 64 k (W_down^T rows of the 128 columns 16 KB, hi
// and lo 2 KB each, c 1 KB) through a ring of 6 LDS stages.  Wavefront w
// owns calibration rows 2 w and 2 w + 1 over all 128 columns: it builds the
// masked A operands of its rows once per stage and multiplies them with the
// 8 column tiles of W_down^T, so that no two wavefronts build the same
// operand.  With PACK = 1 an A tile holds the 16 rows (15 candidates and y)
// of one calibration row; with PACK = 2 (at most 7 candidates) it holds two
// calibration rows of 8 (7 candidates and y), halving the MFMA work; with
// PACK = 4 (at most 4 candidates, ||y||^2 known) four calibration rows of 4
// and no y row, each wavefront over half of the 128 columns.
// W_down enters transposed (W_down^T, [d][d_ff], made by
// cal_transpose_kernel) so that each MFMA B operand is one 16-byte LDS read;
// chunk q of tile row r sits at q ^ (r & 7), so the eight rows read by eight
// consecutive lanes fall in distinct banks.  The operands of the first half
// of stage s + 1 are read and masked at the end of stage s (the stage
// barrier waits for two stages), so every stage starts with MFMAs; the
// second half's operands are masked while the first half's products run.
// Per row (m, r) the kernel writes the sum of the squares of its 128
// outputs, the partial of ||y - y_t||^2 (and ||y||^2, slot 15) for the
// column tile; cal_reduce_kernel finishes the norms.

struct CalErrArgs {
  const uint16_t *ph, *pl;  // [n][d_ff] bf16 hi and lo terms of p
  const uint8_t *cnt;       // [n][d_ff] candidates at or below |g|
  const uint16_t *WdT;      // W_down^T of the layer, [d][d_ff]
  float *part;              // [d / 128][n][16] column-tile sums of squares ([d / 64] with PACK 4)
  int n, d, d_ff;
};

constexpr int kCalRows = 16;  // calibration rows per workgroup (2 per wavefront)

__device__ __forceinline__ int ct_pos(int r, int q) { return q ^ (r & 7); }

// PACK = calibration rows per A tile: 1 (15 candidates and y), 2 (up to 7
// candidates and y), or 4 (up to 4 candidates, no y row: ||y||^2 comes from
// an earlier product).  With PACK 4 wavefront w takes calibration rows
// 4 (w & 3) .. 4 (w & 3) + 3 over the 64 columns of half w >> 2 of the tile,
// and its sums of squares go to part tile 2 blockIdx.x + (w >> 2).
template <int PACK>
__global__ __launch_bounds__(kDenseThreads) void cal_err_kernel(CalErrArgs a) {
  static_assert(PACK == 1 || PACK == 2 || PACK == 4, "one, two or four calibration rows per A tile");
  __shared__ __attribute__((aligned(1024))) uint8_t rg0[kDenseStageBytes], rg1[kDenseStageBytes],
      rg2[kDenseStageBytes], rg3[kDenseStageBytes], rg4[kDenseStageBytes], rg5[kDenseStageBytes];
  constexpr int CT = kDenseDownNT / 16 / (PACK == 4 ? 2 : 1);  // column tiles of 16 per wavefront
  constexpr int NA = PACK == 4 ? 1 : 2 / PACK;                 // A tiles per wavefront
  constexpr int RPT = 16 / PACK;                               // A rows per calibration row
  constexpr bool Y = PACK != 4;                                // the last of them is y
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ch = PACK == 4 ? w >> 2 : 0;  // column half (PACK 4)
  const int g = lane >> 4, l16 = lane & 15;
  const int n0 = blockIdx.x * kDenseDownNT, m0 = blockIdx.y * kCalRows;
  const int K = a.d_ff;
  const int S = K / kDenseKC;
  const __amdgpu_buffer_rsrc_t rsw = dense_rsrc(a.WdT, (uint32_t)((size_t)K * a.d * 2));
  const uint32_t pbytes = (uint32_t)((size_t)a.n * K * 2);
  const __amdgpu_buffer_rsrc_t rsh = dense_rsrc(a.ph, pbytes), rsl = dense_rsrc(a.pl, pbytes);
  const __amdgpu_buffer_rsrc_t rsc = dense_rsrc(a.cnt, (uint32_t)((size_t)a.n * K));
  // W_down^T row tile (128 rows of 128 bytes): wavefront w fills LDS slots
  // 128 w + 64 i + lane (i = 0, 1); slot s holds, at position s & 7 of tile
  // row s >> 3, the chunk whose position is ct_pos
  const int s0 = 128 * w + lane, s1 = s0 + 64;
  const int r0 = s0 >> 3, r1 = s1 >> 3;
  const uint32_t ow0 = (uint32_t)(((size_t)(n0 + r0) * K + 8 * ct_pos(r0, s0 & 7)) * 2);
  const uint32_t ow1 = (uint32_t)(((size_t)(n0 + r1) * K + 8 * ct_pos(r1, s1 & 7)) * 2);
  // hi and lo: wavefronts 0-1 and 2-3, 16 rows x 128 bytes each (lane: row, 16-byte chunk);
  // c: wavefront 4, 16 rows x 64 bytes
  const int ar = 8 * (w & 1) + (lane >> 3), aq = lane & 7;
  const bool arv = m0 + ar < a.n;
  const uint32_t oa = (uint32_t)(((size_t)(m0 + ar) * K + 8 * aq) * 2);
  const int cr = lane >> 2, cq = lane & 3;
  const bool crv = m0 + cr < a.n;
  const uint32_t oc = (uint32_t)((size_t)(m0 + cr) * K + 16 * cq);
  const uint32_t sk = kDenseKC * 2;
  // the third load of every wavefront, chosen without branches (wavefronts
  // 5-7 read zeros past the range into the stage's last 3 KB): a branch
  // around the loads would cost the compiler its record of which LDS buffer
  // each pending load writes, and with it waits on loads of later stages
  const __amdgpu_buffer_rsrc_t r3 = w < 2 ? rsh : (w < 4 ? rsl : rsc);
  const int d3 = w < 4 ? 16384 + w * 1024 : 20480 + (w - 4) * 1024;
  const bool v3 = w < 4 ? arv : (w == 4 && crv);
  const uint32_t o3 = w < 4 ? oa : oc, st3 = w < 4 ? sk : (uint32_t)kDenseKC;
  // A row of this lane: calibration row 2 w + t (tile t; PACK 4: 4 (w & 3) +
  // l16 / 4), candidate lim; with a y row the last row of a calibration row
  // is y (lim 15: every neuron)
  const int rr = l16 % RPT;
  const uint32_t lim = (Y && rr == RPT - 1) ? 15u : (uint32_t)rr;
  f32x4v acc[NA][CT];
#pragma unroll
  for (int t = 0; t < NA; ++t)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[t][ct] = f32x4v{0.f, 0.f, 0.f, 0.f};
  // two operand sets: the products of one half of a stage run while the
  // operands of the next half are read and masked (set 0: first halves)
  bf16x8 ah0[NA], al0[NA], bq0[CT], ah1[NA], al1[NA], bq1[CT];
  // stage buffer BUF, half j: this lane's masked A operands and the B operands
  auto load_ops = [&](const uint8_t *buf, int j, bf16x8(&ah)[NA], bf16x8(&al)[NA], bf16x8(&bq)[CT]) {
    const int k = 32 * j + 8 * g;
#pragma unroll
    for (int t = 0; t < NA; ++t) {
      const int row = PACK == 4 ? 4 * (w & 3) + l16 / RPT : 2 * w + (PACK == 1 ? t : l16 / RPT);
      const u32x4 hv = *reinterpret_cast<const u32x4 *>(buf + 16384 + row * 128 + 2 * k);
      const u32x4 lv = *reinterpret_cast<const u32x4 *>(buf + 18432 + row * 128 + 2 * k);
      const uint2 cv = *reinterpret_cast<const uint2 *>(buf + 20480 + row * 64 + k);
      u32x4 mh, ml;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t cw = q < 2 ? cv.x : cv.y;
        const uint32_t c0 = (cw >> (16 * (q & 1))) & 0xffu, c1 = (cw >> (16 * (q & 1) + 8)) & 0xffu;
        const uint32_t keep = (c0 <= lim ? 0x0000ffffu : 0u) | (c1 <= lim ? 0xffff0000u : 0u);
        mh[q] = hv[q] & keep;
        ml[q] = lv[q] & keep;
      }
      ah[t] = __builtin_bit_cast(bf16x8, mh);
      al[t] = __builtin_bit_cast(bf16x8, ml);
    }
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const int r = 16 * (CT * ch + ct) + l16;
      bq[ct] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(buf + r * 128 + ct_pos(r, 4 * j + g) * 16));
    }
  };
  auto mma = [&](const bf16x8(&ah)[NA], const bf16x8(&al)[NA], const bf16x8(&bq)[CT]) {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int t = 0; t < NA; ++t) acc[t][ct] = mfma16(ah[t], bq[ct], acc[t][ct]);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int t = 0; t < NA; ++t) acc[t][ct] = mfma16(al[t], bq[ct], acc[t][ct]);
  };
  // the schedule of one half: each product followed by a few of the other
  // half's operand instructions (VALU masks, LDS reads), so that the matrix
  // core and the vector unit work at once
  auto interleave = [&]() {
#pragma unroll
    for (int i = 0; i < 2 * NA * CT; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // an LDS read
      __builtin_amdgcn_sched_group_barrier(0x002, PACK == 4 ? 6 : 2, 0);  // VALU (PACK 4: 8 products a half)
    }
  };
#define SATS_CE_ISSUE(BUF, SN)                                                               \
  {                                                                                          \
    const bool v_ = (SN) < S;                                                                \
    const uint32_t ss_ = (uint32_t)(SN);                                                     \
    dma16<0>(rsw, (BUF) + w * 2048, dense_off(v_, ow0 + ss_ * sk, 0));                       \
    dma16<0>(rsw, (BUF) + w * 2048 + 1024, dense_off(v_, ow1 + ss_ * sk, 1));                \
    dma16<0>(r3, (BUF) + d3, dense_off(v_ && v3, o3 + ss_ * st3, 2));                        \
  }
  // step s: wait until stage s + 1 has landed (the loads of s + 2 .. s + 4,
  // nine, may be outstanding) and every wavefront is done with stage s - 1,
  // whose buffer takes stage s + 5; then stage s, whose first-half operands
  // are already in registers, with its second-half operands built under the
  // first half's products and the first-half operands of stage s + 1 under
  // the second half's (read but not used after the last stage)
#define SATS_CE_STEP(CUR, NXT, FREE, P)                                                      \
  {                                                                                          \
    const int s_ = s0_ + (P);                                                                \
    dense_stage_barrier<9>();                                                                \
    SATS_CE_ISSUE(FREE, s_ + 5);                                                             \
    if (s_ < S) {                                                                            \
      load_ops((CUR), 1, ah1, al1, bq1);                                                     \
      mma(ah0, al0, bq0);                                                                    \
      interleave();                                                                          \
      load_ops((NXT), 0, ah0, al0, bq0);                                                     \
      mma(ah1, al1, bq1);                                                                    \
      interleave();                                                                          \
    }                                                                                        \
  }
  SATS_CE_ISSUE(rg0, 0);
  SATS_CE_ISSUE(rg1, 1);
  SATS_CE_ISSUE(rg2, 2);
  SATS_CE_ISSUE(rg3, 3);
  SATS_CE_ISSUE(rg4, 4);
  dense_stage_barrier<12>();  // stage 0 has landed
  load_ops(rg0, 0, ah0, al0, bq0);
  for (int s0_ = 0; s0_ < S; s0_ += 6) {
    SATS_CE_STEP(rg0, rg1, rg5, 0)
    SATS_CE_STEP(rg1, rg2, rg0, 1)
    SATS_CE_STEP(rg2, rg3, rg1, 2)
    SATS_CE_STEP(rg3, rg4, rg2, 3)
    SATS_CE_STEP(rg4, rg5, rg3, 4)
    SATS_CE_STEP(rg5, rg0, rg4, 5)
  }
  __builtin_amdgcn_s_waitcnt(0);  // the zero-filling loads past the range land too
#undef SATS_CE_STEP
#undef SATS_CE_ISSUE
  // sums of squares over the wavefront's columns (128; PACK 4: 64): its
  // column tiles in order within the lane, then the 16 columns of a tile by
  // lane exchange.  Lane (g, l16) of tile t holds A rows 4 g .. 4 g + 3.
#pragma unroll
  for (int t = 0; t < NA; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = 0.0f;
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) v += acc[t][ct][r] * acc[t][ct][r];
#pragma unroll
      for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, 16);
      const int arow = 4 * g + r;
      const int m = m0 + (PACK == 4 ? 4 * (w & 3) + arow / RPT : 2 * w + (PACK == 1 ? t : arow / RPT));
      const int cand = arow % RPT;
      const int slot = (Y && cand == RPT - 1) ? 15 : cand;
      const int tile = PACK == 4 ? 2 * blockIdx.x + ch : blockIdx.x;
      if (l16 == 0 && m < a.n) a.part[((size_t)tile * a.n + m) * 16 + slot] = v;
    }
}

#undef SATS_DENSE_RING
#undef SATS_DENSE_RING_H
#undef SATS_DENSE_RING8_H
#undef SATS_DENSE_RING8
#undef SATS_DENSE_STEP8
#undef SATS_DENSE_STEP

struct GlueArgs {
  const int *ctl;
  const int *perm;
  const float *part;      // [KSPLIT][n_dense][d]
  int ksplit, d;
  uint16_t *out;          // last layer: [n][d] of the pass, rows through perm; else null
  uint16_t *hnext;        // otherwise: next layer input of the dense group, [n_dense][d]
  uint16_t *layer_in;     // optional: inspection copy of the next layer input, rows through perm
  // LoRA (zpart null: none): y += s z B_down for sparse-path rows, z the sum
  // over the nzb column tiles of zpart [nzb][kDenseMaxTokens][rank], in tile order
  const float *zpart;
  const uint16_t *Bd;     // [rank][d] of the layer
  const uint8_t *gbase;
  int rank, nzb;
  float lscale;
};

// one workgroup per dense token (blockIdx.x); thread t owns columns
// 4 t .. 4 t + 3 and issues its loads of every partial at once
constexpr int kGlueThreads = 1024;
__global__ __launch_bounds__(kGlueThreads) void dense_glue_kernel(GlueArgs a) {
  if (!a.ctl[1]) return;
  const int m = blockIdx.x;
  const int nd = a.ctl[0];
  if (m >= nd) return;
  __shared__ float ssw[kGlueThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c = 4 * tid;  // d <= 4096
  const bool on = c < a.d;
  // LoRA, sparse-path row: B_down[k][c .. c + 3] of the first 16 ranks, loaded
  // with the partials (it does not depend on z)
  const bool lora = a.zpart && !a.gbase[m];
  constexpr int kBdPre = 16;
  uint2 bpre[kBdPre];
#pragma unroll
  for (int k = 0; k < kBdPre; ++k)
    bpre[k] = (lora && on && k < a.rank) ? *reinterpret_cast<const uint2 *>(a.Bd + (size_t)k * a.d + c)
                                         : make_uint2(0u, 0u);
  f32x4v v[kDenseMaxKsplit];
#pragma unroll
  for (int q = 0; q < kDenseMaxKsplit; ++q)
    v[q] = (on && q < a.ksplit) ? *reinterpret_cast<const f32x4v *>(a.part + ((size_t)q * nd + m) * a.d + c)
                                : f32x4v{0.f, 0.f, 0.f, 0.f};
  f32x4v y = v[0];
#pragma unroll
  for (int q = 1; q < kDenseMaxKsplit; ++q) y += v[q];  // chunk order
  if (lora) {  // LoRA, sparse-path row: + s z B_down
    __shared__ float zf[kGlueThreads];
    __shared__ float zs[64];
    constexpr int Q = 16;  // tile groups (16 x rank <= 1024 threads)
    const int R = a.rank, i = tid % R, q = tid / R;
    // thread (q, i) adds tiles q, q + Q, ...; then the Q group sums in order
    if (q < Q)
      zf[tid] = (q < a.nzb) ? sum_coherent(a.zpart + ((size_t)q * kDenseMaxTokens + m) * R + i,
                                           (size_t)Q * kDenseMaxTokens * R, (a.nzb - q + Q - 1) / Q)
                            : 0.0f;
    __syncthreads();
    if (tid < R) {
      float zq[Q];
#pragma unroll
      for (int k = 0; k < Q; ++k) zq[k] = zf[k * R + tid];
      float z = 0.0f;
#pragma unroll
      for (int k = 0; k < Q; ++k) z += zq[k];
      zs[tid] = a.lscale * z;
    }
    __syncthreads();
    if (on) {
      f32x4v t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < kBdPre; ++k) {
        if (k < R) {
          t[0] = fmaf(zs[k], bf16_to_f32(bpre[k].x & 0xffffu), t[0]);
          t[1] = fmaf(zs[k], bf16_to_f32(bpre[k].x >> 16), t[1]);
          t[2] = fmaf(zs[k], bf16_to_f32(bpre[k].y & 0xffffu), t[2]);
          t[3] = fmaf(zs[k], bf16_to_f32(bpre[k].y >> 16), t[3]);
        }
      }
#pragma unroll 16
      for (int k = kBdPre; k < R; ++k) {
        const uint2 bw = *reinterpret_cast<const uint2 *>(a.Bd + (size_t)k * a.d + c);
        t[0] = fmaf(zs[k], bf16_to_f32(bw.x & 0xffffu), t[0]);
        t[1] = fmaf(zs[k], bf16_to_f32(bw.x >> 16), t[1]);
        t[2] = fmaf(zs[k], bf16_to_f32(bw.y & 0xffffu), t[2]);
        t[3] = fmaf(zs[k], bf16_to_f32(bw.y >> 16), t[3]);
      }
      y += t;
    }
  }
  const int row = a.perm[m];
  if (a.out) {
    if (on) {
      uint16_t *o = a.out + (size_t)row * a.d + c;
      o[0] = f32_to_bf16(y[0]);
      o[1] = f32_to_bf16(y[1]);
      o[2] = f32_to_bf16(y[2]);
      o[3] = f32_to_bf16(y[3]);
    }
    return;
  }
  float sq = y[0] * y[0];
  sq = fmaf(y[1], y[1], sq);
  sq = fmaf(y[2], y[2], sq);
  sq = fmaf(y[3], y[3], sq);
  sq = wave_sum(sq);
  if (lane == 0) ssw[wv] = sq;
  __syncthreads();
  float tot = 0.0f;
  for (int i = 0; i < kGlueThreads / 64; ++i) tot += ssw[i];
  const float scale = sqrtf(tot / (float)a.d + kGlueEps);
  if (on) {
    uint16_t h[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) h[i] = f32_to_bf16(y[i] / scale);
    const uint2 hv = make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
    *reinterpret_cast<uint2 *>(a.hnext + (size_t)m * a.d + c) = hv;
    if (a.layer_in) *reinterpret_cast<uint2 *>(a.layer_in + (size_t)row * a.d + c) = hv;
  }
}

// ---------------------------------------------------------------- LoRA, batched

// s (h A) for the group rows and both input-side adapters (A_gate, A_up) of
// a layer, the operands of the gate/up epilogue's adapter terms.  Grid
// (kLoraVChunks k chunks, 4 row tiles of 16, 2 adapters), 256 threads:
// thread (k slice, row r, ranks 4 q .. 4 q + 3) sums one of the 64 / R slices
// of its chunk's k in order from LDS copies of the chunk (so every rank keeps
// all 256 threads busy), and the slices are added in order; the chunk
// partials go to vpart, and the last chunk of a (row tile, adapter) to
// arrive adds them in chunk order.  Base-path rows get zeros (their layers
// see the base weights only).
constexpr int kLoraVChunks = 16;
constexpr int kLoraVMaxChunk = 4096 / kLoraVChunks;  // k rows per chunk (d <= 4096)
constexpr int kLoraVMaxRank = 64;    // ranks 8, 16, 32, 64
struct LoraVArgs {
  const int *ctl;          // [0] rows of the group, [1] MFMA path on
  const uint8_t *gbase;
  const uint16_t *H;       // [rows][K] bf16 layer input of the group
  const uint16_t *Ag, *Au; // [K][R] of the layer
  float *vpart;            // [2][4][kLoraVChunks][16][R]
  float *lv;               // [2][kDenseMaxTokens][R]
  unsigned *cnt;           // [8] arrival counts (zero between launches)
  int K, R;
  float s;
};
__global__ __launch_bounds__(256) void lora_v_kernel(LoraVArgs a) {
  __shared__ uint16_t hs[16 * kLoraVMaxChunk];
  __shared__ uint16_t as[kLoraVMaxChunk * kLoraVMaxRank];
  __shared__ int flag;
  if (!a.ctl[1]) return;
  const int nd = min(a.ctl[0], kDenseMaxTokens);
  const int ch = blockIdx.x, mt = blockIdx.y, ad = blockIdx.z, tid = threadIdx.x;
  if (16 * mt >= nd) return;  // the whole (row tile, adapter) returns: no arrivals
  const int R = a.R, kch = a.K / kLoraVChunks, k0 = ch * kch;
  const uint16_t *A = ad ? a.Au : a.Ag;
  // stage the chunk: 16 rows of h (rows past the group as zeros) and kch rows of A, 16 bytes per load
  for (int e = tid; e < 16 * kch / 8; e += 256) {
    const int r = e / (kch / 8), q = e % (kch / 8), m = 16 * mt + r;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (m < nd) v = *reinterpret_cast<const u32x4 *>(a.H + (size_t)m * a.K + k0 + 8 * q);
    *reinterpret_cast<u32x4 *>(hs + r * kch + 8 * q) = v;
  }
  {  // A's chunk: at most kLoraVMaxChunk * kLoraVMaxRank / 8 / 256 = 8 16-byte loads per thread, all issued first
    constexpr int kAPer = kLoraVMaxChunk * kLoraVMaxRank / 8 / 256;
    u32x4 av[kAPer];
#pragma unroll
    for (int j = 0; j < kAPer; ++j) {
      const int e = tid + 256 * j;
      av[j] = e < kch * R / 8 ? *reinterpret_cast<const u32x4 *>(A + (size_t)k0 * R + 8 * e) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < kAPer; ++j) {
      const int e = tid + 256 * j;
      if (e < kch * R / 8) *reinterpret_cast<u32x4 *>(as + 8 * e) = av[j];
    }
  }
  __syncthreads();
  // thread (slice sl of NS, row r, ranks 4 q .. 4 q + 3): NS = 64 / R slices of
  // the chunk's k, each summed in k order; the slices are then added in order
  const int Q4 = R / 4, NS = 64 / R;
  const int sl = tid / (16 * Q4), r = (tid / Q4) % 16, q = tid % Q4;
  // slice bounds on multiples of 8 k (16-byte LDS reads of h); kch is a multiple of 8
  const int kb = (sl * kch / NS) & ~7, ke = (sl == NS - 1) ? kch : ((sl + 1) * kch / NS) & ~7;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  int k = kb;
  for (; k + 8 <= ke; k += 8) {
    const u32x4 hv = *reinterpret_cast<const u32x4 *>(hs + r * kch + k);
    uint2 w[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) w[e] = *reinterpret_cast<const uint2 *>(as + (k + e) * R + 4 * q);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float h = bf16_to_f32((e & 1) ? (hv[e >> 1] >> 16) : (hv[e >> 1] & 0xffffu));
      acc[0] = fmaf(h, bf16_to_f32(w[e].x & 0xffffu), acc[0]);
      acc[1] = fmaf(h, bf16_to_f32(w[e].x >> 16), acc[1]);
      acc[2] = fmaf(h, bf16_to_f32(w[e].y & 0xffffu), acc[2]);
      acc[3] = fmaf(h, bf16_to_f32(w[e].y >> 16), acc[3]);
    }
  }
  for (; k < ke; ++k) {
    const float h = bf16_to_f32(hs[r * kch + k]);
    const uint2 w = *reinterpret_cast<const uint2 *>(as + k * R + 4 * q);
    acc[0] = fmaf(h, bf16_to_f32(w.x & 0xffffu), acc[0]);
    acc[1] = fmaf(h, bf16_to_f32(w.x >> 16), acc[1]);
    acc[2] = fmaf(h, bf16_to_f32(w.y & 0xffffu), acc[2]);
    acc[3] = fmaf(h, bf16_to_f32(w.y >> 16), acc[3]);
  }
  float *red = reinterpret_cast<float *>(as);  // [NS][16][R], after every thread is done with the chunk
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) red[(sl * 16 + r) * R + 4 * q + j] = acc[j];
  __syncthreads();
  const bool act = sl == 0;
  if (act)
    for (int s2 = 1; s2 < NS; ++s2)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] += red[(s2 * 16 + r) * R + 4 * q + j];
  float *vp = a.vpart + ((size_t)(ad * 4 + mt) * kLoraVChunks) * 16 * R;  // [chunk][16][R]
  if (act)
#pragma unroll
    for (int j = 0; j < 4; ++j) store_coherent(vp + ((size_t)ch * 16 + r) * R + 4 * q + j, acc[j]);
  if (!arrive_last(a.cnt + ad * 4 + mt, gridDim.x, &flag)) return;
  const int m = 16 * mt + r;
  if (act && m < nd) {
    float v[4][kLoraVChunks];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int c2 = 0; c2 < kLoraVChunks; ++c2) v[j][c2] = load_coherent(vp + ((size_t)c2 * 16 + r) * R + 4 * q + j);
    const bool base = a.gbase[m];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float t = 0.0f;
#pragma unroll
      for (int c2 = 0; c2 < kLoraVChunks; ++c2) t += v[j][c2];  // chunk order
      a.lv[((size_t)ad * kDenseMaxTokens + m) * R + 4 * q + j] = base ? 0.0f : a.s * t;
    }
  }
}

}  // namespace sats
