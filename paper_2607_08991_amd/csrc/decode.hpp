// Single-token (decode batch 1) path: one layer is one launch plus the
// second reduction stage.
//
//   layer   Workgroup w owns the gate columns [cw w, cw w + cw) (cw <= 64).
//           Its wavefronts read whole rows of W_gate^T, one column's d
//           weights contiguous, and form a_j = h . W_gate[:, j] in a fixed
//           order; then SiLU (Eq. 2) and the keep rule (Eq. 4-5, or every
//           column on the base path, Eq. 13) give the workgroup's own kept
//           list in LDS, and its two halves stream the listed rows of W_up_T
//           and W_down: u_j = W_up_T[j] . h, p_j = g_j u_j (Eq. 1) and
//           p_j W_down[j] summed into the workgroup's partial y.  No value
//           crosses workgroups inside the launch: there is no hand-off to
//           wait for, and the row reads of one workgroup overlap the gate
//           reads of the others.
//   reduce  Workgroup w adds every partial for its own slice of columns in
//           workgroup order: y, or the rounded output on the last layer, and
//           the slice's sum of squares for the next layer's input
//           rho(y / sqrt(mean(y^2) + 1e-6)).
//
// With LoRA adapters (Section 5) a small launch first forms h A_gate and
// h A_up, and the reduction adds the down adapter.
//
// Workgroups have 1024 threads (16 wavefronts per CU keep enough reads in
// flight).  The assignment of work depends only on the data, never on
// timing, so every sum has a fixed order and results are reproducible bit
// for bit.
#pragma once

#include "kernels.hpp"

namespace sats {

// Optional phase timestamps (build with -DSATS_TRACE): per workgroup, wall
// clock at fixed points of the first layer, read back with sats_trace_read().
#ifdef SATS_TRACE
__device__ unsigned long long sats_trace_buf[4096 * 16];
#define SATS_TRACE_POINT(i)                                                               \
  do {                                                                                    \
    if (threadIdx.x == 0 && blockIdx.x < 4096) sats_trace_buf[blockIdx.x * 16 + (i)] = wall_clock64(); \
  } while (0)
#else
#define SATS_TRACE_POINT(i) \
  do {                      \
  } while (0)
#endif

constexpr int kDecodeThreads = 1024;  // layer, LoRA input and LoRA reduce launches
constexpr int kDecodeWaves = kDecodeThreads / 64;
constexpr int kDecodeMaxD = 4096;     // h lives in LDS
constexpr int kDecodeMaxCols = 64;    // gate columns of a workgroup (one wavefront ballot)
constexpr int kDecodeMaxG = 4096;     // layer workgroups (partials of y)
constexpr int kRedThreads = 256, kRedCols = 16;  // second reduction stage: threads and columns per workgroup
constexpr int kGateQ = 4;             // 16-byte loads per lane in one gate piece
constexpr int kWarmRows = 8;          // next-layer W_gate rows an early workgroup warms (stacks)
constexpr int kVRows = 256;           // input rows per workgroup of the LoRA input launch

struct DecodeArgs {
  const void *x;          // [d] call input (storage type)
  void *out;              // [d]
  const void *Wg, *Wu, *Wd;  // stacked weights, each [L][d_ff][d]: W_gate^T, W_up_T, W_down
  const float *thr;       // [L] (unused on the base path)
  const int32_t *ids;
  const uint8_t *lut;
  int route_mode;
  int L, d, d_ff;
  int cw;                 // gate columns per layer workgroup
  float *ypart;           // [G][d]         per-workgroup partial y
  float *ybuf;            // [d]
  float *sspart;          // [nss]          sums of y^2 per 16 columns
  int G, RW;              // layer workgroups (partials of y), reduce workgroups
  int nss;                // slice sums of squares of y per layer: one per 16 columns
  int fused_reduce;       // 1: the last layer workgroup to finish does the second stage (small layers)
  unsigned *done;         // [1] layer workgroups finished (fused_reduce; the last one resets it)
  uint8_t *route_out;     // optional [1]
  uint8_t *keep_out;      // optional [L][d_ff]
  void *layer_in;         // optional [L][...]: layer l's input at layer_in + l * in_stride
  int64_t in_stride;      // elements between the layers' inputs in layer_in
  // LoRA adapters of the sparse path (Ag null: none), stacked per layer like
  // the weights: Ag, Au [d][rank], Bg [rank][d_ff], BuT, Ad [d_ff][rank],
  // Bd [rank][d]; lscale multiplies every adapter product
  const void *Ag, *Bg, *Au, *BuT, *Ad, *Bd;
  int rank;
  float lscale;
  float *vpart;           // [nvc][2][rank] per input row chunk: partial h . A_gate, h . A_up
  int nvc;                // row chunks of the LoRA input launch
  float *zpart;           // [G][rank]      per layer workgroup: sum of p_j A_down[j] over its kept rows
};

constexpr int kLoraMaxRank = 64;  // ranks 8, 16, 32, 64

struct DecodeSmem {
  float hs[kDecodeMaxD];                // layer input (zero past d)
  u32x4 hq[kDecodeMaxD * 4 / 16];       // the same, packed in the storage type (gate reads, 16 bytes a load)
  float red[2 * kDecodeMaxD];           // column sums; rows: parts of u, half sums; reduce: partial groups
  int mj[kDecodeMaxCols];               // kept columns of the workgroup ...
  float mg[kDecodeMaxCols];             // ... and their g values
  int wcnt[kDecodeWaves];
  float scal[kDecodeWaves];
  int flag;
  float lv[2][kDecodeWaves][kLoraMaxRank];  // LoRA: wavefront partials (input launch), gate adapter terms
  float lvg[kLoraMaxRank];                   // LoRA: h . A_gate
  float lz[kLoraMaxRank];                    // LoRA: h . A_up (layer) or z (reduce)
};

// LoRA operands of the workgroup's kept rows (list position i): the up
// adapter's contribution w_i = s (h A_up) . B_up_T[j] and A_down[j].
template <typename T>
struct LoraRows {
  float lw[kDecodeMaxCols];
  T lad[kDecodeMaxCols * kLoraMaxRank];  // [list position][rank]
};

// Four consecutive floats at byte offset voff of buffer r, written through to
// the device-coherent level in one 16-byte store.  (A compiler builtin, not
// inline assembly: the compiler's hazard checks do not see a store written as
// assembly, and a following write to its data registers can then corrupt the
// stored values.)
__device__ __forceinline__ void store_coherent4(__amdgpu_buffer_rsrc_t r, uint32_t voff, float x0, float x1, float x2,
                                                float x3) {
  const f32x4 v = {x0, x1, x2, x3};
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)voff, 0, 16 /* write through */);
}

// Weight reads (and the partial-y writes) go through buffer descriptors: the matrix base lives in
// scalar registers, the row offset in a scalar register and only the lane's
// byte offset in a vector register, so a batch of loads needs no 64-bit
// address per load.  Reads at or past `bytes` return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t weight_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
// Byte offset that is out of range of every buffer here (all are smaller
// than 2 GB): a buffer load at it returns zeros without a memory access.
constexpr uint32_t kOffNone = 0x80000000u;
// s_waitcnt operand for vmcnt(0) alone (expcnt and lgkmcnt at their maxima)
constexpr int kWaitVm0 = 0x0F70;

// 16 bytes at base + soff + voff, not kept in the caches (streamed once).
__device__ __forceinline__ u32x4 load_rsrc(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 2);
}


// Sums of R values over the 64 lanes of a wavefront (R a power of two),
// by halving exchanges: at the step with lane mask m each lane keeps half of
// its values and adds its partner's matching half, then the last values are
// added across the remaining lanes.  Lanes r * (64 / R) ... (r + 1) * (64 / R)
// - 1 return the sum of value r.  17 exchanges for R = 16 instead of 96.
template <int R>
__device__ __forceinline__ float rows_sum(float (&v)[R], int lane) {
  static_assert(R >= 1 && R <= 64 && (R & (R - 1)) == 0, "R must be a power of two");
#pragma unroll
  for (int m = 32, h = R / 2; h >= 1; m >>= 1, h >>= 1) {
    const bool hi = (lane & m) != 0;
#pragma unroll
    for (int i = 0; i < h; ++i) {
      const float send = hi ? v[i] : v[i + h];
      const float keep = hi ? v[i + h] : v[i];
      v[i] = keep + __shfl_xor(send, m, 64);
    }
  }
  float s = v[0];
#pragma unroll
  for (int m = 32 / R; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
  return s;
}

// ------------------------------------------------------------------ layer input

// Layer input h, in two steps so that its loads overlap others: issue()
// starts the loads of the call input (layer 0) or of the previous layer's y
// and the G slice sums of squares; finish() forms
// h = rho(y / sqrt(mean(y^2) + 1e-6)) into LDS (and the inspection copy when
// `record`).
// slice sums of squares (one per 16 columns of y) per thread
template <int THREADS> constexpr int kSlicesPer() { return (kDecodeMaxD / kRedCols + THREADS - 1) / THREADS; }

template <int THREADS>
struct InputRegs {
  u32x4 xv[kDecodeMaxD / (4 * THREADS)];  // layer 0: x, 16 bytes at a time (d <= 4096)
  float yv[kDecodeMaxD / THREADS];
  float ss[kSlicesPer<THREADS>()];
};

template <typename T, int THREADS>
__device__ __forceinline__ void dec_input_issue(const DecodeArgs &a, int l, InputRegs<THREADS> &r) {
  const int G = a.nss;  // slice sums of squares of the previous layer's reduce
  constexpr int VEC = Elem<T>::kVec;
  const int tid = threadIdx.x, d = a.d;
  // every field gets a value on both branches: finish() passes all of them
  // through register constraints
#pragma unroll
  for (int i = 0; i < kDecodeMaxD / (4 * THREADS); ++i) r.xv[i] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
  for (int i = 0; i < kDecodeMaxD / THREADS; ++i) r.yv[i] = 0.0f;
#pragma unroll
  for (int i = 0; i < kSlicesPer<THREADS>(); ++i) r.ss[i] = 0.0f;
  if (l == 0) {
#pragma unroll
    for (int i = 0; i < kDecodeMaxD / (4 * THREADS); ++i) {
      const int k0 = (i * THREADS + tid) * VEC;
      r.xv[i] = (k0 < d) ? *reinterpret_cast<const u32x4 *>(static_cast<const T *>(a.x) + k0)
                         : u32x4{0u, 0u, 0u, 0u};
    }
  } else {
#pragma unroll
    for (int i = 0; i < kDecodeMaxD / THREADS; ++i) r.yv[i] = load_coherent(a.ybuf + min(i * THREADS + tid, d - 1));
#pragma unroll
    for (int i = 0; i < kSlicesPer<THREADS>(); ++i)
      r.ss[i] = (tid + i * THREADS < G) ? load_coherent(a.sspart + tid + i * THREADS) : 0.0f;
  }
}

template <typename T, int THREADS>
__device__ __forceinline__ void dec_input_finish(const DecodeArgs &a, int l, InputRegs<THREADS> &r, DecodeSmem &sm,
                                                 bool record) {
  constexpr int VEC = Elem<T>::kVec, NW = THREADS / 64;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d = a.d;
  // The values are first used here, not earlier: keeps the compiler from
  // hoisting their use (and the wait for their loads) above loads issued in
  // between.
#pragma unroll
  for (int i = 0; i < kDecodeMaxD / THREADS; ++i) asm volatile("" : "+v"(r.yv[i])::"memory");
#pragma unroll
  for (int i = 0; i < kSlicesPer<THREADS>(); ++i) asm volatile("" : "+v"(r.ss[i])::"memory");
#pragma unroll
  for (int i = 0; i < kDecodeMaxD / (4 * THREADS); ++i) asm volatile("" : "+v"(r.xv[i])::"memory");
  if (l == 0) {
#pragma unroll
    for (int i = 0; i < kDecodeMaxD / (4 * THREADS); ++i) {
      const int k0 = (i * THREADS + tid) * VEC;
      if (k0 < d) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) sm.hs[k0 + v] = unpack<T>(r.xv[i], v);
        if (record) *reinterpret_cast<u32x4 *>(static_cast<T *>(a.layer_in) + k0) = r.xv[i];
      }
    }
  } else {
    float s = 0.0f;  // total sum of squares of y, in a fixed order
#pragma unroll
    for (int i = 0; i < kSlicesPer<THREADS>(); ++i) s += r.ss[i];
    s = wave_sum(s);
    if (lane == 0) sm.scal[wv] = s;
    __syncthreads();
    float tot = 0.0f;
    for (int i = 0; i < NW; ++i) tot += sm.scal[i];
    const float scale = sqrtf(tot / (float)d + kGlueEps);
#pragma unroll
    for (int i = 0; i < kDecodeMaxD / THREADS; ++i) {
      const int k = i * THREADS + tid;
      if (k < d) {
        const T hv = Elem<T>::round(r.yv[i] / scale);
        sm.hs[k] = Elem<T>::value(hv);
        if (record) static_cast<T *>(a.layer_in)[(size_t)l * a.in_stride + k] = hv;
      }
    }
  }
  __syncthreads();
}


// ------------------------------------------------------------------ LoRA input

// The sparse path of a fine-tuned routed model adds s A B to each projection
// (Section 5).  h A_gate and h A_up (rank values each) are formed once per
// layer by a launch of their own: workgroup c takes input rows
// [kVRows c, kVRows c + kVRows) of both A matrices and writes its partial
// sums; the layer launch adds the chunks in order.  The gate adapter term
// s (h A_gate) . B_gate[:, j] is added to a_j, the up adapter term
// s (h A_up) . B_up_T[j] to u_j of each kept row, and the down adapter's
// first factor z = sum p_j A_down[j] is summed next to each partial y; the
// second reduction stage adds s z B_down.
template <typename T>
__global__ __launch_bounds__(kDecodeThreads) void dec_lora_v_kernel(DecodeArgs a, int l) {
  __shared__ DecodeSmem sm;
  constexpr int VEC = Elem<T>::kVec;
  constexpr int M = kVRows * kLoraMaxRank / (VEC * kDecodeThreads);  // passes at the largest rank
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int R = a.rank, RQ = R / VEC;  // 16-byte pieces per row of an A matrix
  const int k0 = blockIdx.x * kVRows, kn = max(0, min(a.d, k0 + kVRows) - k0);
  const size_t al = (size_t)a.d * R;
  const __amdgpu_buffer_rsrc_t rg = weight_rsrc(static_cast<const T *>(a.Ag) + (size_t)l * al, (uint32_t)(al * sizeof(T)));
  const __amdgpu_buffer_rsrc_t ru = weight_rsrc(static_cast<const T *>(a.Au) + (size_t)l * al, (uint32_t)(al * sizeof(T)));
  // piece p = tid + kDecodeThreads m: row k0 + p / RQ, ranks VEC (p % RQ) ..
  // (p % RQ = lane % RQ: RQ divides 64)
  u32x4 qg[M], qu[M];
#pragma unroll
  for (int m = 0; m < M; ++m) {
    const int p = tid + m * kDecodeThreads;
    const uint32_t off = p < kn * RQ ? (uint32_t)(((size_t)k0 * R + (size_t)p * VEC) * sizeof(T)) : kOffNone;
    qg[m] = load_rsrc(rg, off, 0);
    qu[m] = load_rsrc(ru, off, 0);
  }
  InputRegs<kDecodeThreads> ir;
  dec_input_issue<T, kDecodeThreads>(a, l, ir);
  dec_input_finish<T, kDecodeThreads>(a, l, ir, sm, false);
  float sg[VEC], su[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) sg[v] = su[v] = 0.0f;
#pragma unroll
  for (int m = 0; m < M; ++m) {
    const int p = tid + m * kDecodeThreads;
    if (p < kn * RQ) {
      const float hv = sm.hs[k0 + p / RQ];
#pragma unroll
      for (int v = 0; v < VEC; ++v) {
        sg[v] = fmaf(hv, unpack<T>(qg[m], v), sg[v]);
        su[v] = fmaf(hv, unpack<T>(qu[m], v), su[v]);
      }
    }
  }
  // lanes of equal lane % RQ hold the same ranks: halving exchanges add them
  for (int msk = 32; msk >= max(RQ, 1); msk >>= 1)
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      sg[v] += __shfl_xor(sg[v], msk, 64);
      su[v] += __shfl_xor(su[v], msk, 64);
    }
  if (lane < RQ) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      sm.lv[0][wv][lane * VEC + v] = sg[v];
      sm.lv[1][wv][lane * VEC + v] = su[v];
    }
  }
  __syncthreads();
  if (tid < 2 * R) {  // the wavefronts' sums in order
    const int ad = tid / R, i = tid % R;
    float s = 0.0f;
    for (int q = 0; q < kDecodeWaves; ++q) s += sm.lv[ad][q][i];
    store_coherent(a.vpart + ((size_t)blockIdx.x * 2 + ad) * R + i, s);
  }
}

// ------------------------------------------------------------------ gate

// The gate columns of a workgroup: wavefront wv takes columns wv, wv + 16,
// ... of the block, each a row of W_gate^T read in pieces of kGateQ 16-byte
// loads per lane (npc pieces per row); P pieces in all for this wavefront.
struct GatePieces {
  int c0, nc, npc, P, wv;
};

template <typename T>
__device__ __forceinline__ void gate_piece_issue(__amdgpu_buffer_rsrc_t wr, const GatePieces &gp, int d, int p,
                                                 u32x4 (&q)[kGateQ]) {
  const int lane = threadIdx.x & 63;
  const int cl = min(gp.wv + 16 * (p / gp.npc), gp.nc - 1), qi = p % gp.npc;  // wavefront-uniform
  const uint32_t row_bytes = (uint32_t)d * (uint32_t)sizeof(T);
  const uint32_t soff = (uint32_t)(gp.c0 + cl) * row_bytes;
#pragma unroll
  for (int u = 0; u < kGateQ; ++u) {
    const uint32_t byte = (uint32_t)((qi * kGateQ + u) * 64 + lane) * 16u;
    q[u] = load_rsrc(wr, (p < gp.P && byte < row_bytes) ? byte : kOffNone, soff);
  }
}

// Adds a piece's products to acc (even and odd elements apart); after a
// column's last piece the wavefront sum (lanes in a fixed order) goes to
// colsum[column] and acc restarts.  Each weight load meets the 16 bytes of
// packed h at the same elements (zero past d; the weights past the row are
// read as zeros).
template <typename T>
__device__ __forceinline__ void gate_piece_use(const DecodeSmem &sm, const GatePieces &gp, int p,
                                               const u32x4 (&q)[kGateQ], float (&acc)[2], float *colsum) {
  constexpr int VEC = Elem<T>::kVec;
  const int lane = threadIdx.x & 63, qi = p % gp.npc;
  u32x4 hv[kGateQ];
#pragma unroll
  for (int u = 0; u < kGateQ; ++u) hv[u] = sm.hq[(qi * kGateQ + u) * 64 + lane];  // at most 16 KB of a row
#pragma unroll
  for (int u = 0; u < kGateQ; ++u)
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v & 1] = fmaf(unpack<T>(hv[u], v), unpack<T>(q[u], v), acc[v & 1]);
  if (qi == gp.npc - 1) {
    const float s = wave_sum(acc[0] + acc[1]);
    if (lane == 0) colsum[gp.wv + 16 * (p / gp.npc)] = s;
    acc[0] = acc[1] = 0.0f;
  }
}

// h (in LDS as float, zero past d) packed in the storage type: exact, h is
// rounded to it.
template <typename T>
__device__ __forceinline__ void pack_input(DecodeSmem &sm) {
  constexpr int VEC = Elem<T>::kVec, NP = kDecodeMaxD * (int)sizeof(T) / 16;
  for (int i = threadIdx.x; i < NP; i += kDecodeThreads) {
    const f32x4 *src = reinterpret_cast<const f32x4 *>(sm.hs + i * VEC);
    u32x4 q;
    if constexpr (sizeof(T) == 2) {
      const f32x4 lo = src[0], hi = src[1];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        q[j] = (uint32_t)f32_to_bf16(lo[2 * j]) | ((uint32_t)f32_to_bf16(lo[2 * j + 1]) << 16);
        q[j + 2] = (uint32_t)f32_to_bf16(hi[2 * j]) | ((uint32_t)f32_to_bf16(hi[2 * j + 1]) << 16);
      }
    } else {
      q = __builtin_bit_cast(u32x4, src[0]);
    }
    sm.hq[i] = q;
  }
}

// ------------------------------------------------------------------ rows

// The workgroup's wavefronts form 16 / HW row groups of HW wavefronts
// (HW = 8 for rows of more than 4 chunks, 4 or 2 for shorter ones, so that
// no wavefront idles on a short row); group gr takes its own part of the
// kept list, and wavefront v of a group owns column chunks v, v + HW, ... of
// d (64 lanes x 16 bytes each) for both projections.

// One batch: loads of this wavefront's chunks of the kept rows
// list[r0 + r], r < R.  Every load is issued: rows at or past `end` (and
// chunks past d) read at kOffNone, zeros without a memory access, so no
// branch or zero fill sits between the loads and nothing waits on them here.
template <typename T, int R, int NCH, int HW>
__device__ __forceinline__ void rows_issue(__amdgpu_buffer_rsrc_t Wu, __amdgpu_buffer_rsrc_t Wd, const DecodeSmem &sm,
                                           int r0, int end, int d, u32x4 (&bu)[R][NCH], u32x4 (&bd)[R][NCH]) {
  constexpr int VEC = Elem<T>::kVec, CH = 64 * VEC;
  const int lane = threadIdx.x & 63, hw = __builtin_amdgcn_readfirstlane((threadIdx.x >> 6) % HW);
  uint32_t soff[R];  // zero for rows past the end (kOffNone is then out of range whatever the row)
#pragma unroll
  for (int r = 0; r < R; ++r)
    soff[r] = r0 + r < end ? (uint32_t)((size_t)__builtin_amdgcn_readfirstlane(sm.mj[r0 + r]) * d * sizeof(T)) : 0u;
  // all rows of W_up_T first: the up products can start while W_down arrives
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int k = (hw + c * HW) * CH + lane * VEC;
      bu[r][c] = load_rsrc(Wu, (k < d && r0 + r < end) ? (uint32_t)(k * sizeof(T)) : kOffNone, soff[r]);
    }
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int k = (hw + c * HW) * CH + lane * VEC;
      bd[r][c] = load_rsrc(Wd, (k < d && r0 + r < end) ? (uint32_t)(k * sizeof(T)) : kOffNone, soff[r]);
    }
}

// Uses one batch: this wavefront's parts of u_j = W_up_T[j] . h go to its
// group's LDS slot `par`; after the barrier every wavefront of the group
// adds the group's parts in wavefront order, p_j = g_j u_j, and accumulates
// p_j times its chunks of W_down[j].
template <typename T, int R, int NCH, int HW>
__device__ __forceinline__ void rows_consume(DecodeSmem &sm, const float (&hreg)[NCH][Elem<T>::kVec],
                                             float (&yacc)[NCH][Elem<T>::kVec], int r0, int end, int par,
                                             const u32x4 (&bu)[R][NCH], const u32x4 (&bd)[R][NCH], bool lora,
                                             const LoraRows<T> &lr, int rank, float &zh) {
  constexpr int VEC = Elem<T>::kVec;
  const int lane = threadIdx.x & 63, hw = __builtin_amdgcn_readfirstlane((threadIdx.x >> 6) % HW);
  const int gr = __builtin_amdgcn_readfirstlane((threadIdx.x >> 6) / HW);
  float *part = sm.red + (gr * 2 + par) * (R * HW);  // [R][HW] parts of u of this group
  float u[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    u[r] = 0.0f;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int v = 0; v < VEC; ++v) u[r] = fmaf(hreg[c][v], unpack<T>(bu[r][c], v), u[r]);
  }
  const float us = rows_sum<R>(u, lane);
  if ((lane & (64 / R - 1)) == 0) part[(lane / (64 / R)) * HW + hw] = us;
  __syncthreads();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    float ut = 0.0f;
#pragma unroll
    for (int q = 0; q < HW; ++q) ut += part[r * HW + q];
    const int li = max(0, min(r0 + r, end - 1));
    if (lora) ut += lr.lw[li];  // the up adapter's term of this kept row
    const float pr = (r0 + r < end) ? sm.mg[li] * ut : 0.0f;
    if (lora && hw == 0 && lane < rank && r0 + r < end)  // z_lane += p_j A_down[j][lane], this group's rows in order
      zh = fmaf(pr, Elem<T>::value(lr.lad[(size_t)li * rank + lane]), zh);
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int v = 0; v < VEC; ++v) yacc[c][v] = fmaf(pr, unpack<T>(bd[r][c], v), yacc[c][v]);
  }
  // the sums are taken here, not sunk to the end of the caller's pass: the
  // batch's registers are then free for the loads that refill them
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int v = 0; v < VEC; ++v) asm volatile("" : "+v"(yacc[c][v]));
}

// LoRA: for the kept rows list[i0 .. i0 + mn), w_i = s (h A_up) .
// B_up_T[j] into lr.lw and A_down[j] into lr.lad (R / VEC adjacent threads
// per row, 16 bytes each).  The loads are issued before the first row
// batches (loads complete in issue order) and used after them; one pass
// covers a workgroup's list (at most 64 rows of R / VEC <= 16 pieces).
template <typename T>
struct LoraPrepRegs {
  u32x4 bu, ad;
};

template <typename T>
__device__ __forceinline__ void lora_prep_load(const DecodeArgs &a, int l, const DecodeSmem &sm, int i0, int mn, int b0,
                                               LoraPrepRegs<T> &pr) {
  constexpr int VEC = Elem<T>::kVec;
  const int R = a.rank, RQ = R / VEC, idx = b0 + (int)threadIdx.x;
  const size_t rl = (size_t)a.d_ff * R;
  const uint32_t bytes = (uint32_t)(rl * sizeof(T));
  const __amdgpu_buffer_rsrc_t rb = weight_rsrc(static_cast<const T *>(a.BuT) + (size_t)l * rl, bytes);
  const __amdgpu_buffer_rsrc_t rd = weight_rsrc(static_cast<const T *>(a.Ad) + (size_t)l * rl, bytes);
  const bool on = idx < mn * RQ;
  const int m = i0 + (on ? idx / RQ : 0), q = idx % RQ;
  const uint32_t off = on ? (uint32_t)(((size_t)sm.mj[m] * R + q * VEC) * sizeof(T)) : kOffNone;
  pr.bu = __builtin_amdgcn_raw_buffer_load_b128(rb, (int)off, 0, 0);
  pr.ad = __builtin_amdgcn_raw_buffer_load_b128(rd, (int)off, 0, 0);
}

template <typename T>
__device__ __forceinline__ void lora_prep_use(const DecodeArgs &a, const DecodeSmem &sm, LoraRows<T> &lr, int i0,
                                              int mn, int b0, const LoraPrepRegs<T> &pr) {
  constexpr int VEC = Elem<T>::kVec;
  const int R = a.rank, RQ = R / VEC, idx = b0 + (int)threadIdx.x;
  const bool on = idx < mn * RQ;
  const int m = i0 + (on ? idx / RQ : 0), q = idx % RQ;
  float w = 0.0f;
#pragma unroll
  for (int v = 0; v < VEC; ++v) w = fmaf(sm.lz[q * VEC + v], unpack<T>(pr.bu, v), w);
  for (int msk = 1; msk < RQ; msk <<= 1) w += __shfl_xor(w, msk, 64);
  if (on) {
    if (q == 0) lr.lw[m] = a.lscale * w;
    *reinterpret_cast<u32x4 *>(&lr.lad[(size_t)m * R + q * VEC]) = pr.ad;
  }
}


// ------------------------------------------------------------------ layer

// Second reduction stage inside the layer launch (small layers: d <=
// kFusedMaxD, G <= kFusedMaxG): the last workgroup to finish adds the G
// partials in the order of dec_reduce_kernel (16 groups, each every 16th
// partial in workgroup order, the groups in order; slice sums of squares by
// the same exchanges), so either form gives the same bits.  Thread t takes
// groups t / 128 and t / 128 + 8 at columns 4 (t % 128) .. + 3, every
// 16-byte partial load issued before any is used.
constexpr int kFusedMaxD = 512, kFusedMaxG = 96;

template <typename T>
__device__ void dec_reduce_all(const DecodeArgs &a, int l, DecodeSmem &sm) {
  constexpr int NG = kRedThreads / kRedCols, FQ = kFusedMaxG / NG, NQ = kFusedMaxD / 4;
  static_assert(NG * kFusedMaxD <= 2 * kDecodeMaxD && 2 * kDecodeThreads == NG * NQ, "fused second stage tiling");
  const int tid = threadIdx.x, lane = tid & 63;
  const int d = a.d, G = a.G;
  const __amdgpu_buffer_rsrc_t yp = weight_rsrc(a.ypart, (uint32_t)((size_t)G * d * sizeof(float)));
  f32x4 v[2][FQ];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int q = 0; q < FQ; ++q) {
      const int it = tid + h * kDecodeThreads, g = it / NQ, c4 = 4 * (it % NQ), k = g + NG * q;
      const uint32_t off = (c4 < d && k < G) ? (uint32_t)(((size_t)k * d + c4) * sizeof(float)) : kOffNone;
      v[h][q] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(yp, (int)off, 0, 16 /* coherent */));
    }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int it = tid + h * kDecodeThreads, g = it / NQ, c4 = 4 * (it % NQ);
    f32x4 s = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int q = 0; q < FQ; ++q)
      if (g + NG * q < G) s += v[h][q];
    if (c4 < d) *reinterpret_cast<f32x4 *>(&sm.red[g * kFusedMaxD + c4]) = s;
  }
  __syncthreads();
  if (tid < kFusedMaxD) {
    const int col = tid;
    const bool on = col < d;
    float y = 0.0f;
    if (on) {
      for (int q = 0; q < NG && q < G; ++q) y += sm.red[q * kFusedMaxD + col];
      if (l == a.L - 1) static_cast<T *>(a.out)[col] = Elem<T>::round(y);
      else store_coherent(a.ybuf + col, y);
    }
    float sq = on ? y * y : 0.0f;
#pragma unroll
    for (int m = 8; m >= 1; m >>= 1) sq += __shfl_xor(sq, m, 64);
    if ((lane & 15) == 0 && on && l < a.L - 1) store_coherent(a.sspart + col / kRedCols, sq);
  }
}

// One layer of one token (see the top of this file); workgroup w writes its
// partial y to ypart[w] (and z to zpart[w] with adapters).
template <typename T, bool LORA, int HW>
__global__ __launch_bounds__(kDecodeThreads) void dec_layer_kernel(DecodeArgs a, int l) {
  __shared__ DecodeSmem sm;
  __shared__ LoraRows<T> lr;
  constexpr int VEC = Elem<T>::kVec;
  constexpr int CH = 64 * VEC;              // elements per chunk (one 16-byte load per lane)
  constexpr int DMAX = HW == 8 ? kDecodeMaxD / CH : HW;  // chunks per row (at most)
  constexpr int NCH = (DMAX + HW - 1) / HW;  // chunks per wavefront of a row group
  constexpr int NGR = kDecodeWaves / HW;    // row groups
  constexpr int R = 8 / NCH;                // rows of two batches (2 x 8 loads in flight per lane)
  constexpr int RB = R > 2 ? R / 4 : 1;     // rows per batch
  static_assert(HW == 2 || HW == 4 || HW == 8, "row group width");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6), hw = wv % HW, gr = wv / HW;
  const int w = blockIdx.x;
  const int d = a.d, d_ff = a.d_ff;
  const size_t wl = (size_t)d * d_ff;
  // the route sets only the keep rule and, with adapters, whether their terms
  // load.  Without adapters the table lookup (the id, then its entry) is two
  // buffer loads that return zero when there is no table: no branch and no
  // wait on them comes before the first weight loads, and the entry is read
  // at the keep list
  const bool lut = !LORA && a.route_mode == ROUTE_LUT;
  const int base0 = LORA ? token_is_base(a.route_mode, a.ids, a.lut, 0) : a.route_mode == ROUTE_BASE;
  if (l == 0) SATS_TRACE_POINT(0);
  const bool lora = LORA && !base0;
  const uint32_t wbytes = (uint32_t)(wl * sizeof(T));
  const __amdgpu_buffer_rsrc_t Wg = weight_rsrc(static_cast<const T *>(a.Wg) + (size_t)l * wl, wbytes);
  const __amdgpu_buffer_rsrc_t Wu = weight_rsrc(static_cast<const T *>(a.Wu) + (size_t)l * wl, wbytes);
  const __amdgpu_buffer_rsrc_t Wd = weight_rsrc(static_cast<const T *>(a.Wd) + (size_t)l * wl, wbytes);

  // ---- gate: wavefront wv reads columns wv, wv + 16, ... of the block
  GatePieces gp;
  gp.c0 = w * a.cw;
  gp.nc = max(1, min(a.cw, d_ff - gp.c0));
  gp.npc = ((d * (int)sizeof(T) + 1023) / 1024 + kGateQ - 1) / kGateQ;
  gp.wv = wv;
  gp.P = (wv < gp.nc ? (gp.nc - wv + 15) / 16 : 0) * gp.npc;
  // the layer input's loads go first: h is formed while the first gate
  // pieces are in flight, not after them (loads complete in issue order)
  InputRegs<kDecodeThreads> ir;
  dec_input_issue<T, kDecodeThreads>(a, l, ir);
  int rid = __builtin_amdgcn_raw_buffer_load_b32(weight_rsrc(a.ids, lut ? 4u : 0u), 0, 0, 0);
  // LoRA: B_gate at the block's columns (thread (c, i): ranks i, i + 16, ...)
  // and every chunk partial of h A_gate, h A_up (all loads issued at once,
  // ahead of the weights); used once h is formed
  constexpr int BQ = kLoraMaxRank / kDecodeWaves, VC = kDecodeMaxD / kVRows;
  float bgv[BQ];
  float vq[VC];
  const int lc = tid & 63, li = tid >> 6;
  if (lora) {
    const T *bg = static_cast<const T *>(a.Bg) + (size_t)l * a.rank * d_ff + gp.c0 + min(lc, gp.nc - 1);
#pragma unroll
    for (int m = 0; m < BQ; ++m) {
      const int i = li + m * kDecodeWaves;
      bgv[m] = (i < a.rank) ? Elem<T>::get(bg + (size_t)i * d_ff) : 0.0f;
    }
    // thread t < 2 rank: adapter t / rank, rank index t % rank, chunk c
#pragma unroll
    for (int c = 0; c < VC; ++c)
      vq[c] = (tid < 2 * a.rank && c < a.nvc)
                  ? load_coherent(a.vpart + ((size_t)c * 2 + tid / a.rank) * a.rank + tid % a.rank)
                  : 0.0f;
  }
  u32x4 qa[kGateQ], qb[kGateQ];
  gate_piece_issue<T>(Wg, gp, d, 0, qa);
  gate_piece_issue<T>(Wg, gp, d, 1, qb);
  for (int k = d + tid; k < kDecodeMaxD; k += kDecodeThreads) sm.hs[k] = 0.0f;  // past d: no products
  dec_input_finish<T, kDecodeThreads>(a, l, ir, sm, a.layer_in != nullptr && w == 0);
  // (rid passed through as a lane value: the entry then stays in a vector
  // register until the keep list instead of being waited for here)
  asm volatile("" : "+v"(rid));
  const int lent = __builtin_amdgcn_raw_buffer_load_b8(weight_rsrc(a.lut, lut ? 0x7fffffffu : 0u), rid, 0, 0);
  // the layer's threshold the same way, read at the keep list (zero on the base path)
  const float thr = __builtin_bit_cast(
      float, __builtin_amdgcn_raw_buffer_load_b32(weight_rsrc(a.thr, base0 ? 0u : (uint32_t)(l + 1) * 4u),
                                                  (int)(l * 4), 0, 0));
  pack_input<T>(sm);
  __syncthreads();
  if (l == 0) SATS_TRACE_POINT(1);
  if (lora) {  // h A_gate into lvg, h A_up into lz; then the gate adapter terms
    if (tid < 2 * a.rank) {  // the chunks in order
      float v = 0.0f;
#pragma unroll
      for (int c = 0; c < VC; ++c)
        if (c < a.nvc) v += vq[c];
      if (tid < a.rank) sm.lvg[tid] = v;
      else sm.lz[tid - a.rank] = v;
    }
    __syncthreads();
    float t = 0.0f;
#pragma unroll
    for (int m = 0; m < BQ; ++m) {
      const int i = li + m * kDecodeWaves;
      if (i < a.rank) t = fmaf(sm.lvg[i], bgv[m], t);
    }
    sm.lv[0][li][lc] = t;
  }
  // the loop issues the next pieces on every pass (past the last piece they
  // read zeros without a memory access) and the last pass is taken out of
  // it: with no branch around a load, both buffers stay in flight, where a
  // conditional issue makes the compiler assume the first buffer may be the
  // newer one and wait for both
  float acc[2] = {0.0f, 0.0f};
  int p = 0;
  for (; p + 2 < gp.P; p += 2) {
    gate_piece_use<T>(sm, gp, p, qa, acc, sm.red);
    gate_piece_issue<T>(Wg, gp, d, p + 2, qa);
    gate_piece_use<T>(sm, gp, p + 1, qb, acc, sm.red);
    gate_piece_issue<T>(Wg, gp, d, p + 3, qb);
  }
  if (p < gp.P) gate_piece_use<T>(sm, gp, p, qa, acc, sm.red);
  if (p + 1 < gp.P) gate_piece_use<T>(sm, gp, p + 1, qb, acc, sm.red);
  // every load of the wavefront has landed here (the last pieces were used and
  // the route entry and threshold came before them); the explicit wait says
  // so to the compiler, which otherwise keeps loads of the loop (and, on the
  // wavefronts that skip the keep list, those two) pending and waits for the
  // first row batches before the second is issued
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  __syncthreads();
  if (l == 0) SATS_TRACE_POINT(2);
  // ---- keep list: one lane per column
  if (wv == 0) {
    const bool on = lane < gp.nc && gp.c0 + lane < d_ff;
    float av = on ? sm.red[lane] : 0.0f;
    if (lora && a.lscale != 0.0f) {
      float t = 0.0f;
      for (int q = 0; q < kDecodeWaves; ++q) t += sm.lv[0][q][lane];
      av += a.lscale * t;
    }
    const float g = silu(av);
    const int base = base0 | (lent != 0);
    const bool keep = on && (base || fabsf(g) >= thr);
    if (a.keep_out && on) a.keep_out[(size_t)l * d_ff + gp.c0 + lane] = (uint8_t)keep;
    const uint64_t bal = __ballot(keep);
    const int rk = __popcll(bal & ((1ull << lane) - 1ull));
    if (keep) {
      sm.mj[rk] = gp.c0 + lane;
      sm.mg[rk] = g;
    }
    if (lane == 0) sm.wcnt[0] = __popcll(bal);
  }
  __syncthreads();
  const int tot = sm.wcnt[0];
  if (l == 0 && w == 0 && tid == 0 && a.route_out) a.route_out[0] = (uint8_t)(base0 | (lent != 0));
  if (l == 0) SATS_TRACE_POINT(4);

  // ---- rows: group gr takes list[b, e)
  const int hn = (tot + NGR - 1) / NGR;
  const int b = gr * hn, e = min(tot, (gr + 1) * hn);
  const int nbt = (hn + RB - 1) / RB;  // batches (every group runs the same number)
  float hreg[NCH][VEC];  // h at this lane's columns
  float yacc[NCH][VEC];
  u32x4 au[RB][NCH], ad[RB][NCH], cu[RB][NCH], cd[RB][NCH];
  LoraPrepRegs<T> lp;
  if (lora) lora_prep_load<T>(a, l, sm, 0, tot, 0, lp);
  rows_issue<T, RB, NCH, HW>(Wu, Wd, sm, b, e, d, au, ad);
  rows_issue<T, RB, NCH, HW>(Wu, Wd, sm, b + RB, e, d, cu, cd);
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      const int k = (hw + c * HW) * CH + lane * VEC + v;
      hreg[c][v] = (k < d) ? sm.hs[k] : 0.0f;
      yacc[c][v] = 0.0f;
    }
  float zh = 0.0f;  // LoRA, lane i < rank of wavefront 0 of each group: z_i over the group's kept rows
  if (lora) {  // the up adapter's terms and A_down of the kept rows
    lora_prep_use<T>(a, sm, lr, 0, tot, 0, lp);
    __syncthreads();
  }
  int par = 0;  // LDS slot parity for the parts of u
  // batches issued on every pass and the last pass taken out, as the gate
  // pieces (past the end they read zeros)
  int i = 0;
  for (; i + 2 < nbt; i += 2) {
    rows_consume<T, RB, NCH, HW>(sm, hreg, yacc, b + i * RB, e, par, au, ad, lora, lr, a.rank, zh);
    par ^= 1;
    // (a batch's loads are not moved above the last uses of the buffer they
    // refill: they then take its registers, with no copy that would wait
    // for them at the end of the pass)
    __builtin_amdgcn_sched_barrier(0);
    rows_issue<T, RB, NCH, HW>(Wu, Wd, sm, b + (i + 2) * RB, e, d, au, ad);
    rows_consume<T, RB, NCH, HW>(sm, hreg, yacc, b + (i + 1) * RB, e, par, cu, cd, lora, lr, a.rank, zh);
    par ^= 1;
    __builtin_amdgcn_sched_barrier(0);
    rows_issue<T, RB, NCH, HW>(Wu, Wd, sm, b + (i + 3) * RB, e, d, cu, cd);
  }
  if (i < nbt) {
    rows_consume<T, RB, NCH, HW>(sm, hreg, yacc, b + i * RB, e, par, au, ad, lora, lr, a.rank, zh);
    par ^= 1;
  }
  if (i + 1 < nbt) rows_consume<T, RB, NCH, HW>(sm, hreg, yacc, b + (i + 1) * RB, e, par, cu, cd, lora, lr, a.rank, zh);
  __syncthreads();
  if (lora) {  // z = the groups' sums, added in group order
    if (hw == 0 && gr > 0 && lane < a.rank) sm.lv[1][gr][lane] = zh;
    __syncthreads();
    if (wv == 0 && lane < a.rank) {
      float z = zh;
      for (int q = 1; q < NGR; ++q) z += sm.lv[1][q][lane];
      store_coherent(a.zpart + (size_t)w * a.rank + lane, z);
    }
  }
  if (l == 0) SATS_TRACE_POINT(5);
  // the groups' sums, added in group order, are this workgroup's partial y
  // (groups 1 .. NGR - 1 pass theirs through LDS: NGR - 1 rows of d)
  static_assert((NGR - 1) * DMAX * CH <= 2 * kDecodeMaxD, "group sums fit the LDS buffer");
  if (gr > 0) {
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int k = (hw + c * HW) * CH + lane * VEC;
      if (k < d) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) sm.red[(gr - 1) * d + k + v] = yacc[c][v];
      }
    }
  }
  __syncthreads();
  if (gr == 0) {
    const __amdgpu_buffer_rsrc_t yr = weight_rsrc(a.ypart + (size_t)w * d, (uint32_t)(d * sizeof(float)));
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int k = (hw + c * HW) * CH + lane * VEC;
      if (k < d) {
        float y[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
          y[v] = yacc[c][v];
          for (int q = 1; q < NGR; ++q) y[v] += sm.red[(q - 1) * d + k + v];
        }
#pragma unroll
        for (int v = 0; v < VEC; v += 4)
          store_coherent4(yr, (uint32_t)((k + v) * sizeof(float)), y[v], y[v + 1], y[v + 2], y[v + 3]);
      }
    }
  }
  // a workgroup that kept fewer than half its columns is done early: in a
  // stack it warms the first rows of its next-layer W_gate block in the MALL
  // (loads that allocate) while the heavier workgroups finish, so the next
  // layer's gate starts on cache hits.  Nothing waits on these loads but the
  // workgroup's own end.
  if (!LORA && !a.fused_reduce && l + 1 < a.L && 2 * tot < gp.nc) {
    constexpr int PFN = kWarmRows * kDecodeMaxD * (int)sizeof(T) / (kDecodeThreads * 16);
    const uint32_t rowb = (uint32_t)(d * sizeof(T));
    const __amdgpu_buffer_rsrc_t wn = weight_rsrc(static_cast<const T *>(a.Wg) + (size_t)(l + 1) * wl, wbytes);
    u32x4 pf[PFN];
#pragma unroll
    for (int i = 0; i < PFN; ++i) {
      const uint32_t byte = (uint32_t)(i * kDecodeThreads + tid) * 16u;
      const int r = (int)(byte / rowb);  // row of the block
      const bool on = r < kWarmRows && r < gp.nc;
      pf[i] = __builtin_amdgcn_raw_buffer_load_b128(wn, on ? (int)((uint32_t)(gp.c0 + r) * rowb + byte % rowb)
                                                           : (int)kOffNone, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < PFN; ++i) asm volatile("" ::"v"(pf[i]));
  }
  if (!LORA && a.fused_reduce && arrive_last(a.done, (unsigned)a.G, &sm.flag)) dec_reduce_all<T>(a, l, sm);
}

// ------------------------------------------------------------------ reduce

// Workgroup w (of RW) and its slice of columns: y = sum of the G partials
// in workgroup order.
template <typename T, bool LORA>
__device__ void dec_reduce(const DecodeArgs &a, int l, int w, DecodeSmem &sm, bool base) {
  const bool lora = LORA && !base;
  constexpr int THREADS = kDecodeThreads, NW = kDecodeWaves;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d = a.d, G = a.G;
  const int cpw = (d + a.RW - 1) / a.RW;  // columns of this workgroup (<= THREADS / ngr: the plan)
  const int cw0 = w * cpw;
  const int nc = max(0, min(cpw, d - cw0));
  // partial groups: every 16th partial in workgroup order, the groups added
  // in order -- the order of dec_reduce_kernel, so that a call with adapters
  // at scale 0 gives the plain call's bits
  constexpr int ngr = kRedThreads / kRedCols;
  const int c = tid % cpw, gr = tid / cpw;
  float s = 0.0f;
  if (c < nc && gr < ngr && gr < G)
    s = sum_coherent(a.ypart + (size_t)gr * d + cw0 + c, (size_t)ngr * d, (G - gr + ngr - 1) / ngr);
  sm.red[tid] = s;
  __syncthreads();
  float y = 0.0f;
  if (tid < nc)
    for (int qg = 0; qg < ngr && qg < G; ++qg) y += sm.red[qg * cpw + tid];
  if (lora) {  // + s z B_down, z summed over the G partials in workgroup order
    const int R = a.rank, Q = THREADS / R;
    // B_down[i][cw0 + c] for every (i, c) of the slice, one element per thread
    // and pass (every load of a pass issued before any is used), into LDS
    float *bsl = sm.red + THREADS;  // [R][cpw] (the partial-group sums use the first THREADS)
    {
      const T *bd = static_cast<const T *>(a.Bd) + (size_t)l * R * d + cw0;
      const int per = max(1, cpw), tot = R * per;
      float bv[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = tid + k * THREADS, i = min(e / per, R - 1), c = min(e % per, max(nc - 1, 0));
        bv[k] = Elem<T>::get(bd + (size_t)i * d + c);
      }
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (tid + k * THREADS < tot) bsl[tid + k * THREADS] = bv[k];
      for (int e = tid + 4 * THREADS; e < tot; e += THREADS) bsl[e] = Elem<T>::get(bd + (size_t)(e / per) * d + min(e % per, max(nc - 1, 0)));
    }
    float *flat = &sm.lv[0][0][0];
    float zs = 0.0f;
    {
      const int i = tid % R, q = tid / R;
      if (q < G) zs = sum_coherent(a.zpart + (size_t)q * R + i, (size_t)Q * R, (G - q + Q - 1) / Q);
    }
    if (l == 0) SATS_TRACE_POINT(12);
    flat[tid] = zs;
    __syncthreads();
    if (l == 0) SATS_TRACE_POINT(14);
    if (tid < R) {
      float z = 0.0f;
      for (int q = 0; q < Q; ++q) z += flat[q * R + tid];
      sm.lz[tid] = a.lscale * z;
    }
    __syncthreads();
    if (l == 0) SATS_TRACE_POINT(11);
    if (tid < nc) {
      float t = 0.0f;
      for (int i = 0; i < R; ++i) t = fmaf(sm.lz[i], bsl[i * cpw + tid], t);
      y += t;
    }
  }
  if (tid < nc) {
    if (l == a.L - 1) static_cast<T *>(a.out)[cw0 + tid] = Elem<T>::round(y);
    else store_coherent(a.ybuf + cw0 + tid, y);
  }
  // sums of squares per 16 columns (the slices of dec_reduce_kernel, added in
  // its order: the cpw <= 64 columns sit in wavefront 0, 16 lanes a slice)
  if (wv == 0 && l < a.L - 1) {
    float sq = (tid < nc) ? y * y : 0.0f;
#pragma unroll
    for (int m = 8; m >= 1; m >>= 1) sq += __shfl_xor(sq, m, 64);
    if ((lane & 15) == 0 && lane < nc) store_coherent(a.sspart + (cw0 + lane) / kRedCols, sq);
  }
  (void)NW;
}


// ------------------------------------------------------------------ kernels

// Second reduction stage with adapters: workgroup w (of RW) takes one slice
// of y and adds s z B_down (z summed over the partials in workgroup order).
template <typename T>
__global__ __launch_bounds__(kDecodeThreads) void dec_reduce_lora_kernel(DecodeArgs a, int l) {
  __shared__ DecodeSmem sm;
  dec_reduce<T, true>(a, l, blockIdx.x, sm, token_is_base(a.route_mode, a.ids, a.lut, 0));
}

// Second reduction stage of a layer without adapters, a launch of its own
// (the kernel boundary orders it after every partial).  Workgroup w owns
// columns [16 w, 16 w + 16):
// 16 groups of threads each add every 16th partial in workgroup order, the
// groups are added in order, and y (or the rounded output on the last layer)
// and the slice's sum of squares for the next layer's input are written.
template <typename T>
__global__ __launch_bounds__(kRedThreads) void dec_reduce_kernel(DecodeArgs a, int l) {
  constexpr int NG = kRedThreads / kRedCols;
  __shared__ float red[kRedThreads];
  const int tid = threadIdx.x, c = tid % kRedCols, g = tid / kRedCols;
  const int d = a.d, G = a.G, col = blockIdx.x * kRedCols + c;
  float s = 0.0f;
  if (col < d && g < G) s = sum_coherent(a.ypart + (size_t)g * d + col, (size_t)NG * d, (G - g + NG - 1) / NG);
  red[tid] = s;
  __syncthreads();
  if (tid < 64) {
    const bool on = tid < kRedCols && blockIdx.x * kRedCols + tid < d;
    float y = 0.0f;
    if (on) {
      for (int q = 0; q < NG && q < G; ++q) y += red[q * kRedCols + tid];
      if (l == a.L - 1) static_cast<T *>(a.out)[blockIdx.x * kRedCols + tid] = Elem<T>::round(y);
      else store_coherent(a.ybuf + blockIdx.x * kRedCols + tid, y);
    }
    const float sq = wave_sum(on ? y * y : 0.0f);  // the slice's sum of squares, fixed order
    if (tid == 0 && l < a.L - 1) store_coherent(a.sspart + blockIdx.x, sq);
  }
}

}  // namespace sats
