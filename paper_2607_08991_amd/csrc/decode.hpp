// Single-token (decode batch 1) path: three plain launches per layer.
//
//   gate    W_gate is cut into tiles one 16-byte load per lane wide (64 lanes:
//           512 bf16 or 256 fp32 columns, 1 KB of each row) by a chunk of
//           rows.  A workgroup forms h . tile for its tile, sums its
//           wavefronts' partials in LDS and writes one partial a per column
//           and row chunk.
//   rows    Work units are (column block, share): every workgroup of a
//           column block adds the block's row-chunk partials in chunk order,
//           applies SiLU (Eq. 2) and the keep rule (Eq. 4-5, or every column
//           on the base path, Eq. 13) and compacts the kept columns in LDS;
//           all of them get the same list, and each takes an even share of
//           it: u_j = W_up_T[j] . h, p_j = g_j u_j (Eq. 1) and
//           p_j W_down[j] accumulated into the workgroup's partial y, the
//           rows of both projections read in the same batches.
//   reduce  Workgroup w adds every partial for its own slice of columns in
//           workgroup order: y, or the rounded output on the last layer, and
//           the slice's sum of squares for the next layer's input
//           rho(y / sqrt(mean(y^2) + 1e-6)).
//
// Workgroups have 1024 threads (16 wavefronts per CU keep more row reads in
// flight than 8).  Partials cross workgroups through device-coherent stores
// and loads; kernel boundaries order the phases.  The assignment of work
// depends only on the data, never on timing, so every sum has a fixed order
// and results are reproducible bit for bit.
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

constexpr int kDecodeThreads = 1024;  // rows and reduce launches
constexpr int kDecodeWaves = kDecodeThreads / 64;
#ifndef SATS_GATE_THREADS
#define SATS_GATE_THREADS 1024
#endif
constexpr int kGateThreads = SATS_GATE_THREADS;  // gate launch
constexpr int kGateBatch = kGateThreads >= 1024 ? 8 : 16;  // 16-byte loads in flight per lane
constexpr int kDecodeMaxD = 4096;  // h lives in LDS
constexpr int kDecodeMaxG = 1024;  // rows / reduce workgroups (partials of y)
constexpr int kRedThreads = 256, kRedCols = 16;  // second reduction stage: threads and columns per workgroup

// Columns of one gate column block (one 16-byte load per lane of a wavefront).
template <typename T> constexpr int dec_block_cols() { return 64 * Elem<T>::kVec; }
// Gate partials of one column are stored contiguously, padded to whole 16 bytes.
__host__ __device__ constexpr int dec_nrcp(int nrc) { return (nrc + 3) & ~3; }

struct DecodeArgs {
  const void *x;          // [d] call input (storage type)
  void *out;              // [d]
  const void *Wg, *Wu, *Wd;  // stacked weights
  const float *thr;       // [L] (unused on the base path)
  const int32_t *ids;
  const uint8_t *lut;
  int route_mode;
  int L, d, d_ff;
  int nblk, nrc;          // gate tiles: column blocks x row chunks
  float *gpart;           // [d_ff][nrcp]   partial a of each row chunk (nrcp = nrc rounded up to 4)
  float *ypart;           // [G][d]         per-workgroup partial y
  float *ybuf;            // [d]
  float *sspart;          // [RW]           per-reduce-workgroup sums of y^2
  int G, RW;              // rows workgroups (partials of y), reduce workgroups
  int nss;                // slice sums of squares of y per layer: one per 16 columns
  int *state;             // [1] the token's route (1: base path), set by the layer-0 gate launch
  unsigned *done;         // [1] rows workgroups whose partial y is written (cleared by the gate launch)
  unsigned *err;          // device error flag (a bounded wait gave up)
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
  float *vpart;           // [nrc][rank] per gate row chunk: partial h . A_up
  float *zpart;           // [G][rank]   per rows workgroup: sum of p_j A_down[j] over its kept rows
};

constexpr int kLoraMaxRank = 64;  // ranks 8, 16, 32, 64

struct DecodeSmem {
  float hs[kDecodeMaxD];                // layer input
  float red[2 * kDecodeMaxD];           // gate: wavefront partials; rows: parts of u, half sums
  int mj[kDecodeThreads / 2];           // kept columns of the current column block ...
  float mg[kDecodeThreads / 2];         // ... and their g values
  int wcnt[kDecodeWaves];
  float scal[kDecodeWaves];
  int flag;
  float lv[2][kDecodeWaves][kLoraMaxRank];  // LoRA: wavefront partials of h . A (gate, up)
  float lz[kLoraMaxRank];                    // LoRA: h . A_up (rows) or z (reduce)
};

// LoRA operands of a rows workgroup's kept rows (list position i): the up
// adapter's contribution w_i = s (h A_up) . B_up_T[j] and A_down[j].
template <typename T>
struct LoraRows {
  float lw[kDecodeThreads / 2];
  T lad[64 * Elem<T>::kVec * kLoraMaxRank];  // [list position][rank]: one column block's list at most
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

// 16 bytes at base + soff + voff, not kept in the caches (streamed once).
__device__ __forceinline__ u32x4 load_rsrc(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 2);
}

// Sum of the nrc gate partials of column `col`, in row-chunk order: 16 bytes
// per load, written through by the gate launch and read from the
// device-coherent level.
__device__ __forceinline__ float gate_sum(__amdgpu_buffer_rsrc_t gp, int col, int nrc) {
  const int nq = dec_nrcp(nrc) / 4;
  const uint32_t base = (uint32_t)col * (uint32_t)(nq * 16);
  float s = 0.0f;
  for (int q0 = 0; q0 < nq; q0 += 4) {
    f32x4 v[4];  // up to 16 partials in flight
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t off = (q0 + i < nq) ? base + (uint32_t)((q0 + i) * 16) : kOffNone;
      v[i] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(gp, (int)off, 0, 16 /* coherent */));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if ((q0 + i) * 4 + j < nrc) s += v[i][j];
  }
  return s;
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
template <int THREADS>
struct InputRegs {
  u32x4 xv[kDecodeMaxD / (4 * THREADS)];  // layer 0: x, 16 bytes at a time (d <= 4096)
  float yv[kDecodeMaxD / THREADS];
  float ss[kDecodeMaxG / THREADS];
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
  for (int i = 0; i < kDecodeMaxG / THREADS; ++i) r.ss[i] = 0.0f;
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
    for (int i = 0; i < kDecodeMaxG / THREADS; ++i)
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
  for (int i = 0; i < kDecodeMaxG / THREADS; ++i) asm volatile("" : "+v"(r.ss[i])::"memory");
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
    for (int i = 0; i < kDecodeMaxG / THREADS; ++i) s += r.ss[i];
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

// ------------------------------------------------------------------ LoRA adapters
//
// The sparse path of a fine-tuned routed model adds s A B to each projection
// (Section 5).  Every product splits over the gate's row chunks: a gate tile
// over rows k0 .. k0 + kn adds s (h[k0..] A_gate[k0..]) B_gate to its partial
// of a, so the row-chunk sums give h (W_gate + s A_gate B_gate) with no step
// of its own; the tiles of column block 0 also write h[k0..] A_up[k0..], whose
// sum the rows launch uses for the up adapter of its kept rows.  The down
// adapter's first factor is summed over the kept rows (z = sum p_j A_down[j])
// next to each rows workgroup's partial y, and the second reduction stage
// adds s z B_down.

constexpr int kLoraPieces = 2;  // 16-byte pieces of an A matrix per thread and pass

template <typename T>
struct LoraGateRegs {
  u32x4 ag[kLoraPieces], au[kLoraPieces];  // A_gate / A_up pieces of one pass over the tile's rows
};

// B_gate rows at the tile's columns, staged in LDS by loads that write LDS
// (no registers held across the tile): row r at lb[r], 16 bytes per lane.
struct LoraGateSmem {
  uint8_t lb[kLoraMaxRank][1024];
};

// One pass of A loads: pieces p0 + tid, p0 + tid + THREADS (16 bytes each) of
// rows k0 .. k0 + kn of A_gate (and of A_up when `up`).
template <typename T>
__device__ __forceinline__ void lora_a_issue(const DecodeArgs &a, int l, int k0, int kn, bool up, int p0,
                                             LoraGateRegs<T> &lr) {
  constexpr int VEC = Elem<T>::kVec;
  const int R = a.rank, tid = threadIdx.x;
  const uint32_t abytes = (uint32_t)((size_t)a.d * R * sizeof(T));
  const __amdgpu_buffer_rsrc_t rg = weight_rsrc(static_cast<const T *>(a.Ag) + (size_t)l * a.d * R, abytes);
  const __amdgpu_buffer_rsrc_t ru = weight_rsrc(static_cast<const T *>(a.Au) + (size_t)l * a.d * R, abytes);
  const int np = kn * R / VEC;
  const uint32_t abase = (uint32_t)((size_t)k0 * R * sizeof(T));
#pragma unroll
  for (int m = 0; m < kLoraPieces; ++m) {
    const int pc = p0 + tid + m * kGateThreads;
    const uint32_t off = pc < np ? abase + (uint32_t)pc * 16u : kOffNone;
    lr.ag[m] = __builtin_amdgcn_raw_buffer_load_b128(rg, (int)off, 0, 0);
    lr.au[m] = up ? __builtin_amdgcn_raw_buffer_load_b128(ru, (int)off, 0, 0) : u32x4{0u, 0u, 0u, 0u};
  }
}

// This wavefront's rows of B_gate (wv, wv + NW, ...) at the lane's columns,
// straight into LDS.
template <typename T>
__device__ __forceinline__ void lora_b_issue(const DecodeArgs &a, int l, int col, LoraGateSmem &ls) {
  constexpr int NW = kGateThreads / 64;
  const int R = a.rank, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const __amdgpu_buffer_rsrc_t rb = weight_rsrc(static_cast<const T *>(a.Bg) + (size_t)l * R * a.d_ff,
                                                (uint32_t)((size_t)R * a.d_ff * sizeof(T)));
  // every row slot is loaded, past the rank from past the buffer (zeros): a
  // branch around these loads would cost the compiler its record of which
  // LDS bytes they write, and with it waits on every load before LDS reads
#pragma unroll
  for (int m = 0; m < kLoraMaxRank / NW; ++m) {
    const int row = wv + m * NW;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (__attribute__((address_space(3))) void *)ls.lb[row], 16,
                                             row < R ? (int)(col * sizeof(T)) : (int)kOffNone,
                                             row < R ? (int)((size_t)row * a.d_ff * sizeof(T)) : 0, 0, 0);
  }
}

// h . A over the tile's rows: each lane adds its pieces of one pass to sv
// (every piece of a thread covers the same rank indices: THREADS pieces
// span whole rows); lora_v_reduce then adds the lanes of equal index by
// halving exchanges, and lanes 0 .. R / VEC - 1 write the wavefront's sums.
template <typename T>
__device__ __forceinline__ void lora_a_acc(const DecodeArgs &a, int k0, int kn, int p0, const u32x4 (&pc)[kLoraPieces],
                                           float (&sv)[Elem<T>::kVec], const DecodeSmem &sm) {
  constexpr int VEC = Elem<T>::kVec;
  const int R = a.rank, np = kn * R / VEC;
#pragma unroll
  for (int m = 0; m < kLoraPieces; ++m) {
    const int p = p0 + threadIdx.x + m * kGateThreads;
    if (p < np) {
      const float hv = sm.hs[k0 + p * VEC / R];
#pragma unroll
      for (int v = 0; v < VEC; ++v) sv[v] = fmaf(hv, unpack<T>(pc[m], v), sv[v]);
    }
  }
}

template <typename T>
__device__ __forceinline__ void lora_v_reduce(const DecodeArgs &a, float (&sv)[Elem<T>::kVec],
                                              float (&out)[kLoraMaxRank]) {
  constexpr int VEC = Elem<T>::kVec;
  const int RQ = a.rank / VEC, lane = threadIdx.x & 63;
  for (int msk = 32; msk >= max(RQ, 1); msk >>= 1)
#pragma unroll
    for (int v = 0; v < VEC; ++v) sv[v] += __shfl_xor(sv[v], msk, 64);
  if (lane < RQ) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) out[lane * VEC + v] = sv[v];
  }
}

// ------------------------------------------------------------------ gate

// One batch of a gate tile: rows k0w + NW (r0 + u), u < GB, of this
// wavefront (past its nr rows the last row is read again and given weight 0).
template <typename T, int GB, int NW>
__device__ __forceinline__ void gate_issue(__amdgpu_buffer_rsrc_t wr, uint32_t row0_bytes, uint32_t stride_bytes,
                                           int r0, int nr, uint32_t lo, u32x4 (&q)[GB]) {
#pragma unroll
  for (int u = 0; u < GB; ++u) q[u] = load_rsrc(wr, lo, row0_bytes + (uint32_t)min(r0 + u, nr - 1) * stride_bytes);
}

template <typename T, int GB, int NW>
__device__ __forceinline__ void gate_consume(const DecodeSmem &sm, int k0w, int r0, int nr, const u32x4 (&q)[GB],
                                             float (&acc)[Elem<T>::kVec]) {
#pragma unroll
  for (int u = 0; u < GB; ++u) {
    const float hv = sm.hs[k0w + min(r0 + u, nr - 1) * NW];
    const float hu = (r0 + u < nr) ? hv : 0.0f;
#pragma unroll
    for (int v = 0; v < Elem<T>::kVec; ++v) acc[v] = fmaf(hu, unpack<T>(q[u], v), acc[v]);
  }
}

// Gate tiles blockIdx.x, blockIdx.x + gridDim.x, ... (tile t: column block
// t % nblk, row chunk t / nblk); forms h in LDS before the first tile's
// products (its loads follow the tile's first weight loads).
template <typename T, bool LORA>
__device__ void dec_gate(const DecodeArgs &a, int l, DecodeSmem &sm, LoraGateSmem &ls, bool record) {
  constexpr int THREADS = kGateThreads, VEC = Elem<T>::kVec, NW = THREADS / 64;
  constexpr int CB = dec_block_cols<T>();
  constexpr int GB = kGateBatch;
  static_assert(NW * CB <= 2 * kDecodeMaxD, "gate partials fit the LDS buffer");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int d = a.d, d_ff = a.d_ff;
  const int rows = (d + a.nrc - 1) / a.nrc;
  const __amdgpu_buffer_rsrc_t wr =
      weight_rsrc(static_cast<const T *>(a.Wg) + (size_t)l * d * d_ff, (uint32_t)((size_t)d * d_ff * sizeof(T)));
  const uint32_t stride = (uint32_t)((size_t)NW * d_ff * sizeof(T));  // between a wavefront's rows
  InputRegs<THREADS> ir;
  bool have_input = false;
  // LoRA: the token's route (base-path tokens use the base weights only)
  constexpr bool lora = LORA;
  const float lsc = !lora ? 0.0f
                          : ((l == 0 ? token_is_base(a.route_mode, a.ids, a.lut, 0) : a.state[0]) ? 0.0f : a.lscale);
  for (int t = blockIdx.x; t < a.nblk * a.nrc; t += gridDim.x) {
    const int cb = t % a.nblk, rc = t / a.nblk;
    const int k0 = rc * rows, kn = max(0, min(d, k0 + rows) - k0);
    const int col = cb * CB + lane * VEC;
    const int nr = (kn - wv + NW - 1) / NW;  // this wavefront's rows: k0 + wv + NW r, r < nr
    // Lanes past d_ff read in-bounds data of the next row (or zeros past the
    // matrix) and their sums are never stored, so only nr guards the loads.
    const bool live = nr > 0;
    const uint32_t row0 = (uint32_t)((size_t)(k0 + wv) * d_ff * sizeof(T));  // wavefront-uniform
    const uint32_t lo = (uint32_t)(col * sizeof(T));
    float acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = 0.0f;
    u32x4 q[GB];
    // LoRA: B_gate rows go to LDS now; the A pieces are loaded with the
    // wavefront's last weight batch and used after it (a wait for them
    // earlier would also wait for the weight loads issued before them)
    LoraGateRegs<T> lr;
    const bool a_early = !live || nr <= GB;
    if constexpr (LORA) {
      lora_b_issue<T>(a, l, col, ls);
      if (a_early) lora_a_issue<T>(a, l, k0, kn, cb == 0, 0, lr);
    }
    if (live) gate_issue<T, GB, NW>(wr, row0, stride, 0, nr, lo, q);
    if (!have_input) {  // h is needed from the first batch on; its loads follow the weights'
      dec_input_issue<T, THREADS>(a, l, ir);
      dec_input_finish<T, THREADS>(a, l, ir, sm, record);
      have_input = true;
      if (l == 0) SATS_TRACE_POINT(1);
    }
    if (live) {
      gate_consume<T, GB, NW>(sm, k0 + wv, 0, nr, q, acc);
      for (int r0 = GB; r0 < nr; r0 += GB) {
        if (LORA && r0 + GB >= nr) lora_a_issue<T>(a, l, k0, kn, cb == 0, 0, lr);
        gate_issue<T, GB, NW>(wr, row0, stride, r0, nr, lo, q);
        gate_consume<T, GB, NW>(sm, k0 + wv, r0, nr, q, acc);
      }
    }
    if constexpr (LORA) {  // this tile's h . A_gate (and h . A_up on column block 0)
      float sg[VEC], su[VEC];
#pragma unroll
      for (int v = 0; v < VEC; ++v) sg[v] = su[v] = 0.0f;
      const int np = kn * a.rank / VEC, pp = kLoraPieces * kGateThreads;
      for (int p0 = 0; p0 < np; p0 += pp) {
        if (p0 > 0) lora_a_issue<T>(a, l, k0, kn, cb == 0, p0, lr);
        lora_a_acc<T>(a, k0, kn, p0, lr.ag, sg, sm);
        if (cb == 0) lora_a_acc<T>(a, k0, kn, p0, lr.au, su, sm);
      }
      lora_v_reduce<T>(a, sg, sm.lv[0][wv]);
      if (cb == 0) lora_v_reduce<T>(a, su, sm.lv[1][wv]);
      __syncthreads();
      if (l == 0) SATS_TRACE_POINT(13);
      if (cb == 0 && tid < a.rank) {
        float v = 0.0f;
#pragma unroll
        for (int q2 = 0; q2 < NW; ++q2) v += sm.lv[1][q2][tid];
        store_coherent(a.vpart + (size_t)rc * a.rank + tid, v);
      }
    }
    if (LORA && lsc != 0.0f) {  // s (h[k0..] A_gate[k0..]) B_gate: this wavefront's rows of B_gate
#pragma unroll
      for (int m = 0; m < kLoraMaxRank / NW; ++m) {
        const int row = wv + m * NW;
        if (row < a.rank) {
          float vg = 0.0f;
#pragma unroll
          for (int q2 = 0; q2 < NW; ++q2) vg += sm.lv[0][q2][row];
          vg *= lsc;
          const u32x4 bq = *reinterpret_cast<const u32x4 *>(&ls.lb[row][lane * 16]);
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc[v] = fmaf(vg, unpack<T>(bq, v), acc[v]);
        }
      }
    }
#pragma unroll
    for (int v = 0; v < VEC; ++v) sm.red[wv * CB + lane * VEC + v] = acc[v];
    __syncthreads();
    if (tid < CB && cb * CB + tid < d_ff) {
      float s = 0.0f;
#pragma unroll
      for (int q2 = 0; q2 < NW; ++q2) s += sm.red[q2 * CB + tid];
      store_coherent(a.gpart + (size_t)(cb * CB + tid) * dec_nrcp(a.nrc) + rc, s);
    }
    __syncthreads();  // LDS reuse by the next tile
  }
}

// ------------------------------------------------------------------ rows

// The workgroup's wavefronts form two halves of 8; half hf takes its own
// rows of the unit, and wavefront v of a half owns column chunks v, v + 8,
// ... of d (64 lanes x 16 bytes each) for both projections.

// One batch: loads of this wavefront's chunks of the kept rows
// list[r0 + r], r < R (rows at or past `end` are not read).
template <typename T, int R, int NCH>
__device__ __forceinline__ void rows_issue(__amdgpu_buffer_rsrc_t Wu, __amdgpu_buffer_rsrc_t Wd, const DecodeSmem &sm,
                                           int r0, int end, int d, u32x4 (&bu)[R][NCH], u32x4 (&bd)[R][NCH]) {
  constexpr int VEC = Elem<T>::kVec, CH = 64 * VEC;
  const int lane = threadIdx.x & 63, hw = __builtin_amdgcn_readfirstlane((threadIdx.x >> 6) & 7);
  uint32_t soff[R];
#pragma unroll
  for (int r = 0; r < R; ++r)
    soff[r] = (uint32_t)((size_t)__builtin_amdgcn_readfirstlane(sm.mj[max(0, min(r0 + r, end - 1))]) * d * sizeof(T));
  // all rows of W_up_T first: the up products can start while W_down arrives
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int k = (hw + c * 8) * CH + lane * VEC;
      bu[r][c] = (k < d && r0 + r < end) ? load_rsrc(Wu, (uint32_t)(k * sizeof(T)), soff[r]) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int k = (hw + c * 8) * CH + lane * VEC;
      bd[r][c] = (k < d && r0 + r < end) ? load_rsrc(Wd, (uint32_t)(k * sizeof(T)), soff[r]) : u32x4{0u, 0u, 0u, 0u};
    }
}

// Uses one batch: this wavefront's parts of u_j = W_up_T[j] . h go to its
// half's LDS slot `par`; after the barrier every wavefront of the half adds
// the half's parts in wavefront order, p_j = g_j u_j, and accumulates p_j
// times its chunks of W_down[j].
template <typename T, int R, int NCH>
__device__ __forceinline__ void rows_consume(DecodeSmem &sm, const float (&hreg)[NCH][Elem<T>::kVec],
                                             float (&yacc)[NCH][Elem<T>::kVec], int r0, int end, int par,
                                             const u32x4 (&bu)[R][NCH], const u32x4 (&bd)[R][NCH], bool lora,
                                             const LoraRows<T> &lr, int rank, float &zh) {
  constexpr int VEC = Elem<T>::kVec;
  const int lane = threadIdx.x & 63, hw = __builtin_amdgcn_readfirstlane((threadIdx.x >> 6) & 7);
  const int hf = __builtin_amdgcn_readfirstlane(threadIdx.x >> 9);
  float *part = sm.red + (hf * 2 + par) * (R * 8);  // [R][8] parts of u of this half
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
  if ((lane & (64 / R - 1)) == 0) part[(lane / (64 / R)) * 8 + hw] = us;
  __syncthreads();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    float ut = 0.0f;
#pragma unroll
    for (int q = 0; q < 8; ++q) ut += part[r * 8 + q];
    const int li = max(0, min(r0 + r, end - 1));
    if (lora) ut += lr.lw[li];  // the up adapter's term of this kept row
    const float pr = (r0 + r < end) ? sm.mg[li] * ut : 0.0f;
    if (lora && hw == 0 && lane < rank && r0 + r < end)  // z_lane += p_j A_down[j][lane], this half's rows in order
      zh = fmaf(pr, Elem<T>::value(lr.lad[(size_t)li * rank + lane]), zh);
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int v = 0; v < VEC; ++v) yacc[c][v] = fmaf(pr, unpack<T>(bd[r][c], v), yacc[c][v]);
  }
}

// LoRA: h . A_up from the gate launch's row-chunk partials, in a fixed
// order: thread (q, i) adds chunks q, q + 8, ... (its first loads are issued
// at the start of the rows launch, ahead of every streaming load of its
// wavefront, since loads complete in issue order), then thread i adds the 8
// groups, into sm.lz.
constexpr int kLoraVG = 8, kLoraVQ = 4;
__device__ __forceinline__ void lora_vu_issue(const DecodeArgs &a, float (&vq)[kLoraVQ]) {
  const int R = a.rank, tid = threadIdx.x, i = tid % R, q = tid / R;
#pragma unroll
  for (int k = 0; k < kLoraVQ; ++k) {
    const int rc = q + kLoraVG * k;
    vq[k] = (q < kLoraVG && rc < a.nrc) ? load_coherent(a.vpart + (size_t)rc * R + i) : 0.0f;
  }
}
__device__ __forceinline__ void lora_vu_finish(const DecodeArgs &a, const float (&vq)[kLoraVQ], DecodeSmem &sm) {
  const int R = a.rank, tid = threadIdx.x, i = tid % R, q = tid / R;
  float *flat = &sm.lv[0][0][0];
  float v = 0.0f;
#pragma unroll
  for (int k = 0; k < kLoraVQ; ++k) v += vq[k];
  const int rest = a.nrc - q - kLoraVG * kLoraVQ;  // chunks past the first loads
  if (q < kLoraVG && rest > 0)
    v += sum_coherent(a.vpart + (size_t)(q + kLoraVG * kLoraVQ) * R + i, (size_t)kLoraVG * R,
                      (rest + kLoraVG - 1) / kLoraVG);
  flat[tid] = v;
  __syncthreads();
  if (tid < R) {
    float u = 0.0f;
#pragma unroll
    for (int g = 0; g < kLoraVG; ++g) u += flat[g * R + tid];
    sm.lz[tid] = u;
  }
}

// LoRA: for the kept rows list[i0 .. i0 + mn) of a unit, w_i = s (h A_up) .
// B_up_T[j] into lr.lw and A_down[j] into lr.lad (R / VEC adjacent threads
// per row, 16 bytes each).  The loads of the first pass are issued before
// the unit's first row batches (loads complete in issue order) and used
// after them; further passes (more than THREADS / (R / VEC) rows) follow.
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

// Rows phase of workgroup w (of G): units w, w + G, ... of nblk x S units
// (S = max(1, G / nblk) shares per column block); writes the workgroup's
// partial y.  h is formed first (its loads overlap the first block's partial
// sums).
template <typename T, bool LORA>
__device__ void dec_rows(const DecodeArgs &a, int l, int base, int G, int w, DecodeSmem &sm, LoraRows<T> &lr) {
  constexpr int VEC = Elem<T>::kVec, NW = kDecodeWaves;
  constexpr int CB = dec_block_cols<T>();
  constexpr int CH = 64 * VEC;              // elements per chunk (one 16-byte load per lane)
  constexpr int DMAX = kDecodeMaxD / CH;    // chunks per row
  constexpr int NCH = (DMAX + 7) / 8;       // chunks per wavefront of a half
  constexpr int R = 8 / NCH;                // rows of two batches (2 x 8 loads in flight per lane)
  constexpr int RB = R > 2 ? R / 4 : 1;     // rows per batch
  static_assert(CB <= kDecodeThreads / 2 && 4 * R * 8 <= 2 * kDecodeMaxD, "single-token tiling");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6), hw = wv & 7, hf = wv >> 3;
  const int d = a.d, d_ff = a.d_ff, nblk = a.nblk;
  const size_t wl = (size_t)d * d_ff;
  const int S = max(1, G / nblk), units = nblk * S;
  const float thr = base ? 0.0f : a.thr[l];
  const __amdgpu_buffer_rsrc_t Wu = weight_rsrc(static_cast<const T *>(a.Wu) + (size_t)l * wl, (uint32_t)(wl * sizeof(T)));
  const __amdgpu_buffer_rsrc_t Wd = weight_rsrc(static_cast<const T *>(a.Wd) + (size_t)l * wl, (uint32_t)(wl * sizeof(T)));
  const __amdgpu_buffer_rsrc_t gp =
      weight_rsrc(a.gpart, (uint32_t)((size_t)d_ff * dec_nrcp(a.nrc) * sizeof(float)));

  InputRegs<kDecodeThreads> ir;
  float hreg[NCH][VEC];  // h at this lane's columns
  float yacc[NCH][VEC];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int v = 0; v < VEC; ++v) hreg[c][v] = yacc[c][v] = 0.0f;
  int par = 0;  // LDS slot parity for the parts of u
  const bool lora = LORA && !base;
  float zh = 0.0f;  // LoRA, lane i < rank of wavefront 0 of each half: z_i over the half's kept rows
  float vq[kLoraVQ];
  if (lora) {
    lora_vu_issue(a, vq);
    asm volatile("" ::: "memory");  // keeps these loads ahead of the partial sums' and the rows'
  }

  for (int un = w; un < units; un += G) {
    const int cb = un % nblk, sub = un / nblk;
    // the block's keep list (every workgroup of the block forms the same one)
    const int gcol = cb * CB + tid;
    bool keep = false;
    float g = 0.0f;
    if (tid < CB && gcol < d_ff) {
      g = silu(gate_sum(gp, gcol, a.nrc));
      keep = base || (fabsf(g) >= thr);
      if (sub == 0 && a.keep_out) a.keep_out[(size_t)l * d_ff + gcol] = (uint8_t)keep;
    }
    // h's loads follow the partials' (the keep list is on the critical path)
    // and are waited for only after the first rows are issued
    if (un == w) dec_input_issue<T, kDecodeThreads>(a, l, ir);
    const uint64_t bal = __ballot(keep);
    const int rank = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) sm.wcnt[wv] = __popcll(bal);
    __syncthreads();
    int off = 0, tot = 0;
    for (int i = 0; i < NW; ++i) {
      off += (i < wv) ? sm.wcnt[i] : 0;
      tot += sm.wcnt[i];
    }
    if (keep) {
      sm.mj[off + rank] = gcol;
      sm.mg[off + rank] = g;
    }
    __syncthreads();
    // this unit's rows: list[i0, i0 + mn); half hf takes [b, e)
    const int i0 = (int)(((int64_t)sub * tot) / S);
    const int mn = (int)(((int64_t)(sub + 1) * tot) / S) - i0;
    const int hn = (mn + 1) / 2;
    const int b = i0 + hf * hn, e = i0 + min(mn, (hf + 1) * hn);
    if (l == 0 && un == w) SATS_TRACE_POINT(4);
    if (lora && un == w) lora_vu_finish(a, vq, sm);
    // batches of RB rows in two register sets: the next batch is always in
    // flight while one is used (both halves run the same number of batches)
    const int nbt = (hn + RB - 1) / RB;
    u32x4 au[RB][NCH], ad[RB][NCH], cu[RB][NCH], cd[RB][NCH];
    LoraPrepRegs<T> lp;
    if (lora) lora_prep_load<T>(a, l, sm, i0, mn, 0, lp);
    if (nbt > 0) rows_issue<T, RB, NCH>(Wu, Wd, sm, b, e, d, au, ad);
    if (nbt > 1) rows_issue<T, RB, NCH>(Wu, Wd, sm, b + RB, e, d, cu, cd);
    if (un == w) {
      dec_input_finish<T, kDecodeThreads>(a, l, ir, sm, false);
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
          const int k = (hw + c * 8) * CH + lane * VEC + v;
          hreg[c][v] = (k < d) ? sm.hs[k] : 0.0f;
        }
    }
    if (lora) {  // the up adapter's terms and A_down of this unit's rows
      if (l == 0 && un == w) SATS_TRACE_POINT(8);
      const int rq = a.rank / VEC;
      lora_prep_use<T>(a, sm, lr, i0, mn, 0, lp);
      for (int b0 = kDecodeThreads; b0 < mn * rq; b0 += kDecodeThreads) {
        lora_prep_load<T>(a, l, sm, i0, mn, b0, lp);
        lora_prep_use<T>(a, sm, lr, i0, mn, b0, lp);
      }
      __syncthreads();
      if (l == 0 && un == w) SATS_TRACE_POINT(9);
    }
    for (int i = 0; i < nbt; i += 2) {
      rows_consume<T, RB, NCH>(sm, hreg, yacc, b + i * RB, e, par, au, ad, lora, lr, a.rank, zh);
      par ^= 1;
      if (i + 2 < nbt) rows_issue<T, RB, NCH>(Wu, Wd, sm, b + (i + 2) * RB, e, d, au, ad);
      if (i + 1 < nbt) {
        rows_consume<T, RB, NCH>(sm, hreg, yacc, b + (i + 1) * RB, e, par, cu, cd, lora, lr, a.rank, zh);
        par ^= 1;
        if (i + 3 < nbt) rows_issue<T, RB, NCH>(Wu, Wd, sm, b + (i + 3) * RB, e, d, cu, cd);
      }
    }
    __syncthreads();  // the next unit rewrites the list
  }
  if (lora) {  // z = half 0's sum + half 1's
    if (wv == 8 && lane < a.rank) lr.lw[lane] = zh;
    __syncthreads();
    if (wv == 0 && lane < a.rank) store_coherent(a.zpart + (size_t)w * a.rank + lane, zh + lr.lw[lane]);
    if (l == 0) SATS_TRACE_POINT(10);
  }
  if (l == 0) SATS_TRACE_POINT(5);
  // the two halves' sums, added in half order, are this workgroup's partial y
  float *hsum = sm.red;  // [d]
  if (hf == 1) {
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int k = (hw + c * 8) * CH + lane * VEC;
      if (k < d) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) hsum[k + v] = yacc[c][v];
      }
    }
  }
  __syncthreads();
  if (hf == 0) {
    const __amdgpu_buffer_rsrc_t yr = weight_rsrc(a.ypart + (size_t)w * d, (uint32_t)(d * sizeof(float)));
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int k = (hw + c * 8) * CH + lane * VEC;
      if (k < d) {
#pragma unroll
        for (int v = 0; v < VEC; v += 4)
          store_coherent4(yr, (uint32_t)((k + v) * sizeof(float)), yacc[c][v] + hsum[k + v],
                          yacc[c][v + 1] + hsum[k + v + 1], yacc[c][v + 2] + hsum[k + v + 2],
                          yacc[c][v + 3] + hsum[k + v + 3]);
      }
    }
  }
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

// Gate tiles (any grid); LORA: with the adapters of the sparse path.
template <typename T, bool LORA>
__global__ __launch_bounds__(kGateThreads) void dec_gate_kernel(DecodeArgs a, int l) {
  __shared__ DecodeSmem sm;
  __shared__ LoraGateSmem ls;
  if (blockIdx.x == 0 && threadIdx.x == 0)  // the previous rows launch has finished
    __hip_atomic_store(a.done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (l == 0 && blockIdx.x == 0 && threadIdx.x == 0) {
    const int base = token_is_base(a.route_mode, a.ids, a.lut, 0);
    a.state[0] = base;
    if (a.route_out) a.route_out[0] = (uint8_t)base;
  }
  if (l == 0) SATS_TRACE_POINT(0);
  dec_gate<T, LORA>(a, l, sm, ls, a.layer_in != nullptr && blockIdx.x == 0);
  if (l == 0) SATS_TRACE_POINT(2);
}

// Rows: G workgroups, each writing its partial y.  Without adapters the
// second reduction stage is a launch of its own (dec_reduce_kernel).  With
// adapters it follows in this launch: the last RW workgroups to finish each
// sum one slice of y (and add s z B_down) over every partial (workgroup
// order).  They wait only for workgroups that are running or done, with
// nothing of their own in flight; the wait is bounded (it raises the device
// error flag instead of hanging).  The count goes back to zero at the start
// of the next gate launch (which always comes before the next rows launch).
constexpr int kSpinLimit = 1 << 20;  // polls of one wait (each a device-coherent load)

template <typename T, bool LORA>
__global__ __launch_bounds__(kDecodeThreads) void dec_rows_kernel(DecodeArgs a, int l) {
  __shared__ DecodeSmem sm;
  __shared__ LoraRows<T> lr;
  if (l == 0) SATS_TRACE_POINT(3);
  const int base = a.state[0];
  dec_rows<T, LORA>(a, l, base, a.G, blockIdx.x, sm, lr);
  if constexpr (!LORA) return;  // the second stage is dec_reduce_kernel
  const int tid = threadIdx.x, G = a.G;
  __builtin_amdgcn_s_waitcnt(0);  // this thread's partial-y stores have completed
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __syncthreads();
  if (tid == 0) sm.flag = (int)__hip_atomic_fetch_add(a.done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  const int ticket = sm.flag;
  if (ticket < G - a.RW) return;
  if (tid == 0) {
    int polls = 0;
    while (__hip_atomic_load(a.done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < (unsigned)G) {
      if (++polls >= kSpinLimit) {
        __hip_atomic_store(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __syncthreads();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  if (l == 0) SATS_TRACE_POINT(6);
  dec_reduce<T, LORA>(a, l, ticket - (G - a.RW), sm, base);
  if (l == 0) SATS_TRACE_POINT(7);
}


// Second reduction stage of a layer without adapters, a launch of its own
// (the kernel boundary orders it after every partial; a hand-off inside the
// rows launch -- last arrivals counted, the reducers waiting for the count --
// measured 2 us slower per layer, its stores and polls queued behind the
// other workgroups' row loads).  Workgroup w owns columns [16 w, 16 w + 16):
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
