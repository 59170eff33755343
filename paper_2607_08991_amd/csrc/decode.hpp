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

constexpr int kDecodeThreads = 1024;  // rows and reduce launches
constexpr int kDecodeWaves = kDecodeThreads / 64;
#ifndef SATS_GATE_THREADS
#define SATS_GATE_THREADS 1024
#endif
constexpr int kGateThreads = SATS_GATE_THREADS;  // gate launch
constexpr int kGateBatch = kGateThreads >= 1024 ? 8 : 16;  // 16-byte loads in flight per lane
constexpr int kDecodeMaxD = 4096;  // h lives in LDS
constexpr int kDecodeMaxG = 1024;  // rows / reduce workgroups (partials of y)

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
  int *state;             // [1] the token's route (1: base path), set by the layer-0 gate launch
  unsigned *done;         // [1] rows workgroups whose partial y is written (cleared by the gate launch)
  unsigned *err;          // device error flag (a bounded wait gave up)
  uint8_t *route_out;     // optional [1]
  uint8_t *keep_out;      // optional [L][d_ff]
  void *layer_in;         // optional [L][d]
};

struct DecodeSmem {
  float hs[kDecodeMaxD];                // layer input
  float red[2 * kDecodeMaxD];           // gate: wavefront partials; rows: parts of u, half sums
  int mj[kDecodeThreads / 2];           // kept columns of the current column block ...
  float mg[kDecodeThreads / 2];         // ... and their g values
  int wcnt[kDecodeWaves];
  float scal[kDecodeWaves];
  int flag;
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
  const int G = a.RW;  // slice sums of squares of the previous layer's reduce
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
        if (record) static_cast<T *>(a.layer_in)[(size_t)l * d + k] = hv;
      }
    }
  }
  __syncthreads();
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
template <typename T>
__device__ void dec_gate(const DecodeArgs &a, int l, DecodeSmem &sm, bool record) {
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
        gate_issue<T, GB, NW>(wr, row0, stride, r0, nr, lo, q);
        gate_consume<T, GB, NW>(sm, k0 + wv, r0, nr, q, acc);
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
                                             const u32x4 (&bu)[R][NCH], const u32x4 (&bd)[R][NCH]) {
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
    const float pr = (r0 + r < end) ? sm.mg[max(0, min(r0 + r, end - 1))] * ut : 0.0f;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int v = 0; v < VEC; ++v) yacc[c][v] = fmaf(pr, unpack<T>(bd[r][c], v), yacc[c][v]);
  }
}

// Rows phase of workgroup w (of G): units w, w + G, ... of nblk x S units
// (S = max(1, G / nblk) shares per column block); writes the workgroup's
// partial y.  h is formed first (its loads overlap the first block's partial
// sums).
template <typename T>
__device__ void dec_rows(const DecodeArgs &a, int l, int base, int G, int w, DecodeSmem &sm) {
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
    // batches of RB rows in two register sets: the next batch is always in
    // flight while one is used (both halves run the same number of batches)
    const int nbt = (hn + RB - 1) / RB;
    u32x4 au[RB][NCH], ad[RB][NCH], cu[RB][NCH], cd[RB][NCH];
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
    for (int i = 0; i < nbt; i += 2) {
      rows_consume<T, RB, NCH>(sm, hreg, yacc, b + i * RB, e, par, au, ad);
      par ^= 1;
      if (i + 2 < nbt) rows_issue<T, RB, NCH>(Wu, Wd, sm, b + (i + 2) * RB, e, d, au, ad);
      if (i + 1 < nbt) {
        rows_consume<T, RB, NCH>(sm, hreg, yacc, b + (i + 1) * RB, e, par, cu, cd);
        par ^= 1;
        if (i + 3 < nbt) rows_issue<T, RB, NCH>(Wu, Wd, sm, b + (i + 3) * RB, e, d, cu, cd);
      }
    }
    __syncthreads();  // the next unit rewrites the list
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
template <typename T>
__device__ void dec_reduce(const DecodeArgs &a, int l, int w, DecodeSmem &sm) {
  constexpr int THREADS = kDecodeThreads, NW = kDecodeWaves;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d = a.d, G = a.G;
  const int cpw = (d + a.RW - 1) / a.RW;  // columns of this workgroup (<= THREADS)
  const int cw0 = w * cpw;
  const int nc = max(0, min(cpw, d - cw0));
  const int ngr = THREADS / cpw;    // partial groups
  const int c = tid % cpw, gr = tid / cpw;
  float s = 0.0f;
  if (c < nc && gr < ngr && gr < G)
    s = sum_coherent(a.ypart + (size_t)gr * d + cw0 + c, (size_t)ngr * d, (G - gr + ngr - 1) / ngr);
  sm.red[tid] = s;
  __syncthreads();
  float y = 0.0f;
  if (tid < nc) {
    for (int qg = 0; qg < ngr && qg < G; ++qg) y += sm.red[qg * cpw + tid];
    if (l == a.L - 1) static_cast<T *>(a.out)[cw0 + tid] = Elem<T>::round(y);
    else store_coherent(a.ybuf + cw0 + tid, y);
  }
  float sq = (tid < nc) ? y * y : 0.0f;  // slice sum of squares, fixed order
  sq = wave_sum(sq);
  if (lane == 0) sm.scal[wv] = sq;
  __syncthreads();
  if (tid == 0 && l < a.L - 1) {
    float tot = 0.0f;
    for (int i = 0; i < NW; ++i) tot += sm.scal[i];
    store_coherent(a.sspart + w, tot);
  }
}

// ------------------------------------------------------------------ kernels

// Gate tiles (any grid).
template <typename T>
__global__ __launch_bounds__(kGateThreads) void dec_gate_kernel(DecodeArgs a, int l) {
  __shared__ DecodeSmem sm;
  if (blockIdx.x == 0 && threadIdx.x == 0)  // the previous rows launch has finished
    __hip_atomic_store(a.done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (l == 0 && blockIdx.x == 0 && threadIdx.x == 0) {
    const int base = token_is_base(a.route_mode, a.ids, a.lut, 0);
    a.state[0] = base;
    if (a.route_out) a.route_out[0] = (uint8_t)base;
  }
  if (l == 0) SATS_TRACE_POINT(0);
  dec_gate<T>(a, l, sm, a.layer_in != nullptr && blockIdx.x == 0);
  if (l == 0) SATS_TRACE_POINT(2);
}

// Rows: G workgroups, then the second reduction stage: the last RW of them
// to finish each sum one slice of y over every partial (workgroup order).
// They wait only for workgroups that are running or done, with nothing of
// their own in flight; the wait is bounded (it raises the device error
// flag instead of hanging).  The count goes back to zero at the start of the
// next gate launch (which always comes before the next rows launch).
constexpr int kSpinLimit = 1 << 20;  // polls of one wait (each a device-coherent load)

template <typename T>
__global__ __launch_bounds__(kDecodeThreads) void dec_rows_kernel(DecodeArgs a, int l) {
  __shared__ DecodeSmem sm;
  if (l == 0) SATS_TRACE_POINT(3);
  dec_rows<T>(a, l, a.state[0], a.G, blockIdx.x, sm);
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
  dec_reduce<T>(a, l, ticket - (G - a.RW), sm);
  if (l == 0) SATS_TRACE_POINT(7);
}


}  // namespace sats
