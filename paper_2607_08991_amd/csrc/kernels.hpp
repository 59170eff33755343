// Device kernels of the routed, threshold-sparsified gated MLP (gfx950).
//
// One layer runs as three kernels over a tile of at most NT tokens
// (blockIdx.z selects the tile):
//
//   gate_kernel   a_j = W_gate_T[j] . h (split over chunks of d), then the last
//                 workgroup to finish a column block sums the row-split
//                 partials in a fixed order and applies SiLU (Eq. 2), the
//                 keep rule |g| >= t (Eq. 4-5; every column for base-path
//                 tokens, Eq. 13) and compacts the kept columns of the block
//                 with a wavefront ballot and an LDS prefix.  The layer input h
//                 is built here: the call's input x for layer 0, otherwise the
//                 previous layer's y normalised by its root mean square.
//   up_kernel     one wavefront per kept row j of W_up_T: u_j = W_up_T[j] . h,
//                 p_j = g_j u_j (Eq. 1), written at the row's compacted position.
//   down_kernel   y = sum_j p_j W_down[j]: split over column slices of W_down
//                 and over chunks of the kept-row list; the last workgroup of a
//                 slice sums the chunk partials in a fixed order and writes y
//                 (or the rounded output for the last layer) and the slice's
//                 sum of squares for the next layer's normalisation.
//
// Cross-workgroup hand-off (partials -> last workgroup) uses device-coherent
// stores and loads and an agent-scope counter; the counters reset themselves
// so no memset is needed between launches.  No floating-point atomics: results are
// deterministic.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sats {

constexpr int kThreads = 256;
constexpr int kGateCols = 64;  // gate columns per column block of the batch kernels
constexpr float kGlueEps = 1e-6f;

// ------------------------------------------------------------------ elements

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// float -> bfloat16 bits, round to nearest even (from the bit layout: add half
// an ulp of the kept part, plus one when the kept part is odd, then truncate)
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Elem;
template <> struct Elem<uint16_t> {  // bfloat16 storage
  static constexpr int kVec = 8;     // elements per 16-byte load
  __device__ __forceinline__ static float get(const uint16_t *p) { return bf16_to_f32(*p); }
  __device__ __forceinline__ static uint16_t round(float f) { return f32_to_bf16(f); }
  __device__ __forceinline__ static float value(uint16_t s) { return bf16_to_f32(s); }
};
template <> struct Elem<float> {
  static constexpr int kVec = 4;
  __device__ __forceinline__ static float get(const float *p) { return *p; }
  __device__ __forceinline__ static float round(float f) { return f; }
  __device__ __forceinline__ static float value(float s) { return s; }
};

// VEC consecutive elements starting at p as float32.  VEC > 1 requires p to be
// 16-byte aligned (the host only selects the vector path when it is).
template <typename T, int VEC>
__device__ __forceinline__ void load_vec(const T *__restrict__ p, float (&w)[VEC]) {
  if constexpr (VEC == 1) {
    w[0] = Elem<T>::get(p);
  } else if constexpr (sizeof(T) == 2) {
    static_assert(VEC == 8, "bf16 vector width");
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      w[2 * i] = __uint_as_float(q[i] << 16);
      w[2 * i + 1] = __uint_as_float(q[i] & 0xffff0000u);
    }
  } else {
    static_assert(VEC == 4, "f32 vector width");
    const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(p));
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  }
}

// Raw 16-byte loads, unpacked element by element where they are used (keeps
// bf16 data packed in registers).
template <typename T>
__device__ __forceinline__ u32x4 load_raw(const T *__restrict__ p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}
template <typename T>
__device__ __forceinline__ float unpack(const u32x4 &q, int v) {
  if constexpr (sizeof(T) == 2) {
    const uint32_t w = q[v >> 1];
    return __uint_as_float((v & 1) ? (w & 0xffff0000u) : (w << 16));
  } else {
    return __uint_as_float(q[v]);
  }
}

// Same for small, reused operands (cached load).
template <typename T, int VEC>
__device__ __forceinline__ void load_vec_cached(const T *__restrict__ p, float (&w)[VEC]) {
  if constexpr (VEC == 1) {
    w[0] = Elem<T>::get(p);
  } else if constexpr (sizeof(T) == 2) {
    const u32x4 v = *reinterpret_cast<const u32x4 *>(p);
    const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      w[2 * i] = __uint_as_float(q[i] << 16);
      w[2 * i + 1] = __uint_as_float(q[i] & 0xffff0000u);
    }
  } else {
    const f32x4 v = *reinterpret_cast<const f32x4 *>(p);
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  }
}

__device__ __forceinline__ float silu(float a) { return a / (1.0f + __expf(-a)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Cross-workgroup hand-off without cache-wide maintenance.  Partials that
// another workgroup will read are written with device-coherent stores
// (agent-scope atomic stores: written through to the device-coherent level)
// and read back with device-coherent loads, so no L2 writeback or invalidate
// is needed.  arrive_last() waits for this thread's stores to complete,
// counts one arrival of the workgroup and reports whether it was the last of
// `expected`; the last arrival resets the counter for the next launch.
__device__ __forceinline__ void store_coherent(float *p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float *p) {
  return __hip_atomic_load(const_cast<float *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// sum_{q < n} p[q * stride], added in index order.  The loads are issued 16 at
// a time before any is used (one memory latency per 16 terms instead of one
// per term); addresses past n are clamped in bounds and their values dropped.
__device__ __forceinline__ float sum_coherent(const float *p, size_t stride, int n) {
  float s = 0.0f;
  for (int q0 = 0; q0 < n; q0 += 16) {
    float v[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) v[q] = load_coherent(p + (size_t)min(q0 + q, n - 1) * stride);
#pragma unroll
    for (int q = 0; q < 16; ++q)
      if (q0 + q < n) s += v[q];
  }
  return s;
}

__device__ __forceinline__ bool arrive_last(unsigned *counter, unsigned expected, int *flag_lds) {
  __builtin_amdgcn_s_waitcnt(0);  // this thread's coherent stores have completed
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = (prev == expected - 1);
    if (last) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *flag_lds = last;
  }
  __syncthreads();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  return *flag_lds != 0;
}

// Route modes: every token sparse, table lookup, every token base.
enum { ROUTE_SPARSE = 0, ROUTE_LUT = 1, ROUTE_BASE = 2 };

__device__ __forceinline__ int token_is_base(int mode, const int32_t *ids, const uint8_t *lut, int tok) {
  if (mode == ROUTE_BASE) return 1;
  if (mode == ROUTE_LUT) return lut[ids[tok]] != 0;
  return 0;
}

// ------------------------------------------------------------------ gate

struct GateArgs {
  const void *W;         // W_gate_T of this layer, [d_ff][d]
  const void *x;         // layer 0: call input [n][d]; otherwise null
  const float *ybuf;     // layer > 0: previous layer's y, [P][d]
  const float *ss;       // layer > 0: per-slice sums of y^2, [tiles][n_slices][NT]
  int n_slices;
  void *hbuf;            // layer input h, [P][d] (written by column block 0)
  void *layer_in;        // optional copy of h for inspection, [n][d]
  const float *thr;      // threshold of this layer (device), unused in base mode
  const int32_t *ids;
  const uint8_t *lut;
  int route_mode;
  uint8_t *route_out;    // optional, [n]
  float *gpart;          // [tiles][KS][NT][d_ff]
  unsigned *gcnt;        // [tiles][nblocks]
  float *gval;           // [tiles][NT][d_ff]
  int *blk_cnt;          // [tiles][nblocks]
  int *blk_idx;          // [tiles][d_ff], block b's entries from b*CB
  uint32_t *blk_mask;    // [tiles][d_ff], bit t = token t keeps the column
  uint8_t *keep_out;     // optional, [tiles][NT][d_ff]
  const uint8_t *skip;   // [n] 1: token done by the dense MFMA path (see dense.hpp)
  const int *ctl;        // [0] tokens on that path
  int n, d, d_ff, KS, KC, nblocks;
};

template <typename T, int VEC, int NT>
__global__ __launch_bounds__(kThreads) void gate_kernel(GateArgs a) {
  constexpr int CB = kGateCols;  // columns per block
  constexpr int STEP = 64 * VEC;  // k covered by one wavefront load
  extern __shared__ float smem[];
  __shared__ int flag;
  __shared__ int wcnt[kThreads / 64];
  __shared__ float tscale[NT];
  __shared__ int tbase[NT];
  __shared__ int tskip[NT];
  const int tid = threadIdx.x;
  const int blk = blockIdx.x, ks = blockIdx.y, tile = blockIdx.z;
  if (a.ctl[0] == a.n && a.skip[0]) return;  // every token is on the dense MFMA path
  const int tok0 = tile * NT;
  const int nt = min(NT, a.n - tok0);
  const int k0 = ks * a.KC;
  const int kc = max(0, min(a.d, k0 + a.KC) - k0);
  const T *__restrict__ W = static_cast<const T *>(a.W);

  // ---- layer input for rows [k0, k0 + kc) of the tile's tokens
  if (tid < NT) {
    float s = 1.0f;
    int base = 0;
    if (tid < nt) {
      if (a.x == nullptr) {
        const float *ssp = a.ss + (size_t)tile * a.n_slices * NT + tid;
        float acc = 0.0f;
        for (int sl = 0; sl < a.n_slices; ++sl) acc += ssp[(size_t)sl * NT];
        s = sqrtf(acc / (float)a.d + kGlueEps);
      }
      base = token_is_base(a.route_mode, a.ids, a.lut, tok0 + tid);
      if (a.route_out && blk == 0 && ks == 0) a.route_out[tok0 + tid] = (uint8_t)base;
    }
    tscale[tid] = s;
    tbase[tid] = base;
    tskip[tid] = (tid < nt) ? a.skip[tok0 + tid] : 1;
  }
  __syncthreads();
  float *hs = smem;  // [NT][KC]
  for (int i = tid; i < NT * a.KC; i += kThreads) {
    const int t = i / a.KC, k = i - t * a.KC;
    float v = 0.0f;
    if (t < nt && k < kc) {
      const size_t off = (size_t)(tok0 + t) * a.d + k0 + k;
      T hv;
      if (a.x != nullptr) {
        hv = static_cast<const T *>(a.x)[off];
      } else {
        hv = Elem<T>::round(a.ybuf[off] / tscale[t]);
      }
      v = Elem<T>::value(hv);
      if (blk == 0) {
        static_cast<T *>(a.hbuf)[off] = hv;
        // a token on the dense MFMA path has its layer inputs written there
        if (a.layer_in && (a.x != nullptr || !tskip[t])) static_cast<T *>(a.layer_in)[off] = hv;
      }
    }
    hs[i] = v;
  }
  __syncthreads();

  // ---- partial gate projection over rows [k0, k0 + kc): wavefront wv takes
  // columns wv, wv + 4, ... of the block, each lane VEC consecutive weights of
  // a row of W_gate_T per load; the lanes are added in a fixed order
  const int lane = tid & 63, wv = tid >> 6;
  for (int cc = wv; cc < CB; cc += kThreads / 64) {
    const int col = blk * CB + cc;
    float u[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) u[t] = 0.0f;
    if (col < a.d_ff) {
      const T *__restrict__ wp = W + (size_t)col * a.d + k0;
      int k = lane * VEC;
      if constexpr (VEC > 1) {
        for (; k + STEP < kc; k += 2 * STEP) {  // two loads in flight
          const u32x4 w0 = load_raw<T>(wp + k), w1 = load_raw<T>(wp + k + STEP);
#pragma unroll
          for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
              u[t] = fmaf(hs[t * a.KC + k + v], unpack<T>(w0, v), u[t]);
              u[t] = fmaf(hs[t * a.KC + k + STEP + v], unpack<T>(w1, v), u[t]);
            }
        }
      }
      for (; k < kc; k += STEP) {
        float w[VEC];
        load_vec<T, VEC>(wp + k, w);
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int v = 0; v < VEC; ++v) u[t] = fmaf(hs[t * a.KC + k + v], w[v], u[t]);
      }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) u[t] = wave_sum(u[t]);
    if (lane == 0 && col < a.d_ff) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
        if (t < nt) store_coherent(a.gpart + (((size_t)tile * a.KS + ks) * NT + t) * a.d_ff + col, u[t]);
    }
  }

  // ---- the last workgroup of this column block finishes it
  if (!arrive_last(a.gcnt + (size_t)tile * a.nblocks + blk, (unsigned)a.KS, &flag)) return;

  const float thr = (a.route_mode == ROUTE_BASE) ? 0.0f : *a.thr;
  uint32_t mask = 0;
  const int col = blk * CB + tid;
  if (tid < CB && col < a.d_ff) {
    for (int t = 0; t < nt; ++t) {
      const float *pp = a.gpart + ((size_t)tile * a.KS * NT + t) * a.d_ff + col;
      const float s = sum_coherent(pp, (size_t)NT * a.d_ff, a.KS);
      const float g = silu(s);
      const bool keep = tbase[t] || (fabsf(g) >= thr);
      a.gval[((size_t)tile * NT + t) * a.d_ff + col] = g;
      mask |= (uint32_t)(keep && !tskip[t]) << t;
      if (a.keep_out && !tskip[t]) a.keep_out[((size_t)tile * NT + t) * a.d_ff + col] = (uint8_t)keep;
    }
  }
  const bool act = mask != 0;
  const uint64_t bal = __ballot(act);
  const int rank = __popcll(bal & ((1ull << lane) - 1ull));
  if (lane == 0) wcnt[wv] = __popcll(bal);
  __syncthreads();
  int off = 0;
  for (int w = 0; w < wv; ++w) off += wcnt[w];
  if (act) {
    const size_t e = (size_t)tile * a.d_ff + (size_t)blk * CB + off + rank;
    a.blk_idx[e] = col;
    a.blk_mask[e] = mask;
  }
  if (tid == 0) {
    int tot = 0;
    for (int w = 0; w < kThreads / 64; ++w) tot += wcnt[w];
    a.blk_cnt[(size_t)tile * a.nblocks + blk] = tot;
  }
}

// ------------------------------------------------------------------ up

struct UpArgs {
  const void *W;          // W_up_T of this layer, [d_ff][d]
  const void *hbuf;       // [P][d]
  const float *gval;      // [tiles][NT][d_ff]
  const int *blk_cnt;     // [tiles][nblocks]
  const int *blk_idx;     // [tiles][d_ff]
  const uint32_t *blk_mask;
  float *pbuf;            // [tiles][NT][d_ff], by compacted position
  int *jlist;             // [tiles][d_ff], row index by compacted position
  int *ucount;            // [tiles]
  const uint8_t *skip;
  const int *ctl;
  int n, d, d_ff, nblocks, CB;
};

template <typename T, int VEC, int NT>
__global__ __launch_bounds__(kThreads) void up_kernel(UpArgs a) {
  extern __shared__ int pref[];  // [nblocks + 1]
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int tile = blockIdx.y;
  if (a.ctl[0] == a.n && a.skip[0]) return;  // every token is on the dense MFMA path
  const int tok0 = tile * NT;
  const int nt = min(NT, a.n - tok0);
  const int *cnt = a.blk_cnt + (size_t)tile * a.nblocks;

  // exclusive prefix of the per-block kept counts (wavefront 0, 64 at a time)
  if (wv == 0) {
    int carry = 0;
    for (int b0 = 0; b0 < a.nblocks; b0 += 64) {
      const int b = b0 + lane;
      const int v = (b < a.nblocks) ? cnt[b] : 0;
      int incl = v;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int u = __shfl_up(incl, o, 64);
        if (lane >= o) incl += u;
      }
      if (b < a.nblocks) pref[b] = carry + incl - v;
      carry += __shfl(incl, 63, 64);
    }
    if (lane == 0) pref[a.nblocks] = carry;
  }
  __syncthreads();
  const int U = pref[a.nblocks];
  if (blockIdx.x == 0 && tid == 0) a.ucount[tile] = U;

  const T *__restrict__ W = static_cast<const T *>(a.W);
  const T *__restrict__ H = static_cast<const T *>(a.hbuf) + (size_t)tok0 * a.d;
  const int nw = gridDim.x * (kThreads / 64);
  for (int pos = blockIdx.x * (kThreads / 64) + wv; pos < U; pos += nw) {
    // block holding compacted position pos: largest b with pref[b] <= pos
    int lo = 0, hi = a.nblocks - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (pref[mid] <= pos) lo = mid; else hi = mid - 1;
    }
    const size_t e = (size_t)tile * a.d_ff + (size_t)lo * a.CB + (pos - pref[lo]);
    const int j = a.blk_idx[e];
    const uint32_t m = a.blk_mask[e];
    const T *__restrict__ wr = W + (size_t)j * a.d;
    float u[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) u[t] = 0.0f;
    int k = lane * VEC;
    if constexpr (VEC > 1) {
      // 8 wavefront-wide loads of the row in flight at a time
      for (; k + 7 * 64 * VEC < a.d; k += 8 * 64 * VEC) {
        u32x4 wq[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) wq[q] = load_raw<T>(wr + k + q * 64 * VEC);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          if (t < nt && ((m >> t) & 1u)) {
#pragma unroll
            for (int q = 0; q < 8; ++q) {
              float h[VEC];
              load_vec_cached<T, VEC>(H + (size_t)t * a.d + k + q * 64 * VEC, h);
#pragma unroll
              for (int v = 0; v < VEC; ++v) u[t] = fmaf(h[v], unpack<T>(wq[q], v), u[t]);
            }
          }
        }
      }
    }
    for (; k < a.d; k += 64 * VEC) {
      float w[VEC];
      load_vec<T, VEC>(wr + k, w);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t < nt && ((m >> t) & 1u)) {
          float h[VEC];
          load_vec_cached<T, VEC>(H + (size_t)t * a.d + k, h);
#pragma unroll
          for (int v = 0; v < VEC; ++v) u[t] = fmaf(h[v], w[v], u[t]);
        }
      }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) u[t] = wave_sum(u[t]);
    if (lane == 0) {
      a.jlist[(size_t)tile * a.d_ff + pos] = j;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const size_t o = ((size_t)tile * NT + t) * a.d_ff;
        const bool on = t < nt && ((m >> t) & 1u);
        a.pbuf[o + pos] = on ? a.gval[o + j] * u[t] : 0.0f;
      }
    }
  }
}

// ------------------------------------------------------------------ down

struct DownArgs {
  const void *W;          // W_down of this layer, [d_ff][d]
  const float *pbuf;      // [tiles][NT][d_ff]
  const int *jlist;       // [tiles][d_ff]
  const int *ucount;      // [tiles]
  float *dpart;           // [tiles][KCH][NT][d]
  unsigned *dcnt;         // [tiles][n_slices]
  float *ybuf;            // [P][d]
  float *ss;              // [tiles][n_slices][NT]
  void *out;              // last layer: [n][d] (storage type); otherwise null
  const uint8_t *skip;    // tokens whose output the dense MFMA path writes
  const int *ctl;
  int n, d, d_ff, KCH, n_slices;
};

template <typename T, int VEC, int NT>
__global__ __launch_bounds__(kThreads) void down_kernel(DownArgs a) {
  constexpr int CL = (VEC == 1) ? 64 : 16;
  constexpr int RG = kThreads / CL;
  constexpr int SW = CL * VEC;  // columns per slice
  extern __shared__ float smem[];
  __shared__ int flag;

  const int tid = threadIdx.x;
  const int slice = blockIdx.x, ch = blockIdx.y, tile = blockIdx.z;
  if (a.ctl[0] == a.n && a.skip[0]) return;  // every token is on the dense MFMA path
  const int tok0 = tile * NT;
  const int nt = min(NT, a.n - tok0);
  const int U = a.ucount[tile];
  const int R = (U + a.KCH - 1) / a.KCH;
  const int p0 = ch * R, p1 = min(U, p0 + R);
  const int cl = tid % CL, rg = tid / CL;
  const int c0 = slice * SW + cl * VEC;
  const T *__restrict__ W = static_cast<const T *>(a.W);
  const int *__restrict__ jl = a.jlist + (size_t)tile * a.d_ff;
  const float *__restrict__ pb = a.pbuf + (size_t)tile * NT * a.d_ff;

  float acc[NT][VEC];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[t][v] = 0.0f;
  if (c0 < a.d) {
    int pos = p0 + rg;
    if constexpr (VEC > 1) {
      // whole batches of 8 rows: row indices, then 8 row loads in flight
      for (; pos + 7 * RG < p1; pos += 8 * RG) {
        int jj[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) jj[u] = jl[pos + u * RG];
        u32x4 wq[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) wq[u] = load_raw<T>(W + (size_t)jj[u] * a.d + c0);
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            const float pv = pb[(size_t)t * a.d_ff + pos + u * RG];
#pragma unroll
            for (int v = 0; v < VEC; ++v) acc[t][v] = fmaf(pv, unpack<T>(wq[u], v), acc[t][v]);
          }
      }
    }
    for (; pos < p1; pos += RG) {
      const int j = jl[pos];
      float w[VEC];
      load_vec<T, VEC>(W + (size_t)j * a.d + c0, w);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const float pv = pb[(size_t)t * a.d_ff + pos];
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[t][v] = fmaf(pv, w[v], acc[t][v]);
      }
    }
  }
  float *red = smem;  // [RG][NT][SW]
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int v = 0; v < VEC; ++v) red[(rg * NT + t) * SW + cl * VEC + v] = acc[t][v];
  __syncthreads();
  for (int o = tid; o < NT * SW; o += kThreads) {
    const int t = o / SW, c = o - t * SW;
    const int col = slice * SW + c;
    if (t < nt && col < a.d) {
      float s = 0.0f;
#pragma unroll
      for (int r = 0; r < RG; ++r) s += red[(r * NT + t) * SW + c];
      store_coherent(a.dpart + (((size_t)tile * a.KCH + ch) * NT + t) * a.d + col, s);
    }
  }

  if (!arrive_last(a.dcnt + (size_t)tile * a.n_slices + slice, (unsigned)a.KCH, &flag)) return;

  float *yv = smem;  // [NT][SW]; red is no longer needed
  __syncthreads();
  for (int o = tid; o < NT * SW; o += kThreads) {
    const int t = o / SW, c = o - t * SW;
    const int col = slice * SW + c;
    float y = 0.0f;
    if (t < nt && col < a.d) {
      const float *pp = a.dpart + ((size_t)tile * a.KCH * NT + t) * a.d + col;
      y = sum_coherent(pp, (size_t)NT * a.d, a.KCH);
      const size_t off = (size_t)(tok0 + t) * a.d + col;
      if (!a.skip[tok0 + t]) {
        if (a.out) static_cast<T *>(a.out)[off] = Elem<T>::round(y);
        else a.ybuf[off] = y;
      }
    }
    yv[o] = y;
  }
  __syncthreads();
  if (a.out == nullptr && tid < NT) {
    float s = 0.0f;
    for (int c = 0; c < SW; ++c) s = fmaf(yv[tid * SW + c], yv[tid * SW + c], s);
    a.ss[((size_t)tile * a.n_slices + slice) * NT + tid] = s;
  }
}

// ------------------------------------------------------------------ inspection

// Ascending list of the kept columns of one token at one layer.
struct CompactArgs {
  const uint8_t *keep;    // [tiles][NT][d_ff] == [P'][d_ff] with P' = tiles*NT
  const uint8_t *skip;    // unused (the MFMA path writes its own keep flags)
  int32_t *idx;           // [n][d_ff] (this layer, offset by the pass)
  int32_t *count;         // [n]
  int n, d_ff;
};

__global__ __launch_bounds__(kThreads) void compact_kernel(CompactArgs a) {
  __shared__ int wsum[kThreads / 64];
  __shared__ int carry_s;
  const int tok = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const uint8_t *kp = a.keep + (size_t)tok * a.d_ff;
  if (tid == 0) carry_s = 0;
  __syncthreads();
  for (int c0 = 0; c0 < a.d_ff; c0 += kThreads) {
    const int c = c0 + tid;
    const bool on = c < a.d_ff && kp[c];
    const uint64_t bal = __ballot(on);
    const int rank = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[wv] = __popcll(bal);
    __syncthreads();
    int off = carry_s;
    for (int w = 0; w < wv; ++w) off += wsum[w];
    if (on && a.idx) a.idx[(size_t)tok * a.d_ff + off + rank] = c;
    __syncthreads();
    if (tid == 0) {
      int s = 0;
      for (int w = 0; w < kThreads / 64; ++w) s += wsum[w];
      carry_s += s;
    }
    __syncthreads();
  }
  if (tid == 0 && a.count) a.count[tok] = carry_s;
}

}  // namespace sats
