// Host side of the C ABI declared in include/sats.h: argument checks,
// workspace management, launch planning and kernel timing.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "../../include/sats.h"
#include "kernels.hpp"
#include "decode.hpp"
#include "dense.hpp"
#include "calib.hpp"
#include "route.hpp"

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess) return fail(SATS_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

// --------------------------------------------------------------- kernel timing

struct Timer {
  bool armed = false;
  int cap = 0, used = 0;
  std::vector<hipEvent_t> start, stop;
};
std::mutex g_timer_mu;
Timer g_timer[SATS_K_COUNT];

// Start and stop events of one timed launch (null when its kind is not
// armed).  They are handed to hipExtLaunchKernelGGL, which takes the
// timestamps from the kernel's own dispatch, so the measured span is the
// kernel's execution and not a separate marker's.
struct TimedLaunch {
  hipEvent_t start = nullptr, stop = nullptr;
  TimedLaunch(int kind, hipStream_t) {  // kind < 0: an untimed launch
    if (kind < 0 || kind >= SATS_K_COUNT) return;
    Timer &tm = g_timer[kind];
    if (tm.armed && tm.used < tm.cap) {
      const int slot = tm.used++;
      start = tm.start[slot];
      stop = tm.stop[slot];
    }
  }
};

// --------------------------------------------------------------- planning

constexpr int kMaxPass = 64;  // tokens per pass through the layers

// d_ff chunks of the dense group's down-projection: about 256 workgroups,
// each chunk a whole number of 64-row stages
int dense_ksplit(int64_t d, int64_t d_ff) {
#ifdef SATS_KS
  return SATS_KS;
#endif
  const int64_t tiles = d / sats::kDenseDownNT;
  int64_t ks = std::max<int64_t>(1, (256 + tiles - 1) / tiles);
  ks = std::min<int64_t>(ks, std::min<int64_t>(sats::kDenseMaxKsplit, std::max<int64_t>(1, d_ff / sats::kDenseKC)));
  return (int)ks;
}

// MFMA kernels specialised on the 16-row tiles that cover a pass of np tokens
typedef void (*DenseKernel)(sats::DenseArgs);
DenseKernel dense_gateup_fn(int np, bool lora = false) {
  using namespace sats;
  const int mt = (np + 15) / 16;
  if (lora)
    return mt <= 1 ? dense_gateup_kernel<1, true> : mt == 2 ? dense_gateup_kernel<2, true>
                                                  : mt == 3 ? dense_gateup_kernel<3, true> : dense_gateup_kernel<4, true>;
  return mt <= 1 ? dense_gateup_kernel<1> : mt == 2 ? dense_gateup_kernel<2> : mt == 3 ? dense_gateup_kernel<3>
                                                                                        : dense_gateup_kernel<4>;
}
DenseKernel dense_down_fn(int np) {
  using namespace sats;
  const int mt = (np + 15) / 16;
  return mt <= 1 ? dense_down_kernel<1> : mt == 2 ? dense_down_kernel<2> : mt == 3 ? dense_down_kernel<3>
                                                                                    : dense_down_kernel<4>;
}

int round_pow2_down(int v) {
  int p = 1;
  while (p * 2 <= v) p *= 2;
  return p;
}

// Execution options of the calling thread (sats_set_options).
thread_local sats_options g_opt{};

// Compacted batch kernels: target workgroup counts of the gate and down
// launches and kept rows per wavefront of the up launch.
constexpr int kGateTarget = 2048, kDownTarget = 512, kUpRowsPerWave = 2;

struct Plan {
  int vec, CL, CB;         // down lanes per row segment; gate columns per block
  int nblocks;             // gate column blocks
  int KS, KC;              // gate row split
  int SW, n_slices, KCH;   // down column slices and list chunks
  int up_grid;             // up workgroups per tile
  int NT;                  // tokens per tile
};

Plan make_plan(int64_t d, int64_t d_ff, int esz, bool vec_ok, int n_pass) {
  Plan p{};
  p.vec = vec_ok ? 16 / esz : 1;
  p.CL = (p.vec == 1) ? 64 : 16;  // down-projection lanes per row segment
  p.CB = sats::kGateCols;
  p.nblocks = (int)((d_ff + p.CB - 1) / p.CB);
  p.NT = (n_pass == 1) ? 1 : 4;
  // gate: d in chunks of whole wavefront loads (64 x vec elements), about
  // kGateTarget workgroups, at most 1024 rows of h per chunk in LDS
  const int64_t step = 64 * (int64_t)p.vec;
  int64_t ks = round_pow2_down(std::max(1, kGateTarget / p.nblocks));
  ks = std::min<int64_t>(ks, std::max<int64_t>(1, d / step));
  ks = std::max<int64_t>(ks, (d + 1023) / 1024);
  p.KC = (int)((((d + ks - 1) / ks) + step - 1) / step * step);
  p.KS = (int)((d + p.KC - 1) / p.KC);
  p.SW = p.CL * p.vec;
  p.n_slices = (int)((d + p.SW - 1) / p.SW);
  p.KCH = std::max(1, kDownTarget / p.n_slices);
  int64_t waves = (d_ff + kUpRowsPerWave - 1) / kUpRowsPerWave;
  p.up_grid = (int)std::min<int64_t>(std::max<int64_t>(1, (waves + 3) / 4), 4096);
  return p;
}

// --------------------------------------------------------------- workspace

size_t align_up(size_t v) { return (v + 255) & ~size_t(255); }

struct Carve {
  char *base;
  size_t off = 0;
  template <typename T> T *take(size_t count) {
    T *p = reinterpret_cast<T *>(base ? base + off : nullptr);
    off += align_up(count * sizeof(T));
    return p;
  }
};

struct Buffers {
  void *hbuf;
  float *ybuf, *ss, *gpart, *gval, *pbuf, *dpart;
  int *blk_cnt, *blk_idx, *jlist, *ucount;
  uint32_t *blk_mask;
  uint8_t *keep;
  float *ypart, *sspart;  // single-token path: per-workgroup partial y and sums of squares
  float *dvpart, *dzpart; // single-token path, LoRA: partial h . A per input row chunk, z per layer workgroup
  int *perm, *ctl;        // batched path: token partition and dense-group control words
  uint8_t *skip, *gbase;
  uint16_t *xd, *hnext, *pdense;  // dense group (MFMA): inputs, next inputs, p
  int prows;                       // ... rows of each of those three
  uint8_t *uflag;                  // dense group: union of the keep sets per column
  float *ddpart;                   // dense group down-projection partials
  float *blv, *blvpart, *blzpart;  // batched LoRA: s (h A) per group row, its chunk partials, z per column tile
};

// Layout for passes of up to `pass` tokens (the counters live in their own
// zero-initialised allocation).
struct DecodePlan {
  int G = 0;           // layer workgroups, one partial y each (0: path not used)
  int cw = 0;          // gate columns per layer workgroup
  int RW = 0;          // reduce workgroups
  int nvc = 0;         // LoRA input launch: row chunks of the adapters' A matrices
  bool fused = false;  // second stage inside the layer launch (no adapters, few partials)
};

size_t layout(char *base, const Plan &p, int64_t pass, int64_t d, int64_t d_ff, int esz, int64_t L,
              const DecodePlan &dp, Buffers *b, int64_t lora_rank = 0) {
  const int64_t Pp = ((pass + 3) / 4) * 4;  // tokens rounded up to whole tiles
  const int64_t tiles = Pp;                  // upper bound over tile sizes
  Carve c{base};
  Buffers t{};
  t.hbuf = c.take<char>(Pp * d * esz);
  t.ybuf = c.take<float>(Pp * d);
  t.ss = c.take<float>(Pp * p.n_slices);
  t.gpart = c.take<float>(Pp * (int64_t)p.KS * d_ff);
  t.gval = c.take<float>(Pp * d_ff);
  t.pbuf = c.take<float>(Pp * d_ff);
  t.dpart = c.take<float>(Pp * (int64_t)p.KCH * d);
  t.blk_cnt = c.take<int>(tiles * p.nblocks);
  t.blk_idx = c.take<int>(tiles * d_ff);
  t.jlist = c.take<int>(tiles * d_ff);
  t.ucount = c.take<int>(tiles);
  t.blk_mask = c.take<uint32_t>(tiles * d_ff);
  t.keep = c.take<uint8_t>(std::max(Pp, L) * d_ff);
  t.ypart = c.take<float>((int64_t)dp.G * d);
  t.sspart = c.take<float>(std::max<int64_t>(std::max(dp.G, dp.RW), (d + sats::kRedCols - 1) / sats::kRedCols));
  t.perm = c.take<int>(Pp);
  t.ctl = c.take<int>(64);
  t.skip = c.take<uint8_t>(Pp);
  t.gbase = c.take<uint8_t>(Pp);
  t.prows = (int)Pp;
  t.xd = c.take<uint16_t>(Pp * d);
  t.hnext = c.take<uint16_t>(Pp * d);
  t.pdense = c.take<uint16_t>(Pp * d_ff);
  t.uflag = c.take<uint8_t>(d_ff);
  t.ddpart = c.take<float>((int64_t)sats::kDenseMaxKsplit * Pp * d);
  t.dvpart = c.take<float>((int64_t)dp.nvc * 2 * sats::kLoraMaxRank);
  t.dzpart = c.take<float>((int64_t)dp.G * sats::kLoraMaxRank);
  if (lora_rank > 0) {  // batched LoRA calls only
    t.blv = c.take<float>(2 * (int64_t)sats::kDenseMaxTokens * lora_rank);
    t.blvpart = c.take<float>(2 * 4 * (int64_t)sats::kLoraVChunks * 16 * lora_rank);
    t.blzpart = c.take<float>((d_ff / 32) * (int64_t)sats::kDenseMaxTokens * lora_rank);  // tiles of >= 32 columns
  }
  if (b) *b = t;
  return c.off;
}

// The counter allocation starts with control words (the device error flag);
// the per-block counters follow.  Every counter is zero whenever no kernel is
// running.
constexpr size_t kCtl = 512;
constexpr size_t kErr = 320;
constexpr size_t kLoraV = 448;  // [8] batched LoRA: arrivals of the s (h A) chunks
constexpr size_t kDecDone = 324;  // single-token layer launch: workgroups finished (small layers)

size_t counter_count(const Plan &p, int64_t pass, const DecodePlan &dp) {
  const int64_t tiles = ((pass + 3) / 4) * 4;
  (void)dp;
  return kCtl + (size_t)std::max<int64_t>(tiles * p.nblocks + tiles * p.n_slices, 2 * (int64_t)p.nblocks + 64);
}

// ------------------------------------------------------- single-token plan

int device_cus();

// Columns per gate/up workgroup: 64, or d_ff spread evenly over the compute
// units (a multiple of 8, at least 32) when tiles of 64 would leave some of
// them idle (Llama shape: 256 tiles of 56; Qwen3: 256 of 48).
int dense_tile_cols(int64_t d_ff) {
  const int cus = std::max(1, device_cus());
  if (d_ff / sats::kDenseNT >= cus) return sats::kDenseNT;
  const int64_t nt = ((d_ff + cus - 1) / cus + 7) / 8 * 8;
  return (int)std::clamp<int64_t>(nt, 32, sats::kDenseNT);
}

int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return cus;
}


// Batch passes of np tokens: whether the matrix-core kernels run (bf16, the
// vector layout, shapes on their tiles and matrices below 2 GB) and whether
// they take every token (else the base-path group only).
bool batch_mfma(int esz, bool vec_ok, int np, bool lora, int64_t d, int64_t d_ff) {
  return esz == 2 && vec_ok && (np >= sats::kMfmaMinTokens || lora) && d % sats::kDenseDownNT == 0 &&
         d_ff % sats::kDenseKC == 0 && d <= 4096 && (uint64_t)d * d_ff * 2 < (1ull << 31) &&
         g_opt.batch_path != SATS_BATCH_COMPACT;
}
bool batch_whole() { return g_opt.batch_path != SATS_BATCH_SPLIT; }

struct Workspace {
  char *mem = nullptr;
  size_t bytes = 0;
  unsigned *counters = nullptr;
  size_t n_counters = 0;
};

std::mutex g_ws_mu;
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;

int ensure_workspace(hipStream_t stream, size_t bytes, size_t n_counters, Workspace **out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lk(g_ws_mu);
  Workspace &w = g_ws[{dev, stream}];
  if (w.bytes < bytes || w.n_counters < n_counters) {
    HIP_TRY(hipStreamSynchronize(stream));  // the old buffers may still be in use
    if (w.mem) HIP_TRY(hipFree(w.mem));
    if (w.counters) HIP_TRY(hipFree(w.counters));
    w = Workspace{};
    const size_t nb = std::max(bytes, (size_t)256);
    const size_t nc = std::max(n_counters, (size_t)64);
    if (hipMalloc(&w.mem, nb) != hipSuccess)
      return fail(SATS_ERR_WORKSPACE, "workspace allocation of %zu bytes failed", nb);
    if (hipMalloc(&w.counters, nc * sizeof(unsigned)) != hipSuccess) {
      (void)hipFree(w.mem);
      w = Workspace{};
      return fail(SATS_ERR_WORKSPACE, "counter allocation failed");
    }
    HIP_TRY(hipMemsetAsync(w.counters, 0, nc * sizeof(unsigned), stream));
    w.bytes = nb;
    w.n_counters = nc;
  }
  *out = &w;
  return SATS_OK;
}

// Single-token plan.  h is held in LDS (d <= kDecodeMaxD).  Layer workgroup
// w owns gate columns [cw w, cw w + cw): cw is the option, else the layer's
// weights (W_gate and about half of the other two) spread over workgroups of
// about kDecWgBytes each, at most one per compute unit, at most 64 columns.
// The second reduction stage: without adapters a launch of 16-column slices,
// or, for small layers (d <= kFusedMaxD, G <= kFusedMaxG), the last layer
// workgroup to finish; with adapters about 64 columns per workgroup (each one also
// sums every partial z), a whole number of 16-column slices.  Returns false
// when the shape does not fit.
constexpr int64_t kDecWgBytes = 64 << 10;

bool make_decode_plan(int64_t d, int64_t d_ff, int esz, DecodePlan *dp, int lora_rank = 0, int cus = -1) {
  DecodePlan q{};
  if (cus < 0) cus = device_cus();
  const int64_t wgs = std::min<int64_t>(std::max(cus, 1), std::max<int64_t>(1, (2 * d * d_ff * esz + kDecWgBytes - 1) / kDecWgBytes));
  int64_t cw = g_opt.dec_block_cols > 0 ? g_opt.dec_block_cols : (d_ff + wgs - 1) / wgs;
  cw = std::min<int64_t>(cw, sats::kDecodeMaxCols);
  q.cw = (int)cw;
  const int64_t G = (d_ff + cw - 1) / cw;
  q.G = (int)std::min<int64_t>(G, sats::kDecodeMaxG + 1);
  q.nvc = (int)((d + sats::kVRows - 1) / sats::kVRows);
  if (lora_rank > 0) {
    // second stage with adapters: slices of 32 columns (128 workgroups at
    // d = 4096; 64-column slices measured 0.6 us slower, 16-column ones 0.2)
    const int64_t rw0 = (d + 31) / 32;
    const int64_t cpw = (((d + rw0 - 1) / rw0 + sats::kRedCols - 1) / sats::kRedCols) * sats::kRedCols;
    q.RW = (int)((d + cpw - 1) / cpw);
  } else {
    q.RW = (int)((d + sats::kRedCols - 1) / sats::kRedCols);
  }
  // buffer descriptors address one layer's matrix with 32-bit offsets, and
  // 0x80000000 is the offset that reads zeros: every matrix must stay below 2 GB
  q.fused = lora_rank == 0 && d <= sats::kFusedMaxD && G <= sats::kFusedMaxG;
  const bool ok = G <= sats::kDecodeMaxG && d <= sats::kDecodeMaxD &&
                  (d + q.RW - 1) / q.RW <= sats::kDecodeThreads / (sats::kRedThreads / sats::kRedCols) &&
                  (uint64_t)d * (uint64_t)d_ff * (uint64_t)esz < (1ull << 31);
  *dp = ok ? q : DecodePlan{};
  return ok;
}

// ------------------------------------------------- allocation-free forward

// Device memory of sats_mlp_forward_noalloc: a fixed array per device (each
// GPU that runs the library holds its own copy until the process ends),
// arrival counters in the first kScratchCounterBytes, the workspace after
// them.  In host code `scratch` is only a stand-in for the symbol: its device
// address is taken once per device with hipGetSymbolAddress and only that
// address is passed to kernels and copies.
constexpr size_t kScratchBytes = (size_t)16 << 20;
constexpr size_t kScratchCounterBytes = (size_t)64 << 10;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
std::map<int, char *> g_scratch;  // device -> device address of its scratch

// The current device's scratch address (taken on the first call on a device).
int scratch_addr(char **out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch.find(dev);
  if (it == g_scratch.end()) {
    char *p = nullptr;
    const hipError_t e = hipGetSymbolAddress((void **)&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(SATS_ERR_HIP, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
    it = g_scratch.emplace(dev, p).first;
  }
  *out = it->second;
  return SATS_OK;
}

// Zeroes counters [0, n) except the device error flag (which keeps a raised
// error until sats_device_status reads it).  A kernel, not a memset, so that
// the call can be captured in a HIP graph.
__global__ void clear_counters_kernel(unsigned *c, int n, int keep) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    if (i != keep) c[i] = 0u;
}

// --------------------------------------------------------------- the call

struct Call {
  const void *x;
  const int32_t *ids;
  const void *Wg, *Wu, *Wd;
  const float *thr;
  const uint8_t *lut;
  void *out;
  int64_t n, d, d_ff, L;
  hipStream_t stream;
  int route_mode;
  // inspection (may be null)
  uint8_t *route_out;
  int32_t *active_count, *active_idx;
  void *layer_in;
  // LoRA adapters of the sparse path (Ag null: none)
  const void *Ag, *Bg, *Au, *BuT, *Ad, *Bd;
  int64_t rank;
  float lscale;
  // token tok of ntot: the single-token path's offsets into the inspection arrays
  int64_t tok, ntot;
  // allocation-free call: the workspace is the library's static scratch array
  bool noalloc;
};


template <typename T, int VEC, int NT>
int run_pass(const Call &c, const Plan &p, const Buffers &b, unsigned *counters, int64_t base, int np) {
  using namespace sats;
  const int tiles = (np + NT - 1) / NT;
  const int64_t d = c.d, d_ff = c.d_ff;
  const size_t wl = (size_t)d * (size_t)d_ff;
  unsigned *gcnt = counters + kCtl;
  unsigned *dcnt = gcnt + (size_t)tiles * p.nblocks;
  const bool inspect_lists = c.active_count || c.active_idx;

  // routing for the pass: partition, dense-group size and whether MFMA takes it
  const bool lora = c.Ag != nullptr;  // batched LoRA: the whole pass on MFMA (checked by the caller)
  const bool mfma = batch_mfma((int)sizeof(T), VEC > 1, np, lora, d, d_ff);
  // whole batch on MFMA (each row applies its own keep rule): known here, so
  // the compacted sparse-path launches are left out
  const bool whole = batch_whole();
  const bool all_mfma = mfma && whole;
  if (lora && !all_mfma) return fail(SATS_ERR_SHAPE, "batched LoRA pass without the MFMA path");
  {
    RouteArgs ra{};
    ra.ids = c.ids ? c.ids + base : nullptr;
    ra.lut = c.lut;
    ra.route_mode = c.route_mode;
    ra.n = np;
    ra.d = (int)d;
    ra.x = static_cast<const uint16_t *>(c.x) + base * d;  // read only on the MFMA path (bf16)
    ra.perm = b.perm;
    ra.ctl = b.ctl;
    ra.skip = b.skip;
    ra.route_out = c.route_out ? c.route_out + base : nullptr;
    ra.xd = b.xd;
    ra.layer_in0 = c.layer_in ? static_cast<uint16_t *>(c.layer_in) + base * d : nullptr;
    ra.gbase = b.gbase;
    ra.mfma = mfma ? 1 : 0;
    ra.whole = whole ? 1 : 0;
    ra.min_group = lora ? 1 : kMfmaMinTokens;  // a LoRA pass has no other path for its tokens
    hipLaunchKernelGGL(route_kernel, dim3(np), dim3(kThreads), 0, c.stream, ra);
    HIP_TRY(hipGetLastError());
  }

  const int nt_gu = mfma ? dense_tile_cols(d_ff) : sats::kDenseNT;  // gate/up columns per workgroup
  for (int64_t l = 0; l < c.L; ++l) {
    if (mfma) {
      // base-path group on MFMA (kernels return at once when the group is small)
      DenseArgs da{};
      da.ctl = b.ctl;
      da.gbase = b.gbase;
      da.perm = b.perm;
      da.thr = c.thr ? c.thr + l : nullptr;
      da.keep_out = inspect_lists ? b.keep : nullptr;
      da.uflag = b.uflag;
      da.H = (l == 0) ? b.xd : b.hnext;
      da.Wg = static_cast<const uint16_t *>(c.Wg) + l * wl;
      da.Wt = static_cast<const uint16_t *>(c.Wu) + l * wl;
      da.P = b.pdense;
      da.K = (int)d;
      da.N = (int)d_ff;
      da.nt = nt_gu;
      da.hcap = b.prows;
      const size_t al = (size_t)d * c.rank;   // elements of A_gate, A_up (per layer)
      const size_t bl = (size_t)d_ff * c.rank;  // elements of B_gate, B_up_T, A_down (per layer)
      if (lora) {
        LoraVArgs va{};
        va.ctl = b.ctl;
        va.gbase = b.gbase;
        va.H = da.H;
        va.Ag = static_cast<const uint16_t *>(c.Ag) + l * al;
        va.Au = static_cast<const uint16_t *>(c.Au) + l * al;
        va.vpart = b.blvpart;
        va.lv = b.blv;
        va.cnt = counters + kLoraV;
        va.K = (int)d;
        va.R = (int)c.rank;
        va.s = c.lscale;
        {
          TimedLaunch tl(SATS_K_LORA_V, c.stream);
          hipExtLaunchKernelGGL(lora_v_kernel, dim3(kLoraVChunks, 4, 2), dim3(256), 0, c.stream, tl.start, tl.stop,
                                0, va);
        }
        HIP_TRY(hipGetLastError());
        da.lv = b.blv;
        da.Bg = static_cast<const uint16_t *>(c.Bg) + l * bl;
        da.BuT = static_cast<const uint16_t *>(c.BuT) + l * bl;
        da.Ad = static_cast<const uint16_t *>(c.Ad) + l * bl;
        da.zpart = b.blzpart;
        da.rank = (int)c.rank;
      }
      {
        TimedLaunch tl(SATS_K_DENSE, c.stream);
        hipExtLaunchKernelGGL(dense_gateup_fn(np, lora), dim3((unsigned)((d_ff + da.nt - 1) / da.nt)),
                              dim3(kDenseThreads), 0, c.stream, tl.start, tl.stop, 0, da);
      }
      HIP_TRY(hipGetLastError());
      DenseArgs dd{};
      dd.ctl = b.ctl;
      dd.H = b.pdense;
      dd.hcap = b.prows;
      dd.Wb = static_cast<const uint16_t *>(c.Wd) + l * wl;
      dd.part = b.ddpart;
      dd.uflag = b.uflag;
      dd.K = (int)d_ff;
      dd.N = (int)d;
      const int ks = dense_ksplit(d, d_ff);
      dd.kchunk = (int)(((d_ff + ks - 1) / ks + kDenseKC - 1) / kDenseKC * kDenseKC);
      {
        TimedLaunch tl(SATS_K_DENSE_DOWN, c.stream);
        hipExtLaunchKernelGGL(dense_down_fn(np), dim3(d / kDenseDownNT * ks), dim3(kDenseThreads), 0, c.stream,
                              tl.start, tl.stop, 0, dd);
      }
      HIP_TRY(hipGetLastError());
      GlueArgs ga{};
      ga.ctl = b.ctl;
      ga.perm = b.perm;
      ga.part = b.ddpart;
      ga.ksplit = ks;
      ga.d = (int)d;
      ga.out = (l == c.L - 1) ? static_cast<uint16_t *>(c.out) + base * d : nullptr;
      ga.hnext = b.hnext;
      ga.layer_in = (c.layer_in && l + 1 < c.L) ? static_cast<uint16_t *>(c.layer_in) + ((l + 1) * c.n + base) * d
                                                 : nullptr;
      if (lora) {
        ga.zpart = b.blzpart;
        ga.Bd = static_cast<const uint16_t *>(c.Bd) + l * (size_t)c.rank * d;
        ga.gbase = b.gbase;
        ga.rank = (int)c.rank;
        ga.nzb = (int)((d_ff + nt_gu - 1) / nt_gu);
        ga.lscale = c.lscale;
      }
      hipLaunchKernelGGL(dense_glue_kernel, dim3(np), dim3(kGlueThreads), 0, c.stream, ga);
      HIP_TRY(hipGetLastError());
    }
    auto compact = [&]() -> int {
      CompactArgs ca{};
      ca.keep = b.keep;
      ca.skip = b.skip;
      ca.idx = c.active_idx ? c.active_idx + (l * c.n + base) * d_ff : nullptr;
      ca.count = c.active_count ? c.active_count + l * c.n + base : nullptr;
      ca.n = np;
      ca.d_ff = (int)d_ff;
      TimedLaunch tl(SATS_K_INSPECT, c.stream);
      hipExtLaunchKernelGGL(compact_kernel, dim3(np), dim3(kThreads), 0, c.stream, tl.start, tl.stop, 0, ca);
      HIP_TRY(hipGetLastError());
      return SATS_OK;
    };
    if (all_mfma) {
      if (inspect_lists && compact() != SATS_OK) return SATS_ERR_HIP;
      continue;
    }
    GateArgs g{};
    g.W = static_cast<const T *>(c.Wg) + l * wl;
    g.x = (l == 0) ? static_cast<const void *>(static_cast<const T *>(c.x) + base * d) : nullptr;
    g.ybuf = b.ybuf;
    g.ss = b.ss;
    g.n_slices = p.n_slices;
    g.hbuf = b.hbuf;
    g.layer_in = c.layer_in ? static_cast<void *>(static_cast<T *>(c.layer_in) + (l * c.n + base) * d) : nullptr;
    g.thr = c.thr ? c.thr + l : nullptr;
    g.ids = c.ids ? c.ids + base : nullptr;
    g.lut = c.lut;
    g.route_mode = c.route_mode;
    g.route_out = (l == 0 && c.route_out) ? c.route_out + base : nullptr;
    g.gpart = b.gpart;
    g.gcnt = gcnt;
    g.gval = b.gval;
    g.blk_cnt = b.blk_cnt;
    g.blk_idx = b.blk_idx;
    g.blk_mask = b.blk_mask;
    g.keep_out = inspect_lists ? b.keep : nullptr;
    g.skip = b.skip;
    g.ctl = b.ctl;
    g.n = np;
    g.d = (int)d;
    g.d_ff = (int)d_ff;
    g.KS = p.KS;
    g.KC = p.KC;
    g.nblocks = p.nblocks;
    const size_t gate_lds = sizeof(float) * (size_t)NT * p.KC;
    {
      TimedLaunch tl(SATS_K_GATE, c.stream);
      hipExtLaunchKernelGGL((gate_kernel<T, VEC, NT>), dim3(p.nblocks, p.KS, tiles), dim3(kThreads), gate_lds,
                            c.stream, tl.start, tl.stop, 0, g);
    }
    HIP_TRY(hipGetLastError());

    if (inspect_lists && compact() != SATS_OK) return SATS_ERR_HIP;

    UpArgs u{};
    u.W = static_cast<const T *>(c.Wu) + l * wl;
    u.hbuf = b.hbuf;
    u.gval = b.gval;
    u.blk_cnt = b.blk_cnt;
    u.blk_idx = b.blk_idx;
    u.blk_mask = b.blk_mask;
    u.pbuf = b.pbuf;
    u.jlist = b.jlist;
    u.ucount = b.ucount;
    u.skip = b.skip;
    u.ctl = b.ctl;
    u.n = np;
    u.d = (int)d;
    u.d_ff = (int)d_ff;
    u.nblocks = p.nblocks;
    u.CB = p.CB;
    {
      TimedLaunch tl(SATS_K_UP, c.stream);
      hipExtLaunchKernelGGL((up_kernel<T, VEC, NT>), dim3(p.up_grid, tiles), dim3(kThreads),
                            sizeof(int) * (p.nblocks + 1), c.stream, tl.start, tl.stop, 0, u);
    }
    HIP_TRY(hipGetLastError());

    DownArgs dn{};
    dn.W = static_cast<const T *>(c.Wd) + l * wl;
    dn.pbuf = b.pbuf;
    dn.jlist = b.jlist;
    dn.ucount = b.ucount;
    dn.dpart = b.dpart;
    dn.dcnt = dcnt;
    dn.ybuf = b.ybuf;
    dn.ss = b.ss;
    dn.out = (l == c.L - 1) ? static_cast<void *>(static_cast<T *>(c.out) + base * d) : nullptr;
    dn.skip = b.skip;
    dn.ctl = b.ctl;
    dn.n = np;
    dn.d = (int)d;
    dn.d_ff = (int)d_ff;
    dn.KCH = p.KCH;
    dn.n_slices = p.n_slices;
    {
      TimedLaunch tl(SATS_K_DOWN, c.stream);
      hipExtLaunchKernelGGL((down_kernel<T, VEC, NT>), dim3(p.n_slices, p.KCH, tiles), dim3(kThreads),
                            sizeof(float) * (size_t)(kThreads / p.CL) * NT * p.SW, c.stream, tl.start, tl.stop, 0,
                            dn);
    }
    HIP_TRY(hipGetLastError());
  }
  return SATS_OK;
}

// The layer kernel for this call: with or without adapters, and rows split
// over groups of 2, 4 or 8 wavefronts by the number of 16-byte chunks per row.
template <typename T>
void (*dec_layer_fn(bool lora, int64_t d))(sats::DecodeArgs, int) {
  using namespace sats;
  const int64_t chunks = (d * (int64_t)sizeof(T) + 1023) / 1024;
  if (chunks <= 2) return lora ? dec_layer_kernel<T, true, 2> : dec_layer_kernel<T, false, 2>;
  if (chunks <= 4) return lora ? dec_layer_kernel<T, true, 4> : dec_layer_kernel<T, false, 4>;
  return lora ? dec_layer_kernel<T, true, 8> : dec_layer_kernel<T, false, 8>;
}

template <typename T>
int run_decode(const Call &c, const DecodePlan &dp, const Buffers &b, unsigned *counters) {
  using namespace sats;
  DecodeArgs a{};
  a.x = c.x;
  a.out = c.out;
  a.Wg = c.Wg;
  a.Wu = c.Wu;
  a.Wd = c.Wd;
  a.thr = c.thr;
  a.ids = c.ids;
  a.lut = c.lut;
  a.route_mode = c.route_mode;
  a.L = (int)c.L;
  a.d = (int)c.d;
  a.d_ff = (int)c.d_ff;
  a.cw = dp.cw;
  a.G = dp.G;
  a.RW = dp.RW;
  a.ypart = b.ypart;
  a.nss = (int)((c.d + kRedCols - 1) / kRedCols);
  a.fused_reduce = (dp.fused && !c.Ag) ? 1 : 0;
  a.done = counters + kDecDone;
  a.ybuf = b.ybuf;
  a.sspart = b.sspart;
  a.route_out = c.route_out;
  const bool lists = c.active_count || c.active_idx;
  a.keep_out = lists ? b.keep : nullptr;
  a.layer_in = c.layer_in;
  a.in_stride = std::max<int64_t>(1, c.ntot) * c.d;
  a.Ag = c.Ag;
  a.Bg = c.Bg;
  a.Au = c.Au;
  a.BuT = c.BuT;
  a.Ad = c.Ad;
  a.Bd = c.Bd;
  a.rank = (int)c.rank;
  a.lscale = c.lscale;
  a.vpart = b.dvpart;
  a.nvc = dp.nvc;
  a.zpart = b.dzpart;
  // per layer: [LoRA input] -> layer -> second reduction stage; kernel
  // boundaries order the phases
  for (int l = 0; l < (int)c.L; ++l) {
    if (c.Ag) {
      TimedLaunch tl(SATS_K_DEC_LORA_V, c.stream);
      hipExtLaunchKernelGGL(dec_lora_v_kernel<T>, dim3(dp.nvc), dim3(kDecodeThreads), 0, c.stream, tl.start,
                            tl.stop, 0, a, l);
      HIP_TRY(hipGetLastError());
    }
    {
      TimedLaunch tl(SATS_K_DEC_LAYER, c.stream);
      auto kern = dec_layer_fn<T>(c.Ag != nullptr, c.d);
      hipExtLaunchKernelGGL(kern, dim3(dp.G), dim3(kDecodeThreads), 0, c.stream, tl.start, tl.stop, 0, a, l);
    }
    HIP_TRY(hipGetLastError());
    if (a.fused_reduce) continue;
    if (c.Ag) {
      TimedLaunch tl(SATS_K_DEC_REDUCE_LORA, c.stream);
      hipExtLaunchKernelGGL(dec_reduce_lora_kernel<T>, dim3(dp.RW), dim3(kDecodeThreads), 0, c.stream, tl.start,
                            tl.stop, 0, a, l);
    } else {
      TimedLaunch tl(SATS_K_DEC_REDUCE, c.stream);
      hipExtLaunchKernelGGL(dec_reduce_kernel<T>, dim3(dp.RW), dim3(kRedThreads), 0, c.stream, tl.start, tl.stop, 0,
                            a, l);
    }
    HIP_TRY(hipGetLastError());
  }
  if (lists) {
    for (int64_t l = 0; l < c.L; ++l) {
      CompactArgs ca{};
      const int64_t nt = std::max<int64_t>(1, c.ntot);
      ca.keep = b.keep + l * c.d_ff;
      ca.idx = c.active_idx ? c.active_idx + (l * nt + c.tok) * c.d_ff : nullptr;
      ca.count = c.active_count ? c.active_count + l * nt + c.tok : nullptr;
      ca.n = 1;
      ca.d_ff = (int)c.d_ff;
      TimedLaunch tl(SATS_K_INSPECT, c.stream);
      hipExtLaunchKernelGGL(compact_kernel, dim3(1), dim3(kThreads), 0, c.stream, tl.start, tl.stop, 0, ca);
      HIP_TRY(hipGetLastError());
    }
  }
  return SATS_OK;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int lora_check(const Call &c) {
  if (!c.Bg || !c.Au || !c.BuT || !c.Ad || !c.Bd) return fail(SATS_ERR_NULL, "all six adapter matrices are required");
  if (c.rank != 8 && c.rank != 16 && c.rank != 32 && c.rank != 64)
    return fail(SATS_ERR_SHAPE, "LoRA rank must be 8, 16, 32 or 64 (got %lld)", (long long)c.rank);
  for (const void *q : {c.Ag, c.Bg, c.Au, c.BuT, c.Ad, c.Bd})
    if (!aligned16(q)) return fail(SATS_ERR_ARG, "adapter matrices must be 16-byte aligned");
  if (!std::isfinite(c.lscale)) return fail(SATS_ERR_ARG, "LoRA scale must be finite");
  return SATS_OK;
}

// Batches of bf16 LoRA calls run the batched passes with the whole pass on
// MFMA (the adapters enter the gate/up epilogue and the glue); everything
// else runs the single-token path token after token.
bool lora_batched(const Call &c, int esz, bool vec_ok) {
  return c.n >= sats::kMfmaMinTokens && batch_mfma(esz, vec_ok, (int)std::min<int64_t>(c.n, kMaxPass), true, c.d, c.d_ff) &&
         batch_whole() && !g_opt.lora_per_token;
}

// LoRA calls on the single-token path, token after token (each token takes
// its own route; the inspection outputs are written at the token's offsets).
template <typename T>
int run_lora(const Call &c, bool vec_ok) {
  const int esz = (int)sizeof(T);
  DecodePlan dp;
  if (!vec_ok || g_opt.single_token == SATS_SINGLE_OFF ||
      !make_decode_plan(c.d, c.d_ff, esz, &dp, (int)c.rank))
    return fail(SATS_ERR_SHAPE,
                "LoRA calls need the single-token layout: d <= %d, d and d_ff multiples of %d, 16-byte aligned arrays",
                sats::kDecodeMaxD, 16 / esz);
  if ((uint64_t)c.d_ff * c.rank * esz >= (1ull << 31) || (uint64_t)c.d * c.rank * esz >= (1ull << 31))
    return fail(SATS_ERR_SHAPE, "adapter matrices past 2 GB");
  if (c.rank * ((c.d + dp.RW - 1) / dp.RW) > 2 * sats::kDecodeMaxD - sats::kDecodeThreads)
    return fail(SATS_ERR_SHAPE, "LoRA: B_down slices of the second reduction stage do not fit LDS");
  const Plan p = make_plan(c.d, c.d_ff, esz, vec_ok, 1);
  const size_t bytes = layout(nullptr, p, 1, c.d, c.d_ff, esz, c.L, dp, nullptr);
  Workspace *ws = nullptr;
  int rc = ensure_workspace(c.stream, bytes, counter_count(p, 1, dp), &ws);
  if (rc) return rc;
  Buffers b{};
  layout(ws->mem, p, 1, c.d, c.d_ff, esz, c.L, dp, &b);
  for (int64_t i = 0; i < c.n; ++i) {
    Call ci = c;
    ci.x = static_cast<const T *>(c.x) + i * c.d;
    ci.out = static_cast<T *>(c.out) + i * c.d;
    ci.ids = c.ids ? c.ids + i : nullptr;
    ci.route_out = c.route_out ? c.route_out + i : nullptr;
    ci.layer_in = c.layer_in ? static_cast<void *>(static_cast<T *>(c.layer_in) + i * c.d) : nullptr;
    ci.n = 1;
    ci.tok = i;
    ci.ntot = c.n;
    if ((rc = run_decode<T>(ci, dp, b, ws->counters))) return rc;
  }
  return SATS_OK;
}

template <typename T>
int run(const Call &c) {
  if (!c.x || !c.Wg || !c.Wu || !c.Wd || !c.out) return fail(SATS_ERR_NULL, "x, weights and out must be non-null");
  if (c.route_mode != sats::ROUTE_BASE && !c.thr) return fail(SATS_ERR_NULL, "thresholds must be non-null");
  if (c.route_mode == sats::ROUTE_LUT && !c.ids) return fail(SATS_ERR_NULL, "token_ids must be non-null when route_lut is given");
  if (c.d < 1 || c.d_ff < 1 || c.L < 1 || c.n < 0)
    return fail(SATS_ERR_SHAPE, "need d >= 1, d_ff >= 1, n_layers >= 1, n_tokens >= 0 (got %lld, %lld, %lld, %lld)",
                (long long)c.d, (long long)c.d_ff, (long long)c.L, (long long)c.n);
  if (c.d > (1 << 24) || c.d_ff > (1 << 24) || c.n > ((int64_t)1 << 40))
    return fail(SATS_ERR_SHAPE, "d and d_ff must be at most 2^24");
  if (c.n == 0) return SATS_OK;
  const int esz = (int)sizeof(T);
  {
    const char *xb = static_cast<const char *>(c.x), *ob = static_cast<const char *>(c.out);
    const size_t bytes = (size_t)c.n * c.d * esz;
    if (xb != ob && xb < ob + bytes && ob < xb + bytes)
      return fail(SATS_ERR_ARG, "out overlaps x without being equal to it");
  }
  const int vec = 16 / esz;
  const bool vec_ok = c.d % vec == 0 && c.d_ff % vec == 0 && aligned16(c.x) && aligned16(c.out) &&
                      aligned16(c.Wg) && aligned16(c.Wu) && aligned16(c.Wd) &&
                      (!c.layer_in || aligned16(c.layer_in));
  const int pass = (int)std::min<int64_t>(c.n, kMaxPass);
  const Plan p = make_plan(c.d, c.d_ff, esz, vec_ok, pass);
  if (c.Ag) {
    int rc = lora_check(c);
    if (rc) return rc;
    if (!lora_batched(c, esz, vec_ok)) return run_lora<T>(c, vec_ok);
  }
  const int64_t lrank = c.Ag ? c.rank : 0;
  // single-token path: one token, vector layout, h fits the LDS copy
  bool decode = c.n == 1 && vec_ok && g_opt.single_token != SATS_SINGLE_OFF;
  DecodePlan dp;
  if (decode) decode = make_decode_plan(c.d, c.d_ff, esz, &dp);
  const size_t bytes = layout(nullptr, p, pass, c.d, c.d_ff, esz, c.L, dp, nullptr, lrank);
  Workspace *ws = nullptr;
  size_t ncount = counter_count(p, pass, dp);
  Workspace fixed{};
  int rc = 0;
  if (c.noalloc) {
    if (bytes > kScratchBytes - kScratchCounterBytes || ncount * sizeof(unsigned) > kScratchCounterBytes)
      return fail(SATS_ERR_WORKSPACE,
                  "the call needs %zu bytes of workspace and %zu counters; the allocation-free forward has %zu and %zu",
                  bytes, ncount, kScratchBytes - kScratchCounterBytes, kScratchCounterBytes / sizeof(unsigned));
    char *base = nullptr;
    if ((rc = scratch_addr(&base))) return rc;
    fixed.counters = reinterpret_cast<unsigned *>(base);
    fixed.n_counters = kScratchCounterBytes / sizeof(unsigned);
    fixed.mem = base + kScratchCounterBytes;
    fixed.bytes = kScratchBytes - kScratchCounterBytes;
    hipLaunchKernelGGL(clear_counters_kernel, dim3(8), dim3(256), 0, c.stream, fixed.counters, (int)ncount, (int)kErr);
    HIP_TRY(hipGetLastError());
    ws = &fixed;
  } else if ((rc = ensure_workspace(c.stream, bytes, ncount, &ws))) {
    return rc;
  }
  Buffers b{};
  layout(ws->mem, p, pass, c.d, c.d_ff, esz, c.L, dp, &b, lrank);
  if (decode) return run_decode<T>(c, dp, b, ws->counters);

  for (int64_t base = 0; base < c.n; base += kMaxPass) {
    const int np = (int)std::min<int64_t>(kMaxPass, c.n - base);
    const Plan pp = (np == pass) ? p : make_plan(c.d, c.d_ff, esz, vec_ok, np);
    constexpr int V = 16 / sizeof(T);
    if (pp.vec == 1) {
      rc = (pp.NT == 1) ? run_pass<T, 1, 1>(c, pp, b, ws->counters, base, np)
                        : run_pass<T, 1, 4>(c, pp, b, ws->counters, base, np);
    } else {
      rc = (pp.NT == 1) ? run_pass<T, V, 1>(c, pp, b, ws->counters, base, np)
                        : run_pass<T, V, 4>(c, pp, b, ws->counters, base, np);
    }
    if (rc) return rc;
  }
  return SATS_OK;
}

Call make_call(const void *x, const int32_t *ids, const void *Wg, const void *Wu, const void *Wd,
               const float *thr, const uint8_t *lut, void *out, int64_t n, int64_t d, int64_t d_ff,
               int64_t L, hipStream_t s, int mode) {
  Call c{};
  c.x = x; c.ids = ids; c.Wg = Wg; c.Wu = Wu; c.Wd = Wd; c.thr = thr; c.lut = lut; c.out = out;
  c.n = n; c.d = d; c.d_ff = d_ff; c.L = L; c.stream = s; c.route_mode = mode;
  return c;
}

int route_mode_of(const uint8_t *lut) { return lut ? sats::ROUTE_LUT : sats::ROUTE_SPARSE; }


// --------------------------------------------------------------- SATS calibration

// Device buffers of one calibration call (allocated per call: calibration is
// an offline step, and its buffers are sized by the calibration set).
struct CalBuffers {
  float *G = nullptr;              // [n][d_ff] g
  uint16_t *ph = nullptr, *pl = nullptr;  // [n][d_ff] p as bf16 hi + lo
  uint8_t *cnt = nullptr;          // [n][d_ff] candidates at or below |g|
  uint16_t *WdT = nullptr;         // [d][d_ff] W_down^T of the layer
  float *part = nullptr;           // [d / 64][n][16] (products with a y row use the first d / 128 tiles)
  uint32_t *hpart = nullptr, *hist = nullptr, *prefix = nullptr, *rank = nullptr;
  float *tk = nullptr, *thr15 = nullptr;
  unsigned long long *ge15 = nullptr;  // #{|g| >= t_r} of a product's candidates
  double *errsum = nullptr;
  double *rsum = nullptr;          // [ceil(n / 64)][16] workgroup sums of the Eq. 6 terms
  float *ny2 = nullptr;            // [n] ||y||^2 of each row (from the first product)
  int *ctl = nullptr;              // [passes][2] rows of each gate/up pass, MFMA on
};

// The calibration buffers are kept per device from call to call (grown when
// a call needs more, freed by sats_release): a call allocates nothing once
// they are large enough, where allocating and freeing ~250 MB per call cost
// more than a millisecond.  Calls hold g_cal_mu throughout and synchronise
// their stream before they return, so two calls never share them at once.
struct CalCache {
  CalBuffers b;
  size_t cap[17] = {};  // elements of each buffer, in the order of cal_buffers
};
std::mutex g_cal_mu;
std::map<int, CalCache> g_cal;

template <typename P> int cal_alloc(P **p, size_t *cap, size_t count) {
  if (*p && *cap >= count) return SATS_OK;
  if (*p) HIP_TRY(hipFree(*p));
  *p = nullptr;
  *cap = 0;
  if (hipMalloc((void **)p, std::max<size_t>(count, 1) * sizeof(P)) != hipSuccess)
    return fail(SATS_ERR_WORKSPACE, "calibration buffer of %zu bytes failed", count * sizeof(P));
  *cap = count;
  return SATS_OK;
}

// A call's own temporary buffer (freed by the call).
template <typename P> int cal_tmp_alloc(P **p, size_t count) {
  if (hipMalloc((void **)p, std::max<size_t>(count, 1) * sizeof(P)) != hipSuccess)
    return fail(SATS_ERR_WORKSPACE, "calibration buffer of %zu bytes failed", count * sizeof(P));
  return SATS_OK;
}

int cal_release_all() {
  std::lock_guard<std::mutex> lk(g_cal_mu);
  for (auto &kv : g_cal) {
    HIP_TRY(hipSetDevice(kv.first));
    HIP_TRY(hipDeviceSynchronize());
    const CalBuffers &b = kv.second.b;
    for (void *q : {(void *)b.G, (void *)b.ph, (void *)b.pl, (void *)b.cnt, (void *)b.WdT, (void *)b.part,
                    (void *)b.hpart, (void *)b.hist, (void *)b.prefix, (void *)b.rank, (void *)b.tk, (void *)b.thr15,
                    (void *)b.ge15, (void *)b.errsum, (void *)b.ctl, (void *)b.rsum, (void *)b.ny2})
      if (q) HIP_TRY(hipFree(q));
  }
  g_cal.clear();
  return SATS_OK;
}

constexpr int kCalHistParts = 256;  // workgroups of a radix pass (each writes its own histogram)

// Rank m = ceil(q N) of the Eq. 3 order statistic at level q (q taken to 1e-6).
uint64_t level_rank(double q, uint64_t N) {
  if (!(q > 0.0)) return 0;
  const uint64_t qi = (uint64_t)std::llround(std::min(q, 1.0) * 1e6);
  const unsigned __int128 num = (unsigned __int128)qi * N + 999999u;
  const uint64_t m = (uint64_t)(num / 1000000u);
  return std::max<uint64_t>(1, std::min<uint64_t>(m, N));
}

int cal_check_shape(int64_t n, int64_t d, int64_t d_ff) {
  if (n < 1 || d < 1 || d_ff < 1)
    return fail(SATS_ERR_SHAPE, "calibration needs n, d, d_ff >= 1");
  if (d % sats::kDenseDownNT || d % sats::kDenseKC || d_ff % sats::kDenseNT || d_ff % sats::kDenseKC || d > 4096)
    return fail(SATS_ERR_SHAPE, "calibration needs d a multiple of 128 (at most 4096) and d_ff of 64");
  if ((uint64_t)d * d_ff * 2 >= (1ull << 31) || (uint64_t)n * d_ff * 2 >= (1ull << 31))
    return fail(SATS_ERR_SHAPE, "calibration buffers past 2 GB");
  return SATS_OK;
}

// g and p of n calibration rows (MFMA, 64 rows per pass) into G, ph, pl.
int cal_gate_up(const uint16_t *h, const uint16_t *Wg, const uint16_t *Wu, int64_t n, int64_t d, int64_t d_ff,
                CalBuffers &cb, hipStream_t s) {
  using namespace sats;
  const int64_t passes = (n + kDenseMaxTokens - 1) / kDenseMaxTokens;
  std::vector<int> ctl(2 * passes);
  for (int64_t i = 0; i < passes; ++i) {
    ctl[2 * i] = (int)std::min<int64_t>(kDenseMaxTokens, n - i * kDenseMaxTokens);
    ctl[2 * i + 1] = 1;
  }
  HIP_TRY(hipMemcpyAsync(cb.ctl, ctl.data(), ctl.size() * sizeof(int), hipMemcpyHostToDevice, s));
  // every pass in one launch, the passes of a column tile side by side on
  // one XCD so that its weights come from HBM about once (see DenseArgs)
  DenseArgs da{};
  da.ctl = cb.ctl;
  da.H = h;
  da.Wg = Wg;
  da.Wt = Wu;
  da.K = (int)d;
  da.N = (int)d_ff;
  da.nt = dense_tile_cols(d_ff);
  da.hcap = (int)n;  // calibration rows from pass 0's first on
  da.cal_g = cb.G;
  da.cal_ph = cb.ph;
  da.cal_pl = cb.pl;
  da.cal_passes = (int)passes;
  da.cal_tiles = (int)((d_ff + da.nt - 1) / da.nt);
  const int64_t grid = (int64_t)((da.cal_tiles + 7) / 8) * 8 * passes;
  TimedLaunch tl(SATS_K_CAL_GATEUP, s);
  hipExtLaunchKernelGGL(dense_gateup_kernel<4, false, true>, dim3((unsigned)grid), dim3(kDenseThreads), 0, s, tl.start,
                        tl.stop, 0, da);
  HIP_TRY(hipGetLastError());
  return SATS_OK;
}

// Eq. 3 order statistics of |g| at `levels` (up to kCalMaxLevels) into t (host).
int cal_quantiles(CalBuffers &cb, uint64_t N, const double *levels, int K, float *t, hipStream_t s) {
  using namespace sats;
  std::vector<uint32_t> rank(K), zero(K, 0u);
  for (int k = 0; k < K; ++k) rank[k] = (uint32_t)level_rank(levels[k], N);
  HIP_TRY(hipMemcpyAsync(cb.rank, rank.data(), K * sizeof(uint32_t), hipMemcpyHostToDevice, s));
  HIP_TRY(hipMemcpyAsync(cb.prefix, zero.data(), K * sizeof(uint32_t), hipMemcpyHostToDevice, s));
  // passes: bits 31..20 (one histogram for every level), 19..12, 11..4, 3..0
  static const int kShift[4] = {20, 12, 4, 0}, kBits[4] = {12, 8, 8, 4};
  for (int pass = 0; pass < 4; ++pass) {
    const int kh = pass == 0 ? 1 : K, nh = kh << kBits[pass];
    hipLaunchKernelGGL(cal_hist_kernel, dim3(kCalHistParts), dim3(kCalHistThreads), 0, s, cb.G, (size_t)N,
                       cb.prefix, kh, kShift[pass], kBits[pass], cb.hpart);
    hipLaunchKernelGGL(cal_hist_reduce_kernel, dim3((nh + kCalHRBins - 1) / kCalHRBins), dim3(kCalHistThreads), 0, s,
                       cb.hpart, kCalHistParts, nh, cb.hist);
    hipLaunchKernelGGL(cal_select_kernel, dim3(K), dim3(kCalSelThreads), 0, s, cb.hist,
                       pass == 0 ? (size_t)0 : ((size_t)1 << kBits[pass]), 1 << kBits[pass], kBits[pass], cb.prefix,
                       cb.rank, pass == 3 ? cb.tk : (float *)nullptr);
  }
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipMemcpyAsync(t, cb.tk, K * sizeof(float), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  return SATS_OK;
}

// Eq. 6 error and sparsity of ascending candidates t[0..K) (any K), 15 per
// product.  err_rows (device, [n][K]) is optional; without err only the
// sparsities are computed.  Candidates at or below 0 remove no neuron (no
// |g| is below them): their error and sparsity are 0 exactly, and the
// products start at the first positive candidate.  The first product carries
// y and keeps ||y||^2 per row; a later product of at most 4 candidates takes
// it from there and packs four calibration rows per MFMA tile.
int cal_curves(CalBuffers &cb, const uint16_t *Wd, int64_t n, int64_t d, int64_t d_ff, const float *t, int K,
               double *err, double *sp, float *err_rows, hipStream_t s) {
  using namespace sats;
  const uint64_t N = (uint64_t)n * d_ff;
  const int grid = (int)std::max<uint64_t>(1, std::min<uint64_t>(2048, (N / 4 + kCalThreads - 1) / kCalThreads));
  if (err) {
    hipLaunchKernelGGL(cal_transpose_kernel, dim3(d / 64, d_ff / 64), dim3(kCalThreads), 0, s, Wd, (int)d_ff,
                       (int)d, cb.WdT);
    HIP_TRY(hipGetLastError());
  }
  int z = 0;
  while (z < K && t[z] <= 0.0f) ++z;
  for (int k = 0; k < z; ++k) {
    if (err) err[k] = 0.0;
    sp[k] = 0.0;
  }
  if (err && err_rows && z > 0) {
    hipLaunchKernelGGL(cal_zero_cols_kernel, dim3((unsigned)std::min<int64_t>(1024, (n * z + kCalThreads - 1) / kCalThreads)),
                       dim3(kCalThreads), 0, s, err_rows, (size_t)n, K, z);
    HIP_TRY(hipGetLastError());
  }
  bool have_y = false;  // ||y||^2 of every row is in cb.ny2
  for (int k0 = z; k0 < K; k0 += kCalCand) {
    const int kc = std::min(kCalCand, K - k0);
    const bool pack4 = have_y && kc <= 4;
    float thr[kCalCand];
    for (int r = 0; r < kCalCand; ++r) thr[r] = r < kc ? t[k0 + r] : INFINITY;
    HIP_TRY(hipMemcpyAsync(cb.thr15, thr, sizeof thr, hipMemcpyHostToDevice, s));
    HIP_TRY(hipMemsetAsync(cb.ge15, 0, kCalCand * sizeof(unsigned long long), s));
    hipLaunchKernelGGL(cal_bucket_kernel, dim3(grid), dim3(kCalThreads), 0, s, cb.G, (size_t)N, cb.thr15, cb.cnt,
                       cb.ge15);
    if (err) {
      CalErrArgs ce{};
      ce.ph = cb.ph;
      ce.pl = cb.pl;
      ce.cnt = cb.cnt;
      ce.WdT = cb.WdT;
      ce.part = cb.part;
      ce.n = (int)n;
      ce.d = (int)d;
      ce.d_ff = (int)d_ff;
      {
        TimedLaunch tl(SATS_K_CAL_ERR, s);
        // at most 4 candidates and ||y||^2 known: four calibration rows per
        // MFMA tile, no y row; at most 7: two per tile
        if (pack4)
          hipExtLaunchKernelGGL(cal_err_kernel<4>, dim3(d / kDenseDownNT, (n + kCalRows - 1) / kCalRows),
                                dim3(kDenseThreads), 0, s, tl.start, tl.stop, 0, ce);
        else if (kc <= 7)
          hipExtLaunchKernelGGL(cal_err_kernel<2>, dim3(d / kDenseDownNT, (n + kCalRows - 1) / kCalRows),
                                dim3(kDenseThreads), 0, s, tl.start, tl.stop, 0, ce);
        else
          hipExtLaunchKernelGGL(cal_err_kernel<1>, dim3(d / kDenseDownNT, (n + kCalRows - 1) / kCalRows),
                                dim3(kDenseThreads), 0, s, tl.start, tl.stop, 0, ce);
      }
      const int rblocks = (int)((n + 63) / 64);
      hipLaunchKernelGGL(cal_reduce_kernel, dim3(rblocks), dim3(64 * kCalRedWaves), 0, s, cb.part,
                         (int)(d / kDenseDownNT) * (pack4 ? 2 : 1), (int)n, kc,
                         err_rows ? err_rows + k0 : (float *)nullptr, K, cb.rsum,
                         pack4 ? (const float *)cb.ny2 : (const float *)nullptr, have_y ? (float *)nullptr : cb.ny2);
      have_y = true;
      hipLaunchKernelGGL(cal_reduce_sum_kernel, dim3(1), dim3(64), 0, s, cb.rsum, rblocks, kc, cb.errsum);
    }
    HIP_TRY(hipGetLastError());
    double es[kCalCand];
    unsigned long long ge[kCalCand];
    if (err) HIP_TRY(hipMemcpyAsync(es, cb.errsum, kc * sizeof(double), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(ge, cb.ge15, kc * sizeof(unsigned long long), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    for (int r = 0; r < kc; ++r) {
      if (err) err[k0 + r] = es[r] / (double)n;
      sp[k0 + r] = (double)(N - ge[r]) / (double)N;  // #{|g| < t_r} / N
    }
  }
  return SATS_OK;
}

// The buffers of a call with n rows of d x d_ff into cb, from the current
// device's cache (the caller holds g_cal_mu).
int cal_buffers(CalBuffers &cb, int64_t n, int64_t d, int64_t d_ff) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  CalCache &c = g_cal[dev];
  CalBuffers &b = c.b;
  size_t *k = c.cap;
  const size_t N = (size_t)n * d_ff;
  int rc = 0;
  if ((rc = cal_alloc(&b.G, &k[0], N)) || (rc = cal_alloc(&b.ph, &k[1], N)) || (rc = cal_alloc(&b.pl, &k[2], N)) ||
      (rc = cal_alloc(&b.cnt, &k[3], N)) || (rc = cal_alloc(&b.WdT, &k[4], (size_t)d * d_ff)) ||
      (rc = cal_alloc(&b.part, &k[5], (size_t)(d / sats::kDenseDownNT) * 2 * n * 16)) ||
      (rc = cal_alloc(&b.hpart, &k[6], (size_t)kCalHistParts * sats::kCalHistLds)) ||
      (rc = cal_alloc(&b.hist, &k[7], sats::kCalHistLds)) || (rc = cal_alloc(&b.prefix, &k[8], sats::kCalMaxLevels)) ||
      (rc = cal_alloc(&b.rank, &k[9], sats::kCalMaxLevels)) || (rc = cal_alloc(&b.tk, &k[10], sats::kCalMaxLevels)) ||
      (rc = cal_alloc(&b.thr15, &k[11], sats::kCalCand)) || (rc = cal_alloc(&b.ge15, &k[12], sats::kCalCand)) ||
      (rc = cal_alloc(&b.errsum, &k[13], sats::kCalCand)) ||
      (rc = cal_alloc(&b.ctl, &k[14], 2 * ((n + sats::kDenseMaxTokens - 1) / sats::kDenseMaxTokens))) ||
      (rc = cal_alloc(&b.rsum, &k[15], (size_t)((n + 63) / 64) * 16)) || (rc = cal_alloc(&b.ny2, &k[16], (size_t)n)))
    return rc;
  cb = b;
  return SATS_OK;
}

// One layer: candidates at `levels` and their curves (host outputs).
int cal_layer(CalBuffers &cb, const uint16_t *h, const uint16_t *Wg, const uint16_t *Wu, const uint16_t *Wd, int64_t n,
              int64_t d, int64_t d_ff, const double *levels, int K, float *t, double *err, double *sp, float *err_rows,
              hipStream_t s, bool gate_up = true) {
  int rc = 0;
  if (gate_up && (rc = cal_gate_up(h, Wg, Wu, n, d, d_ff, cb, s))) return rc;
  for (int k0 = 0; k0 < K; k0 += sats::kCalMaxLevels)
    if ((rc = cal_quantiles(cb, (uint64_t)n * d_ff, levels + k0, std::min(sats::kCalMaxLevels, K - k0), t + k0, s)))
      return rc;
  return cal_curves(cb, Wd, n, d, d_ff, t, K, err, sp, err_rows, s);
}

struct CalCurve {
  std::vector<double> level, t, err, sp;
};

// b* over the breakpoints of S(b) (Eq. 7-10): for each distinct error value
// b (and 0), every free layer takes its largest candidate with Err <= b; S
// is the mean sparsity over all layers (fixed ones at their own); the
// budget whose S is nearest the target wins, the smallest on ties.
void cal_select(const std::vector<CalCurve> &cv, const std::vector<int> &fixed, const std::vector<double> &fixed_sp,
                double s_tar, double *b_out, std::vector<int> *idx_out, double *s_out) {
  const size_t L = cv.size();
  std::vector<double> budgets{0.0};
  for (size_t l = 0; l < L; ++l)
    if (!fixed[l]) budgets.insert(budgets.end(), cv[l].err.begin(), cv[l].err.end());
  std::sort(budgets.begin(), budgets.end());
  budgets.erase(std::unique(budgets.begin(), budgets.end()), budgets.end());
  bool have = false;
  for (double b : budgets) {
    std::vector<int> idx(L, -1);
    double S = 0.0;
    for (size_t l = 0; l < L; ++l) {
      if (fixed[l]) {
        S += fixed_sp[l];
        continue;
      }
      int best = -1;  // the largest admissible threshold (t = 0, Err = 0, is always admissible)
      for (size_t k = 0; k < cv[l].t.size(); ++k)
        if (cv[l].err[k] <= b && (best < 0 || cv[l].t[k] > cv[l].t[best])) best = (int)k;
      best = std::max(best, 0);
      idx[l] = best;
      S += cv[l].sp[best];
    }
    S /= (double)L;
    if (!have || std::fabs(S - s_tar) < std::fabs(*s_out - s_tar)) {
      have = true;
      *b_out = b;
      *idx_out = idx;
      *s_out = S;
    }
  }
}

// candidate levels: 0 and step, 2 step, ... below 1
std::vector<double> cal_coarse(double step) {
  std::vector<double> v{0.0};
  const int n = (int)std::lround(1.0 / step);
  for (int i = 1; i < n; ++i) v.push_back(std::round(i * step * 1e10) / 1e10);
  return v;
}
// levels fine apart strictly between the coarse neighbours of the coarse level q
std::vector<double> cal_fine(double q, const std::vector<double> &coarse, double fine) {
  double lo = 0.0, hi = 1.0;
  for (double c : coarse) {
    if (c > 0.0 && c < q - 1e-12) lo = std::max(lo, c);
    if (c > q + 1e-12) hi = std::min(hi, c);
  }
  std::vector<double> v;
  for (int i = 1; lo + i * fine < hi - 1e-9; ++i) v.push_back(std::round((lo + i * fine) * 1e10) / 1e10);
  return v;
}

int cal_stack(const uint16_t *x, int64_t n, const uint16_t *Wg, const uint16_t *Wu, const uint16_t *Wd, int64_t d,
              int64_t d_ff, int64_t L, double s_tar, double coarse_step, double fine_step, int guardrail,
              float *thresholds, double *budget, double *realized, hipStream_t s) {
  int rc = cal_check_shape(n, d, d_ff);
  if (rc) return rc;
  // held until the temporaries below are freed (hipFree synchronises the
  // device), so the kept buffers are idle when the next call takes them
  std::lock_guard<std::mutex> lk(g_cal_mu);
  if (L < 1 || !(coarse_step > 0.0 && coarse_step < 1.0) || !(fine_step > 0.0) || !(s_tar >= 0.0 && s_tar <= 1.0))
    return fail(SATS_ERR_ARG, "calibration needs L >= 1, 0 < coarse_step < 1, fine_step > 0, 0 <= s_tar <= 1");
  const size_t wl = (size_t)d * d_ff;
  // every layer's input on the base path (the stack's own forward, inputs exported)
  uint16_t *hin = nullptr, *out = nullptr;
  if ((rc = cal_tmp_alloc(&hin, (size_t)L * n * d)) || (rc = cal_tmp_alloc(&out, (size_t)n * d))) {
    if (hin) (void)hipFree(hin);
    return rc;
  }
  struct Free {
    uint16_t *a, *b;
    ~Free() { (void)hipFree(a); (void)hipFree(b); }
  } fr{hin, out};
  Call c = make_call(x, nullptr, Wg, Wu, Wd, nullptr, nullptr, out, n, d, d_ff, L, s, sats::ROUTE_BASE);
  c.layer_in = hin;
  if ((rc = run<uint16_t>(c))) return rc;
  CalBuffers cb;
  if ((rc = cal_buffers(cb, n, d, d_ff))) return rc;
  const std::vector<double> coarse = cal_coarse(coarse_step);
  std::vector<CalCurve> cv(L);
  std::vector<int> fixed(L, 0);
  std::vector<double> fixed_sp(L, 0.0);
  std::vector<float> fixed_t(L, 0.0f);
  // with_err false: thresholds and sparsities only (the guardrail layer)
  auto layer_curves = [&](int64_t l, const std::vector<double> &lv, CalCurve &out_c, bool gate_up,
                          bool with_err = true) -> int {
    const int K = (int)lv.size();
    std::vector<float> t(K);
    std::vector<double> err(K, 0.0), sp(K);
    const int r = cal_layer(cb, hin + (size_t)l * n * d, Wg + l * wl, Wu + l * wl, Wd + l * wl, n, d, d_ff, lv.data(),
                            K, t.data(), with_err ? err.data() : nullptr, sp.data(), nullptr, s, gate_up);
    if (r) return r;
    for (int k = 0; k < K; ++k) {
      out_c.level.push_back(lv[k]);
      out_c.t.push_back(t[k]);
      out_c.err.push_back(err[k]);
      out_c.sp.push_back(sp[k]);
    }
    return SATS_OK;
  };
  // stage 1: the coarse grid on every layer; the guardrail layer keeps its
  // CATS threshold at the target sparsity
  for (int64_t l = 0; l < L; ++l) {
    if ((rc = layer_curves(l, coarse, cv[l], true))) return rc;
    if (guardrail && L > 1 && l == L - 1) {
      CalCurve g1;
      if ((rc = layer_curves(l, {s_tar}, g1, false, false))) return rc;
      fixed[l] = 1;
      fixed_sp[l] = g1.sp[0];
      fixed_t[l] = (float)g1.t[0];
    }
  }
  double b1 = 0.0, s1 = 0.0;
  std::vector<int> idx1;
  cal_select(cv, fixed, fixed_sp, s_tar, &b1, &idx1, &s1);
  // stage 2: finer levels on both sides of each free layer's choice (between
  // the coarse levels adjacent to the level it was chosen at: the smallest
  // level of its threshold, since the selection keeps the first of equal
  // thresholds), added to its candidates
  for (int64_t l = 0; l < L; ++l) {
    if (fixed[l]) continue;
    const double q = cv[l].level[idx1[l]];
    const std::vector<double> fl = cal_fine(q, coarse, fine_step);
    if (fl.empty()) continue;
    if ((rc = layer_curves(l, fl, cv[l], true))) return rc;
  }
  double b2 = 0.0, s2 = 0.0;
  std::vector<int> idx2;
  cal_select(cv, fixed, fixed_sp, s_tar, &b2, &idx2, &s2);
  for (int64_t l = 0; l < L; ++l) thresholds[l] = fixed[l] ? fixed_t[l] : (float)cv[l].t[idx2[l]];
  if (budget) *budget = b2;
  if (realized) *realized = s2;
  return SATS_OK;
}

template <typename T>
int forward_lora(const T *x, const int32_t *token_ids, const T *W_gate, const T *W_up_T, const T *W_down,
                 const T *A_gate, const T *B_gate, const T *A_up, const T *B_up_T, const T *A_down, const T *B_down,
                 int64_t rank, float scale, const float *thresholds, const uint8_t *route_lut, T *out,
                 int64_t n_tokens, int64_t d, int64_t d_ff, int64_t n_layers, hipStream_t stream,
                 uint8_t *route_out, int32_t *active_count, int32_t *active_idx, T *layer_in) {
  g_err.clear();
  if (!A_gate) return fail(SATS_ERR_NULL, "all six adapter matrices are required");
  Call c = make_call(x, token_ids, W_gate, W_up_T, W_down, thresholds, route_lut, out, n_tokens, d,
                     d_ff, n_layers, stream, route_mode_of(route_lut));
  c.route_out = route_out;
  c.active_count = active_count;
  c.active_idx = active_idx;
  c.layer_in = layer_in;
  c.Ag = A_gate;
  c.Bg = B_gate;
  c.Au = A_up;
  c.BuT = B_up_T;
  c.Ad = A_down;
  c.Bd = B_down;
  c.rank = rank;
  c.lscale = scale;
  return run<T>(c);
}
// --------------------------------------------------------------- routing table

// Device buffers of the routing-table construction, kept from call to call
// per device (grown when a call needs more; freed by sats_release).  Calls
// hold g_route_mu throughout (each call synchronises its stream before it
// returns), so two calls never share them at once.
struct RouteBuffers {
  size_t ent = 0, off = 0, parts = 0, vocab = 0;  // capacities: entries, offsets, part words, ids
  sats::u32x4 *pent = nullptr;
  uint32_t *poff = nullptr;
  unsigned *cnt = nullptr, *hcnt = nullptr, *htot = nullptr;
  unsigned *err = nullptr;  // inside out (its third word)
  unsigned long long *sum = nullptr, *sel = nullptr;
  double *score = nullptr, *out = nullptr;
};
std::mutex g_route_mu;
std::map<int, RouteBuffers> g_route;

template <typename P> int route_grow(P **p, size_t *cap, size_t need) {
  if (*p && *cap >= need) return SATS_OK;
  if (*p) HIP_TRY(hipFree(*p));
  *p = nullptr;
  *cap = 0;
  if (hipMalloc((void **)p, std::max<size_t>(need, 1) * sizeof(P)) != hipSuccess)
    return fail(SATS_ERR_WORKSPACE, "routing-table buffer of %zu bytes failed", need * sizeof(P));
  *cap = need;
  return SATS_OK;
}

int route_release_all() {
  std::lock_guard<std::mutex> lk(g_route_mu);
  for (auto &kv : g_route) {
    HIP_TRY(hipSetDevice(kv.first));
    HIP_TRY(hipDeviceSynchronize());
    RouteBuffers &b = kv.second;
    for (void *q : {(void *)b.pent, (void *)b.poff, (void *)b.cnt, (void *)b.hcnt, (void *)b.htot, (void *)b.sum,
                    (void *)b.sel, (void *)b.score, (void *)b.out})
      if (q) HIP_TRY(hipFree(q));
  }
  g_route.clear();
  return SATS_OK;
}

// The routing-table construction of Eq. 11-14 (synchronous).
int route_build(const float *lb, const float *ls, const int32_t *ids, int64_t n, const int32_t *hids, int64_t nh,
                int64_t vocab, double r_tar, uint8_t *table, double *score_out, double *tau_out,
                double *realized_out, hipStream_t s) {
  using namespace sats;
  if (!table || (n > 0 && (!lb || !ls || !ids)) || (nh > 0 && !hids))
    return fail(SATS_ERR_NULL, "route_lut, and the losses and ids of a non-empty split, must be non-null");
  if (n < 0 || nh < 0 || vocab < 1 || vocab > (1ll << 31) - 1 || n > (1ll << 40) || nh > (1ll << 40))
    return fail(SATS_ERR_SHAPE, "need n_tokens, n_heldout >= 0 and 1 <= vocab < 2^31");
  if (!(r_tar >= 0.0 && r_tar <= 1.0)) return fail(SATS_ERR_ARG, "r_tar must be in [0, 1]");
  const size_t V = (size_t)vocab;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lk(g_route_mu);
  RouteBuffers &b = g_route[dev];
  // partitioned sums (ranges of 2^rbits ids, at most kRouteRanges of them),
  // or per-chunk atomics into kRouteCopies copies past kRoutePartMaxVocab
  const bool part = vocab <= kRoutePartMaxVocab;
  int rbits = 10;
  while (((vocab + (1ll << rbits) - 1) >> rbits) > kRouteRanges) ++rbits;
  const int nr = (int)((vocab + (1ll << rbits) - 1) >> rbits);
  const int64_t nc = (n + kRouteChunk - 1) / kRouteChunk, nhc = (nh + kRouteChunk - 1) / kRouteChunk;
  if (nc > INT32_MAX || nhc > INT32_MAX) return fail(SATS_ERR_SHAPE, "too many occurrences");
  const int P = part ? kRouteParts : kRouteCopies;
  const int64_t mc = std::max<int64_t>(nc, nhc);
  int rc = 0;
  size_t cap_sum = b.parts, cap_h = b.parts, cap_v = b.vocab, cap_v2 = b.vocab, cap_sel = kSelWords, cap_o = 2,
         cap_e = 1;
  if ((part && ((rc = route_grow(&b.pent, &b.ent, (size_t)mc * kRouteChunk)) ||
                (rc = route_grow(&b.poff, &b.off, (size_t)(nr + 1) * mc)))) ||
      (rc = route_grow(&b.cnt, &b.parts, (size_t)P * V)) || (rc = route_grow(&b.sum, &cap_sum, (size_t)P * V)) ||
      (rc = route_grow(&b.hcnt, &cap_h, (size_t)P * V)) || (rc = route_grow(&b.htot, &b.vocab, V)) ||
      (rc = route_grow(&b.score, &cap_v, V)))
    return rc;
  (void)cap_v2;
  // out: tau*, R(tau*) and the error flag (one copy back)
  if (!b.sel && ((rc = route_grow(&b.sel, &cap_sel, (size_t)kSelWords)) || (rc = route_grow(&b.out, &cap_o, 3))))
    return rc;
  b.err = reinterpret_cast<unsigned *>(b.out + 2);
  (void)cap_e;
  double *score = score_out ? score_out : b.score;
  hipLaunchKernelGGL(route_clear_kernel, dim3(8), dim3(256), 0, s, b.sel, (int)kSelWords, b.err);
  if (part) {
    // each split: entries per chunk, then the merge of every range (the
    // merge also runs for an empty split: zero totals)
    for (int split = 0; split < 2; ++split) {
      const bool dmg = split == 0;
      const int64_t nn = dmg ? n : nh, ch = dmg ? nc : nhc;
      if (nn > 0) {
        RoutePartArgs pa{dmg ? ids : hids, lb, ls, nn, (int)vocab, rbits, nr, (int)ch, b.pent, b.poff, b.err};
        TimedLaunch tl(dmg ? SATS_K_ROUTE_ACCUM : -1, s);
        hipExtLaunchKernelGGL(dmg ? route_part_kernel<true> : route_part_kernel<false>, dim3((unsigned)ch),
                              dim3(kRouteThreads), 0, s, tl.start, tl.stop, 0, pa);
        HIP_TRY(hipGetLastError());
      }
      RouteMergeArgs ma{b.pent, b.poff, (int)ch, rbits, nr, (int)vocab, P, dmg ? b.cnt : b.hcnt, b.sum};
      TimedLaunch tl(dmg ? SATS_K_ROUTE_MERGE : -1, s);
      hipExtLaunchKernelGGL(dmg ? route_merge_kernel<true> : route_merge_kernel<false>, dim3(nr, P),
                            dim3(kRouteThreads), 0, s, tl.start, tl.stop, 0, ma);
      HIP_TRY(hipGetLastError());
    }
  } else {
    HIP_TRY(hipMemsetAsync(b.sum, 0, (size_t)P * V * sizeof(unsigned long long), s));
    HIP_TRY(hipMemsetAsync(b.cnt, 0, (size_t)P * V * sizeof(unsigned), s));
    HIP_TRY(hipMemsetAsync(b.hcnt, 0, (size_t)P * V * sizeof(unsigned), s));
    if (n > 0) {
      RouteAccumArgs ra{ids, lb, ls, n, (int)vocab, b.sum, b.cnt, b.err};
      TimedLaunch tl(SATS_K_ROUTE_ACCUM, s);
      hipExtLaunchKernelGGL(route_accum_kernel<true>, dim3((unsigned)nc), dim3(kRouteThreads), 0, s, tl.start,
                            tl.stop, 0, ra);
    }
    if (nh > 0) {
      RouteAccumArgs ra{hids, nullptr, nullptr, nh, (int)vocab, nullptr, b.hcnt, b.err};
      hipLaunchKernelGGL(route_accum_kernel<false>, dim3((unsigned)nhc), dim3(kRouteThreads), 0, s, ra);
    }
    HIP_TRY(hipGetLastError());
  }
  const unsigned vb = (unsigned)((V + 255) / 256), vk = (unsigned)((V + 1023) / 1024);
  hipLaunchKernelGGL(route_score_kernel, dim3(vb), dim3(256), 0, s, b.sum, b.cnt, b.hcnt, P, (int)vocab, score,
                     b.htot, b.sel);
  // Eq. 14 on the device
  RouteSelArgs sa{score, b.htot, (int)vocab, (long long)nh, r_tar, b.sel, b.out, b.err};
  for (int k = 1; k < 8; ++k)
    hipLaunchKernelGGL(route_select_pass_kernel, dim3(vk), dim3(1024), 0, s, sa, k);
  hipLaunchKernelGGL(route_select_final_kernel, dim3(vk), dim3(1024), 0, s, sa);
  hipLaunchKernelGGL(route_table_kernel, dim3(vb), dim3(256), 0, s, score, (int)vocab, b.out, b.err, table);
  HIP_TRY(hipGetLastError());
  double res[3] = {0.0, 0.0, 0.0};  // tau*, R(tau*), the error flag in the low word of the third
  HIP_TRY(hipMemcpyAsync(res, b.out, sizeof res, hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  unsigned herr = 0;
  std::memcpy(&herr, &res[2], sizeof herr);
  if (herr == 1) return fail(SATS_ERR_ARG, "a token id is outside [0, vocab)");
  if (herr == 2) return fail(SATS_ERR_ARG, "a loss difference is NaN or at least 2^31");
  if (herr) return fail(SATS_ERR_DEVICE, "routing table: a chunk's id table overflowed");
  if (tau_out) *tau_out = res[0];
  if (realized_out) *realized_out = res[1];
  return SATS_OK;
}
}  // namespace

// =============================================================== C ABI

extern "C" {

int sats_mlp_forward(const sats_bf16 *x, const int32_t *token_ids, const sats_bf16 *W_gate,
                     const sats_bf16 *W_up_T, const sats_bf16 *W_down, const float *thresholds,
                     const uint8_t *route_lut, sats_bf16 *out, int64_t n_tokens, int64_t d,
                     int64_t d_ff, int64_t n_layers, hipStream_t stream) {
  g_err.clear();
  return run<uint16_t>(make_call(x, token_ids, W_gate, W_up_T, W_down, thresholds, route_lut, out,
                                 n_tokens, d, d_ff, n_layers, stream, route_mode_of(route_lut)));
}

int sats_mlp_forward_noalloc(const sats_bf16 *x, const int32_t *token_ids, const sats_bf16 *W_gate,
                             const sats_bf16 *W_up_T, const sats_bf16 *W_down, const float *thresholds,
                             const uint8_t *route_lut, sats_bf16 *out, int64_t n_tokens, int64_t d,
                             int64_t d_ff, int64_t n_layers, hipStream_t stream) {
  g_err.clear();
  Call c = make_call(x, token_ids, W_gate, W_up_T, W_down, thresholds, route_lut, out, n_tokens, d, d_ff,
                     n_layers, stream, route_mode_of(route_lut));
  c.noalloc = true;
  return run<uint16_t>(c);
}

int sats_mlp_dense(const sats_bf16 *x, const sats_bf16 *W_gate, const sats_bf16 *W_up_T,
                   const sats_bf16 *W_down, sats_bf16 *out, int64_t n_tokens, int64_t d,
                   int64_t d_ff, int64_t n_layers, hipStream_t stream) {
  g_err.clear();
  return run<uint16_t>(make_call(x, nullptr, W_gate, W_up_T, W_down, nullptr, nullptr, out, n_tokens,
                                 d, d_ff, n_layers, stream, sats::ROUTE_BASE));
}

int sats_mlp_forward_f32(const float *x, const int32_t *token_ids, const float *W_gate,
                         const float *W_up_T, const float *W_down, const float *thresholds,
                         const uint8_t *route_lut, float *out, int64_t n_tokens, int64_t d,
                         int64_t d_ff, int64_t n_layers, hipStream_t stream) {
  g_err.clear();
  return run<float>(make_call(x, token_ids, W_gate, W_up_T, W_down, thresholds, route_lut, out,
                              n_tokens, d, d_ff, n_layers, stream, route_mode_of(route_lut)));
}

int sats_mlp_dense_f32(const float *x, const float *W_gate, const float *W_up_T, const float *W_down,
                       float *out, int64_t n_tokens, int64_t d, int64_t d_ff, int64_t n_layers,
                       hipStream_t stream) {
  g_err.clear();
  return run<float>(make_call(x, nullptr, W_gate, W_up_T, W_down, nullptr, nullptr, out, n_tokens, d,
                              d_ff, n_layers, stream, sats::ROUTE_BASE));
}

int sats_mlp_forward_inspect(const sats_bf16 *x, const int32_t *token_ids, const sats_bf16 *W_gate,
                             const sats_bf16 *W_up_T, const sats_bf16 *W_down, const float *thresholds,
                             const uint8_t *route_lut, sats_bf16 *out, int64_t n_tokens, int64_t d,
                             int64_t d_ff, int64_t n_layers, hipStream_t stream, uint8_t *route_out,
                             int32_t *active_count, int32_t *active_idx, sats_bf16 *layer_in) {
  g_err.clear();
  Call c = make_call(x, token_ids, W_gate, W_up_T, W_down, thresholds, route_lut, out, n_tokens, d,
                     d_ff, n_layers, stream, route_mode_of(route_lut));
  c.route_out = route_out;
  c.active_count = active_count;
  c.active_idx = active_idx;
  c.layer_in = layer_in;
  return run<uint16_t>(c);
}

int sats_mlp_forward_inspect_f32(const float *x, const int32_t *token_ids, const float *W_gate,
                                 const float *W_up_T, const float *W_down, const float *thresholds,
                                 const uint8_t *route_lut, float *out, int64_t n_tokens, int64_t d,
                                 int64_t d_ff, int64_t n_layers, hipStream_t stream,
                                 uint8_t *route_out, int32_t *active_count, int32_t *active_idx,
                                 float *layer_in) {
  g_err.clear();
  Call c = make_call(x, token_ids, W_gate, W_up_T, W_down, thresholds, route_lut, out, n_tokens, d,
                     d_ff, n_layers, stream, route_mode_of(route_lut));
  c.route_out = route_out;
  c.active_count = active_count;
  c.active_idx = active_idx;
  c.layer_in = layer_in;
  return run<float>(c);
}


int sats_mlp_forward_lora(const sats_bf16 *x, const int32_t *token_ids, const sats_bf16 *W_gate,
                          const sats_bf16 *W_up_T, const sats_bf16 *W_down, const sats_bf16 *A_gate,
                          const sats_bf16 *B_gate, const sats_bf16 *A_up, const sats_bf16 *B_up_T,
                          const sats_bf16 *A_down, const sats_bf16 *B_down, int64_t rank, float scale,
                          const float *thresholds, const uint8_t *route_lut, sats_bf16 *out, int64_t n_tokens,
                          int64_t d, int64_t d_ff, int64_t n_layers, hipStream_t stream, uint8_t *route_out,
                          int32_t *active_count, int32_t *active_idx, sats_bf16 *layer_in) {
  return forward_lora<uint16_t>(x, token_ids, W_gate, W_up_T, W_down, A_gate, B_gate, A_up, B_up_T, A_down, B_down,
                                rank, scale, thresholds, route_lut, out, n_tokens, d, d_ff, n_layers, stream,
                                route_out, active_count, active_idx, layer_in);
}

int sats_mlp_forward_lora_f32(const float *x, const int32_t *token_ids, const float *W_gate, const float *W_up_T,
                              const float *W_down, const float *A_gate, const float *B_gate, const float *A_up,
                              const float *B_up_T, const float *A_down, const float *B_down, int64_t rank,
                              float scale, const float *thresholds, const uint8_t *route_lut, float *out,
                              int64_t n_tokens, int64_t d, int64_t d_ff, int64_t n_layers, hipStream_t stream,
                              uint8_t *route_out, int32_t *active_count, int32_t *active_idx, float *layer_in) {
  return forward_lora<float>(x, token_ids, W_gate, W_up_T, W_down, A_gate, B_gate, A_up, B_up_T, A_down, B_down,
                             rank, scale, thresholds, route_lut, out, n_tokens, d, d_ff, n_layers, stream,
                             route_out, active_count, active_idx, layer_in);
}

int sats_route_table(const float *loss_base, const float *loss_sparse, const int32_t *token_ids, int64_t n_tokens,
                     const int32_t *heldout_ids, int64_t n_heldout, int64_t vocab, double r_tar,
                     uint8_t *route_lut, double *scores, double *tau_out, double *realized_out, hipStream_t stream) {
  g_err.clear();
  return route_build(loss_base, loss_sparse, token_ids, n_tokens, heldout_ids, n_heldout, vocab, r_tar, route_lut,
                     scores, tau_out, realized_out, stream);
}

int sats_reserve(int64_t max_tokens, int64_t d, int64_t d_ff, int64_t n_layers, int elem_bytes,
                 hipStream_t stream) {
  g_err.clear();
  if (elem_bytes != 2 && elem_bytes != 4) return fail(SATS_ERR_ARG, "elem_bytes must be 2 or 4");
  if (d < 1 || d_ff < 1 || max_tokens < 1 || n_layers < 1 || d > (1 << 24) || d_ff > (1 << 24))
    return fail(SATS_ERR_SHAPE, "bad shape for sats_reserve");
  const int pass = (int)std::min<int64_t>(max_tokens, kMaxPass);
  size_t bytes = 0, nc = 0;
  int cus = device_cus();
  if (cus < 1) return fail(SATS_ERR_HIP, "no device");
  DecodePlan dps[2]{};  // the plain single-token plan and the one of LoRA calls at the largest rank
  (void)make_decode_plan(d, d_ff, elem_bytes, &dps[0], 0, cus);
  (void)make_decode_plan(d, d_ff, elem_bytes, &dps[1], sats::kLoraMaxRank, cus);
  for (const DecodePlan &dp : dps)
    for (int v = 0; v < 2; ++v)
      for (int np : {1, pass}) {
        const Plan p = make_plan(d, d_ff, elem_bytes, v == 1, np);
        bytes = std::max(bytes, layout(nullptr, p, pass, d, d_ff, elem_bytes, n_layers, dp, nullptr,
                                       elem_bytes == 2 ? sats::kLoraMaxRank : 0));
        nc = std::max(nc, counter_count(p, pass, dp));
      }
  Workspace *ws = nullptr;
  return ensure_workspace(stream, bytes, nc, &ws);
}

int sats_release(void) {
  g_err.clear();
  std::lock_guard<std::mutex> lk(g_ws_mu);
  int cur = 0;
  HIP_TRY(hipGetDevice(&cur));
  for (auto &kv : g_ws) {
    HIP_TRY(hipSetDevice(kv.first.first));
    HIP_TRY(hipDeviceSynchronize());
    if (kv.second.mem) HIP_TRY(hipFree(kv.second.mem));
    if (kv.second.counters) HIP_TRY(hipFree(kv.second.counters));
  }
  g_ws.clear();
  HIP_TRY(hipSetDevice(cur));
  int rc = route_release_all();
  if (!rc) rc = cal_release_all();
  HIP_TRY(hipSetDevice(cur));
  return rc;
}

int sats_calibration_curves(const sats_bf16 *h, const sats_bf16 *W_gate, const sats_bf16 *W_up_T,
                            const sats_bf16 *W_down, int64_t n, int64_t d, int64_t d_ff, const double *levels,
                            int64_t n_levels, float *t_out, double *err_out, double *sp_out, float *err_rows,
                            hipStream_t stream) {
  g_err.clear();
  if (!h || !W_gate || !W_up_T || !W_down || !levels || !t_out || !err_out || !sp_out)
    return fail(SATS_ERR_NULL, "h, weights, levels and the outputs must be non-null");
  if (n_levels < 1 || n_levels > 4096) return fail(SATS_ERR_ARG, "1 <= n_levels <= 4096");
  for (int64_t k = 0; k < n_levels; ++k)
    if (!(levels[k] >= 0.0 && levels[k] <= 1.0) || (k && levels[k] < levels[k - 1]))
      return fail(SATS_ERR_ARG, "levels must be ascending in [0, 1]");
  int rc = cal_check_shape(n, d, d_ff);
  if (rc) return rc;
  std::lock_guard<std::mutex> lk(g_cal_mu);
  CalBuffers cb;
  if ((rc = cal_buffers(cb, n, d, d_ff))) return rc;
  rc = cal_layer(cb, h, W_gate, W_up_T, W_down, n, d, d_ff, levels, (int)n_levels, t_out, err_out, sp_out, err_rows,
                 stream);
  const hipError_t se = hipStreamSynchronize(stream);  // also on an error: the next call reuses the buffers
  if (!rc && se != hipSuccess) return fail(SATS_ERR_HIP, "%s", hipGetErrorString(se));
  return rc;
}

int sats_calibrate_sats(const sats_bf16 *x_cal, int64_t n_cal, const sats_bf16 *W_gate, const sats_bf16 *W_up_T,
                        const sats_bf16 *W_down, int64_t d, int64_t d_ff, int64_t n_layers, double s_tar,
                        double coarse_step, double fine_step, int guardrail, float *thresholds_out,
                        double *budget_out, double *realized_out, hipStream_t stream) {
  g_err.clear();
  if (!x_cal || !W_gate || !W_up_T || !W_down || !thresholds_out)
    return fail(SATS_ERR_NULL, "x_cal, weights and thresholds_out must be non-null");
  const int rc = cal_stack(x_cal, n_cal, W_gate, W_up_T, W_down, d, d_ff, n_layers, s_tar, coarse_step, fine_step,
                           guardrail, thresholds_out, budget_out, realized_out, stream);
  if (!rc) HIP_TRY(hipStreamSynchronize(stream));
  return rc;
}

const char *sats_last_error(void) { return g_err.c_str(); }

int sats_set_options(const sats_options *opt) {
  g_err.clear();
  if (!opt) {
    g_opt = sats_options{};
    return SATS_OK;
  }
  if (opt->batch_path < SATS_BATCH_AUTO || opt->batch_path > SATS_BATCH_COMPACT ||
      opt->single_token < SATS_SINGLE_AUTO || opt->single_token > SATS_SINGLE_OFF || opt->dec_block_cols < 0 ||
      opt->dec_block_cols > sats::kDecodeMaxCols || opt->lora_per_token < 0 || opt->lora_per_token > 1)
    return fail(SATS_ERR_ARG, "an option is outside its range");
  g_opt = *opt;
  return SATS_OK;
}

int sats_query_path(int64_t n_tokens, int64_t d, int64_t d_ff, int elem_bytes, int aligned16, int n_cus,
                    int *path) {
  g_err.clear();
  if (!path) return fail(SATS_ERR_NULL, "path must be non-null");
  if (elem_bytes != 2 && elem_bytes != 4) return fail(SATS_ERR_ARG, "elem_bytes must be 2 or 4");
  if (n_cus < 0) return fail(SATS_ERR_ARG, "n_cus must be >= 0");
  if (d < 1 || d_ff < 1 || n_tokens < 0 || d > (1 << 24) || d_ff > (1 << 24) || n_tokens > ((int64_t)1 << 40))
    return fail(SATS_ERR_SHAPE, "need d >= 1, d_ff >= 1, n_tokens >= 0, d and d_ff at most 2^24");
  *path = 0;
  if (n_tokens == 0) return SATS_OK;
  const int vec = 16 / elem_bytes;
  const bool vec_ok = aligned16 && d % vec == 0 && d_ff % vec == 0;
  const int cus = n_cus > 0 ? n_cus : device_cus();
  DecodePlan dp;
  if (n_tokens == 1 && vec_ok && g_opt.single_token != SATS_SINGLE_OFF &&
      make_decode_plan(d, d_ff, elem_bytes, &dp, 0, cus)) {
    *path = SATS_PATH_SINGLE_TOKEN;
    return SATS_OK;
  }
  const int np = (int)std::min<int64_t>(n_tokens, kMaxPass);
  if (!batch_mfma(elem_bytes, vec_ok, np, false, d, d_ff)) *path = SATS_PATH_BATCH_COMPACT;
  else *path = batch_whole() ? SATS_PATH_BATCH_MFMA : SATS_PATH_BATCH_SPLIT;
  return SATS_OK;
}

int sats_device_status(hipStream_t stream) {
  g_err.clear();
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  HIP_TRY(hipStreamSynchronize(stream));
  // the flags of this stream's workspace and of the device's allocation-free scratch
  std::vector<unsigned *> flags;
  {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    auto it = g_ws.find({dev, stream});
    if (it != g_ws.end() && it->second.counters) flags.push_back(it->second.counters + kErr);
  }
  {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    auto it = g_scratch.find(dev);
    if (it != g_scratch.end()) flags.push_back(reinterpret_cast<unsigned *>(it->second) + kErr);
  }
  bool raised = false;
  for (unsigned *f : flags) {
    unsigned flag = 0;
    HIP_TRY(hipMemcpy(&flag, f, sizeof flag, hipMemcpyDeviceToHost));
    if (flag) {
      const unsigned zero = 0;
      HIP_TRY(hipMemcpy(f, &zero, sizeof zero, hipMemcpyHostToDevice));
      raised = true;
    }
  }
  if (raised) return fail(SATS_ERR_DEVICE, "a bounded device-side wait gave up (results of the affected call are invalid)");
  return SATS_OK;
}

int sats_timing_begin(int kind, int capacity) {
  g_err.clear();
  if (kind < 0 || kind >= SATS_K_COUNT || capacity < 1) return fail(SATS_ERR_ARG, "bad timing request");
  std::lock_guard<std::mutex> lk(g_timer_mu);
  Timer &t = g_timer[kind];
  while ((int)t.start.size() < capacity) {
    hipEvent_t a, b;
    HIP_TRY(hipEventCreate(&a));
    HIP_TRY(hipEventCreate(&b));
    t.start.push_back(a);
    t.stop.push_back(b);
  }
  t.cap = capacity;
  t.used = 0;
  t.armed = true;
  return SATS_OK;
}

int sats_timing_end(int kind, double *total_ms, int64_t *count) {
  g_err.clear();
  if (kind < 0 || kind >= SATS_K_COUNT) return fail(SATS_ERR_ARG, "bad timing kind");
  std::lock_guard<std::mutex> lk(g_timer_mu);
  Timer &t = g_timer[kind];
  t.armed = false;
  double sum = 0.0;
  for (int i = 0; i < t.used; ++i) {
    HIP_TRY(hipEventSynchronize(t.stop[i]));
    float ms = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, t.start[i], t.stop[i]));
    sum += ms;
  }
  if (total_ms) *total_ms = sum;
  if (count) *count = t.used;
  t.used = 0;
  return SATS_OK;
}

#ifdef SATS_TRACE
int sats_trace_read(unsigned long long *host, int64_t count) {
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpyFromSymbol(host, HIP_SYMBOL(sats::sats_trace_buf),
                              sizeof(unsigned long long) * (size_t)std::min<int64_t>(count, 4096 * 16)));
  return SATS_OK;
}
#endif

const char *sats_kernel_name(int kind) {
  switch (kind) {
    case SATS_K_GATE: return "gate_kernel";
    case SATS_K_UP: return "up_kernel";
    case SATS_K_DOWN: return "down_kernel";
    case SATS_K_INSPECT: return "compact_kernel";
    case SATS_K_DENSE: return "dense_gateup_kernel";
    case SATS_K_DENSE_DOWN: return "dense_down_kernel";
    case SATS_K_ROUTE_ACCUM: return "route_part_kernel";
    case SATS_K_ROUTE_MERGE: return "route_merge_kernel";
    case SATS_K_LORA_V: return "lora_v_kernel";
    case SATS_K_DEC_LAYER: return "dec_layer_kernel";
    case SATS_K_DEC_LORA_V: return "dec_lora_v_kernel";
    case SATS_K_DEC_REDUCE: return "dec_reduce_kernel";
    case SATS_K_DEC_REDUCE_LORA: return "dec_reduce_lora_kernel";
    case SATS_K_CAL_ERR: return "cal_err_kernel";
    case SATS_K_CAL_GATEUP: return "dense_gateup_kernel (calibration)";
    default: return "";
  }
}

}  // extern "C"
