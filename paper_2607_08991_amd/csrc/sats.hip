// Host side of the C ABI declared in include/sats.h: argument checks,
// workspace management, launch planning and kernel timing.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
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
  TimedLaunch(int kind, hipStream_t) {
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
  const int64_t tiles = d / sats::kDenseDownNT;
  int64_t ks = std::max<int64_t>(1, (256 + tiles - 1) / tiles);
  ks = std::min<int64_t>(ks, std::min<int64_t>(sats::kDenseMaxKsplit, std::max<int64_t>(1, d_ff / sats::kDenseKC)));
  return (int)ks;
}

// MFMA kernels specialised on the 16-row tiles that cover a pass of np tokens
typedef void (*DenseKernel)(sats::DenseArgs);
DenseKernel dense_gateup_fn(int np) {
  using namespace sats;
  const int mt = (np + 15) / 16;
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

int env_int(const char *name, int dflt) {
  const char *s = getenv(name);
  if (!s || !*s) return dflt;
  int v = atoi(s);
  return v > 0 ? v : dflt;
}

struct Plan {
  int vec, CL, RG, CB;     // down lanes per row segment; gate row groups and columns per block
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
  const int gate_cl = (p.vec == 1) ? 64 : sats::kGateLanes;
  p.RG = sats::kThreads / gate_cl;
  p.CB = gate_cl * p.vec;
  p.nblocks = (int)((d_ff + p.CB - 1) / p.CB);
  p.NT = (n_pass == 1) ? 1 : 4;
  const int gate_target = env_int("SATS_GATE_WGS", 2048);
  int ks = round_pow2_down(std::max(1, gate_target / p.nblocks));
  ks = std::min<int64_t>(ks, std::max<int64_t>(1, d / p.RG));
  ks = std::max<int64_t>(ks, (d + 1023) / 1024);
  p.KC = (int)((d + ks - 1) / ks);
  p.KS = (int)((d + p.KC - 1) / p.KC);
  p.SW = p.CL * p.vec;
  p.n_slices = (int)((d + p.SW - 1) / p.SW);
  const int down_target = env_int("SATS_DOWN_WGS", 512);
  p.KCH = std::max(1, down_target / p.n_slices);
  const int rows_per_wave = env_int("SATS_UP_ROWS_PER_WAVE", 2);
  int64_t waves = (d_ff + rows_per_wave - 1) / rows_per_wave;
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
  float *dgpart;          // single-token path: partial gate sums per row chunk
  int *dstate;            // single-token path: the token's route
  int *perm, *ctl;        // batched path: token partition and dense-group control words
  uint8_t *skip, *gbase;
  uint16_t *xd, *hnext, *pdense;  // dense group (MFMA): inputs, next inputs, p
  float *ddpart;                   // dense group down-projection partials
};

// Layout for passes of up to `pass` tokens (the counters live in their own
// zero-initialised allocation).
struct DecodePlan {
  int G = 0;           // rows workgroups, one partial y each (0: path not used)
  int RW = 0;          // reduce workgroups (128-byte column slices where d allows)
  int nblk = 0;        // gate column blocks
  int nrc = 0;         // gate row chunks
  int gate_grid = 0;   // workgroups of the gate launch
};

size_t layout(char *base, const Plan &p, int64_t pass, int64_t d, int64_t d_ff, int esz, int64_t L,
              const DecodePlan &dp, Buffers *b) {
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
  t.sspart = c.take<float>(std::max(dp.G, dp.RW));
  t.perm = c.take<int>(Pp);
  t.ctl = c.take<int>(64);
  t.skip = c.take<uint8_t>(Pp);
  t.gbase = c.take<uint8_t>(Pp);
  t.xd = c.take<uint16_t>(Pp * d);
  t.hnext = c.take<uint16_t>(Pp * d);
  t.pdense = c.take<uint16_t>(Pp * d_ff);
  t.ddpart = c.take<float>((int64_t)sats::kDenseMaxKsplit * Pp * d);
  t.dgpart = c.take<float>((int64_t)sats::dec_nrcp(dp.nrc) * d_ff);
  t.dstate = c.take<int>(64);
  if (b) *b = t;
  return c.off;
}

// The counter allocation starts with control words (the device error flag);
// the per-block counters follow.  Every counter is zero whenever no kernel is
// running.
constexpr size_t kCtl = 512;
constexpr size_t kErr = 320;
constexpr size_t kDone = 322;  // single-token rows launch: partials written (second-stage reduction)

size_t counter_count(const Plan &p, int64_t pass, const DecodePlan &dp) {
  const int64_t tiles = ((pass + 3) / 4) * 4;
  (void)dp;
  return kCtl + (size_t)std::max<int64_t>(tiles * p.nblocks + tiles * p.n_slices, 2 * (int64_t)p.nblocks + 64);
}

// ------------------------------------------------------- single-token plan

int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return cus;
}

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

// Single-token plan.  h is held in LDS (d <= kDecodeMaxD); `G` workgroups
// (at most kDecodeMaxG) take the rows and reduce phases, each reduce
// workgroup owning at most one column per thread; gate tiles are one column
// block by about d / nrc rows.  Returns false when the shape does not fit.
bool make_decode_plan(int64_t d, int64_t d_ff, int esz, int G, DecodePlan *dp) {
  DecodePlan q{};
  const int64_t cb = (int64_t)(16 / esz) * 64;
  q.G = G;
  q.nblk = (int)((d_ff + cb - 1) / cb);
  const int64_t tiles = env_int("SATS_DEC_GATE_WGS", 256);
  int64_t nrc = std::max<int64_t>(1, tiles / q.nblk);
  nrc = std::min<int64_t>(nrc, std::max<int64_t>(1, d / (sats::kGateThreads / 64)));  // a row per wavefront
  q.nrc = (int)nrc;
  q.gate_grid = q.nblk * q.nrc;
  // second reduction stage: the last RW rows workgroups to finish take one
  // slice of y each, 32 columns (128 bytes of each partial) or more; RW is
  // kept to a quarter of the CUs so that the reducers, which wait for the
  // others, never fill the device
  q.RW = (int)std::min<int64_t>(std::max<int64_t>(1, (d + 31) / 32), std::max(1, device_cus() / 4));
  q.RW = std::min(q.RW, G);
  const bool ok = G >= 1 && G <= sats::kDecodeMaxG && d <= sats::kDecodeMaxD &&
                  (d + q.RW - 1) / q.RW <= sats::kDecodeThreads;
  *dp = ok ? q : DecodePlan{};
  return ok;
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
  const bool mfma = sizeof(T) == 2 && VEC > 1 && np >= kMfmaMinTokens &&
                    d % kDenseDownNT == 0 && d_ff % kDenseKC == 0 && d <= 4096 &&
                    (uint64_t)d * d_ff * 2 < (1ull << 31) &&
                    !getenv("SATS_NO_MFMA");
  // whole batch on MFMA (each row applies its own keep rule): known here, so
  // the compacted sparse-path launches are left out
  const bool whole = !getenv("SATS_MFMA_BASE_GROUP_ONLY");
  const bool all_mfma = mfma && whole;
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
    hipLaunchKernelGGL(route_kernel, dim3(np), dim3(kThreads), 0, c.stream, ra);
    HIP_TRY(hipGetLastError());
  }

  for (int64_t l = 0; l < c.L; ++l) {
    if (mfma) {
      // base-path group on MFMA (kernels return at once when the group is small)
      DenseArgs da{};
      da.ctl = b.ctl;
      da.gbase = b.gbase;
      da.perm = b.perm;
      da.thr = c.thr ? c.thr + l : nullptr;
      da.keep_out = inspect_lists ? b.keep : nullptr;
      da.H = (l == 0) ? b.xd : b.hnext;
      da.Wb = static_cast<const uint16_t *>(c.Wg) + l * wl;
      da.Wt = static_cast<const uint16_t *>(c.Wu) + l * wl;
      da.P = b.pdense;
      da.K = (int)d;
      da.N = (int)d_ff;
      {
        TimedLaunch tl(SATS_K_DENSE, c.stream);
        hipExtLaunchKernelGGL(dense_gateup_fn(np), dim3(d_ff / kDenseNT), dim3(kDenseThreads), 0, c.stream,
                              tl.start, tl.stop, 0, da);
      }
      HIP_TRY(hipGetLastError());
      DenseArgs dd{};
      dd.ctl = b.ctl;
      dd.H = b.pdense;
      dd.Wb = static_cast<const uint16_t *>(c.Wd) + l * wl;
      dd.part = b.ddpart;
      dd.K = (int)d_ff;
      dd.N = (int)d;
      const int ks = dense_ksplit(d, d_ff);
      dd.kchunk = (int)(((d_ff + ks - 1) / ks + kDenseKC - 1) / kDenseKC * kDenseKC);
      {
        TimedLaunch tl(SATS_K_DENSE, c.stream);
        hipExtLaunchKernelGGL(dense_down_fn(np), dim3(d / kDenseDownNT, ks), dim3(kDenseThreads), 0, c.stream,
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
    const size_t gate_lds = sizeof(float) * std::max<size_t>((size_t)NT * p.KC, (size_t)p.RG * NT * p.CB);
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
  a.nblk = dp.nblk;
  a.nrc = dp.nrc;
  a.gpart = b.dgpart;
  a.state = b.dstate;
  a.G = dp.G;
  a.RW = dp.RW;
  a.ypart = b.ypart;
  a.done = counters + kDone;
  a.err = counters + kErr;
  a.ybuf = b.ybuf;
  a.sspart = b.sspart;
  a.route_out = c.route_out;
  const bool lists = c.active_count || c.active_idx;
  a.keep_out = lists ? b.keep : nullptr;
  a.layer_in = c.layer_in;
  // two plain launches per layer (the rows launch ends with the second
  // reduction stage); kernel boundaries order the phases
  for (int l = 0; l < (int)c.L; ++l) {
    {
      TimedLaunch tl(SATS_K_DEC_GATE, c.stream);
      hipExtLaunchKernelGGL((dec_gate_kernel<T>), dim3(dp.gate_grid), dim3(kGateThreads), 0, c.stream,
                            tl.start, tl.stop, 0, a, l);
    }
    HIP_TRY(hipGetLastError());
    {
      TimedLaunch tl(SATS_K_DEC_ROWS, c.stream);
      hipExtLaunchKernelGGL((dec_rows_kernel<T>), dim3(dp.G), dim3(kDecodeThreads), 0, c.stream,
                            tl.start, tl.stop, 0, a, l);
    }
    HIP_TRY(hipGetLastError());
  }
  if (lists) {
    for (int64_t l = 0; l < c.L; ++l) {
      CompactArgs ca{};
      ca.keep = b.keep + l * c.d_ff;
      ca.idx = c.active_idx ? c.active_idx + l * c.d_ff : nullptr;
      ca.count = c.active_count ? c.active_count + l : nullptr;
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
  // single-token path: one token, vector layout, h fits the LDS copy
  bool decode = c.n == 1 && vec_ok && !getenv("SATS_NO_DECODE");
  DecodePlan dp;
  if (decode) decode = make_decode_plan(c.d, c.d_ff, esz, env_int("SATS_DEC_ROWS_WGS", device_cus()), &dp);
  const size_t bytes = layout(nullptr, p, pass, c.d, c.d_ff, esz, c.L, dp, nullptr);
  Workspace *ws = nullptr;
  size_t ncount = counter_count(p, pass, dp);
  int rc = ensure_workspace(c.stream, bytes, ncount, &ws);
  if (rc) return rc;
  Buffers b{};
  layout(ws->mem, p, pass, c.d, c.d_ff, esz, c.L, dp, &b);
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
  DecodePlan dp{};
  (void)make_decode_plan(d, d_ff, elem_bytes, env_int("SATS_DEC_ROWS_WGS", cus), &dp);
  for (int v = 0; v < 2; ++v)
    for (int np : {1, pass}) {
      const Plan p = make_plan(d, d_ff, elem_bytes, v == 1, np);
      bytes = std::max(bytes, layout(nullptr, p, pass, d, d_ff, elem_bytes, n_layers, dp, nullptr));
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
  return SATS_OK;
}

const char *sats_last_error(void) { return g_err.c_str(); }

int sats_device_status(hipStream_t stream) {
  g_err.clear();
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  HIP_TRY(hipStreamSynchronize(stream));
  std::lock_guard<std::mutex> lk(g_ws_mu);
  auto it = g_ws.find({dev, stream});
  if (it == g_ws.end() || !it->second.counters) return SATS_OK;
  unsigned flag = 0;
  HIP_TRY(hipMemcpy(&flag, it->second.counters + kErr, sizeof flag, hipMemcpyDeviceToHost));
  if (flag) {
    const unsigned zero = 0;
    HIP_TRY(hipMemcpy(it->second.counters + kErr, &zero, sizeof zero, hipMemcpyHostToDevice));
    return fail(SATS_ERR_DEVICE, "a bounded device-side wait gave up (results of the affected call are invalid)");
  }
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
                              sizeof(unsigned long long) * (size_t)std::min<int64_t>(count, 4096 * 8)));
  return SATS_OK;
}
#endif

const char *sats_kernel_name(int kind) {
  switch (kind) {
    case SATS_K_GATE: return "gate_kernel";
    case SATS_K_UP: return "up_kernel";
    case SATS_K_DOWN: return "down_kernel";
    case SATS_K_INSPECT: return "compact_kernel";
    case SATS_K_DENSE: return "dense_mfma_kernels";
    case SATS_K_DEC_GATE: return "dec_gate_kernel";
    case SATS_K_DEC_ROWS: return "dec_rows_kernel";
    default: return "";
  }
}

}  // extern "C"
