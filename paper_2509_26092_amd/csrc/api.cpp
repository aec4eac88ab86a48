// Step executor and C ABI of the ResNet-18 training-step library.
//
// The host side builds, once per (N,H,W), a plan: every layer's shapes, the
// workspace offset of every saved tensor, and the split counts of the weight
// gradients. A step is then a fixed sequence of kernel launches on the
// context's stream with no host synchronisation.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/rn18.h"
#include "../../include/rn18_ops.h"
#include "kernels.h"

using namespace rn18;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIPCHK(x)                                                              \
  do {                                                                         \
    hipError_t e_ = (x);                                                       \
    if (e_ != hipSuccess) return fail(RN18_EHIP, "%s: %s", #x, hipGetErrorString(e_)); \
  } while (0)
#define LCHK(x)                                                                \
  do {                                                                         \
    int r_ = (x);                                                              \
    if (r_ != 0) return fail(RN18_EHIP, "launch failed: %s (%s)", #x, hipGetErrorString(hipGetLastError())); \
  } while (0)

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
inline int out_size(int h, int k, int s, int p) { return (h + 2 * p - k) / s + 1; }
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The convolution kernels address each tensor with 32-bit byte offsets:
// buffer resources sized to the tensor, an out-of-range sentinel of 2^31, and
// unsigned offset arithmetic that may run a tile (< 1 MiB) past the end. A
// convolution launch therefore sees tensors below 2^31 bytes minus a 16 MiB
// margin: a training step launches each convolution over batch chunks that
// fit, and the single-operator entry points reject larger tensors.
constexpr size_t kMaxTensorBytes = ((size_t)1 << 31) - ((size_t)1 << 24);
// The other kernels index whole tensors by 16-byte chunk in 32-bit integers
// (or by element in 64-bit ones): every tensor of a step stays below 16 times
// the bound above.
constexpr size_t kMaxWholeTensorBytes = 16 * kMaxTensorBytes;

// fp16 loss scaling defaults: initial scale and growth interval (steps)
constexpr float kLossScaleInit = 65536.0f;
constexpr unsigned kLossScaleInterval = 2000;

// ----------------------------------------------------------------------------
// Architecture
// ----------------------------------------------------------------------------
struct ConvL {
  int cin, cout, k, s, p;
  int cin_p;               // channels of the NHWC input tensor (padded for the stem)
  long w, g, b, rm, rv;    // offsets in the flat state (floats)
  long wf, wd;             // element offsets in the weight shadows (wd = -1: none)
};
struct BlockL { int c1, c2, ds; };

struct Arch {
  std::vector<ConvL> convs;
  std::vector<BlockL> blocks;
  int feat = 0, classes = 0;
  bool imagenet = false;
  long fc_w = 0, fc_b = 0, P = 0, R = 0;
  long wf_total = 0, wd_total = 0;
  long wf_s2d = -1;      // ImageNet stem as a 4x4 conv over its space-to-depth input: [64][16][16]
};

bool build_arch(const rn18_config& c, Arch* a) {
  if (c.num_classes < 1 || c.arch < 0 || c.arch > 2 || c.prec < 0 || c.prec > 2) return false;
  const int cp = prec_vw(c.prec);
  int stem_c, stem_k, stem_s, stem_p;
  std::vector<int> widths, nblk, fstride;
  if (c.arch == RN18_TINY) {
    stem_c = 16; stem_k = 3; stem_s = 1; stem_p = 1;
    widths = {16}; nblk = {1}; fstride = {1};
  } else {
    stem_c = 64;
    if (c.arch == RN18_IMAGENET) { stem_k = 7; stem_s = 2; stem_p = 3; }
    else { stem_k = 3; stem_s = 1; stem_p = 1; }
    widths = {64, 128, 256, 512}; nblk = {2, 2, 2, 2}; fstride = {1, 2, 2, 2};
  }
  a->imagenet = c.arch == RN18_IMAGENET;
  a->convs.clear();
  a->blocks.clear();
  a->convs.push_back(ConvL{3, stem_c, stem_k, stem_s, stem_p, cp});
  int cin = stem_c;
  for (size_t si = 0; si < widths.size(); ++si)
    for (int bi = 0; bi < nblk[si]; ++bi) {
      const int s = bi == 0 ? fstride[si] : 1, w = widths[si];
      BlockL b;
      b.c1 = (int)a->convs.size(); a->convs.push_back(ConvL{cin, w, 3, s, 1, cin});
      b.c2 = (int)a->convs.size(); a->convs.push_back(ConvL{w, w, 3, 1, 1, w});
      b.ds = -1;
      if (s != 1 || cin != w) { b.ds = (int)a->convs.size(); a->convs.push_back(ConvL{cin, w, 1, s, 0, cin}); }
      a->blocks.push_back(b);
      cin = w;
    }
  a->feat = cin;
  a->classes = c.num_classes;
  long o = 0;
  for (auto& L : a->convs) {
    L.w = o; o += (long)L.cout * L.cin * L.k * L.k;
    L.g = o; o += L.cout;
    L.b = o; o += L.cout;
  }
  a->fc_w = o; o += (long)c.num_classes * a->feat;
  a->fc_b = o; o += c.num_classes;
  a->P = o;
  for (auto& L : a->convs) {
    L.rm = o; o += L.cout;
    L.rv = o; o += L.cout;
  }
  a->R = o - a->P;
  long f = 0, d = 0;
  for (size_t i = 0; i < a->convs.size(); ++i) {
    ConvL& L = a->convs[i];
    L.wf = f; f += (long)L.cout * L.k * L.k * L.cin_p;
    if (i == 0) L.wd = -1;
    else { L.wd = d; d += (long)L.cout * L.k * L.k * L.cin_p; }
  }
  if (a->imagenet) {
    a->wf_s2d = f;
    f += (long)a->convs[0].cout * 16 * 16;
  }
  a->wf_total = f;
  a->wd_total = d;
  return true;
}

// ----------------------------------------------------------------------------
// Plan for one (N,H,W)
// ----------------------------------------------------------------------------
struct ConvP {
  int Hin, Win, Ho, Wo;         // stored input and output sizes
  int k, s, p, cin;             // conv as computed: kernel, stride, pad, stored input channels
  long wf;                      // its forward weight shadow offset
  bool s2d;                     // ImageNet stem computed as a 4x4 conv over a space-to-depth input
  long M;                       // N*Ho*Wo
  size_t x, y;                  // workspace offsets of input and output
  size_t mean, rstd, scale, shift, coef;
  int nb;                       // images per launch (batch chunk whose tensors fit 32-bit offsets)
  int splits, pps;              // weight-gradient split-K of a full chunk of nb images
  int splits_r, pps_r;          // ... and of the last, shorter chunk (N % nb images), if any
  int wslots;                   // split-K partial slots over all chunks
};
// mbits: ReLU mask bytes of the block output (one byte per 16-byte chunk)
struct BlockP { size_t in, z1, out, mbits; };

constexpr size_t kSplitScratchBytes = (size_t)64 << 20;
constexpr size_t kFuseBwdMaxBytes = (size_t)16 << 20;   // largest BN tensor whose backward partials a data gradient writes

struct Plan {
  int N, H, W;
  std::vector<ConvP> cp;
  std::vector<BlockP> bp;
  size_t x0, zstem, pool, parg;
  int Hs, Ws, Hp, Wp;           // stem output and pool output sizes
  int Hf, Wf;                   // final feature map
  size_t f, logits, dlogits, df, rowloss, lossbuf;
  // gy[p], gy2[p]: dY of the second and first conv of the blocks of index
  // parity p (gy[1] also takes the stem's dY); gyd: dY of a projection
  size_t gA, gB, gz, gy[2], gy2[2], gyd;
  size_t part, wpart, grad;
  size_t bnst;                  // forward conv epilogue BN partials (one entry per 32 rows at most)
  size_t bnst2, part2;          // the same scratch for the projection convs, which run on the side stream
  size_t gsplit, gsplit_bytes;  // split-K partials of the forward and data-gradient convs (caller's stream)
  size_t total;
};

struct Ctx {
  rn18_config cfg;
  Arch arch;
  int prec;
  int es;                       // element size of activations
  hipStream_t stream;
  float* momentum = nullptr;
  void* wf = nullptr;
  void* wd = nullptr;
  RepackEntry* tab = nullptr;   // element-wise repack entries, then the tiled ones (one allocation)
  int ntab = 0, nttab = 0, ntiles = 0;
  long tab_total = 0;           // elements over the element-wise entries
  unsigned* err = nullptr;
  LossScale* ls = nullptr;      // fp16 contexts: dynamic loss scale (device)
  // dropout before the classifier: on iff the rate is > 0, keep threshold,
  // scale, and the Philox key and step counter of the next training step
  bool drop_on = false;
  uint32_t drop_thresh = 0;
  float drop_scale = 1.f;
  uint64_t drop_seed = 0, drop_step = 0;
  // weight gradients run on a second stream (default priority) beside the
  // data-gradient chain: events hand each dY buffer over and back
  hipStream_t side = nullptr;
  // ev_blk[p]: end of the side-stream weight gradients of the last block of
  // index parity p
  hipEvent_t ev_fork = nullptr, ev_join = nullptr, ev_ds = nullptr, ev_blk[2] = {nullptr, nullptr};
  void* ws = nullptr;
  size_t ws_bytes = 0;
  bool ws_owned = false;
  std::map<std::tuple<int, int, int>, Plan> plans;
  int dbg_stop_blocks = -1;     // debugging: end the backward pass after this many blocks
  int dbg_chunk = 0;            // debugging: at most this many images per convolution launch (0 = as needed)
  bool dbg_serial = false;      // debugging: every launch on the caller's stream (no side stream)
  struct Capture { int kind, index; void* dst; size_t bytes; };
  std::vector<Capture> captures; // debugging: copies of backward tensors
  // optional per-launch timing with HIP events on the context stream
  struct ProfEv { int cls, layer, tile; const char* name; double flops, bytes; hipEvent_t a, b; };
  bool prof_on = false;
  std::vector<ProfEv> prof;
  std::vector<hipEvent_t> prof_spare;
};

hipEvent_t prof_event(Ctx* c) {
  if (!c->prof_spare.empty()) {
    hipEvent_t e = c->prof_spare.back();
    c->prof_spare.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Start a timed launch group; returns its index or -1 when profiling is off.
int prof_begin(Ctx* c, int cls, int layer, int tile, const char* name, double flops, double bytes) {
  if (!c || !c->prof_on) return -1;
  Ctx::ProfEv ev{cls, layer, tile, name, flops, bytes, prof_event(c), prof_event(c)};
  if (!ev.a || !ev.b || hipEventRecord(ev.a, c->stream) != hipSuccess) return -1;
  c->prof.push_back(ev);
  return (int)c->prof.size() - 1;
}
void prof_end(Ctx* c, int idx) {
  if (idx >= 0) (void)hipEventRecord(c->prof[idx].b, c->stream);
}
#define TIMED(cls, layer, tile, name, fl, by, expr)             \
  do {                                                          \
    const int pi_ = prof_begin(c, cls, layer, tile, name, fl, by); \
    LCHK(expr);                                \
    prof_end(c, pi_);                          \
  } while (0)

// Enqueue the debugging copies registered for (kind, index) from `src`.
int run_captures(Ctx* c, int kind, int index, const void* src, size_t avail) {
  for (const auto& cp : c->captures) {
    if (cp.kind != kind || cp.index != index) continue;
    if (cp.bytes > avail) return fail(RN18_EINVAL, "capture of %zu bytes exceeds the %zu-byte tensor", cp.bytes, avail);
    HIPCHK(hipMemcpyAsync(cp.dst, src, cp.bytes, hipMemcpyDeviceToDevice, c->stream));
  }
  return RN18_OK;
}

ConvGather gather_fwd(const void* x, const void* w, void* y, int N, int Hin, int Win, int Cin, int Ho, int Wo,
                      int Cout, int k, int s, int p) {
  ConvGather g{};
  g.A = x; g.B = w; g.C = y;
  g.N = N; g.Hin = Hin; g.Win = Win; g.Cin = Cin;
  g.Hm = Ho; g.Wm = Wo; g.M = N * Ho * Wo;
  g.Hout = Ho; g.Wout = Wo; g.Cols = Cout;
  g.os = 1; g.oph = 0; g.opw = 0;
  g.is = s; g.ip = p;
  g.nth = k; g.ntw = k;
  g.dh0 = 0; g.dhs = 1; g.dw0 = 0; g.dws = 1;
  g.wkh0 = 0; g.wkhs = 1; g.wkw0 = 0; g.wkws = 1; g.KW = k; g.KHW = k * k;
  g.K = k * k * Cin;
  g.mode = 0;
  return g;
}

// Data gradient of a stride-1 conv (input [N][H][W][Cin], output
// [N][Ho][Wo][Cout]) as a forward conv of dY with the taps mirrored.
ConvGather gather_dgrad1(const void* dy, const void* wd, void* dx, int N, int H, int W, int Cin, int Ho, int Wo,
                         int Cout, int k, int p, int mode, const void* R, const void* Rm) {
  ConvGather g{};
  g.A = dy; g.B = wd; g.C = dx; g.R = R; g.Rm = Rm;
  g.N = N; g.Hin = Ho; g.Win = Wo; g.Cin = Cout;
  g.Hm = H; g.Wm = W; g.M = N * H * W;
  g.Hout = H; g.Wout = W; g.Cols = Cin;
  g.os = 1; g.oph = 0; g.opw = 0;
  g.is = 1; g.ip = k - 1 - p;
  g.nth = k; g.ntw = k;
  g.dh0 = 0; g.dhs = 1; g.dw0 = 0; g.dws = 1;
  g.wkh0 = k - 1; g.wkhs = -1; g.wkw0 = k - 1; g.wkws = -1; g.KW = k; g.KHW = k * k;
  g.K = k * k * Cout;
  g.mode = mode;
  return g;
}

int build_plan(const Ctx& c, int N, int H, int W, Plan* pl, std::string* why) {
  const Arch& a = c.arch;
  const int es = c.es;
  char buf[256];
  if (N < 1 || H < 1 || W < 1) { *why = "N, H and W must be >= 1"; return RN18_EINVAL; }
  if ((long)N * H * W >= (1l << 31)) { *why = "input too large"; return RN18_EINVAL; }
  pl->N = N; pl->H = H; pl->W = W;
  size_t off = 0, max_tensor = (size_t)N * 3 * H * W * 4;  // the caller's NCHW fp32 images
  auto alloc = [&](size_t bytes) {
    if (bytes > max_tensor) max_tensor = bytes;
    size_t o = off;
    off += align256(bytes);
    return o;
  };
  auto act = [&](int h, int w, int ch) { return alloc((size_t)N * h * w * ch * es); };
  pl->cp.assign(a.convs.size(), ConvP{});
  pl->bp.assign(a.blocks.size(), BlockP{});
  size_t max_blockio = 0, max_z1 = 0, max_y = 0, max_yb = 0, max_yd = 0, max_wpart = 0;
  long max_partC = 0;

  auto conv_plan = [&](int li, int hin, int win, size_t xin) -> bool {
    const ConvL& L = a.convs[li];
    ConvP& P = pl->cp[li];
    P.Hin = hin; P.Win = win;
    P.Ho = out_size(hin, L.k, L.s, L.p);
    P.Wo = out_size(win, L.k, L.s, L.p);
    P.k = L.k; P.s = L.s; P.p = L.p; P.cin = L.cin_p; P.wf = L.wf; P.s2d = false;
    if (li == 0 && a.wf_s2d >= 0 && hin % 2 == 0 && win % 2 == 0) {
      // 7x7 stride-2 pad-3 stem == 4x4 stride-1 conv over the 2x2 space-to-depth
      // input (H/2 x W/2 x 16), padded by 2 before and 1 after
      P.s2d = true;
      P.Hin = hin / 2; P.Win = win / 2;
      P.k = 4; P.s = 1; P.p = 2; P.cin = 16; P.wf = a.wf_s2d;
    }
    if (P.Ho < 1 || P.Wo < 1) {
      snprintf(buf, sizeof buf, "conv %d: empty output for input %dx%d", li, hin, win);
      *why = buf;
      return false;
    }
    P.M = (long)N * P.Ho * P.Wo;
    if (P.M < 2) {
      snprintf(buf, sizeof buf, "batch norm after conv %d sees a single value per channel (N*Ho*Wo = 1)", li);
      *why = buf;
      return false;
    }
    {
      const size_t in_img = (size_t)P.Hin * P.Win * P.cin * es, out_img = (size_t)P.Ho * P.Wo * L.cout * es;
      const size_t per_img = std::max(in_img, out_img);
      if (per_img > kMaxTensorBytes) {
        snprintf(buf, sizeof buf, "one image of conv %d needs %zu bytes, beyond the per-launch limit", li, per_img);
        *why = buf;
        return false;
      }
      long nb = std::min((long)N, (long)(kMaxTensorBytes / per_img));
      if (c.dbg_chunk > 0) nb = std::min(nb, (long)c.dbg_chunk);
      P.nb = (int)nb;
    }
    P.x = xin;
    P.y = act(P.Ho, P.Wo, L.cout);
    P.mean = alloc(L.cout * 4); P.rstd = alloc(L.cout * 4);
    P.scale = alloc(L.cout * 4); P.shift = alloc(L.cout * 4);
    P.coef = alloc(3 * L.cout * 4);
    const size_t ybytes = (size_t)P.M * L.cout * es;
    if (ybytes > max_y) max_y = ybytes;
    if (li > 0 && ybytes > max_yb) max_yb = ybytes;   // block convs (not the stem)
    {
      ConvWgrad wg{};
      wg.N = P.nb; wg.H = P.Hin; wg.W = P.Win; wg.Cin = P.cin; wg.Ho = P.Ho; wg.Wo = P.Wo; wg.Cout = L.cout;
      wg.KH = P.k; wg.KW = P.k; wg.stride = P.s; wg.pad = P.p;
      P.splits = conv_wgrad_splits_shape(c.prec, wg, &P.pps);
      const int rem = N % P.nb;
      P.splits_r = P.pps_r = 0;
      if (rem) {
        wg.N = rem;
        P.splits_r = conv_wgrad_splits_shape(c.prec, wg, &P.pps_r);
      }
      P.wslots = (N / P.nb) * P.splits + P.splits_r;
    }
    const size_t wp = (size_t)P.wslots * L.cout * P.k * P.k * P.cin * 4;
    if (wp > max_wpart) max_wpart = wp;
    // backward partials (2 floats per block and channel) or the forward
    // statistics' chunk sums (3 doubles per chunk and channel, <= 64 chunks)
    long pc = (long)bn_bwd_partial_blocks(c.prec, P.M, L.cout) * L.cout * 2;
    if (li == 0 && a.imagenet)
      pc = std::max(pc, (long)bn_bwd_partial_pool_blocks(c.prec, N, P.Ho, P.Wo, L.cout) * L.cout * 2);
    pc = std::max(pc, 64l * L.cout * 6);
    if (pc > max_partC) max_partC = pc;
    return true;
  };

  const bool s2d = a.wf_s2d >= 0 && H % 2 == 0 && W % 2 == 0;
  pl->x0 = s2d ? act(H / 2, W / 2, 16) : act(H, W, a.convs[0].cin_p);
  if (!conv_plan(0, H, W, pl->x0)) return RN18_EINVAL;
  pl->Hs = pl->cp[0].Ho; pl->Ws = pl->cp[0].Wo;
  pl->zstem = act(pl->Hs, pl->Ws, a.convs[0].cout);
  size_t zs_bytes = (size_t)N * pl->Hs * pl->Ws * a.convs[0].cout * es;
  max_blockio = zs_bytes;
  size_t cur = pl->zstem;
  int h = pl->Hs, w = pl->Ws;
  if (a.imagenet) {
    pl->Hp = out_size(h, 3, 2, 1); pl->Wp = out_size(w, 3, 2, 1);
    pl->pool = act(pl->Hp, pl->Wp, a.convs[0].cout);
    pl->parg = alloc((size_t)N * pl->Hp * pl->Wp * a.convs[0].cout);
    cur = pl->pool; h = pl->Hp; w = pl->Wp;
  } else {
    pl->Hp = h; pl->Wp = w; pl->pool = pl->zstem; pl->parg = 0;
  }
  for (size_t bi = 0; bi < a.blocks.size(); ++bi) {
    const BlockL& B = a.blocks[bi];
    BlockP& bp = pl->bp[bi];
    bp.in = cur;
    if (!conv_plan(B.c1, h, w, cur)) return RN18_EINVAL;
    const ConvP& p1 = pl->cp[B.c1];
    bp.z1 = act(p1.Ho, p1.Wo, a.convs[B.c1].cout);
    const size_t z1b = (size_t)p1.M * a.convs[B.c1].cout * es;
    if (z1b > max_z1) max_z1 = z1b;
    if (!conv_plan(B.c2, p1.Ho, p1.Wo, bp.z1)) return RN18_EINVAL;
    if (B.ds >= 0) {
      if (!conv_plan(B.ds, h, w, cur)) return RN18_EINVAL;
      const size_t ydb = (size_t)pl->cp[B.ds].M * a.convs[B.ds].cout * es;
      if (ydb > max_yd) max_yd = ydb;
    }
    const ConvP& p2 = pl->cp[B.c2];
    bp.out = act(p2.Ho, p2.Wo, a.convs[B.c2].cout);
    bp.mbits = alloc((size_t)p2.M * a.convs[B.c2].cout * es / 16);
    const size_t ob = (size_t)p2.M * a.convs[B.c2].cout * es;
    const size_t ib = (size_t)N * h * w * a.convs[B.c1].cin * es;
    if (ob > max_blockio) max_blockio = ob;
    if (ib > max_blockio) max_blockio = ib;
    cur = bp.out; h = p2.Ho; w = p2.Wo;
  }
  pl->Hf = h; pl->Wf = w;
  const int C = a.classes;
  pl->f = alloc((size_t)N * a.feat * 4);
  pl->logits = alloc((size_t)N * C * 4);
  pl->dlogits = alloc((size_t)N * C * 4);
  pl->df = alloc((size_t)N * a.feat * 4);
  pl->rowloss = alloc((size_t)N * 4);
  pl->lossbuf = alloc(4);
  pl->gA = alloc(max_blockio);
  pl->gB = alloc(max_blockio);
  pl->gz = alloc(max_z1 ? max_z1 : 16);
  pl->gy[0] = alloc(max_yb ? max_yb : 16);
  pl->gy2[0] = alloc(max_yb ? max_yb : 16);
  pl->gy[1] = alloc(max_y);
  pl->gy2[1] = alloc(max_yb ? max_yb : 16);
  pl->gyd = alloc(max_yd ? max_yd : 16);
  pl->part = alloc((size_t)max_partC * 4);
  size_t max_bnst = 0;
  for (size_t li = 0; li < a.convs.size(); ++li) {
    // at most one entry per 32 GEMM rows of each launch
    const ConvP& P = pl->cp[li];
    const size_t b = (size_t)(ceil_div(P.M, 32) + ceil_div(N, P.nb)) * a.convs[li].cout * 4 * 4;
    if (b > max_bnst) max_bnst = b;
  }
  pl->bnst = alloc(max_bnst);
  {
    size_t mb = 16, mp = 16;
    for (const BlockL& B : a.blocks) {
      if (B.ds < 0) continue;
      const ConvP& P = pl->cp[B.ds];
      const size_t cout = a.convs[B.ds].cout;
      mb = std::max(mb, (size_t)(ceil_div(P.M, 32) + ceil_div(N, P.nb)) * cout * 16);
      mp = std::max(mp, (size_t)64 * cout * 3 * 8);
    }
    pl->bnst2 = alloc(mb);
    pl->part2 = alloc(mp);
  }
  // (kernels address the split-K scratch with 64-bit offsets: not a tensor
  // under the per-tensor limit)
  // Split-K scratch of one fixed size at every shape, so that the workspace
  // stays linear in the batch (the memory model of Sec. 5.3). It holds the
  // largest automatic split (3 ranges of 284 fp32 tiles of 128x128, 56 MB);
  // the launcher cuts a larger forced split to fit. Kernels address it with
  // 64-bit offsets: it is not a tensor under the per-tensor limit.
  pl->gsplit_bytes = kSplitScratchBytes;
  pl->gsplit = off;
  off += align256(kSplitScratchBytes);
  // the weight-gradient split-K scratch also holds the classifier's split-K
  // partials (the classifier runs before any weight gradient)
  for (size_t hw : {gemm_f32_workspace(N, C, a.feat), gemm_f32_workspace(C, a.feat, N),
                    gemm_f32_workspace(N, a.feat, C)})
    if (hw > max_wpart) max_wpart = hw;
  pl->wpart = alloc(max_wpart);
  pl->grad = alloc((size_t)a.P * 4);
  pl->total = off;
  if (max_tensor > kMaxWholeTensorBytes) {
    snprintf(buf, sizeof buf, "a %zu-byte tensor exceeds the kernels' per-tensor limit of %zu bytes", max_tensor,
             kMaxWholeTensorBytes);
    *why = buf;
    return RN18_EINVAL;
  }
  return RN18_OK;
}

// ----------------------------------------------------------------------------
// Conv launch helpers
// ----------------------------------------------------------------------------

// Data gradient of a conv with input [N][H][W][Cin] and output [N][Ho][Wo][Cout].
// mode: 0 store, 1 accumulate, 2 add masked residual (R, Rm).
// dy2, wd2 (stride 2 only): the data gradient of a 1x1 stride-2 pad-0
// projection of the same input ([N][Ho][Wo][Cout] and [Cin][Cout]) is added
// inside the GEMM of parity phase (0,0), the only phase it reaches, so the
// block-input gradient is rounded once.
// The BN whose backward pass the data gradient feeds (see ConvGather::bstats):
// its partials go to `out`, and the launch adds the entries it wrote to
// *entries, or clears *ok when the kernels it runs do not compute them.
struct BwdFeed {
  float* out;
  const void* y;
  const uint8_t* mask;
  const float* mean;
  const float* rstd;
  const float* sc;
  const float* sf;
  int* entries;
  bool* ok;
};

int launch_dgrad(int prec, const void* dy, const void* wd, void* dx, int N, int H, int W, int Cin, int Ho, int Wo,
                 int Cout, int k, int s, int p, int mode, const void* R, const void* Rm, hipStream_t st,
                 Ctx* c = nullptr, int layer = -1, int cin_real = 0, const void* dy2 = nullptr,
                 const void* wd2 = nullptr, void* sws = nullptr, size_t sws_bytes = 0,
                 const BwdFeed* feed = nullptr) {
  const double creal = cin_real > 0 ? cin_real : Cin;
  if (dy2 && (s != 2 || !wd2)) return -1;
  if (s == 1) {
    ConvGather g = gather_dgrad1(dy, wd, dx, N, H, W, Cin, Ho, Wo, Cout, k, p, mode, R, Rm);
    g.ws = sws; g.ws_bytes = sws_bytes;
    if (feed && conv_gather_bwd_ok(prec, g)) {
      g.bstats = feed->out; g.by = feed->y; g.bmask = feed->mask;
      g.bmean = feed->mean; g.brstd = feed->rstd; g.bsc = feed->sc; g.bsf = feed->sf;
      *feed->entries += conv_gather_bwd_entries(prec, g);
    } else if (feed) {
      *feed->ok = false;
    }
    const int pi = prof_begin(c, RN18_K_CONV_DGRAD, layer, conv_gather_tile(prec, g), conv_gather_kernel_name(prec, g), 2.0 * g.M * creal * g.K, 0.0);
    const int r = conv_gather_launch(prec, g, st);
    prof_end(c, pi);
    return r;
  }
  if (s != 2) return -1;
  // the four parity phases, launched together
  ConvGather ph4[4];
  int np = 0;
  double flops = 0.0;
  for (int ph = 0; ph < 2; ++ph)
    for (int pw = 0; pw < 2; ++pw) {
      const int Hm = (H - ph + 1) / 2, Wm = (W - pw + 1) / 2;
      if (Hm <= 0 || Wm <= 0) continue;
      const int kh0 = (ph + p) & 1, kw0 = (pw + p) & 1;
      const int nth = kh0 < k ? (k - kh0 + 1) / 2 : 0;
      const int ntw = kw0 < k ? (k - kw0 + 1) / 2 : 0;
      ConvGather g{};
      g.A = dy; g.B = wd; g.C = dx; g.R = R; g.Rm = Rm;
      g.N = N; g.Hin = Ho; g.Win = Wo; g.Cin = Cout;
      g.Hm = Hm; g.Wm = Wm; g.M = N * Hm * Wm;
      g.Hout = H; g.Wout = W; g.Cols = Cin;
      g.os = 2; g.oph = ph; g.opw = pw;
      g.is = 1; g.ip = 0;
      g.nth = nth; g.ntw = ntw;
      g.dh0 = (ph + p - kh0) / 2; g.dhs = -1; g.dw0 = (pw + p - kw0) / 2; g.dws = -1;
      g.wkh0 = kh0; g.wkhs = 2; g.wkw0 = kw0; g.wkws = 2; g.KW = k; g.KHW = k * k;
      g.K = nth * ntw * Cout;
      g.mode = mode;
      g.ws = sws; g.ws_bytes = sws_bytes;
      if (dy2 && ph == 0 && pw == 0) {
        // output pixel (2i, 2j) of the projection's data gradient is dy2[i][j] x wd2
        g.A2 = dy2; g.B2 = wd2; g.K2 = Cout;
      }
      if (g.K == 0 && g.K2 == 0) {
        if (mode == 1) continue;   // nothing to add
        g.nth = 1; g.ntw = 1;      // K = 0: the kernel writes acc = 0 (+ residual)
      }
      if (feed) {
        g.bstats = feed->out; g.by = feed->y; g.bmask = feed->mask;
        g.bmean = feed->mean; g.brstd = feed->rstd; g.bsc = feed->sc; g.bsf = feed->sf;
      }
      flops += 2.0 * g.M * creal * (g.K + g.K2);
      ph4[np++] = g;
    }
  if (np == 0) return 0;
  if (feed && conv_gather_bwd_ok_multi(prec, ph4, np)) {
    // the phases partition the output pixels: one entry row per row tile of each
    *feed->entries += conv_gather_bwd_entries_multi(prec, ph4, np);
  } else if (feed) {
    *feed->ok = false;
    for (int i = 0; i < np; ++i) ph4[i].bstats = nullptr;
  }
  const int pi = prof_begin(c, RN18_K_CONV_DGRAD, layer, conv_gather_tile_multi(prec, ph4, np),
                            conv_gather_kernel_name_multi(prec, ph4, np),
                            flops, 0.0);
  const int r = conv_gather_launch_multi(prec, ph4, np, st);
  prof_end(c, pi);
  return r;
}

// s2d: the operands are the space-to-depth stem's (k = 4, Cin = 16) and the
// result is mapped back to the 7x7 stem weights; flops are then those of the
// 7x7 conv.
// Weight-gradient split-K partials of one launch into wpart[splits][Cout][k*k*Cin].
int launch_wgrad_part(int prec, const void* dy, const void* x, float* wpart, int N, int H, int W, int Cin,
                      int cin_real, int Ho, int Wo, int Cout, int k, int s, int p, int splits, int pps,
                      hipStream_t st, Ctx* c = nullptr, int layer = -1, bool s2d = false) {
  ConvWgrad g{};
  g.DY = dy; g.X = x; g.P = wpart;
  g.N = N; g.H = H; g.W = W; g.Cin = Cin; g.Ho = Ho; g.Wo = Wo; g.Cout = Cout;
  g.KH = k; g.KW = k; g.stride = s; g.pad = p;
  g.Mpix = N * Ho * Wo;
  g.Kcols = k * k * Cin;
  g.pix_per_split = pps;
  g.splits = splits;
  const double mpix = (double)N * Ho * Wo;
  int pi = prof_begin(c, RN18_K_CONV_WGRAD, layer, conv_wgrad_tile(prec, Cout, g.Kcols), conv_wgrad_kernel_name_shape(prec, g),
                      2.0 * Cout * (s2d ? 49 : k * k) * cin_real * mpix,
                      (double)splits * Cout * g.Kcols * 4);
  int r = conv_wgrad_launch(prec, g, st);
  prof_end(c, pi);
  return r;
}

// Sum of `splits` partial slots into the OIHW fp32 weight gradient.
int launch_wgrad_reduce(const float* wpart, int splits, int Cout, int k, int Cin, int cin_real, float* out, bool s2d,
                        hipStream_t st, Ctx* c = nullptr, int layer = -1) {
  const double kcols = (double)k * k * Cin;
  const int pi = prof_begin(c, RN18_K_WGRAD_REDUCE, layer, 0, "wgrad_reduce_kernel", 0.0,
                            ((double)splits + 1.0) * Cout * kcols * 4);
  const int r = wgrad_reduce_launch(wpart, splits, Cout, k * k, Cin, cin_real, out, s2d ? 1 : 0, st);
  prof_end(c, pi);
  return r;
}

int launch_wgrad_full(int prec, const void* dy, const void* x, float* out, float* wpart, int N, int H, int W, int Cin,
                      int cin_real, int Ho, int Wo, int Cout, int k, int s, int p, int splits, int pps,
                      hipStream_t st, Ctx* c = nullptr, int layer = -1, bool s2d = false) {
  const int r = launch_wgrad_part(prec, dy, x, wpart, N, H, W, Cin, cin_real, Ho, Wo, Cout, k, s, p, splits, pps, st, c,
                                  layer, s2d);
  if (r) return r;
  return launch_wgrad_reduce(wpart, splits, Cout, k, Cin, cin_real, out, s2d, st, c, layer);
}

// ----------------------------------------------------------------------------
// Forward / backward
// ----------------------------------------------------------------------------
int ensure_ws(Ctx* c, const Plan& pl) {
  if (c->ws_bytes >= pl.total) return RN18_OK;
  if (!c->ws_owned && c->ws)
    return fail(RN18_ENOMEM, "workspace of %zu bytes is smaller than the %zu this shape needs", c->ws_bytes, pl.total);
  if (c->ws) {
    HIPCHK(hipStreamSynchronize(c->stream));
    HIPCHK(hipFree(c->ws));
    c->ws = nullptr;
    c->ws_bytes = 0;
  }
  if (hipMalloc(&c->ws, pl.total) != hipSuccess) {
    c->ws = nullptr;
    return fail(RN18_ENOMEM, "cannot allocate a %zu-byte workspace", pl.total);
  }
  c->ws_bytes = pl.total;
  c->ws_owned = true;
  return RN18_OK;
}

int get_plan(Ctx* c, int N, int H, int W, const Plan** out) {
  auto key = std::make_tuple(N, H, W);
  auto it = c->plans.find(key);
  if (it == c->plans.end()) {
    Plan pl;
    std::string why;
    int r = build_plan(*c, N, H, W, &pl, &why);
    if (r) return fail(r, "%s", why.c_str());
    it = c->plans.emplace(key, pl).first;
  }
  *out = &it->second;
  return RN18_OK;
}

void destroy_side(Ctx& c) {
  if (c.side) {
    (void)hipStreamSynchronize(c.side);
    (void)hipStreamDestroy(c.side);
    c.side = nullptr;
  }
  for (hipEvent_t* e : {&c.ev_fork, &c.ev_join, &c.ev_ds, &c.ev_blk[0], &c.ev_blk[1]})
    if (*e) { (void)hipEventDestroy(*e); *e = nullptr; }
}

int run_forward(Ctx* c, const Plan& pl, const float* state_c, float* state_rs, const float* images, bool train) {
  const Arch& a = c->arch;
  char* ws = (char*)c->ws;
  hipStream_t st = c->stream;
  const int prec = c->prec;
  const int N = pl.N;
  const float eps = c->cfg.bn_eps, mom = c->cfg.bn_momentum;
  auto W = [&](int li) { return (const char*)c->wf + (size_t)pl.cp[li].wf * c->es; };

  const double es = c->es;
  TIMED(RN18_K_PREP, -1, 2, kernel_instance_name("repack_tiled_kernel", prec), 0.0,
        (double)(a.wf_total - c->tab_total) * (4.0 + 2.0 * es),
        repack_tiled_launch(prec, state_c, c->wf, c->wd, c->tab + c->ntab, c->nttab, c->ntiles, st));
  if (c->tab_total > 0)
    TIMED(RN18_K_PREP, -1, 0, kernel_instance_name("repack_kernel", prec), 0.0, (double)c->tab_total * (4.0 + 2.0 * es),
          repack_launch(prec, state_c, c->wf, c->wd, c->tab, c->ntab, c->tab_total, st));
  if (pl.cp[0].s2d)
    TIMED(RN18_K_PREP, -1, 1, kernel_instance_name("ingest_s2d_kernel", prec), 0.0,
          (double)N * pl.H * pl.W * (12.0 + 4.0 * es),
          ingest_s2d_launch(prec, images, ws + pl.x0, N, pl.H, pl.W, c->err, st));
  else
    TIMED(RN18_K_PREP, -1, 1, kernel_instance_name("ingest_kernel", prec), 0.0,
          (double)N * pl.H * pl.W * (12.0 + a.convs[0].cin_p * es),
          ingest_launch(prec, images, ws + pl.x0, N, pl.H, pl.W, a.convs[0].cin_p, c->err, st));

  // conv + BN statistics of layer li on stream cs with the BN scratch at
  // bnst_off / part_off
  auto conv_bn_on = [&](int li, hipStream_t cs, size_t bnst_off, size_t part_off, bool split) -> int {
    const ConvL& L = a.convs[li];
    const ConvP& P = pl.cp[li];
    // training: the conv epilogue also writes per-tile BN partials of its
    // output; the batch chunks append their entries one after another
    float* tstats = (float*)(ws + bnst_off);
    const size_t in_img = (size_t)P.Hin * P.Win * P.cin * es, out_img = (size_t)P.Ho * P.Wo * L.cout * es;
    long ntiles = 0;
    for (int n0 = 0; n0 < N; n0 += P.nb) {
      const int nc = std::min(P.nb, N - n0);
      ConvGather g = gather_fwd(ws + P.x + n0 * in_img, W(li), ws + P.y + n0 * out_img, nc, P.Hin, P.Win, P.cin,
                                P.Ho, P.Wo, L.cout, P.k, P.s, P.p);
      if (train) g.stats = tstats + ntiles * L.cout * 4;
      if (split) { g.ws = ws + pl.gsplit; g.ws_bytes = pl.gsplit_bytes; }
      const double mc = (double)nc * P.Ho * P.Wo;
      TIMED(RN18_K_CONV_FWD, li, conv_gather_tile(prec, g), conv_gather_kernel_name(prec, g),
            2.0 * mc * L.cout * L.k * L.k * L.cin,
            (double)nc * (in_img + out_img) + (double)L.cout * P.k * P.k * P.cin * es, conv_gather_launch(prec, g, cs));
      if (train) ntiles += conv_gather_stat_entries(prec, g);
    }
    float* mean = (float*)(ws + P.mean);
    float* rstd = (float*)(ws + P.rstd);
    float* sc = (float*)(ws + P.scale);
    float* sf = (float*)(ws + P.shift);
    if (train) {
      TIMED(RN18_K_BN_STATS, li, 1, "bn_stats_tiles_reduce_kernel", 0.0, (double)ntiles * L.cout * 16,
            bn_stats_tiles_final_launch(tstats, (int)ntiles, L.cout, (double*)(ws + part_off), state_c + L.g,
                                        state_c + L.b, eps, mom,
                                        state_rs + L.rm, state_rs + L.rv, mean, rstd, sc, sf, cs));
    } else {
      LCHK(bn_eval_coef_launch(state_c + L.g, state_c + L.b, state_c + L.rm, state_c + L.rv, eps, L.cout, sc, sf, cs));
    }
    return 0;
  };
  auto conv_bn = [&](int li) -> int { return conv_bn_on(li, st, pl.bnst, pl.part, true); };
  // the projection conv of a downsampling block reads only the block input:
  // with the side stream it runs there beside the block's first two convs
  const bool ovf = c->side && !c->dbg_serial && !c->prof_on && c->captures.empty();
  // mb: offset of the mask bytes to write (block outputs of a training step), or 0
  auto apply = [&](int li, int relu, int res_mode, size_t r, int li2, size_t z, size_t mb = 0) -> int {
    const ConvL& L = a.convs[li];
    const ConvP& P = pl.cp[li];
    const float* sc2 = li2 >= 0 ? (const float*)(ws + pl.cp[li2].scale) : nullptr;
    const float* sf2 = li2 >= 0 ? (const float*)(ws + pl.cp[li2].shift) : nullptr;
    const double tb = (double)P.M * L.cout * es;
    TIMED(RN18_K_BN_APPLY, li, res_mode, kernel_instance_name("bn_apply_kernel", prec), 0.0,
          tb * (res_mode ? 3 : 2) + (mb ? tb / 16 : 0.0),
          bn_apply_launch(prec, ws + P.y, (float*)(ws + P.scale), (float*)(ws + P.shift), relu, res_mode,
                          res_mode ? ws + r : nullptr, sc2, sf2, ws + z, P.M, L.cout, st,
                          mb ? (uint8_t*)(ws + mb) : nullptr));
    return 0;
  };

  int r;
  if ((r = conv_bn(0))) return r;
  if (a.imagenet) {
    // stem BN-apply + ReLU + max pool in one pass from the conv output
    const ConvP& P0 = pl.cp[0];
    TIMED(RN18_K_MAXPOOL, 0, 0, kernel_instance_name("bn_apply_pool_kernel", prec), 0.0,
          (double)N * a.convs[0].cout * ((double)pl.Hs * pl.Ws * es + (double)pl.Hp * pl.Wp * (es + 1)),
          bn_apply_pool_launch(prec, ws + P0.y, (const float*)(ws + P0.scale), (const float*)(ws + P0.shift),
                               ws + pl.pool, (uint8_t*)(ws + pl.parg), N, pl.Hs, pl.Ws, a.convs[0].cout, pl.Hp,
                               pl.Wp, st));
  } else if ((r = apply(0, 1, 0, 0, -1, pl.zstem))) {
    return r;
  }
  for (size_t bi = 0; bi < a.blocks.size(); ++bi) {
    const BlockL& B = a.blocks[bi];
    const BlockP& bp = pl.bp[bi];
    const bool side_ds = ovf && B.ds >= 0;
    if (side_ds) {
      HIPCHK(hipEventRecord(c->ev_fork, st));
      HIPCHK(hipStreamWaitEvent(c->side, c->ev_fork, 0));
      if ((r = conv_bn_on(B.ds, c->side, pl.bnst2, pl.part2, false))) return r;
      HIPCHK(hipEventRecord(c->ev_ds, c->side));
    }
    if ((r = conv_bn(B.c1))) return r;
    if ((r = apply(B.c1, 1, 0, 0, -1, bp.z1))) return r;
    if ((r = conv_bn(B.c2))) return r;
    if (B.ds >= 0) {
      if (side_ds) {
        HIPCHK(hipStreamWaitEvent(st, c->ev_ds, 0));
      } else if ((r = conv_bn(B.ds))) {
        return r;
      }
      if ((r = apply(B.c2, 1, 2, pl.cp[B.ds].y, B.ds, bp.out, train ? bp.mbits : 0))) return r;
    } else {
      if ((r = apply(B.c2, 1, 1, bp.in, -1, bp.out, train ? bp.mbits : 0))) return r;
    }
  }
  const size_t last = pl.bp.back().out;
  TIMED(RN18_K_AVGPOOL, 0, 0, kernel_instance_name("avgpool_fwd_kernel", prec), 0.0, (double)N * a.feat * ((double)pl.Hf * pl.Wf * es + 4),
        avgpool_fwd_launch(prec, ws + last, (float*)(ws + pl.f), N, pl.Hf * pl.Wf, a.feat, st));
  return RN18_OK;
}

int run_train(Ctx* c, const Plan& pl, float* state, const float* images, const int32_t* labels, float lr,
              float* loss) {
  const Arch& a = c->arch;
  char* ws = (char*)c->ws;
  hipStream_t st = c->stream;
  const int prec = c->prec;
  const int N = pl.N, C = a.classes, F = a.feat;
  int r;
  if ((r = run_forward(c, pl, state, state, images, true))) return r;
  float* f = (float*)(ws + pl.f);
  float* logits = (float*)(ws + pl.logits);
  float* dlog = (float*)(ws + pl.dlogits);
  float* df = (float*)(ws + pl.df);
  float* grad = (float*)(ws + pl.grad);
  const double fcf = 2.0 * N * C * F;
  float* hpart = (float*)(ws + pl.wpart);
  const bool drop = c->drop_on;
  if (drop)
    TIMED(RN18_K_HEAD, 5, 0, "dropout_kernel", 0.0, 8.0 * N * F,
          dropout_launch(f, (long)N * F, c->drop_seed, c->drop_step, c->drop_thresh, c->drop_scale, st));
  TIMED(RN18_K_HEAD, 0, 0, "gemm_f32_kernel", fcf, 0.0, gemm_f32_launch(f, F, 1, state + a.fc_w, 1, F, state + a.fc_b, logits, N, C, F, hpart, st));
  TIMED(RN18_K_HEAD, 1, 0, "softmax_ce_kernel", 0.0, 8.0 * N * C,
        softmax_ce_launch(logits, labels, N, C, dlog, (float*)(ws + pl.rowloss),
                          loss ? loss : (float*)(ws + pl.lossbuf), c->err, st, c->ls));
  // classifier backward: dW = dz^T f, db = sum dz, df = dz W
  TIMED(RN18_K_HEAD, 2, 0, "gemm_f32_kernel", fcf, 0.0, gemm_f32_launch(dlog, 1, C, f, F, 1, nullptr, grad + a.fc_w, C, F, N, hpart, st));
  TIMED(RN18_K_HEAD, 3, 0, "colsum_kernel", 0.0, 4.0 * N * C, colsum_launch(dlog, N, C, grad + a.fc_b, st));
  TIMED(RN18_K_HEAD, 4, 0, "gemm_f32_kernel", fcf, 0.0, gemm_f32_launch(dlog, C, 1, state + a.fc_w, F, 1, nullptr, df, N, F, C, hpart, st));
  if (drop)  // the same mask on the classifier-input gradient
    TIMED(RN18_K_HEAD, 6, 0, "dropout_kernel", 0.0, 8.0 * N * F,
          dropout_launch(df, (long)N * F, c->drop_seed, c->drop_step, c->drop_thresh, c->drop_scale, st));
  size_t gA = pl.gA, gB = pl.gB;
  const size_t es = c->es;
  TIMED(RN18_K_AVGPOOL, 1, 0, kernel_instance_name("avgpool_bwd_kernel", prec), 0.0, (double)N * F * ((double)pl.Hf * pl.Wf * es + 4),
        avgpool_bwd_launch(prec, df, ws + gA, N, pl.Hf * pl.Wf, F, st));
  if (!c->captures.empty() && (r = run_captures(c, RN18_CAP_DA_AVG, 0, ws + gA, (size_t)N * pl.Hf * pl.Wf * F * es)))
    return r;

  auto W_d = [&](int li) { return (const char*)c->wd + (size_t)a.convs[li].wd * c->es; };
  // BN backward of conv li: dz (with a ReLU mask) -> dy written to `dy`
  // mb: the ReLU mask bytes of the block output, or RECOMPUTE when the mask
  // is that of relu(bn(y)) of this layer itself (recomputed from y)
  const size_t RECOMPUTE = ~(size_t)0;
  int fed_li = -1, fed_entries = 0;   // BN whose backward partials the last data gradient wrote, and their count
  // done (optional): an event the apply launch itself completes
  auto bn_back = [&](int li, size_t dz, size_t mb, size_t dy, hipEvent_t done = nullptr) -> int {
    const ConvL& L = a.convs[li];
    const ConvP& P = pl.cp[li];
    int nblk = 0;
    float* part = (float*)(ws + pl.part);
    const double tb = (double)P.M * L.cout * es;
    const bool rc = mb == RECOMPUTE;
    const uint8_t* mzp = rc ? nullptr : (const uint8_t*)(ws + mb);
    const float* msc = rc ? (const float*)(ws + P.scale) : nullptr;
    const float* msf = rc ? (const float*)(ws + P.shift) : nullptr;
    if (fed_li == li) {
      // the data gradient that produced dz wrote this BN's partials
      part = (float*)(ws + pl.bnst);
      nblk = fed_entries;
      fed_li = -1;
    } else {
      TIMED(RN18_K_BN_BWD_REDUCE, li, 0, kernel_instance_name("bn_bwd_partial_kernel", prec), 0.0,
            2 * tb + (rc ? 0.0 : tb / 16),
            bn_bwd_partial_launch(prec, ws + dz, mzp, ws + P.y, (float*)(ws + P.mean), (float*)(ws + P.rstd), P.M,
                                  L.cout, part, &nblk, st, msc, msf));
    }
    TIMED(RN18_K_BN_BWD_REDUCE, li, 1, "bn_bwd_final_kernel", 0.0, 0.0,
          bn_bwd_final_launch(part, nblk, P.M, L.cout, state + L.g, (float*)(ws + P.rstd), grad + L.g, grad + L.b,
                              (float*)(ws + P.coef), st));
    TIMED(RN18_K_BN_BWD_APPLY, li, 0, kernel_instance_name("bn_bwd_apply_kernel", prec), 0.0,
          3 * tb + (rc ? 0.0 : tb / 16),
          bn_bwd_apply_launch(prec, ws + dz, mzp, ws + P.y, (float*)(ws + P.mean), (float*)(ws + P.coef), ws + dy,
                              P.M, L.cout, st, msc, msf, done));
    if (!c->captures.empty()) return run_captures(c, RN18_CAP_DY, li, ws + dy, (size_t)P.M * L.cout * es);
    return 0;
  };
  // weight gradient: every batch chunk writes its split-K partials to slots
  // of its own, and one reduction sums all of them
  auto wgrad_on = [&](int li, size_t dy, hipStream_t ws_st) -> int {
    const ConvL& L = a.convs[li];
    const ConvP& P = pl.cp[li];
    const size_t in_img = (size_t)P.Hin * P.Win * P.cin * es, out_img = (size_t)P.Ho * P.Wo * L.cout * es;
    const size_t slot = (size_t)L.cout * P.k * P.k * P.cin;
    float* wpart = (float*)(ws + pl.wpart);
    int used = 0;
    for (int n0 = 0; n0 < N; n0 += P.nb) {
      const int nc = std::min(P.nb, N - n0);
      const bool full = nc == P.nb;
      LCHK(launch_wgrad_part(prec, ws + dy + n0 * out_img, ws + P.x + n0 * in_img, wpart + used * slot, nc, P.Hin,
                             P.Win, P.cin, L.cin, P.Ho, P.Wo, L.cout, P.k, P.s, P.p, full ? P.splits : P.splits_r,
                             full ? P.pps : P.pps_r, ws_st, c, li, P.s2d));
      used += full ? P.splits : P.splits_r;
    }
    if (used != P.wslots) return fail(RN18_EINVAL, "conv %d: %d weight-gradient partials, planned %d", li, used, P.wslots);
    LCHK(launch_wgrad_reduce(wpart, used, L.cout, P.k, P.cin, L.cin, grad + L.w, P.s2d, ws_st, c, li));
    return 0;
  };
  // With the side stream (not while profiling or capturing): the weight
  // gradients of a block run on it once their dY buffers are written. The
  // blocks alternate between two pairs of dY buffers by index parity, so the
  // main stream next writes a block's buffers two blocks later and waits
  // for that block's weight gradients only then (one wait per block); the
  // stem's dY goes to the pair of block 1. Each event record or wait costs
  // the queue several microseconds. With 16-bit storage the side stream has
  // slack and a block's weight gradients start together, after its second
  // BN backward (one fork per block). In fp32 the convolutions are bound by
  // the slower fp32 MFMAs and the data gradients they would overlap slow
  // down as much as the weight gradients gain, so each weight gradient
  // starts as soon as its dY is written, overlapping the memory-bound BN
  // passes (measured, CIFAR batch 128: one fork per block 5.15 -> 5.41 ms).
  // The weight gradients only read dY, the forward activations and their
  // own split-K scratch, and write their own slices of the gradient, so the
  // data-gradient chain runs on meanwhile. The stem's weight gradient runs
  // on the main stream after a join, since it shares that scratch.
  const bool ov = c->side && !c->dbg_serial && !c->prof_on && c->captures.empty();
  const bool fork_each = prec == PREC_F32;
  const int nblocks = (int)a.blocks.size();
  int done_from = nblocks;          // side work of blocks >= done_from is known complete on the main stream
  int rec_blk[2] = {nblocks, nblocks};   // block whose side work ev_blk[p] marks the end of
  bool forked = false;
  // main stream: wait until the side work of block k (and of every block
  // forked before it) is complete
  auto need_done = [&](int k) -> int {
    if (!ov || k >= done_from || k >= nblocks) return 0;
    const int p = k & 1;
    if (rec_blk[p] > k) return 0;   // block k did not fork onto the side stream
    HIPCHK(hipStreamWaitEvent(st, c->ev_blk[p], 0));
    done_from = rec_blk[p];
    return 0;
  };
  // weight gradients of block bi from their dY buffers; last: the block's
  // final ones (its end is then recorded for need_done); bound: ev_fork
  // was already bound to the launch that wrote the last dY buffer
  auto fork = [&](int bi, const int* li, const size_t* dy, int n, bool last, bool bound = false) -> int {
    if (!ov) {
      for (int k = 0; k < n; ++k)
        if (int r2 = wgrad_on(li[k], dy[k], st)) return r2;
      return 0;
    }
    if (!bound) HIPCHK(hipEventRecord(c->ev_fork, st));
    HIPCHK(hipStreamWaitEvent(c->side, c->ev_fork, 0));
    forked = true;
    for (int k = 0; k < n; ++k)
      if (int r2 = wgrad_on(li[k], dy[k], c->side)) return r2;
    if (last) {
      HIPCHK(hipEventRecord(c->ev_blk[bi & 1], c->side));
      rec_blk[bi & 1] = bi;
    }
    return 0;
  };
  auto join = [&]() -> int {
    if (!forked) return 0;
    HIPCHK(hipEventRecord(c->ev_join, c->side));
    HIPCHK(hipStreamWaitEvent(st, c->ev_join, 0));
    forked = false;
    done_from = 0;
    return 0;
  };
  // data gradient over the batch chunks; R (shaped like dx) and its mask
  // bytes Rm (1/16 of its size) are cut at the same images. With lds >= 0
  // (the block's projection conv, dY in dys) the projection's data gradient
  // is summed into the same GEMM (phase (0,0) of the stride-2 data gradient).
  // bn_li >= 0: the data gradient is the input of conv bn_li's BN backward
  // (ReLU mask from the mask bytes at bn_mb, or recomputed when bn_mb is
  // RECOMPUTE); where the kernels allow it, the launch also writes that
  // BN's partial sums (to pl.bnst, free during the backward pass) and
  // bn_back then only combines them.
  auto dgrad = [&](int li, size_t dy, size_t dx, int mode, size_t R, size_t Rm, int lds = -1,
                   size_t dys = 0, int bn_li = -1, size_t bn_mb = 0) -> int {
    const ConvL& L = a.convs[li];
    const ConvP& P = pl.cp[li];
    const size_t in_img = (size_t)P.Hin * P.Win * L.cin_p * es, out_img = (size_t)P.Ho * P.Wo * L.cout * es;
    // Only where the BN's tensor is small: the epilogue's y loads cost about
    // what a standalone reduction pass costs, so the fusion pays by the
    // launch it removes (measured at batch 256, 224x224: +25-30 us per
    // stage-2 data gradient against a 27 us reduction, +13-16 us at stage 3
    // against 20 us; at batch 64 every BN tensor is at most 12.8 MB).
    const bool feed_on = bn_li >= 0 && (size_t)pl.cp[bn_li].M * a.convs[bn_li].cout * es <= kFuseBwdMaxBytes;
    bool feed_ok = true;
    int entries = 0;
    if (lds >= 0) {
      const ConvL& D = a.convs[lds];
      const ConvP& PD = pl.cp[lds];
      if (L.s != 2 || D.k != 1 || D.s != 2 || D.p != 0 || D.cin != L.cin || D.cout != L.cout || PD.Ho != P.Ho ||
          PD.Wo != P.Wo || PD.nb != P.nb)
        return fail(RN18_EINVAL, "conv %d: projection %d cannot join its data gradient", li, lds);
    }
    for (int n0 = 0; n0 < N; n0 += P.nb) {
      const int nc = std::min(P.nb, N - n0);
      BwdFeed feed{};
      if (feed_on) {
        const ConvP& PB = pl.cp[bn_li];
        const bool rc = bn_mb == RECOMPUTE;
        feed = BwdFeed{(float*)(ws + pl.bnst) + (size_t)entries * L.cin_p * 2, ws + PB.y + n0 * in_img,
                       rc ? nullptr : (const uint8_t*)(ws + bn_mb + n0 * in_img / 16), (const float*)(ws + PB.mean),
                       (const float*)(ws + PB.rstd), rc ? (const float*)(ws + PB.scale) : nullptr,
                       rc ? (const float*)(ws + PB.shift) : nullptr, &entries, &feed_ok};
      }
      LCHK(launch_dgrad(prec, ws + dy + n0 * out_img, W_d(li), ws + dx + n0 * in_img, nc, P.Hin, P.Win, L.cin_p,
                        P.Ho, P.Wo, L.cout, L.k, L.s, L.p, mode, mode == 2 ? ws + R + n0 * in_img : nullptr,
                        mode == 2 ? ws + Rm + n0 * in_img / 16 : nullptr, st, c, li, L.cin,
                        lds >= 0 ? ws + dys + n0 * out_img : nullptr, lds >= 0 ? W_d(lds) : nullptr,
                        ws + pl.gsplit, pl.gsplit_bytes, feed_on ? &feed : nullptr));
    }
    // every batch chunk must have written its partials
    if (feed_on && feed_ok) { fed_li = bn_li; fed_entries = entries; }
    return 0;
  };

  int done = 0, prev_ds = -1;
  for (int bi = nblocks - 1; bi >= 0; --bi) {
    if (c->dbg_stop_blocks >= 0 && done++ == c->dbg_stop_blocks) return join();
    const BlockL& B = a.blocks[bi];
    const BlockP& bp = pl.bp[bi];
    const size_t gy = pl.gy[bi & 1], gy2 = pl.gy2[bi & 1];
    // this block's dY buffers were last read by the weight gradients of
    // block bi + 2, the projection's by those of the previous projection block
    if ((r = need_done(bi + 2)) || (B.ds >= 0 && prev_ds >= 0 && (r = need_done(prev_ds)))) return join(), r;
    // gA = gradient wrt the block output (before its ReLU mask)
    if ((r = bn_back(B.c2, gA, bp.mbits, gy))) return join(), r;
    if (B.ds >= 0 && (r = bn_back(B.ds, gA, bp.mbits, pl.gyd))) return join(), r;
    const int li_a[2] = {B.c2, B.ds};
    const size_t dy_a[2] = {gy, pl.gyd};
    if (fork_each && (r = fork(bi, li_a, dy_a, B.ds >= 0 ? 2 : 1, false))) return join(), r;
    if ((r = dgrad(B.c2, gy, pl.gz, 0, 0, 0, -1, 0, B.c1, RECOMPUTE))) return join(), r;
    const size_t z1b = (size_t)pl.cp[B.c1].M * a.convs[B.c1].cout * es;
    const size_t inb = (size_t)N * pl.cp[B.c1].Hin * pl.cp[B.c1].Win * a.convs[B.c1].cin_p * es;
    if (!c->captures.empty() && (r = run_captures(c, RN18_CAP_DZ1, bi, ws + pl.gz, z1b))) return r;
    // the BN apply that writes gy2 also completes the fork event
    if ((r = bn_back(B.c1, pl.gz, RECOMPUTE, gy2, ov ? c->ev_fork : nullptr))) return join(), r;
    if (fork_each) {
      if ((r = fork(bi, &B.c1, &gy2, 1, true, ov))) return join(), r;
    } else {
      const int li[3] = {B.c2, B.c1, B.ds};
      const size_t dy[3] = {gy, gy2, pl.gyd};
      if ((r = fork(bi, li, dy, B.ds >= 0 ? 3 : 2, true, ov))) return join(), r;
    }
    // gB enters the previous block's second BN (its output mask), or the
    // CIFAR stem's BN (mask recomputed); the ImageNet stem takes the pool path
    const int nbn = bi > 0 ? a.blocks[bi - 1].c2 : a.imagenet ? -1 : 0;
    const size_t nmb = bi > 0 ? pl.bp[bi - 1].mbits : RECOMPUTE;
    if (B.ds >= 0) {
      if ((r = dgrad(B.c1, gy2, gB, 0, 0, 0, B.ds, pl.gyd, nbn, nmb))) return join(), r;
      prev_ds = bi;
    } else {
      if ((r = dgrad(B.c1, gy2, gB, 2, gA, bp.mbits, -1, 0, nbn, nmb))) return join(), r;
    }
    if (!c->captures.empty() && (r = run_captures(c, RN18_CAP_DX, bi, ws + gB, inb))) return r;
    std::swap(gA, gB);
  }
  // the stem's dY goes to gy[1], last read by the weight gradients of block 1
  const size_t gys = pl.gy[1];
  if ((r = need_done(1))) return join(), r;
  if (a.imagenet) {
    // stem BN backward straight from the pooled gradient (gA) and the argmax
    const ConvL& L = a.convs[0];
    const ConvP& P = pl.cp[0];
    const int C0 = L.cout;
    const uint8_t* parg = (const uint8_t*)(ws + pl.parg);
    if (!c->captures.empty()) {
      // debugging only: materialise the pool's input gradient to capture it
      LCHK(maxpool_bwd_launch(prec, ws + gA, parg, ws + gB, N, pl.Hs, pl.Ws, C0, pl.Hp, pl.Wp, st));
      if ((r = run_captures(c, RN18_CAP_DA_POOL, 0, ws + gB, (size_t)N * pl.Hs * pl.Ws * C0 * es))) return r;
    }
    int nblk = 0;
    float* part = (float*)(ws + pl.part);
    const float* sc = (const float*)(ws + P.scale);
    const float* sf = (const float*)(ws + P.shift);
    const double yb = (double)P.M * C0 * es, pb = (double)N * pl.Hp * pl.Wp * C0 * (es + 1);
    TIMED(RN18_K_BN_BWD_REDUCE, 0, 0, kernel_instance_name("bn_bwd_partial_pool_kernel", prec), 0.0, yb + pb,
          bn_bwd_partial_pool_launch(prec, ws + gA, parg, ws + P.y, sc, sf, (float*)(ws + P.mean),
                                     (float*)(ws + P.rstd), N, pl.Hs, pl.Ws, C0, pl.Hp, pl.Wp, part, &nblk, st));
    TIMED(RN18_K_BN_BWD_REDUCE, 0, 1, "bn_bwd_final_kernel", 0.0, 0.0,
          bn_bwd_final_launch(part, nblk, P.M, C0, state + L.g, (float*)(ws + P.rstd), grad + L.g, grad + L.b,
                              (float*)(ws + P.coef), st));
    TIMED(RN18_K_BN_BWD_APPLY, 0, 0, kernel_instance_name("bn_bwd_apply_pool_kernel", prec), 0.0, 2 * yb + pb,
          bn_bwd_apply_pool_launch(prec, ws + gA, parg, ws + P.y, sc, sf, (float*)(ws + P.mean),
                                   (float*)(ws + P.coef), ws + gys, N, pl.Hs, pl.Ws, C0, pl.Hp, pl.Wp, st));
    if (!c->captures.empty() && (r = run_captures(c, RN18_CAP_DY, 0, ws + gys, (size_t)P.M * C0 * es))) return r;
  } else if ((r = bn_back(0, gA, RECOMPUTE, gys))) {
    return join(), r;
  }
  if ((r = join()) || (r = wgrad_on(0, gys, st))) return join(), r;
  if (c->ls) TIMED(RN18_K_SGD, 1, 0, "grad_check_kernel", 0.0, 4.0 * a.P, grad_check_launch(grad, a.P, c->ls, st));
  TIMED(RN18_K_SGD, 0, 0, "sgd_kernel", 0.0, 20.0 * a.P,
        sgd_launch(state, grad, c->momentum, a.P, lr, c->cfg.momentum, c->cfg.weight_decay, st, c->ls));
  if (c->ls) TIMED(RN18_K_SGD, 2, 0, "loss_scale_update_kernel", 0.0, 0.0, loss_scale_update_launch(c->ls, st));
  return RN18_OK;
}

// Host-side He-normal initial state (splitmix64 + Box-Muller).
struct HostRng {
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  double uniform() { return ((next() >> 11) + 0.5) * (1.0 / 9007199254740992.0); }
  double normal() {
    const double u1 = uniform(), u2 = uniform();
    return sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
  }
};

void host_init(const Arch& a, uint64_t seed, std::vector<float>& st) {
  st.assign(a.P + a.R, 0.f);
  HostRng rng{seed};
  for (const auto& L : a.convs) {
    const double sd = sqrt(2.0 / (L.cin * L.k * L.k));
    const long n = (long)L.cout * L.cin * L.k * L.k;
    for (long i = 0; i < n; ++i) st[L.w + i] = (float)(rng.normal() * sd);
    for (int i = 0; i < L.cout; ++i) { st[L.g + i] = 1.f; st[L.rv + i] = 1.f; }
  }
  const double sd = sqrt(2.0 / a.feat);
  for (long i = 0; i < (long)a.classes * a.feat; ++i) st[a.fc_w + i] = (float)(rng.normal() * sd);
}

int check_cfg(const rn18_config* cfg) {
  if (!cfg) return fail(RN18_EINVAL, "config is NULL");
  if (cfg->arch < 0 || cfg->arch > 2) return fail(RN18_EINVAL, "unknown arch %d", cfg->arch);
  if (cfg->prec < 0 || cfg->prec > 2) return fail(RN18_EINVAL, "unknown precision %d", cfg->prec);
  if (cfg->num_classes < 1) return fail(RN18_EINVAL, "num_classes must be >= 1");
  if (!isfinite(cfg->momentum) || !isfinite(cfg->weight_decay) || !isfinite(cfg->bn_eps) ||
      !isfinite(cfg->bn_momentum) || cfg->bn_eps < 0.f)
    return fail(RN18_EINVAL, "non-finite or negative hyper-parameter");
  return RN18_OK;
}

}  // namespace

struct rn18_ctx {
  Ctx c;
};

extern "C" {

const char* rn18_last_error(void) { return g_err.c_str(); }

size_t rn18_state_floats(const rn18_config* cfg, size_t* n_trainable) {
  Arch a;
  if (!cfg || !build_arch(*cfg, &a)) return 0;
  if (n_trainable) *n_trainable = (size_t)a.P;
  return (size_t)(a.P + a.R);
}

int rn18_init(const rn18_config* cfg, uint64_t seed, void* hip_stream, float* state_out, rn18_ctx** out) {
  if (!out) return fail(RN18_EINVAL, "ctx out-pointer is NULL");
  *out = nullptr;
  int r = check_cfg(cfg);
  if (r) return r;
  if (state_out && !aligned16(state_out)) return fail(RN18_EINVAL, "state must be 16-byte aligned");
  rn18_ctx* h = new (std::nothrow) rn18_ctx();
  if (!h) return fail(RN18_ENOMEM, "out of host memory");
  Ctx& c = h->c;
  c.cfg = *cfg;
  build_arch(*cfg, &c.arch);
  c.prec = cfg->prec;
  c.es = prec_bytes(cfg->prec);
  c.stream = (hipStream_t)hip_stream;
  const Arch& a = c.arch;
  auto bail = [&](int code, const char* what) {
    if (c.momentum) (void)hipFree(c.momentum);
    if (c.wf) (void)hipFree(c.wf);
    if (c.wd) (void)hipFree(c.wd);
    if (c.tab) (void)hipFree(c.tab);
    if (c.err) (void)hipFree(c.err);
    if (c.ls) (void)hipFree(c.ls);
    delete h;
    return fail(code, "%s", what);
  };
  if (hipMalloc(&c.momentum, a.P * 4) != hipSuccess) return bail(RN18_ENOMEM, "momentum allocation failed");
  if (hipMalloc(&c.wf, a.wf_total * c.es + 16) != hipSuccess) return bail(RN18_ENOMEM, "weight shadow allocation failed");
  if (hipMalloc(&c.wd, a.wd_total * c.es + 16) != hipSuccess) return bail(RN18_ENOMEM, "weight shadow allocation failed");
  if (hipMalloc(&c.err, 256) != hipSuccess) return bail(RN18_ENOMEM, "flag allocation failed");
  if (cfg->prec == RN18_FP16) {
    if (hipMalloc(&c.ls, 256) != hipSuccess) return bail(RN18_ENOMEM, "loss-scale allocation failed");
    const LossScale init{kLossScaleInit, 1.0f / kLossScaleInit, 0u, 0u, kLossScaleInterval, 0u};
    if (hipMemcpy(c.ls, &init, sizeof init, hipMemcpyHostToDevice) != hipSuccess)
      return bail(RN18_EHIP, "loss-scale upload failed");
  }
  if (hipStreamCreateWithFlags(&c.side, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&c.ev_fork, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c.ev_join, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c.ev_ds, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c.ev_blk[0], hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c.ev_blk[1], hipEventDisableTiming) != hipSuccess) {
    destroy_side(c);
    return bail(RN18_EHIP, "stream or event creation failed");
  }
  std::vector<RepackEntry> tab, ttab;
  long pre = 0, tpre = 0;
  for (const auto& L : a.convs) {
    RepackEntry e;
    e.src = L.w; e.dst_f = L.wf; e.dst_d = L.wd;
    e.Cout = L.cout; e.Cin = L.cin; e.Cin_p = L.cin_p; e.KHW = L.k * L.k;
    e.mode = 0; e.pad_ = 0;
    if (repack_tiled_fits(e.KHW)) {
      e.n = repack_tiles(e.Cout, e.Cin_p);
      e.nprefix = tpre;
      tpre += e.n;
      ttab.push_back(e);
      continue;
    }
    e.n = (long)L.cout * L.k * L.k * L.cin_p;
    e.nprefix = pre;
    pre += e.n;
    tab.push_back(e);
  }
  if (a.wf_s2d >= 0) {
    const ConvL& L = a.convs[0];
    RepackEntry e;
    e.src = L.w; e.dst_f = a.wf_s2d; e.dst_d = -1;
    e.Cout = L.cout; e.Cin = 3; e.Cin_p = 16; e.KHW = 16;
    e.n = (long)L.cout * 16 * 16;
    e.nprefix = pre;
    e.mode = 1; e.pad_ = 0;
    pre += e.n;
    tab.push_back(e);
  }
  c.ntab = (int)tab.size();
  c.nttab = (int)ttab.size();
  c.ntiles = (int)tpre;
  c.tab_total = pre;
  if (c.ntab > 24 || c.nttab > 24) return bail(RN18_EINVAL, "too many repack entries");
  tab.insert(tab.end(), ttab.begin(), ttab.end());
  if (hipMalloc(&c.tab, sizeof(RepackEntry) * tab.size()) != hipSuccess) return bail(RN18_ENOMEM, "table allocation failed");
  if (hipMemcpy(c.tab, tab.data(), sizeof(RepackEntry) * tab.size(), hipMemcpyHostToDevice) != hipSuccess)
    return bail(RN18_EHIP, "table upload failed");
  if (fill_zero_launch(c.momentum, a.P * 4, c.stream) || fill_zero_launch(c.err, 256, c.stream))
    return bail(RN18_EHIP, "initial fill failed");
  if (state_out) {
    std::vector<float> host;
    host_init(a, seed, host);
    if (hipMemcpyAsync(state_out, host.data(), host.size() * 4, hipMemcpyHostToDevice, c.stream) != hipSuccess ||
        hipStreamSynchronize(c.stream) != hipSuccess)
      return bail(RN18_EHIP, "state upload failed");
  }
  *out = h;
  return RN18_OK;
}

size_t rn18_workspace_bytes(rn18_ctx* h, int N, int H, int W) {
  if (!h) return 0;
  const Plan* pl = nullptr;
  if (get_plan(&h->c, N, H, W, &pl)) return 0;
  return pl->total;
}

int rn18_set_workspace(rn18_ctx* h, void* dev, size_t bytes) {
  if (!h) return fail(RN18_EINVAL, "ctx is NULL");
  if (!dev || !bytes) return fail(RN18_EINVAL, "workspace pointer or size is 0");
  if (((uintptr_t)dev & 255u) != 0) return fail(RN18_EINVAL, "workspace must be 256-byte aligned");
  Ctx& c = h->c;
  if (c.ws_owned && c.ws) {
    HIPCHK(hipStreamSynchronize(c.stream));
    HIPCHK(hipFree(c.ws));
  }
  c.ws = dev;
  c.ws_bytes = bytes;
  c.ws_owned = false;
  return RN18_OK;
}

int rn18_train_step(rn18_ctx* h, float* state, const float* images, const int32_t* labels, int N, int H, int W,
                    float lr, float* loss) {
  if (!h) return fail(RN18_EINVAL, "ctx is NULL");
  if (!state || !images || !labels) return fail(RN18_EINVAL, "state, images and labels must be non-NULL");
  if (!aligned16(state) || !aligned16(images) || (loss && ((uintptr_t)loss & 3u)))
    return fail(RN18_EINVAL, "misaligned pointer");
  if (!isfinite(lr)) return fail(RN18_EINVAL, "lr is not finite");
  Ctx& c = h->c;
  const Plan* pl = nullptr;
  int r = get_plan(&c, N, H, W, &pl);
  if (r) return r;
  if ((r = ensure_ws(&c, *pl))) return r;
  if ((r = run_train(&c, *pl, state, images, labels, lr, loss))) return r;
  ++c.drop_step;
  return RN18_OK;
}

int rn18_set_loss_scale(rn18_ctx* h, float scale, unsigned growth_interval) {
  if (!h) return fail(RN18_EINVAL, "ctx is NULL");
  Ctx& c = h->c;
  if (!c.ls) return fail(RN18_EINVAL, "loss scaling belongs to fp16 contexts");
  int e = 0;
  const float m = frexpf(scale, &e);
  if (!(scale >= 1.0f && scale <= 16777216.0f) || m != 0.5f)
    return fail(RN18_EINVAL, "the loss scale must be a power of two in [1, 2^24]");
  if (growth_interval < 1) return fail(RN18_EINVAL, "the growth interval must be >= 1");
  const LossScale x{scale, 1.0f / scale, 0u, 0u, growth_interval, 0u};
  HIPCHK(hipStreamSynchronize(c.stream));
  HIPCHK(hipMemcpy(c.ls, &x, sizeof x, hipMemcpyHostToDevice));
  return RN18_OK;
}

int rn18_get_loss_scale(rn18_ctx* h, float* scale, uint64_t* skipped_steps) {
  if (!h) return fail(RN18_EINVAL, "ctx is NULL");
  Ctx& c = h->c;
  if (!c.ls) return fail(RN18_EINVAL, "loss scaling belongs to fp16 contexts");
  LossScale x{};
  HIPCHK(hipStreamSynchronize(c.stream));
  HIPCHK(hipMemcpy(&x, c.ls, sizeof x, hipMemcpyDeviceToHost));
  if (scale) *scale = x.scale;
  if (skipped_steps) *skipped_steps = x.skipped;
  return RN18_OK;
}

int rn18_set_dropout(rn18_ctx* h, float p, uint64_t seed, uint64_t step) {
  if (!h) return fail(RN18_EINVAL, "ctx is NULL");
  if (!(p >= 0.f && p < 1.f)) return fail(RN18_EINVAL, "dropout rate must be in [0, 1)");
  Ctx& c = h->c;
  c.drop_on = p > 0.f;
  c.drop_thresh = (uint32_t)floor((double)p * 16777216.0);
  c.drop_scale = (float)(1.0 / (1.0 - (double)p));
  c.drop_seed = seed;
  c.drop_step = step;
  return RN18_OK;
}

int rn18_eval_logits(rn18_ctx* h, const float* state, const float* images, int N, int H, int W, float* logits) {
  if (!h) return fail(RN18_EINVAL, "ctx is NULL");
  if (!state || !images || !logits) return fail(RN18_EINVAL, "state, images and logits must be non-NULL");
  if (!aligned16(state) || !aligned16(images)) return fail(RN18_EINVAL, "misaligned pointer");
  Ctx& c = h->c;
  const Plan* pl = nullptr;
  int r = get_plan(&c, N, H, W, &pl);
  if (r) return r;
  if ((r = ensure_ws(&c, *pl))) return r;
  if ((r = run_forward(&c, *pl, state, nullptr, images, false))) return r;
  char* ws = (char*)c.ws;
  const Arch& a = c.arch;
  Ctx* cp_ = &c;
  {
    Ctx* c = cp_;
    TIMED(RN18_K_HEAD, 0, 0, "gemm_f32_kernel", 2.0 * N * a.classes * a.feat, 0.0,
          gemm_f32_launch((float*)(ws + pl->f), a.feat, 1, state + a.fc_w, 1, a.feat, state + a.fc_b, logits, N,
                          a.classes, a.feat, (float*)(ws + pl->wpart), c->stream));
  }
  return RN18_OK;
}

int ps_dual_merge(float* state, const float* g_small, const float* g_large, size_t n, float factor, void* hip_stream) {
  if (!state || !g_small || !g_large) return fail(RN18_EINVAL, "NULL pointer");
  if (!aligned16(state) || !aligned16(g_small) || !aligned16(g_large)) return fail(RN18_EINVAL, "misaligned pointer");
  if (!isfinite(factor)) return fail(RN18_EINVAL, "factor is not finite");
  if ((const float*)state == g_small || (const float*)state == g_large)
    return fail(RN18_EINVAL, "state must not alias an update vector");
  if (n == 0) return RN18_OK;
  LCHK(merge_launch(state, g_small, g_large, (long)n, factor, (hipStream_t)hip_stream));
  return RN18_OK;
}

int ps_worker_delta(const float* pulled, const float* local, float* delta, size_t n, void* hip_stream) {
  if (!pulled || !local || !delta) return fail(RN18_EINVAL, "NULL pointer");
  if (!aligned16(pulled) || !aligned16(local) || !aligned16(delta)) return fail(RN18_EINVAL, "misaligned pointer");
  if (n == 0) return RN18_OK;
  LCHK(delta_launch(pulled, local, delta, (long)n, (hipStream_t)hip_stream));
  return RN18_OK;
}

int rn18_sync_status(rn18_ctx* h) {
  if (!h) return fail(RN18_EINVAL, "ctx is NULL");
  Ctx& c = h->c;
  unsigned e = 0;
  HIPCHK(hipMemcpyAsync(&e, c.err, 4, hipMemcpyDeviceToHost, c.stream));
  HIPCHK(hipStreamSynchronize(c.stream));
  if (e) {
    LCHK(fill_zero_launch(c.err, 4, c.stream));
    HIPCHK(hipStreamSynchronize(c.stream));
  }
  if (e & DEVERR_LABEL) return fail(RN18_ELABEL, "a label was outside [0, num_classes)");
  if (e & DEVERR_NONFINITE) return fail(RN18_ENONFINITE, "the loss was not finite");
  return RN18_OK;
}

int rn18_get_momentum(rn18_ctx* h, float* dst) {
  if (!h || !dst) return fail(RN18_EINVAL, "NULL pointer");
  HIPCHK(hipMemcpyAsync(dst, h->c.momentum, h->c.arch.P * 4, hipMemcpyDeviceToDevice, h->c.stream));
  return RN18_OK;
}

int rn18_set_momentum(rn18_ctx* h, const float* src) {
  if (!h || !src) return fail(RN18_EINVAL, "NULL pointer");
  HIPCHK(hipMemcpyAsync(h->c.momentum, src, h->c.arch.P * 4, hipMemcpyDeviceToDevice, h->c.stream));
  return RN18_OK;
}

void rn18_destroy(rn18_ctx* h) {
  if (!h) return;
  Ctx& c = h->c;
  (void)hipStreamSynchronize(c.stream);
  if (c.momentum) (void)hipFree(c.momentum);
  if (c.wf) (void)hipFree(c.wf);
  if (c.wd) (void)hipFree(c.wd);
  if (c.tab) (void)hipFree(c.tab);
  if (c.err) (void)hipFree(c.err);
  if (c.ls) (void)hipFree(c.ls);
  if (c.ws_owned && c.ws) (void)hipFree(c.ws);
  destroy_side(c);
  for (auto& ev : c.prof) { (void)hipEventDestroy(ev.a); (void)hipEventDestroy(ev.b); }
  for (auto e : c.prof_spare) (void)hipEventDestroy(e);
  delete h;
}

int rn18_profile_enable(rn18_ctx* h, int on) {
  if (!h) return fail(RN18_EINVAL, "ctx is NULL");
  h->c.prof_on = on != 0;
  return RN18_OK;
}

int rn18_profile_read(rn18_ctx* h, rn18_prof_rec* out, int max, int* count) {
  if (!h || !count) return fail(RN18_EINVAL, "NULL pointer");
  Ctx& c = h->c;
  HIPCHK(hipStreamSynchronize(c.stream));
  int n = 0;
  for (auto& ev : c.prof) {
    float ms = -1.f;
    if (hipEventElapsedTime(&ms, ev.a, ev.b) != hipSuccess) ms = -1.f;
    if (out && n < max) {
      rn18_prof_rec& o = out[n];
      o = rn18_prof_rec{};
      o.cls = ev.cls; o.layer = ev.layer; o.tile = ev.tile;
      o.flops = ev.flops; o.bytes = ev.bytes; o.ms = ms;
      snprintf(o.kernel, sizeof o.kernel, "%s", ev.name ? ev.name : "");
    }
    ++n;
    c.prof_spare.push_back(ev.a);
    c.prof_spare.push_back(ev.b);
  }
  (void)hipGetLastError();
  c.prof.clear();
  *count = n;
  return RN18_OK;
}

int rn18_debug_set(rn18_ctx* h, int key, long value) {
  if (key == RN18_DBG_GATHER_CONFIG) {
    if (conv_gather_override((int)value)) return fail(RN18_EINVAL, "unknown gather configuration %ld", value);
    return RN18_OK;
  }
  if (key == RN18_DBG_WGRAD_CONFIG) {
    if (conv_wgrad_override((int)value)) return fail(RN18_EINVAL, "unknown wgrad configuration %ld", value);
    return RN18_OK;
  }
  if (key == RN18_DBG_GATHER_SPLIT) {
    if (conv_gather_split_override((int)value)) return fail(RN18_EINVAL, "bad split count %ld", value);
    return RN18_OK;
  }
  if (!h) return fail(RN18_EINVAL, "ctx is NULL");
  if (key == RN18_DBG_CONV_CHUNK) {
    if (value < 0 || value > (1l << 30)) return fail(RN18_EINVAL, "bad chunk size %ld", value);
    // plans size their scratch for the chunking: drop the ones built so far
    HIPCHK(hipStreamSynchronize(h->c.stream));
    h->c.plans.clear();
    h->c.dbg_chunk = (int)value;
    return RN18_OK;
  }
  if (key == RN18_DBG_SERIAL) {
    h->c.dbg_serial = value != 0;
    return RN18_OK;
  }
  if (key != RN18_DBG_STOP_BLOCKS) return fail(RN18_EINVAL, "unknown debug key %d", key);
  h->c.dbg_stop_blocks = (int)value;
  return RN18_OK;
}

int rn18_debug_capture(rn18_ctx* h, int kind, int index, void* dst, size_t bytes) {
  if (!h) return fail(RN18_EINVAL, "ctx is NULL");
  if (!dst) { h->c.captures.clear(); return RN18_OK; }
  if (kind < RN18_CAP_DY || kind > RN18_CAP_DA_POOL || kind == 2)
    return fail(RN18_EINVAL, "unknown capture kind %d", kind);
  h->c.captures.push_back(Ctx::Capture{kind, index, dst, bytes});
  return RN18_OK;
}

int rn18_debug_copy(rn18_ctx* h, int N, int H, int W, int which, int index, void* dst, size_t bytes) {
  if (!h || !dst) return fail(RN18_EINVAL, "NULL pointer");
  Ctx& c = h->c;
  const Plan* pl = nullptr;
  int r = get_plan(&c, N, H, W, &pl);
  if (r) return r;
  const Arch& a = c.arch;
  const int nconv = (int)a.convs.size(), nblk = (int)a.blocks.size();
  const void* src = nullptr;
  char* ws = (char*)c.ws;
  auto conv_ok = [&]() { return index >= 0 && index < nconv; };
  auto blk_ok = [&]() { return index >= 0 && index < nblk; };
  switch (which) {
    case RN18_DBG_Y: if (conv_ok()) src = ws + pl->cp[index].y; break;
    case RN18_DBG_Z1: if (blk_ok()) src = ws + pl->bp[index].z1; break;
    case RN18_DBG_OUT: if (blk_ok()) src = ws + pl->bp[index].out; break;
    case RN18_DBG_GA: src = ws + pl->gA; break;
    case RN18_DBG_GB: src = ws + pl->gB; break;
    case RN18_DBG_GZ: src = ws + pl->gz; break;
    case RN18_DBG_GY: src = ws + pl->gy[1]; break;
    case RN18_DBG_GYD: src = ws + pl->gyd; break;
    case RN18_DBG_GRAD: src = ws + pl->grad; break;
    case RN18_DBG_WF: if (conv_ok()) src = (char*)c.wf + (size_t)a.convs[index].wf * c.es; break;
    case RN18_DBG_WD: if (conv_ok() && index > 0) src = (char*)c.wd + (size_t)a.convs[index].wd * c.es; break;
    case RN18_DBG_MEAN: if (conv_ok()) src = ws + pl->cp[index].mean; break;
    case RN18_DBG_RSTD: if (conv_ok()) src = ws + pl->cp[index].rstd; break;
    case RN18_DBG_ZSTEM:
      src = ws + pl->zstem;
      if (a.imagenet && ws) {
        // the fused stem never stores its ReLU output; recompute it from the
        // stem conv output with the coefficients of the last forward pass
        const ConvP& P0 = pl->cp[0];
        if (bn_apply_launch(c.prec, ws + P0.y, (const float*)(ws + P0.scale), (const float*)(ws + P0.shift), 1, 0,
                            nullptr, nullptr, nullptr, ws + pl->zstem, P0.M, a.convs[0].cout, c.stream))
          return fail(RN18_EHIP, "stem activation recompute failed");
      }
      break;
    case RN18_DBG_PARG: if (a.imagenet) src = ws + pl->parg; break;
    default: break;
  }
  if (!src || !ws) return fail(RN18_EINVAL, "no such debug tensor (%d, %d)", which, index);
  size_t limit;
  if (which == RN18_DBG_WF) limit = (size_t)a.wf_total * c.es - (size_t)a.convs[index].wf * c.es;
  else if (which == RN18_DBG_WD) limit = (size_t)a.wd_total * c.es - (size_t)a.convs[index].wd * c.es;
  else limit = c.ws_bytes - (size_t)((const char*)src - ws);
  if (bytes > limit) return fail(RN18_EINVAL, "debug copy of %zu bytes exceeds the tensor's buffer", bytes);
  HIPCHK(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, c.stream));
  return RN18_OK;
}

// ---------------------------------------------------------------------------
// Single-operator entry points
// ---------------------------------------------------------------------------
static int op_check(int prec, int N, int H, int W, int Cin, int Cout, int k, int s, int p, int* Ho, int* Wo) {
  if (prec != RN18_FP32 && prec != RN18_BF16 && prec != RN18_FP16) return fail(RN18_EINVAL, "bad precision");
  const int vw = prec_vw(prec);
  if (N < 1 || H < 1 || W < 1 || Cin < 1 || Cout < 1 || k < 1 || s < 1 || p < 0)
    return fail(RN18_EINVAL, "non-positive size");
  if (Cin % vw || Cout % vw) return fail(RN18_EINVAL, "channel counts must be multiples of %d", vw);
  if (s > 2) return fail(RN18_EINVAL, "stride must be 1 or 2");
  *Ho = out_size(H, k, s, p);
  *Wo = out_size(W, k, s, p);
  if (*Ho < 1 || *Wo < 1) return fail(RN18_EINVAL, "empty output");
  const size_t es = prec_bytes(prec);
  const size_t pix = std::max((size_t)H * W, (size_t)*Ho * *Wo), ch = std::max(Cin, Cout);
  if ((size_t)N * pix * ch * es > kMaxTensorBytes || (size_t)Cout * k * k * Cin * es > kMaxTensorBytes)
    return fail(RN18_EINVAL, "tensor larger than the kernels' per-tensor limit of %zu bytes", kMaxTensorBytes);
  return RN18_OK;
}

int rn18op_conv2d_fwd(int prec, const void* x, const void* w, void* y, int N, int H, int W, int Cin, int Cout, int k,
                      int s, int p, void* stream) {
  int Ho, Wo;
  int r = op_check(prec, N, H, W, Cin, Cout, k, s, p, &Ho, &Wo);
  if (r) return r;
  if (!x || !w || !y || !aligned16(x) || !aligned16(w) || !aligned16(y)) return fail(RN18_EINVAL, "bad pointer");
  ConvGather g = gather_fwd(x, w, y, N, H, W, Cin, Ho, Wo, Cout, k, s, p);
  LCHK(conv_gather_launch(prec, g, (hipStream_t)stream));
  return RN18_OK;
}

int rn18op_conv2d_dgrad(int prec, const void* dy, const void* w, void* dx, int N, int H, int W, int Cin, int Cout,
                        int k, int s, int p, void* stream) {
  int Ho, Wo;
  int r = op_check(prec, N, H, W, Cin, Cout, k, s, p, &Ho, &Wo);
  if (r) return r;
  if (!dy || !w || !dx || !aligned16(dy) || !aligned16(w) || !aligned16(dx)) return fail(RN18_EINVAL, "bad pointer");
  LCHK(launch_dgrad(prec, dy, w, dx, N, H, W, Cin, Ho, Wo, Cout, k, s, p, 0, nullptr, nullptr, (hipStream_t)stream));
  return RN18_OK;
}

namespace {
int wgrad_op_splits(int prec, int N, int H, int W, int Cin, int Ho, int Wo, int Cout, int k, int s, int p, int* pps) {
  ConvWgrad wg{};
  wg.N = N; wg.H = H; wg.W = W; wg.Cin = Cin; wg.Ho = Ho; wg.Wo = Wo; wg.Cout = Cout;
  wg.KH = k; wg.KW = k; wg.stride = s; wg.pad = p;
  return conv_wgrad_splits_shape(prec, wg, pps);
}
}  // namespace

size_t rn18op_conv2d_wgrad_workspace(int prec, int N, int H, int W, int Cin, int Cout, int k, int s, int p) {
  int Ho, Wo;
  if (op_check(prec, N, H, W, Cin, Cout, k, s, p, &Ho, &Wo)) return 0;
  int pps;
  const int splits = wgrad_op_splits(prec, N, H, W, Cin, Ho, Wo, Cout, k, s, p, &pps);
  return (size_t)splits * Cout * k * k * Cin * 4;
}

int rn18op_conv2d_wgrad(int prec, const void* dy, const void* x, float* dw, int N, int H, int W, int Cin, int cin_real,
                        int Cout, int k, int s, int p, void* ws, size_t ws_bytes, void* stream) {
  int Ho, Wo;
  int r = op_check(prec, N, H, W, Cin, Cout, k, s, p, &Ho, &Wo);
  if (r) return r;
  if (cin_real < 1 || cin_real > Cin) return fail(RN18_EINVAL, "cin_real must be in [1, Cin]");
  if (!dy || !x || !dw || !ws || !aligned16(dy) || !aligned16(x) || !aligned16(ws)) return fail(RN18_EINVAL, "bad pointer");
  int pps;
  const int splits = wgrad_op_splits(prec, N, H, W, Cin, Ho, Wo, Cout, k, s, p, &pps);
  if (ws_bytes < (size_t)splits * Cout * k * k * Cin * 4) return fail(RN18_ENOMEM, "workspace too small");
  LCHK(launch_wgrad_full(prec, dy, x, dw, (float*)ws, N, H, W, Cin, cin_real, Ho, Wo, Cout, k, s, p, splits, pps,
                         (hipStream_t)stream));
  return RN18_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Allocation-free weight gradient: the split-K partials live in a static
// device array of the library instead of a caller workspace. Every GPU the
// library runs on holds its own copy of the array until the process ends.
// ---------------------------------------------------------------------------
namespace {
constexpr size_t kNoAllocScratchBytes = (size_t)48 << 20;
__device__ __align__(256) unsigned char g_noalloc_scratch[kNoAllocScratchBytes];
constexpr int kMaxDevices = 64;
void* g_noalloc_ptr[kMaxDevices] = {};
std::mutex g_noalloc_mu;

// Device address of this GPU's copy of the scratch array, looked up once per
// device with that device current. (The array's name in host code is a host
// stand-in, never a device address.)
int noalloc_scratch(void** out) {
  int dev = -1;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(RN18_EINVAL, "device %d beyond the %d the library tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  if (!g_noalloc_ptr[dev]) {
    void* p = nullptr;
    HIPCHK(hipGetSymbolAddress(&p, HIP_SYMBOL(g_noalloc_scratch)));
    if (!p || ((uintptr_t)p & 255u)) return fail(RN18_EHIP, "static scratch has no usable device address");
    g_noalloc_ptr[dev] = p;
  }
  *out = g_noalloc_ptr[dev];
  return RN18_OK;
}
}  // namespace

extern "C" {

size_t rn18op_conv2d_wgrad_noalloc_limit(void) { return kNoAllocScratchBytes; }

int rn18op_conv2d_wgrad_noalloc(int prec, const void* dy, const void* x, float* dw, int N, int H, int W, int Cin,
                                int cin_real, int Cout, int k, int s, int p, void* stream) {
  int Ho, Wo;
  int r = op_check(prec, N, H, W, Cin, Cout, k, s, p, &Ho, &Wo);
  if (r) return r;
  if (cin_real < 1 || cin_real > Cin) return fail(RN18_EINVAL, "cin_real must be in [1, Cin]");
  if (!dy || !x || !dw || !aligned16(dy) || !aligned16(x)) return fail(RN18_EINVAL, "bad pointer");
  int pps;
  const int splits = wgrad_op_splits(prec, N, H, W, Cin, Ho, Wo, Cout, k, s, p, &pps);
  const size_t need = (size_t)splits * Cout * k * k * Cin * 4;
  if (need > kNoAllocScratchBytes)
    return fail(RN18_EINVAL, "this shape needs %zu bytes of split-K scratch, beyond the %zu-byte static scratch", need,
                kNoAllocScratchBytes);
  void* scratch = nullptr;
  if ((r = noalloc_scratch(&scratch))) return r;
  LCHK(launch_wgrad_full(prec, dy, x, dw, (float*)scratch, N, H, W, Cin, cin_real, Ho, Wo, Cout, k, s, p, splits, pps,
                         (hipStream_t)stream));
  return RN18_OK;
}

int rn18op_maxpool_fwd(int prec, const void* x, void* y, uint8_t* arg, int N, int H, int W, int C, void* stream) {
  int Ho, Wo;
  int r = op_check(prec, N, H, W, C, C, 3, 2, 1, &Ho, &Wo);
  if (r) return r;
  if (!x || !y || !arg || !aligned16(x) || !aligned16(y)) return fail(RN18_EINVAL, "bad pointer");
  LCHK(maxpool_fwd_launch(prec, x, y, arg, N, H, W, C, Ho, Wo, (hipStream_t)stream));
  return RN18_OK;
}

int rn18op_maxpool_bwd(int prec, const void* dy, const uint8_t* arg, void* dx, int N, int H, int W, int C,
                       void* stream) {
  int Ho, Wo;
  int r = op_check(prec, N, H, W, C, C, 3, 2, 1, &Ho, &Wo);
  if (r) return r;
  if (!dy || !dx || !arg || !aligned16(dy) || !aligned16(dx)) return fail(RN18_EINVAL, "bad pointer");
  LCHK(maxpool_bwd_launch(prec, dy, arg, dx, N, H, W, C, Ho, Wo, (hipStream_t)stream));
  return RN18_OK;
}

int rn18op_round_bf16(const float* x, uint16_t* y, size_t n, void* stream) {
  if (!x || !y || !aligned16(x) || !aligned16(y)) return fail(RN18_EINVAL, "bad pointer");
  if (n % 8 || n > (size_t)1 << 40) return fail(RN18_EINVAL, "n must be a multiple of 8");
  LCHK(round_bf16_launch(x, y, (long)n, (hipStream_t)stream));
  return RN18_OK;
}

}  // extern "C"
