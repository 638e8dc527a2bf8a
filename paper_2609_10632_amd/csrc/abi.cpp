// C ABI of the conv / BN / SiLU hot path: descriptor validation, workspace sizing and
// kernel dispatch.  Every check runs before anything is enqueued; a call that returns
// an error has launched nothing.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstddef>
#include <cstdlib>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/numbat_conv.h"
#include "kernels.h"

using namespace numbat;

// ---------------------------------------------------------------------------
// Optional launch timing: each kernel launch carries a start / stop event pair that takes
// the dispatch's own begin and end timestamps.
namespace {

struct TimingRec {
  int cls;
  hipEvent_t begin, end;
};

std::mutex g_tmu;
bool g_timing = false;
std::vector<TimingRec> g_recs;
std::vector<hipEvent_t> g_pool;
size_t g_pool_used = 0;
thread_local int g_cls = -1;  // the class of the launches in progress on this thread

hipEvent_t pool_event() {
  if (g_pool_used == g_pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) {
      (void)hipGetLastError();  // timing is best-effort; the launch status stays the kernel's
      return nullptr;
    }
    g_pool.push_back(e);
  }
  return g_pool[g_pool_used++];
}

const char* const kClassNames[KC_COUNT] = {
    "conv_fwd_igemm", "stats_merge", "dgrad_weight_relayout", "conv_dgrad_igemm", "wgrad_igemm",
    "wgrad_splitk_reduce", "bn_stats", "bn_silu_fwd_apply", "bn_silu_bwd_reduce", "bn_silu_bwd_finalize",
    "bn_silu_bwd_apply", "narrow_input_pack", "opt_sumsq", "opt_update", "pool_upsample"};

}  // namespace

namespace numbat {

void trace_begin(int cls) { g_cls = cls; }

void trace_end(int) { g_cls = -1; }

bool timing_events(hipEvent_t* start, hipEvent_t* stop) {
  if (!g_timing || g_cls < 0) return false;
  std::lock_guard<std::mutex> lk(g_tmu);
  hipEvent_t e0 = pool_event(), e1 = pool_event();
  if (e0 == nullptr || e1 == nullptr) return false;  // timing is best-effort: launch untimed
  g_recs.push_back(TimingRec{g_cls, e0, e1});
  *start = e0;
  *stop = e1;
  return true;
}

}  // namespace numbat

namespace {

thread_local std::string g_err;

numbat_status fail(numbat_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

numbat_status ok() {
  g_err.clear();
  return NUMBAT_OK;
}

numbat_status hip_fail(hipError_t e, const char* what) {
  return fail(NUMBAT_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Every non-empty workspace begins with a 256-byte header of counters for the kernels'
// grid-wide synchronisation (zero before a workspace's first use; every call leaves it
// zero); the op's own data follows.
constexpr size_t kWsHeader = 256;
size_t with_header(size_t body) { return body ? body + kWsHeader : 0; }
void* ws_body(void* ws) { return ws ? static_cast<char*>(ws) + kWsHeader : nullptr; }

constexpr int64_t kMaxIndex = (1ll << 31) - 1;

// ---------------------------------------------------------------------------
struct ConvDesc {
  int32_t n, h, w, ci, co, kh, kw, sh, sw, ph, pw, ho, wo;
  int64_t x_pix, y_pix;
  int64_t m;  // n*ho*wo
};

numbat_status check_conv(const numbat_conv_problem* p, ConvDesc* d) {
  if (p == nullptr) return fail(NUMBAT_ERR_NULL, "problem descriptor is NULL");
  if (p->struct_size != sizeof(numbat_conv_problem))
    return fail(NUMBAT_ERR_VERSION, "numbat_conv_problem.struct_size is %u, this library expects %zu",
                p->struct_size, sizeof(numbat_conv_problem));
  if (p->n < 1 || p->h < 1 || p->w < 1 || p->c_in < 1 || p->c_out < 1 || p->kh < 1 || p->kw < 1)
    return fail(NUMBAT_ERR_BAD_DESC, "sizes must be >= 1 (n=%d h=%d w=%d c_in=%d c_out=%d kh=%d kw=%d)", p->n, p->h,
                p->w, p->c_in, p->c_out, p->kh, p->kw);
  if (p->stride_h < 1 || p->stride_w < 1)
    return fail(NUMBAT_ERR_BAD_DESC, "strides must be >= 1 (%d, %d)", p->stride_h, p->stride_w);
  if (p->pad_h < 0 || p->pad_w < 0)
    return fail(NUMBAT_ERR_BAD_DESC, "padding must be >= 0 (%d, %d)", p->pad_h, p->pad_w);
  if (p->pad_h >= p->kh || p->pad_w >= p->kw)
    return fail(NUMBAT_ERR_UNSUPPORTED, "padding must be smaller than the kernel (pad %d,%d kernel %d,%d)", p->pad_h,
                p->pad_w, p->kh, p->kw);
  const int64_t hp = (int64_t)p->h + 2 * p->pad_h - p->kh, wp = (int64_t)p->w + 2 * p->pad_w - p->kw;
  if (hp < 0 || wp < 0) return fail(NUMBAT_ERR_BAD_DESC, "kernel larger than the padded input");
  if (p->kh > 5 || p->kw > 5)
    return fail(NUMBAT_ERR_UNSUPPORTED, "kernel sides above 5 are not provided (%d x %d)", p->kh, p->kw);
  if (p->stride_h > 4 || p->stride_w > 4) return fail(NUMBAT_ERR_UNSUPPORTED, "strides above 4 are not provided");
  if (p->c_out % 8 != 0) return fail(NUMBAT_ERR_UNSUPPORTED, "c_out = %d is not a multiple of 8", p->c_out);
  if (p->c_in % 8 != 0 && p->c_in > 8)
    return fail(NUMBAT_ERR_UNSUPPORTED, "c_in = %d: only multiples of 8, or fewer than 8 channels", p->c_in);
  d->n = p->n;
  d->h = p->h;
  d->w = p->w;
  d->ci = p->c_in;
  d->co = p->c_out;
  d->kh = p->kh;
  d->kw = p->kw;
  d->sh = p->stride_h;
  d->sw = p->stride_w;
  d->ph = p->pad_h;
  d->pw = p->pad_w;
  d->ho = (int32_t)(hp / p->stride_h + 1);
  d->wo = (int32_t)(wp / p->stride_w + 1);
  d->x_pix = p->x_pixel_stride ? p->x_pixel_stride : p->c_in;
  d->y_pix = p->y_pixel_stride ? p->y_pixel_stride : p->c_out;
  if (d->x_pix < d->ci) return fail(NUMBAT_ERR_BAD_DESC, "x_pixel_stride %lld < c_in %d", (long long)d->x_pix, d->ci);
  if (d->y_pix < d->co) return fail(NUMBAT_ERR_BAD_DESC, "y_pixel_stride %lld < c_out %d", (long long)d->y_pix, d->co);
  if (d->ci % 8 == 0 && d->x_pix % 8 != 0)
    return fail(NUMBAT_ERR_ALIGN, "x_pixel_stride %lld is not a multiple of 8", (long long)d->x_pix);
  if (d->y_pix % 8 != 0) return fail(NUMBAT_ERR_ALIGN, "y_pixel_stride %lld is not a multiple of 8", (long long)d->y_pix);
  d->m = (int64_t)d->n * d->ho * d->wo;
  const int64_t npix_in = (int64_t)d->n * d->h * d->w;
  if (d->m > kMaxIndex || npix_in > kMaxIndex)
    return fail(NUMBAT_ERR_UNSUPPORTED, "more than 2^31-1 pixels (in %lld, out %lld)", (long long)npix_in,
                (long long)d->m);
  if ((int64_t)d->co * d->kh * d->kw * d->ci > kMaxIndex) return fail(NUMBAT_ERR_UNSUPPORTED, "weight too large");
  // per-tap element offsets inside a gather are 32-bit
  if (((int64_t)d->kh * d->w + d->kw) * d->x_pix > kMaxIndex || ((int64_t)d->kh * d->wo + d->kw) * d->y_pix > kMaxIndex)
    return fail(NUMBAT_ERR_UNSUPPORTED, "row too wide for 32-bit tap offsets");
  return NUMBAT_OK;
}

// Inputs with fewer than 8 channels (the RGB image) have kernels of their own for the
// forward (reduction packed densely) and the data gradient (one thread per input pixel);
// the weight gradient repacks the input into 8-channel pixels in the workspace (channels
// ci..7 zero) and runs the 16-byte-vector kernel.
bool narrow(const ConvDesc& d) { return d.ci % 8 != 0; }
size_t x8_bytes(const ConvDesc& d) { return round_up((size_t)d.n * d.h * d.w * 16, 256); }

// 3x3, stride-1, padding-1 problems whose reduction channels (c_in for the forward, c_out
// for the data gradient) are 16-multiples of at least 32 run the halo kernel: it stages each
// tile's input halo once per 32-channel chunk instead of gathering every tap
bool halo_geometry(const ConvDesc& d) {
  bool on = d.kh == 3 && d.kw == 3 && d.sh == 1 && d.sw == 1 && d.ph == 1 && d.pw == 1;
#ifdef NUMBAT_TUNING
  if (const char* e = getenv("NUMBAT_HALO")) on = on && atoi(e) != 0;
#endif
  return on;
}
TileCfg halo_tile(const ConvDesc& d, int cs, int nout, bool bt) {
  if (!halo_geometry(d) || cs % 16 != 0 || cs < 32 || (int64_t)nout * 9 * cs * 2 >= ((int64_t)1 << 31) - 16)
    return TileCfg{0, 0, -1, kVariantGeneric};
  return convhalo_pick(d.m, nout, d.h, d.w, bt);
}

TileCfg fwd_tile(const ConvDesc& d) {
  if (narrow(d)) return narrow_pick(d.co);
  const TileCfg h = halo_tile(d, d.ci, d.co, false);
  if (h.variant == kVariantHalo) return h;
  return convgemm_pick(d.m, d.co, d.ci, d.kh * d.kw * d.ci, 1, false);
}

// the prologue-fused forward's tile: the halo kernel on any grid (kVariantGeneric when
// the problem is not one the halo kernel takes)
TileCfg prologue_tile(const ConvDesc& d) {
  if (!halo_geometry(d) || narrow(d) || d.ci % 16 != 0 || d.ci < 32 || d.ci > kProMaxC ||
      (int64_t)d.co * 9 * d.ci * 2 >= ((int64_t)1 << 31) - 16)
    return TileCfg{0, 0, -1, kVariantGeneric};
  return convhalo_pick(d.m, d.co, d.h, d.w, false, true);
}

// the data gradient with the BN + SiLU backward prologue: the halo kernel's tile for the
// problem (kVariantGeneric when the kernel does not take it)
TileCfg bwd_prologue_tile(const ConvDesc& d) {
  if (d.co > kProMaxC || narrow(d)) return TileCfg{0, 0, -1, kVariantGeneric};
  return halo_tile(d, d.co, d.ci, true);
}

// per-tile statistics partials, sized for the forward's tile and the prologue-fused
// forward's (one workspace serves both)
size_t fwd_stats_bytes(const ConvDesc& d) {
  const TileCfg t = fwd_tile(d), tp = prologue_tile(d);
  int64_t mt = (d.m + t.bm - 1) / t.bm;
  if (tp.variant == kVariantHalo) {
    const int64_t mp = (d.m + tp.bm - 1) / tp.bm;
    mt = mp > mt ? mp : mt;
  }
  return round_up((size_t)mt * d.co * sizeof(float2), 256);
}

size_t fwd_ws(const ConvDesc& d) { return fwd_stats_bytes(d); }

// data gradient: the weights re-laid out per stride phase (as fp32 [kh][kw][co][ci] for a
// narrow input)
size_t bwd_data_ws(const ConvDesc& d) {
  return narrow(d) ? round_up((size_t)d.kh * d.kw * d.co * d.ci * sizeof(float), 256)
                   : round_up((size_t)d.kh * d.kw * d.ci * d.co * 2, 256);
}

size_t dw8_bytes(const ConvDesc& d) { return round_up((size_t)d.co * d.kh * d.kw * 8 * sizeof(float), 256); }

// the RGB image layer's shape, whose weight gradient has a kernel of its own
bool stem_wgrad(const ConvDesc& d) {
  return d.ci == 3 && d.kh == 3 && d.kw == 3 && d.sh == 2 && d.sw == 2 && d.ph == 1 && d.pw == 1 && d.co <= 64 &&
         d.co % 8 == 0 && d.ho % 4 == 0 && d.wo % 64 == 0;
}
int64_t stem_wgrad_blocks(const ConvDesc& d) {
  const int64_t np = (int64_t)d.n * (d.ho / 4) * (d.wo / 64);
  return np < 512 ? np : 512;
}

// the geometry fields of a weight-gradient launch
WgradArgs wgrad_geometry(const ConvDesc& d) {
  WgradArgs a;
  std::memset(&a, 0, sizeof a);
  a.x_pix = d.x_pix;
  a.dy_pix = d.y_pix;
  a.n = d.n;
  a.h = d.h;
  a.w = d.w;
  a.ci = d.ci;
  a.co = d.co;
  a.kh = d.kh;
  a.kw = d.kw;
  a.sh = d.sh;
  a.sw = d.sw;
  a.ph = d.ph;
  a.pw = d.pw;
  a.ho = d.ho;
  a.wo = d.wo;
  a.m = d.m;
  a.ktot = d.kh * d.kw * d.ci;
  return a;
}

// 3x3 stride-1 and 1x1 layers whose weight gradient takes the patch-staged kernel: its
// splits and patches (pixel steps) per split
bool halo_wgrad(const ConvDesc& d, int* splits, int64_t* pps) {
  int s = 0;
  int64_t p = 0;
  if (narrow(d) || !wgrad_halo_plan(wgrad_geometry(d), &s, &p)) return false;
  if (splits) *splits = s;
  if (pps) *pps = p;
  return true;
}

size_t bwd_weight_ws(const ConvDesc& d, int* splits, int64_t* rps) {
  {
    int s = 0;
    int64_t p = 0;
    if (halo_wgrad(d, &s, &p)) {  // partials [splits][c_out][kh kw c_in]
      if (splits) *splits = s;
      if (rps) *rps = p;
      return s > 1 ? round_up((size_t)s * d.co * d.kh * d.kw * d.ci * sizeof(float), 256) : 0;
    }
  }
  if (stem_wgrad(d)) {  // per-block partials [blocks][c_out][27]
    if (splits) *splits = 0;
    if (rps) *rps = 0;
    return round_up((size_t)stem_wgrad_blocks(d) * d.co * 27 * sizeof(float), 256);
  }
  const int ci = narrow(d) ? 8 : d.ci;
  const int ktot = d.kh * d.kw * ci;
  int64_t r = 0;
  const int s = wgrad_pick_splits(d.m, d.co, ktot, &r);
  if (splits) *splits = s;
  if (rps) *rps = r;
  const size_t part = s > 1 ? round_up((size_t)s * d.co * ktot * sizeof(float), 256) : 0;
  return part + (narrow(d) ? x8_bytes(d) + dw8_bytes(d) : 0);
}

// ---------------------------------------------------------------------------
struct BnDesc {
  BnArgs a;
};

numbat_status check_bn(const numbat_bn_problem* p, BnDesc* d) {
  if (p == nullptr) return fail(NUMBAT_ERR_NULL, "problem descriptor is NULL");
  if (p->struct_size != sizeof(numbat_bn_problem))
    return fail(NUMBAT_ERR_VERSION, "numbat_bn_problem.struct_size is %u, this library expects %zu", p->struct_size,
                sizeof(numbat_bn_problem));
  if (p->c < 1 || p->m < 2) return fail(NUMBAT_ERR_BAD_DESC, "need c >= 1 and m >= 2 (c=%d m=%lld)", p->c, (long long)p->m);
  if (!(p->eps >= 0.0f)) return fail(NUMBAT_ERR_BAD_DESC, "eps must be >= 0");
  if (!(p->momentum >= 0.0f && p->momentum <= 1.0f)) return fail(NUMBAT_ERR_BAD_DESC, "momentum must be in [0, 1]");
  if (p->c % 8 != 0) return fail(NUMBAT_ERR_UNSUPPORTED, "c = %d is not a multiple of 8", p->c);
  if (p->c > 2048) return fail(NUMBAT_ERR_UNSUPPORTED, "c = %d exceeds 2048", p->c);
  if (p->m * (p->c / 8) > kMaxIndex) return fail(NUMBAT_ERR_UNSUPPORTED, "m * c / 8 exceeds 2^31-1");
  BnArgs& a = d->a;
  a.c = p->c;
  a.m = p->m;
  a.eps = p->eps;
  a.momentum = p->momentum;
  a.y_pix = p->y_pixel_stride ? p->y_pixel_stride : p->c;
  a.a_pix = p->a_pixel_stride ? p->a_pixel_stride : p->c;
  a.r_pix = p->r_pixel_stride ? p->r_pixel_stride : p->c;
  a.dy_pix = p->dy_pixel_stride ? p->dy_pixel_stride : p->c;
  const int64_t s[4] = {a.y_pix, a.a_pix, a.r_pix, a.dy_pix};
  for (int i = 0; i < 4; ++i) {
    if (s[i] < a.c) return fail(NUMBAT_ERR_BAD_DESC, "a pixel stride (%lld) is smaller than c (%d)", (long long)s[i], a.c);
    if (s[i] % 8 != 0) return fail(NUMBAT_ERR_ALIGN, "pixel stride %lld is not a multiple of 8", (long long)s[i]);
  }
  return NUMBAT_OK;
}

size_t bn_fwd_ws(const BnDesc& d) {
  const int nb = bn_reduce_blocks(d.a.m, d.a.c);
  return round_up((size_t)nb * d.a.c * sizeof(float2), 256) + round_up(2 * d.a.c * sizeof(float), 256);
}

size_t bn_bwd_ws(const BnDesc& d) {
  const int nb = bn_reduce_blocks(d.a.m, d.a.c);
  return round_up((size_t)nb * d.a.c * sizeof(float2), 256) + round_up(4 * d.a.c * sizeof(float), 256);
}

numbat_status check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return NUMBAT_OK;
  if (ws == nullptr) return fail(NUMBAT_ERR_WORKSPACE, "workspace of %zu bytes required, got NULL", need);
  if (have < need) return fail(NUMBAT_ERR_WORKSPACE, "workspace of %zu bytes required, got %zu", need, have);
  if (!aligned16(ws)) return fail(NUMBAT_ERR_ALIGN, "workspace must be 16-byte aligned");
  return NUMBAT_OK;
}

// the checks of numbat_conv_fwd that do not involve the workspace
numbat_status check_conv_fwd(const numbat_conv_problem* p, const void* x, const void* w, const void* y,
                             const float* batch_stats, ConvDesc* dp) {
  ConvDesc& d = *dp;
  numbat_status st = check_conv(p, &d);
  if (st != NUMBAT_OK) return st;
  if (x == nullptr || w == nullptr || y == nullptr) return fail(NUMBAT_ERR_NULL, "x, w and y are required");
  const bool vec_in = !narrow(d);
  if ((vec_in && (!aligned16(x) || !aligned16(w))) || !aligned16(y))
    return fail(NUMBAT_ERR_ALIGN, "x, w, y must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(w)) & 1u)
    return fail(NUMBAT_ERR_ALIGN, "x and w must be 2-byte aligned");
  if (batch_stats != nullptr && (reinterpret_cast<uintptr_t>(batch_stats) & 3u))
    return fail(NUMBAT_ERR_ALIGN, "batch_stats must be 4-byte aligned");
  return NUMBAT_OK;
}

// the forward's launches, once every check has passed; ws holds at least fwd_stats_bytes(d)
// bytes when batch_stats is given
// epilogue operation of the inference entry points (none for the training forward)
struct PostOp {
  int32_t kind = kPostNone;
  float eps = 0.f;
  const float *bias = nullptr, *gamma = nullptr, *beta = nullptr, *mean = nullptr, *var = nullptr;
};
// prologue of the fused forward: the previous layer's BN + SiLU applied to the source
struct ProOp {
  const float *gamma = nullptr, *beta = nullptr, *mean = nullptr, *var = nullptr;
  float eps = 0.f;
};

numbat_status conv_fwd_launch(const ConvDesc& d, const void* x, const void* w, void* y, float* batch_stats, void* ws,
                              void* stream, const PostOp& post = PostOp(), const ProOp* pro = nullptr) {
  const bool vec_in = !narrow(d);
  const TileCfg t = pro ? prologue_tile(d) : fwd_tile(d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  char* wsp = static_cast<char*>(ws);
  float2* part = batch_stats ? reinterpret_cast<float2*>(wsp) : nullptr;
  const bf16_t* src = static_cast<const bf16_t*>(x);
  const bf16_t* wt = static_cast<const bf16_t*>(w);
  const int64_t src_pix = d.x_pix;
  const int cs = d.ci;
  ConvGemmArgs g;
  std::memset(&g, 0, sizeof g);
  g.src = src;
  g.src_pix = src_pix;
  g.hs = d.h;
  g.ws = d.w;
  g.cs = cs;
  g.nout = d.co;
  g.nimg = d.n;
  g.gstride_h = d.sh;
  g.gstride_w = d.sw;
  g.dst = static_cast<bf16_t*>(y);
  g.dst_pix = d.y_pix;
  g.hd = d.ho;
  g.wd = d.wo;
  g.dstep_h = g.dstep_w = 1;
  g.stats_part = part;
  g.post = post.kind;
  g.post_eps = post.eps;
  g.post_bias = post.bias;
  g.post_gamma = post.gamma;
  g.post_beta = post.beta;
  g.post_mean = post.mean;
  g.post_var = post.var;
  if (pro) {
    g.pro_kind = kProFwd;
    g.pro_gamma = pro->gamma;
    g.pro_beta = pro->beta;
    g.pro_mean = pro->mean;
    g.pro_var = pro->var;
    g.pro_eps = pro->eps;
  }
  g.nphase = 1;
  GemmPhase& P = g.ph[0];
  P.wt = wt;
  P.taps = d.kh * d.kw;
  P.ktot = P.taps * cs;
  P.gh = d.ho;
  P.gw = d.wo;
  P.m = (int32_t)d.m;
  P.div_gw = make_fastdiv((uint32_t)d.wo);
  P.div_ghw = make_fastdiv((uint32_t)(d.ho * d.wo));
  for (int r = 0; r < d.kh; ++r)
    for (int q = 0; q < d.kw; ++q)
      P.off[r * d.kw + q] = (int32_t)((uint32_t)(uint16_t)(int16_t)(r - d.ph) | ((uint32_t)(q - d.pw) << 16));
  if (t.variant == kVariantHalo)
    e = convhalo_launch(g, t, s, KC_CONV_FWD);
  else
    e = vec_in ? convgemm_launch(g, t, s, KC_CONV_FWD) : convnarrow_launch(g, t, s);
  if (e != hipSuccess) return hip_fail(e, "conv forward launch");
  if (batch_stats) {
    const int mt = (int)((d.m + t.bm - 1) / t.bm);
    e = stats_merge_launch(part, mt, t.bm, d.m, d.co, batch_stats, s);
    if (e != hipSuccess) return hip_fail(e, "batch statistics merge launch");
  }
  return ok();
}

// ---------------------------------------------------------------------------
// Static scratch for numbat_conv_fwd_noalloc: a file-scope device array (each GPU holds its
// own copy for the life of the process).  Its device address is looked up once per device
// with that device current; host code uses only that address, never the array's name.
constexpr size_t kScratchBytes = (size_t)8 << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

// (calls that use it on one GPU share it: overlapping calls race)
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

numbat_status scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(NUMBAT_ERR_DEVICE, "device index %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "static scratch address (hipGetSymbolAddress)");
    if (ptr == nullptr) return fail(NUMBAT_ERR_DEVICE, "static scratch address (hipGetSymbolAddress) is NULL");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return NUMBAT_OK;
}

}  // namespace

extern "C" {

uint32_t numbat_abi_version(void) { return NUMBAT_ABI_VERSION; }

int numbat_kernel_class_count(void) { return KC_COUNT; }

const char* numbat_kernel_class_name(int kernel_class) {
  return (kernel_class >= 0 && kernel_class < KC_COUNT) ? kClassNames[kernel_class] : "";
}

numbat_status numbat_timing_enable(int enable) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing = enable != 0;
  g_recs.clear();
  g_pool_used = 0;
  return ok();
}

numbat_status numbat_timing_read(int kernel_class, double* total_ms, int64_t* launches) {
  if (total_ms == nullptr || launches == nullptr) return fail(NUMBAT_ERR_NULL, "total_ms / launches is NULL");
  if (kernel_class < 0 || kernel_class >= KC_COUNT) return fail(NUMBAT_ERR_BAD_DESC, "unknown kernel class %d", kernel_class);
  std::lock_guard<std::mutex> lk(g_tmu);
  double t = 0;
  int64_t n = 0;
  for (const TimingRec& r : g_recs) {
    if (r.cls != kernel_class) continue;
    hipError_t e = hipEventSynchronize(r.end);
    if (e != hipSuccess) return hip_fail(e, "timing event");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.begin, r.end);
    if (e != hipSuccess) return hip_fail(e, "timing elapsed");
    t += ms;
    ++n;
  }
  *total_ms = t;
  *launches = n;
  return ok();
}

const char* numbat_last_error(void) { return g_err.c_str(); }

const char* numbat_status_string(numbat_status s) {
  switch (s) {
    case NUMBAT_OK: return "NUMBAT_OK";
    case NUMBAT_ERR_NULL: return "NUMBAT_ERR_NULL";
    case NUMBAT_ERR_BAD_DESC: return "NUMBAT_ERR_BAD_DESC";
    case NUMBAT_ERR_UNSUPPORTED: return "NUMBAT_ERR_UNSUPPORTED";
    case NUMBAT_ERR_ALIGN: return "NUMBAT_ERR_ALIGN";
    case NUMBAT_ERR_WORKSPACE: return "NUMBAT_ERR_WORKSPACE";
    case NUMBAT_ERR_DEVICE: return "NUMBAT_ERR_DEVICE";
    case NUMBAT_ERR_VERSION: return "NUMBAT_ERR_VERSION";
  }
  return "NUMBAT_STATUS_UNKNOWN";
}

numbat_status numbat_conv_output_shape(const numbat_conv_problem* p, int32_t* ho, int32_t* wo) {
  ConvDesc d;
  numbat_status st = check_conv(p, &d);
  if (st != NUMBAT_OK) return st;
  if (ho == nullptr || wo == nullptr) return fail(NUMBAT_ERR_NULL, "ho / wo output pointer is NULL");
  *ho = d.ho;
  *wo = d.wo;
  return ok();
}

numbat_status numbat_workspace_size(numbat_op op, const void* problem, size_t* bytes) {
  if (bytes == nullptr) return fail(NUMBAT_ERR_NULL, "bytes output pointer is NULL");
  switch (op) {
    case NUMBAT_OP_CONV_FWD:
    case NUMBAT_OP_CONV_BWD_DATA:
    case NUMBAT_OP_CONV_BWD_WEIGHT: {
      ConvDesc d;
      numbat_status st = check_conv(static_cast<const numbat_conv_problem*>(problem), &d);
      if (st != NUMBAT_OK) return st;
      *bytes = with_header(op == NUMBAT_OP_CONV_FWD        ? fwd_ws(d)
                           : op == NUMBAT_OP_CONV_BWD_DATA ? bwd_data_ws(d)
                                                           : bwd_weight_ws(d, nullptr, nullptr));
      return ok();
    }
    case NUMBAT_OP_CLIP_SGD_NESTEROV:
      *bytes = with_header(round_up((size_t)kOptBlocks * sizeof(double), 256));
      return ok();
    case NUMBAT_OP_CONV_BWD_DATA_BN_SILU: {
      ConvDesc d;
      numbat_status st = check_conv(static_cast<const numbat_conv_problem*>(problem), &d);
      if (st != NUMBAT_OK) return st;
      if (bwd_prologue_tile(d).variant != kVariantHalo)
        return fail(NUMBAT_ERR_UNSUPPORTED, "the BN + SiLU backward prologue does not take this problem");
      *bytes = 0;
      return ok();
    }
    case NUMBAT_OP_BN_SILU_FWD:
    case NUMBAT_OP_BN_SILU_BWD: {
      BnDesc d;
      numbat_status st = check_bn(static_cast<const numbat_bn_problem*>(problem), &d);
      if (st != NUMBAT_OK) return st;
      *bytes = with_header(op == NUMBAT_OP_BN_SILU_FWD ? bn_fwd_ws(d) : bn_bwd_ws(d));
      return ok();
    }
  }
  return fail(NUMBAT_ERR_BAD_DESC, "unknown op %d", (int)op);
}

numbat_status numbat_conv_fwd(const numbat_conv_problem* p, const void* x, const void* w, void* y,
                              float* batch_stats, void* ws, size_t ws_bytes, void* stream) {
  ConvDesc d;
  numbat_status st = check_conv_fwd(p, x, w, y, batch_stats, &d);
  if (st != NUMBAT_OK) return st;
  st = check_ws(ws, ws_bytes, with_header(batch_stats ? fwd_stats_bytes(d) : 0));
  if (st != NUMBAT_OK) return st;
  return conv_fwd_launch(d, x, w, y, batch_stats, batch_stats ? ws_body(ws) : nullptr, stream);
}

numbat_status numbat_conv_fwd_noalloc(const numbat_conv_problem* p, const void* x, const void* w, void* y,
                                      float* batch_stats, void* stream) {
  ConvDesc d;
  numbat_status st = check_conv_fwd(p, x, w, y, batch_stats, &d);
  if (st != NUMBAT_OK) return st;
  const size_t need = with_header(batch_stats ? fwd_stats_bytes(d) : 0);
  if (need > kScratchBytes)
    return fail(NUMBAT_ERR_WORKSPACE,
                "problem needs %zu bytes of scratch; the static scratch of numbat_conv_fwd_noalloc holds %zu "
                "(use numbat_conv_fwd with a workspace)", need, kScratchBytes);
  void* ws = nullptr;
  if (need > 0) {
    st = scratch_of_current_device(&ws);
    if (st != NUMBAT_OK) return st;
  }
  return conv_fwd_launch(d, x, w, y, batch_stats, ws_body(ws), stream);
}

numbat_status numbat_conv_fwd_bn_silu_prologue(const numbat_conv_problem* p, const void* y_prev,
                                               const float* prev_stats, const float* gamma, const float* beta,
                                               float eps, const void* w, void* y, float* batch_stats, void* ws,
                                               size_t ws_bytes, void* stream) {
  ConvDesc d;
  numbat_status st = check_conv_fwd(p, y_prev, w, y, batch_stats, &d);
  if (st != NUMBAT_OK) return st;
  if (prev_stats == nullptr || gamma == nullptr || beta == nullptr)
    return fail(NUMBAT_ERR_NULL, "prev_stats, gamma and beta are required");
  if ((reinterpret_cast<uintptr_t>(prev_stats) | reinterpret_cast<uintptr_t>(gamma) |
       reinterpret_cast<uintptr_t>(beta)) & 3u)
    return fail(NUMBAT_ERR_ALIGN, "prev_stats, gamma and beta must be 4-byte aligned");
  if (!(eps >= 0.0f)) return fail(NUMBAT_ERR_BAD_DESC, "eps must be >= 0");
  if (prologue_tile(d).variant != kVariantHalo)
    return fail(NUMBAT_ERR_UNSUPPORTED,
                "the prologue-fused forward takes 3x3 stride-1 pad-1 problems with c_in a multiple of 16 in "
                "32 .. %d on images the halo kernel takes (%dx%d, c_in %d)", kProMaxC, d.h, d.w, d.ci);
  st = check_ws(ws, ws_bytes, with_header(batch_stats ? fwd_stats_bytes(d) : 0));
  if (st != NUMBAT_OK) return st;
  ProOp pro;
  pro.gamma = gamma;
  pro.beta = beta;
  pro.mean = prev_stats;
  pro.var = prev_stats + d.ci;
  pro.eps = eps;
  return conv_fwd_launch(d, y_prev, w, y, batch_stats, batch_stats ? ws_body(ws) : nullptr, stream, PostOp(), &pro);
}

numbat_status numbat_conv_fwd_bias(const numbat_conv_problem* p, const void* x, const void* w, const float* bias,
                                   void* y, void* stream) {
  ConvDesc d;
  numbat_status st = check_conv_fwd(p, x, w, y, nullptr, &d);
  if (st != NUMBAT_OK) return st;
  if (bias == nullptr) return fail(NUMBAT_ERR_NULL, "bias is required");
  if (reinterpret_cast<uintptr_t>(bias) & 3u) return fail(NUMBAT_ERR_ALIGN, "bias must be 4-byte aligned");
  PostOp op;
  op.kind = kPostBias;
  op.bias = bias;
  return conv_fwd_launch(d, x, w, y, nullptr, nullptr, stream, op);
}

numbat_status numbat_conv_bn_silu_infer(const numbat_conv_problem* p, const void* x, const void* w,
                                        const float* gamma, const float* beta, const float* running_mean,
                                        const float* running_var, float eps, void* y, void* stream) {
  ConvDesc d;
  numbat_status st = check_conv_fwd(p, x, w, y, nullptr, &d);
  if (st != NUMBAT_OK) return st;
  if (gamma == nullptr || beta == nullptr || running_mean == nullptr || running_var == nullptr)
    return fail(NUMBAT_ERR_NULL, "gamma, beta, running_mean and running_var are required");
  if ((reinterpret_cast<uintptr_t>(gamma) | reinterpret_cast<uintptr_t>(beta) |
       reinterpret_cast<uintptr_t>(running_mean) | reinterpret_cast<uintptr_t>(running_var)) & 3u)
    return fail(NUMBAT_ERR_ALIGN, "gamma, beta, running_mean and running_var must be 4-byte aligned");
  if (!(eps >= 0.0f)) return fail(NUMBAT_ERR_BAD_DESC, "eps must be >= 0");
  PostOp op;
  op.kind = kPostBnSilu;
  op.eps = eps;
  op.gamma = gamma;
  op.beta = beta;
  op.mean = running_mean;
  op.var = running_var;
  return conv_fwd_launch(d, x, w, y, nullptr, nullptr, stream, op);
}

// a 3x3 stride-1 data gradient is the forward convolution of dy (src, pixel stride src_pix)
// with the flipped, transposed weights, which the halo kernel reads in place
static ConvGemmArgs halo_dgrad_args(const ConvDesc& d, const void* src, int64_t src_pix, const void* w, void* dx,
                                    int accumulate) {
  ConvGemmArgs g;
  std::memset(&g, 0, sizeof g);
  g.src = static_cast<const bf16_t*>(src);
  g.src_pix = src_pix;
  g.hs = d.ho;
  g.ws = d.wo;
  g.cs = d.co;
  g.nout = d.ci;
  g.nimg = d.n;
  g.gstride_h = g.gstride_w = 1;
  g.dst = static_cast<bf16_t*>(dx);
  g.dst_pix = d.x_pix;
  g.hd = d.h;
  g.wd = d.w;
  g.dstep_h = g.dstep_w = 1;
  g.accumulate = accumulate ? 1 : 0;
  g.nphase = 1;
  g.bt = 1;
  GemmPhase& P = g.ph[0];
  P.wt = static_cast<const bf16_t*>(w);
  P.taps = 9;
  P.ktot = 9 * d.co;
  P.gh = d.h;
  P.gw = d.w;
  P.m = (int32_t)((int64_t)d.n * d.h * d.w);
  P.div_gw = make_fastdiv((uint32_t)d.w);
  P.div_ghw = make_fastdiv((uint32_t)(d.h * d.w));
  return g;
}

numbat_status numbat_conv_bwd_data(const numbat_conv_problem* p, const void* dy, const void* w, void* dx,
                                   int accumulate, void* ws, size_t ws_bytes, void* stream) {
  ConvDesc d;
  numbat_status st = check_conv(p, &d);
  if (st != NUMBAT_OK) return st;
  if (dy == nullptr || w == nullptr || dx == nullptr) return fail(NUMBAT_ERR_NULL, "dy, w and dx are required");
  if (!aligned16(dy)) return fail(NUMBAT_ERR_ALIGN, "dy must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(w) | reinterpret_cast<uintptr_t>(dx)) & 1u)
    return fail(NUMBAT_ERR_ALIGN, "w and dx must be 2-byte aligned");
  if (d.ci % 8 == 0 && !aligned16(dx)) return fail(NUMBAT_ERR_ALIGN, "dx must be 16-byte aligned");
  st = check_ws(ws, ws_bytes, with_header(bwd_data_ws(d)));
  if (st != NUMBAT_OK) return st;
  ws = ws_body(ws);

  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (narrow(d)) {
    NarrowDgradArgs na;
    na.dy = static_cast<const bf16_t*>(dy);
    na.dy_pix = d.y_pix;
    na.wt = static_cast<const bf16_t*>(w);
    na.dx = static_cast<bf16_t*>(dx);
    na.dx_pix = d.x_pix;
    na.n = d.n;
    na.h = d.h;
    na.w = d.w;
    na.co = d.co;
    na.kh = d.kh;
    na.kw = d.kw;
    na.sh = d.sh;
    na.sw = d.sw;
    na.ph = d.ph;
    na.pw = d.pw;
    na.ho = d.ho;
    na.wo = d.wo;
    na.accumulate = accumulate ? 1 : 0;
    e = dgrad_narrow_launch(na, d.ci, static_cast<float*>(ws), s);
    if (e != hipSuccess) return hip_fail(e, "data-gradient launch");
    return ok();
  }

  const TileCfg ht = halo_tile(d, d.co, d.ci, true);
  if (ht.variant == kVariantHalo) {
    ConvGemmArgs g = halo_dgrad_args(d, dy, d.y_pix, w, dx, accumulate);
    e = convhalo_launch(g, ht, s, KC_CONV_DGRAD);
    if (e != hipSuccess) return hip_fail(e, "data-gradient launch");
    return ok();
  }

  // stride phases (a, b): input rows h = a + sh*i read output rows p = i + (a + ph - r) / sh
  const int cpad = d.ci;
  PhaseTaps ph[16];
  int first[16];
  int nphase = 0, total = 0;
  int offh[16][kMaxTaps], offw[16][kMaxTaps];
  for (int pa = 0; pa < d.sh; ++pa)
    for (int pb = 0; pb < d.sw; ++pb) {
      PhaseTaps& f = ph[nphase];
      f.count = 0;
      for (int r = 0; r < d.kh; ++r) {
        const int th = pa + d.ph - r;
        if (((th % d.sh) + d.sh) % d.sh != 0) continue;
        for (int s = 0; s < d.kw; ++s) {
          const int tw = pb + d.pw - s;
          if (((tw % d.sw) + d.sw) % d.sw != 0) continue;
          f.r[f.count] = r;
          f.s[f.count] = s;
          offh[nphase][f.count] = (th - ((th % d.sh) + d.sh) % d.sh) / d.sh;  // exact
          offw[nphase][f.count] = (tw - ((tw % d.sw) + d.sw) % d.sw) / d.sw;
          ++f.count;
        }
      }
      first[nphase] = total * cpad * d.co;
      total += f.count;
      ++nphase;
    }
  // all stride phases in launches of up to kMaxPhases phases (blockIdx.z = phase)
  ConvGemmArgs g;
  std::memset(&g, 0, sizeof g);
  g.src = static_cast<const bf16_t*>(dy);
  g.src_pix = d.y_pix;
  g.hs = d.ho;
  g.ws = d.wo;
  g.cs = d.co;
  g.nout = cpad;
  g.nimg = d.n;
  g.gstride_h = g.gstride_w = 1;
  g.dst = static_cast<bf16_t*>(dx);
  g.dst_pix = d.x_pix;
  g.hd = d.h;
  g.wd = d.w;
  g.dstep_h = d.sh;
  g.dstep_w = d.sw;
  g.accumulate = accumulate ? 1 : 0;
  ConvGemmArgs groups[16];
  TileCfg tiles[16];
  int ngroups = 0;
  int f = 0;
  int64_t mmax = 0;
  int ktmax = 0;
  const int64_t wpix2 = (int64_t)d.ci * 2;
  for (int pa = 0; pa < d.sh; ++pa)
    for (int pb = 0; pb < d.sw; ++pb, ++f) {
      const int gh = pa < d.h ? (d.h - pa + d.sh - 1) / d.sh : 0;
      const int gw = pb < d.w ? (d.w - pb + d.sw - 1) / d.sw : 0;
      const bool last = (pa == d.sh - 1 && pb == d.sw - 1);
      if (gh > 0 && gw > 0) {
        GemmPhase& P = g.ph[g.nphase++];
        const PhaseTaps& T = ph[f];
        P.wt = static_cast<const bf16_t*>(ws) + first[f];  // re-laid-out copy (K-major)
        P.taps = T.count;
        P.ktot = P.taps * d.co;
        P.gh = gh;
        P.gw = gw;
        P.m = d.n * gh * gw;
        P.div_gw = make_fastdiv((uint32_t)gw);
        P.div_ghw = make_fastdiv((uint32_t)(gh * gw));
        P.doff_h = pa;
        P.doff_w = pb;
        for (int t = 0; t < T.count; ++t)
          P.off[t] = (int32_t)((uint32_t)(uint16_t)(int16_t)offh[f][t] | ((uint32_t)offw[f][t] << 16));
        // the OHWI weights read in place: taps in rows of equal r (the same grid as the
        // gather offsets), byte steps between them
        P.wostep = (int32_t)((int64_t)d.kh * d.kw * wpix2);
        if (T.count > 0) {
          int tw = 1;
          while (tw < T.count && T.r[tw] == T.r[0]) ++tw;
          P.wtoff0 = (int32_t)((T.r[0] * d.kw + T.s[0]) * wpix2);
          P.wcstep = tw > 1 ? (int32_t)((T.s[1] - T.s[0]) * wpix2) : 0;
          P.wrstep = T.count > tw
                         ? (int32_t)(((T.r[tw] - T.r[tw - 1]) * d.kw + (T.s[tw] - T.s[tw - 1])) * wpix2)
                         : 0;
        }
        mmax = P.m > mmax ? P.m : mmax;
        ktmax = P.ktot > ktmax ? P.ktot : ktmax;
      }
      if (g.nphase > 0 && (g.nphase == kMaxPhases || last)) {
        groups[ngroups] = g;
        tiles[ngroups] = convgemm_pick(mmax, cpad, d.co, ktmax, g.nphase, true);
        ++ngroups;
        g.nphase = 0;
        mmax = 0;
        ktmax = 0;
      }
    }
  // the direct-to-LDS kernel reads the weights in place; any other kernel takes them
  // re-laid out per phase (K-major) in the workspace
  bool direct = (int64_t)d.co * d.kh * d.kw * wpix2 < (int64_t)1 << 31;
  for (int i = 0; i < ngroups && direct; ++i) {
    ConvGemmArgs c = groups[i];
    c.bt = 1;
    for (int q = 0; q < c.nphase; ++q) c.ph[q].wt = static_cast<const bf16_t*>(w);
    direct = convgemm_direct(c, tiles[i]);
  }
  if (direct) {
    for (int i = 0; i < ngroups; ++i) {
      groups[i].bt = 1;
      for (int q = 0; q < groups[i].nphase; ++q) groups[i].ph[q].wt = static_cast<const bf16_t*>(w);
    }
  } else {
    bf16_t* wt = static_cast<bf16_t*>(ws);
    e = dgrad_weights_launch(static_cast<const bf16_t*>(w), wt, d.co, d.kh, d.kw, d.ci, cpad, first, ph, nphase, s);
    if (e != hipSuccess) return hip_fail(e, "data-gradient weight re-layout launch");
  }
  for (int i = 0; i < ngroups; ++i) {
    e = convgemm_launch(groups[i], tiles[i], s, KC_CONV_DGRAD);
    if (e != hipSuccess) return hip_fail(e, "data-gradient launch");
  }
  return ok();
}

numbat_status numbat_conv_bwd_data_bn_silu_prologue(const numbat_conv_problem* p, const void* g,
                                                    int64_t g_pixel_stride, const void* y, const float* save_mean,
                                                    const float* save_rstd, const float* gamma, const float* beta,
                                                    const float* dgamma, const float* dbeta, const void* w, void* dx,
                                                    void* dy, int accumulate, void* stream) {
  ConvDesc d;
  numbat_status st = check_conv(p, &d);
  if (st != NUMBAT_OK) return st;
  if (g == nullptr || y == nullptr || w == nullptr || dx == nullptr || dy == nullptr)
    return fail(NUMBAT_ERR_NULL, "g, y, w, dx and dy are required");
  if (save_mean == nullptr || save_rstd == nullptr || gamma == nullptr || beta == nullptr || dgamma == nullptr ||
      dbeta == nullptr)
    return fail(NUMBAT_ERR_NULL, "save_mean, save_rstd, gamma, beta, dgamma and dbeta are required");
  const int64_t g_pix = g_pixel_stride == 0 ? d.co : g_pixel_stride;
  if (g_pix < d.co) return fail(NUMBAT_ERR_BAD_DESC, "g_pixel_stride %lld < c_out %d", (long long)g_pix, d.co);
  if (bwd_prologue_tile(d).variant != kVariantHalo)
    return fail(NUMBAT_ERR_UNSUPPORTED,
                "the BN + SiLU backward prologue takes 3x3 stride-1 pad-1 problems with c_out a multiple of 16 in "
                "32 .. %d on images the halo kernel takes (%dx%d, c_out %d)", kProMaxC, d.ho, d.wo, d.co);
  if (!aligned16(g) || !aligned16(y) || !aligned16(dy) || !aligned16(dx) || g_pix % 8 != 0 || d.y_pix % 8 != 0)
    return fail(NUMBAT_ERR_ALIGN, "g, y, dy and dx must be 16-byte aligned with pixel strides multiples of 8");
  if (reinterpret_cast<uintptr_t>(w) & 1u) return fail(NUMBAT_ERR_ALIGN, "w must be 2-byte aligned");
  if ((reinterpret_cast<uintptr_t>(save_mean) | reinterpret_cast<uintptr_t>(save_rstd) |
       reinterpret_cast<uintptr_t>(gamma) | reinterpret_cast<uintptr_t>(beta) | reinterpret_cast<uintptr_t>(dgamma) |
       reinterpret_cast<uintptr_t>(dbeta)) & 3u)
    return fail(NUMBAT_ERR_ALIGN, "save_mean, save_rstd, gamma, beta, dgamma and dbeta must be 4-byte aligned");
  ConvGemmArgs a = halo_dgrad_args(d, g, g_pix, w, dx, accumulate);
  a.pro_kind = kProBwd;
  a.pro_gamma = gamma;
  a.pro_beta = beta;
  a.pro_mean = save_mean;
  a.pro_rstd = save_rstd;
  a.pro_dgamma = dgamma;
  a.pro_dbeta = dbeta;
  a.pro_y = static_cast<const bf16_t*>(y);
  a.pro_y_pix = d.y_pix;
  a.pro_dy = static_cast<bf16_t*>(dy);
  a.pro_dy_pix = d.y_pix;
  a.pro_m = d.m;
  const hipError_t e = convhalo_launch(a, bwd_prologue_tile(d), static_cast<hipStream_t>(stream), KC_CONV_DGRAD);
  if (e != hipSuccess) return hip_fail(e, "data-gradient launch");
  return ok();
}

numbat_status numbat_conv_bwd_weight(const numbat_conv_problem* p, const void* x, const void* dy, float* dw,
                                     int accumulate, void* ws, size_t ws_bytes, void* stream) {
  ConvDesc d;
  numbat_status st = check_conv(p, &d);
  if (st != NUMBAT_OK) return st;
  if (x == nullptr || dy == nullptr || dw == nullptr) return fail(NUMBAT_ERR_NULL, "x, dy and dw are required");
  if ((!narrow(d) && !aligned16(x)) || !aligned16(dy)) return fail(NUMBAT_ERR_ALIGN, "x and dy must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(x) & 1u) || (reinterpret_cast<uintptr_t>(dw) & 3u))
    return fail(NUMBAT_ERR_ALIGN, "x must be 2-byte and dw 4-byte aligned");
  {
    // the gather of one 64-pixel step addresses its images with 32-bit offsets
    const int64_t xp = narrow(d) ? 8 : d.x_pix;
    const int64_t imgs = 64 / ((int64_t)d.ho * d.wo) + 2;
    if (imgs * d.h * d.w * xp * 2 >= (1ll << 31) - (1ll << 24))
      return fail(NUMBAT_ERR_UNSUPPORTED, "input images too large for the weight-gradient gather (%lld bytes each)",
                  (long long)(d.h * (int64_t)d.w * xp * 2));
  }
  int splits = 1;
  int64_t rps = 0;
  const size_t need = bwd_weight_ws(d, &splits, &rps);
  st = check_ws(ws, ws_bytes, with_header(need));
  if (st != NUMBAT_OK) return st;
  ws = ws_body(ws);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (stem_wgrad(d)) {
    WgradArgs a;
    std::memset(&a, 0, sizeof a);
    a.x = static_cast<const bf16_t*>(x);
    a.x_pix = d.x_pix;
    a.dy = static_cast<const bf16_t*>(dy);
    a.dy_pix = d.y_pix;
    a.n = d.n;
    a.h = d.h;
    a.w = d.w;
    a.ci = d.ci;
    a.co = d.co;
    a.kh = d.kh;
    a.kw = d.kw;
    a.sh = d.sh;
    a.sw = d.sw;
    a.ph = d.ph;
    a.pw = d.pw;
    a.ho = d.ho;
    a.wo = d.wo;
    a.m = d.m;
    a.ktot = 27;
    a.out = dw;
    a.accumulate = accumulate ? 1 : 0;
    e = wgrad_stem_launch(a, static_cast<float*>(ws), s);
    if (e != hipSuccess) return hip_fail(e, "image-layer weight-gradient launch");
    return ok();
  }
  const int ci = narrow(d) ? 8 : d.ci;
  const int ktot = d.kh * d.kw * ci;
  char* wsp = static_cast<char*>(ws);
  const size_t part_bytes = splits > 1 ? round_up((size_t)splits * d.co * ktot * sizeof(float), 256) : 0;
  const bf16_t* xs = static_cast<const bf16_t*>(x);
  int64_t x_pix = d.x_pix;
  float* target = dw;  // where the weight-gradient GEMM (or its split reduction) writes
  int acc = accumulate ? 1 : 0;
  if (narrow(d)) {
    bf16_t* x8 = reinterpret_cast<bf16_t*>(wsp + part_bytes);
    target = reinterpret_cast<float*>(wsp + part_bytes + x8_bytes(d));
    e = pack8_launch(xs, d.x_pix, d.ci, (int64_t)d.n * d.h * d.w, x8, s);
    if (e != hipSuccess) return hip_fail(e, "input repack launch");
    xs = x8;
    x_pix = 8;
    acc = 0;
  }
  WgradArgs a;
  std::memset(&a, 0, sizeof a);
  a.x = xs;
  a.x_pix = x_pix;
  a.dy = static_cast<const bf16_t*>(dy);
  a.dy_pix = d.y_pix;
  a.n = d.n;
  a.h = d.h;
  a.w = d.w;
  a.ci = ci;
  a.co = d.co;
  a.kh = d.kh;
  a.kw = d.kw;
  a.sh = d.sh;
  a.sw = d.sw;
  a.ph = d.ph;
  a.pw = d.pw;
  a.ho = d.ho;
  a.wo = d.wo;
  a.m = d.m;
  a.ktot = ktot;
  a.splits = splits;
  a.rows_per_split = rps;
  a.out = splits > 1 ? reinterpret_cast<float*>(wsp) : target;
  a.accumulate = acc;
  e = halo_wgrad(d, nullptr, nullptr) ? wgrad_halo_launch(a, s) : wgrad_launch(a, s);
  if (e != hipSuccess) return hip_fail(e, "weight-gradient launch");
  if (splits > 1) {
    e = splitk_reduce_launch(reinterpret_cast<const float*>(wsp), splits, (int64_t)d.co * ktot, target, acc, s);
    if (e != hipSuccess) return hip_fail(e, "weight-gradient reduction launch");
  }
  if (narrow(d)) {
    e = unpack_dw_launch(target, dw, (int64_t)d.co * d.kh * d.kw, d.ci, accumulate ? 1 : 0, s);
    if (e != hipSuccess) return hip_fail(e, "weight-gradient channel extraction launch");
  }
  return ok();
}

numbat_status numbat_bn_silu_fwd(const numbat_bn_problem* p, const void* y, const float* batch_stats,
                                 const float* gamma, const float* beta, const void* residual, void* out,
                                 float* save_mean, float* save_rstd, float* running_mean, float* running_var,
                                 void* ws, size_t ws_bytes, void* stream) {
  BnDesc d;
  numbat_status st = check_bn(p, &d);
  if (st != NUMBAT_OK) return st;
  if (y == nullptr || gamma == nullptr || beta == nullptr || out == nullptr || save_mean == nullptr ||
      save_rstd == nullptr)
    return fail(NUMBAT_ERR_NULL, "y, gamma, beta, out, save_mean and save_rstd are required");
  if ((running_mean == nullptr) != (running_var == nullptr))
    return fail(NUMBAT_ERR_NULL, "running_mean and running_var must both be given or both be NULL");
  if (!aligned16(y) || !aligned16(out) || (residual && !aligned16(residual)))
    return fail(NUMBAT_ERR_ALIGN, "y, out and residual must be 16-byte aligned");
  const size_t need = batch_stats ? 0 : bn_fwd_ws(d);
  st = check_ws(ws, ws_bytes, with_header(need));
  if (st != NUMBAT_OK) return st;
  ws = ws_body(ws);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const float* mv = batch_stats;
  if (mv == nullptr) {
    const int nb = bn_reduce_blocks(d.a.m, d.a.c);
    float* part = static_cast<float*>(ws);
    float* mean_var = reinterpret_cast<float*>(static_cast<char*>(ws) + round_up((size_t)nb * d.a.c * sizeof(float2), 256));
    hipError_t e = bn_stats_launch(d.a, static_cast<const bf16_t*>(y), part, nb, mean_var, s);
    if (e != hipSuccess) return hip_fail(e, "batch statistics launch");
    mv = mean_var;
  }
  hipError_t e = bn_fwd_launch(d.a, static_cast<const bf16_t*>(y), mv, mv + d.a.c, gamma, beta,
                               static_cast<const bf16_t*>(residual), static_cast<bf16_t*>(out), save_mean, save_rstd,
                               running_mean, running_var, s);
  if (e != hipSuccess) return hip_fail(e, "BN+SiLU forward launch");
  return ok();
}

numbat_status numbat_bn_silu_infer(const numbat_bn_problem* p, const void* y, const float* running_mean,
                                   const float* running_var, const float* gamma, const float* beta,
                                   const void* residual, void* out, void* stream) {
  BnDesc d;
  numbat_status st = check_bn(p, &d);
  if (st != NUMBAT_OK) return st;
  if (y == nullptr || running_mean == nullptr || running_var == nullptr || gamma == nullptr || beta == nullptr ||
      out == nullptr)
    return fail(NUMBAT_ERR_NULL, "y, running_mean, running_var, gamma, beta and out are required");
  if (!aligned16(y) || !aligned16(out) || (residual && !aligned16(residual)))
    return fail(NUMBAT_ERR_ALIGN, "y, out and residual must be 16-byte aligned");
  hipError_t e = bn_fwd_launch(d.a, static_cast<const bf16_t*>(y), running_mean, running_var, gamma, beta,
                               static_cast<const bf16_t*>(residual), static_cast<bf16_t*>(out), nullptr, nullptr,
                               nullptr, nullptr, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "BN+SiLU inference launch");
  return ok();
}

numbat_status numbat_bn_silu_bwd(const numbat_bn_problem* p, const void* g, const void* y,
                                 const float* save_mean, const float* save_rstd, const float* gamma,
                                 const float* beta, void* dy, float* dgamma, float* dbeta, void* residual_grad,
                                 void* ws, size_t ws_bytes, void* stream) {
  BnDesc d;
  numbat_status st = check_bn(p, &d);
  if (st != NUMBAT_OK) return st;
  if (g == nullptr || y == nullptr || save_mean == nullptr || save_rstd == nullptr || gamma == nullptr ||
      beta == nullptr || dgamma == nullptr || dbeta == nullptr)
    return fail(NUMBAT_ERR_NULL, "g, y, save_mean, save_rstd, gamma, beta, dgamma and dbeta are required");
  if (dy == nullptr && residual_grad != nullptr)
    return fail(NUMBAT_ERR_NULL, "residual_grad needs dy (without dy only dgamma and dbeta are formed)");
  if (!aligned16(g) || !aligned16(y) || (dy && !aligned16(dy)) || (residual_grad && !aligned16(residual_grad)))
    return fail(NUMBAT_ERR_ALIGN, "g, y, dy and residual_grad must be 16-byte aligned");
  st = check_ws(ws, ws_bytes, with_header(bn_bwd_ws(d)));
  if (st != NUMBAT_OK) return st;
  ws = ws_body(ws);
  const int nb = bn_reduce_blocks(d.a.m, d.a.c);
  float* part = static_cast<float*>(ws);
  float* coef = reinterpret_cast<float*>(static_cast<char*>(ws) + round_up((size_t)nb * d.a.c * sizeof(float2), 256));
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = bn_bwd_launch(d.a, static_cast<const bf16_t*>(g), static_cast<const bf16_t*>(y), save_mean, save_rstd,
                               gamma, beta, static_cast<bf16_t*>(dy), dgamma, dbeta, static_cast<bf16_t*>(residual_grad),
                               part, nb, coef, s);
  if (e != hipSuccess) return hip_fail(e, "BN+SiLU backward launch");
  return ok();
}

static_assert(sizeof(numbat_param_tensor) == sizeof(OptTensor) && offsetof(numbat_param_tensor, n) == offsetof(OptTensor, n) &&
                  offsetof(numbat_param_tensor, group) == offsetof(OptTensor, group),
              "numbat_param_tensor and OptTensor share one layout");

numbat_status numbat_clip_sgd_nesterov(const numbat_param_tensor* tensors, int32_t count,
                                       const numbat_sgd_group* groups, int32_t ngroups, float momentum_factor,
                                       float max_norm, float* total_norm, void* ws, size_t ws_bytes, void* stream) {
  if (tensors == nullptr || groups == nullptr) return fail(NUMBAT_ERR_NULL, "tensors and groups are required");
  if (reinterpret_cast<uintptr_t>(tensors) & 7u) return fail(NUMBAT_ERR_ALIGN, "tensors must be 8-byte aligned");
  if (total_norm != nullptr && (reinterpret_cast<uintptr_t>(total_norm) & 3u))
    return fail(NUMBAT_ERR_ALIGN, "total_norm must be 4-byte aligned");
  if (count < 1 || count > kOptMaxTensors)
    return fail(NUMBAT_ERR_BAD_DESC, "count = %d: 1 .. %d tensors", count, kOptMaxTensors);
  if (ngroups < 1 || ngroups > kOptMaxGroups)
    return fail(NUMBAT_ERR_BAD_DESC, "ngroups = %d: 1 .. %d groups", ngroups, kOptMaxGroups);
  if (!(momentum_factor >= 0.0f && momentum_factor < 1.0f))
    return fail(NUMBAT_ERR_BAD_DESC, "momentum_factor must be in [0, 1)");
  if (!(max_norm > 0.0f && max_norm < 3.0e38f)) return fail(NUMBAT_ERR_BAD_DESC, "max_norm must be positive and finite");
  OptGroups g;
  std::memset(&g, 0, sizeof g);
  g.count = ngroups;
  for (int i = 0; i < ngroups; ++i) {
    const float lr = groups[i].lr, wd = groups[i].weight_decay;
    if (!(lr >= 0.0f && lr < 3.0e38f) || !(wd >= 0.0f && wd < 3.0e38f))
      return fail(NUMBAT_ERR_BAD_DESC, "group %d: lr and weight_decay must be finite and >= 0", i);
    g.lr[i] = lr;
    g.wd[i] = wd;
  }
  numbat_status st = check_ws(ws, ws_bytes, with_header(round_up((size_t)kOptBlocks * sizeof(double), 256)));
  if (st != NUMBAT_OK) return st;
  ws = ws_body(ws);
  const hipError_t e = opt_clip_sgd_launch(reinterpret_cast<const OptTensor*>(tensors), count, g, momentum_factor, max_norm,
                                           total_norm, static_cast<double*>(ws), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "optimiser step launch");
  return ok();
}

// ---------------------------------------------------------------------------
// SPPF max pool and neck upsampling
namespace {
numbat_status check_pool(const numbat_pool_problem* p, PoolArgs* a) {
  if (p == nullptr) return fail(NUMBAT_ERR_NULL, "problem descriptor is NULL");
  if (p->struct_size != sizeof(numbat_pool_problem))
    return fail(NUMBAT_ERR_VERSION, "numbat_pool_problem.struct_size is %u, this library expects %zu", p->struct_size,
                sizeof(numbat_pool_problem));
  if (p->n < 1 || p->h < 1 || p->w < 1 || p->c < 1)
    return fail(NUMBAT_ERR_BAD_DESC, "sizes must be >= 1 (n=%d h=%d w=%d c=%d)", p->n, p->h, p->w, p->c);
  if (p->c % 8 != 0) return fail(NUMBAT_ERR_UNSUPPORTED, "c = %d is not a multiple of 8", p->c);
  a->n = p->n;
  a->h = p->h;
  a->w = p->w;
  a->c = p->c;
  a->x_pix = p->x_pixel_stride ? p->x_pixel_stride : p->c;
  a->y_pix = p->y_pixel_stride ? p->y_pixel_stride : p->c;
  if (a->x_pix < a->c || a->y_pix < a->c) return fail(NUMBAT_ERR_BAD_DESC, "a pixel stride is smaller than c");
  if (a->x_pix % 8 != 0 || a->y_pix % 8 != 0) return fail(NUMBAT_ERR_ALIGN, "pixel strides must be multiples of 8");
  if ((int64_t)p->n * p->h * p->w * 4 > kMaxIndex) return fail(NUMBAT_ERR_UNSUPPORTED, "more than 2^29 pixels");
  return NUMBAT_OK;
}
}  // namespace

numbat_status numbat_maxpool5_fwd(const numbat_pool_problem* p, const void* x, void* y, uint8_t* idx, void* stream) {
  PoolArgs a;
  numbat_status st = check_pool(p, &a);
  if (st != NUMBAT_OK) return st;
  if (x == nullptr || y == nullptr) return fail(NUMBAT_ERR_NULL, "x and y are required");
  if (!aligned16(x) || !aligned16(y)) return fail(NUMBAT_ERR_ALIGN, "x and y must be 16-byte aligned");
  if (idx != nullptr && (reinterpret_cast<uintptr_t>(idx) & 7u)) return fail(NUMBAT_ERR_ALIGN, "idx must be 8-byte aligned");
  const hipError_t e = maxpool5_fwd_launch(a, static_cast<const bf16_t*>(x), static_cast<bf16_t*>(y), idx,
                                           static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "max pool launch");
  return ok();
}

numbat_status numbat_maxpool5_bwd(const numbat_pool_problem* p, const void* dy, const uint8_t* idx, void* dx,
                                  int accumulate, void* stream) {
  PoolArgs a;
  numbat_status st = check_pool(p, &a);
  if (st != NUMBAT_OK) return st;
  if (dy == nullptr || idx == nullptr || dx == nullptr) return fail(NUMBAT_ERR_NULL, "dy, idx and dx are required");
  if (!aligned16(dy) || !aligned16(dx) || (reinterpret_cast<uintptr_t>(idx) & 7u))
    return fail(NUMBAT_ERR_ALIGN, "dy and dx must be 16-byte and idx 8-byte aligned");
  const hipError_t e = maxpool5_bwd_launch(a, static_cast<const bf16_t*>(dy), idx, static_cast<bf16_t*>(dx),
                                           accumulate ? 1 : 0, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "max pool backward launch");
  return ok();
}

numbat_status numbat_upsample2x_fwd(const numbat_pool_problem* p, const void* x, void* y, void* stream) {
  PoolArgs a;
  numbat_status st = check_pool(p, &a);
  if (st != NUMBAT_OK) return st;
  if (x == nullptr || y == nullptr) return fail(NUMBAT_ERR_NULL, "x and y are required");
  if (!aligned16(x) || !aligned16(y)) return fail(NUMBAT_ERR_ALIGN, "x and y must be 16-byte aligned");
  const hipError_t e = upsample2x_fwd_launch(a, static_cast<const bf16_t*>(x), static_cast<bf16_t*>(y),
                                             static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "upsample launch");
  return ok();
}

numbat_status numbat_upsample2x_bwd(const numbat_pool_problem* p, const void* dy, void* dx, int accumulate,
                                    void* stream) {
  PoolArgs a;
  numbat_status st = check_pool(p, &a);
  if (st != NUMBAT_OK) return st;
  if (dy == nullptr || dx == nullptr) return fail(NUMBAT_ERR_NULL, "dy and dx are required");
  if (!aligned16(dy) || !aligned16(dx)) return fail(NUMBAT_ERR_ALIGN, "dy and dx must be 16-byte aligned");
  const hipError_t e = upsample2x_bwd_launch(a, static_cast<const bf16_t*>(dy), static_cast<bf16_t*>(dx),
                                             accumulate ? 1 : 0, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "upsample backward launch");
  return ok();
}

}  // extern "C"
