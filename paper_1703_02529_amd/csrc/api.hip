// Entry points of libnsc (declared in include/nsc.h): argument validation on
// the host, workspace layout, weight packing and the ordering of the kernels
// of the cascade on one stream.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <new>
#include <vector>

#include "nsc_internal.h"

namespace nsc {

static thread_local char g_err[512];

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

size_t conv_lds_bytes(const CnnLayer& L, bool bf16, int32_t* cin_lds, int32_t* w_lds,
                      int32_t* band_w, int32_t* band_tiles, int32_t* seg_tiles,
                      int32_t max_bt = 0);

namespace {

constexpr size_t kAlign = 256;
constexpr size_t kMaxLds = 160 * 1024;
constexpr int64_t kMaxFrames = 0x7FFFFFFF;

#define NSC_REQUIRE(cond, code, ...) \
  do {                               \
    if (!(cond)) return ::nsc::fail(code, __VA_ARGS__); \
  } while (0)

int check_area(int32_t in_h, int32_t in_w, int32_t out_h, int32_t out_w) {
  NSC_REQUIRE(in_h >= 1 && in_w >= 1, NSC_E_SHAPE, "frame size %dx%d must be positive", in_h, in_w);
  NSC_REQUIRE(out_h >= 1 && out_w >= 1 && out_h <= in_h && out_w <= in_w, NSC_E_SHAPE,
              "grid %dx%d must satisfy 1 <= grid <= frame %dx%d", out_h, out_w, in_h, in_w);
  const Axis ay = Axis::make(in_h, out_h), ax = Axis::make(in_w, out_w);
  const int64_t den = (int64_t)ay.p * ax.p;
  NSC_REQUIRE(255 * den < ((int64_t)1 << 31), NSC_E_SHAPE,
              "area denominator %lld overflows 32-bit sums", (long long)den);
  return NSC_OK;
}

int check_cfg(const nsc_cascade_cfg* c) {
  NSC_REQUIRE(c != nullptr, NSC_E_INVAL, "cfg is NULL");
  if (int rc = check_area(c->in_h, c->in_w, c->dd_h, c->dd_w)) return rc;
  NSC_REQUIRE(c->frame_stride >= (int64_t)c->in_h * c->in_w * 3, NSC_E_INVAL,
              "frame_stride %lld is below one frame (%lld bytes)", (long long)c->frame_stride,
              (long long)c->in_h * c->in_w * 3);
  NSC_REQUIRE(c->cnn_h >= 1 && c->cnn_w >= 1 && c->dd_h % c->cnn_h == 0 && c->dd_w % c->cnn_w == 0,
              NSC_E_SHAPE, "CNN grid %dx%d must divide the detector grid %dx%d", c->cnn_h, c->cnn_w,
              c->dd_h, c->dd_w);
  const int64_t den = nsc_area_den(c->in_h, c->in_w, c->dd_h, c->dd_w);
  const int64_t f = (int64_t)(c->dd_h / c->cnn_h) * (c->dd_w / c->cnn_w);
  NSC_REQUIRE(255 * den * f < ((int64_t)1 << 31), NSC_E_SHAPE,
              "CNN input sums overflow 32 bits (den %lld x %lld cells)", (long long)den, (long long)f);
  NSC_REQUIRE(c->ref_mode == NSC_REF_PREV || c->ref_mode == NSC_REF_FIXED, NSC_E_INVAL,
              "ref_mode %d is neither NSC_REF_PREV nor NSC_REF_FIXED", c->ref_mode);
  if (c->ref_mode == NSC_REF_PREV)
    NSC_REQUIRE(c->delta >= 1 && c->delta <= NSC_MAX_DELTA, NSC_E_INVAL,
                "delta %d outside 1..%d", c->delta, NSC_MAX_DELTA);
  else
    NSC_REQUIRE(c->ref_sums != nullptr, NSC_E_INVAL, "fixed-reference mode needs ref_sums");
  NSC_REQUIRE(c->grid_h >= 1 && c->grid_w >= 1 && c->grid_h <= c->dd_h && c->grid_w <= c->dd_w,
              NSC_E_SHAPE, "block grid %dx%d must lie within the detector grid %dx%d", c->grid_h,
              c->grid_w, c->dd_h, c->dd_w);
  NSC_REQUIRE((int64_t)c->grid_h * c->grid_w <= NSC_MAX_BLOCKS, NSC_E_SHAPE,
              "block grid of %d blocks exceeds %d", c->grid_h * c->grid_w, NSC_MAX_BLOCKS);
  if (c->grid_h * c->grid_w > 1) {
    NSC_REQUIRE(c->lr_w != nullptr, NSC_E_INVAL, "blocked detector needs lr_w");
    NSC_REQUIRE(isfinite(c->lr_b), NSC_E_INVAL, "lr_b must be finite");
  }
  NSC_REQUIRE(!isnan(c->delta_diff), NSC_E_INVAL, "delta_diff is NaN");
  NSC_REQUIRE(!isnan(c->c_low) && !isnan(c->c_high) && c->c_low >= 0.0 && c->c_high <= 1.0 &&
                  c->c_low <= c->c_high,
              NSC_E_INVAL, "need 0 <= c_low (%g) <= c_high (%g) <= 1", c->c_low, c->c_high);
  NSC_REQUIRE(c->check_stride >= 0 && c->check_stride <= NSC_MAX_STRIDE, NSC_E_INVAL,
              "check_stride %d outside 0..%d", c->check_stride, NSC_MAX_STRIDE);
  if (c->ref_mode == NSC_REF_PREV && c->check_stride > 1)
    NSC_REQUIRE(c->delta % c->check_stride == 0, NSC_E_INVAL,
                "delta %d must be a multiple of check_stride %d (the compared frame is a checked "
                "one)", c->delta, c->check_stride);
  NSC_REQUIRE(c->frame_stride <= ((int64_t)1 << 62) / (c->check_stride > 1 ? c->check_stride : 1),
              NSC_E_INVAL, "frame_stride x check_stride overflows");
  NSC_REQUIRE(c->metric >= NSC_METRIC_MSE && c->metric <= NSC_METRIC_PSNR, NSC_E_INVAL,
              "metric %d is not one of NSC_METRIC_MSE / SAD / NRMSE / PSNR", c->metric);
  NSC_REQUIRE(!(c->metric == NSC_METRIC_PSNR && c->grid_h * c->grid_w > 1), NSC_E_INVAL,
              "the blocked detector takes MSE, SAD or NRMSE (an unchanged block's -PSNR is "
              "-inf)");
  NSC_REQUIRE(c->fuse_prev == 0 || c->fuse_prev == 1, NSC_E_INVAL, "fuse_prev %d is not 0 or 1",
              c->fuse_prev);
  // exact int64 squared-difference sums (and sums of squared reference values)
  const double emax = (255.0 * (double)den) * (255.0 * (double)den) * (double)c->dd_h * c->dd_w * 3;
  NSC_REQUIRE(emax < 9.0e18, NSC_E_SHAPE, "squared-difference sums may overflow 64 bits");
  return NSC_OK;
}

// Layer shapes of a CNN description; fills `cnn` (no device memory).
int plan_cnn(const nsc_cnn_desc* d, Cnn* cnn) {
  NSC_REQUIRE(d != nullptr, NSC_E_INVAL, "CNN description is NULL");
  NSC_REQUIRE(d->dtype == NSC_F32 || d->dtype == NSC_BF16 || d->dtype == NSC_BF16_PAIRS,
              NSC_E_DTYPE, "dtype %d is unknown",
              d->dtype);
  NSC_REQUIRE(d->n_conv >= 1 && d->n_conv <= NSC_MAX_CONV, NSC_E_SHAPE,
              "n_conv %d outside 1..%d", d->n_conv, NSC_MAX_CONV);
  NSC_REQUIRE(d->in_h >= 2 && d->in_w >= 2, NSC_E_SHAPE, "CNN input %dx%d too small", d->in_h,
              d->in_w);
  NSC_REQUIRE(d->dense >= 16 && d->dense <= 256 && d->dense % 16 == 0 && (d->dense / 16) != 3 &&
                  ((d->dense / 16) & (d->dense / 16 - 1)) == 0,
              NSC_E_SHAPE, "dense width %d must be 16, 32, 64, 128 or 256", d->dense);
  const bool bf16 = d->dtype == NSC_BF16 || d->dtype == NSC_BF16_PAIRS;
  Cnn c{};
  c.desc = *d;
  c.bf16 = bf16;
  c.h16 = d->dtype == NSC_BF16;
  c.n_layers = d->n_conv;
  int cin = 3, h = d->in_h, w = d->in_w;
  size_t woff = 0, boff = 0, act = 0;
  for (int l = 0; l < d->n_conv; ++l) {
    const int co = d->conv_out[l];
    const int nt = co / 16;
    NSC_REQUIRE(co >= 16 && co % 16 == 0 && (nt <= 4 || nt == 6 || nt == 8 || nt == 16),
                NSC_E_SHAPE, "conv layer %d: %d output channels unsupported", l, co);
    if (l > 0)
      NSC_REQUIRE(cin % (bf16 ? 32 : 4) == 0, NSC_E_SHAPE,
                  "conv layer %d: %d input channels must be a multiple of %d", l, cin,
                  bf16 ? 32 : 4);
    const bool pool = (d->pool_after_mask >> l) & 1u;
    NSC_REQUIRE(!pool || (h >= 2 && w >= 2), NSC_E_SHAPE, "conv layer %d pools a %dx%d map", l, h,
                w);
    CnnLayer& L = c.layers[l];
    L.cin = cin;
    L.cout = co;
    L.h = h;
    L.w = w;
    L.pool = pool;
    // layer 0: K = (dy, dx of 4, c of 4) = 48, padded with zero weights to whole MFMA steps
    L.kpad = l == 0 ? (bf16 ? 64 : 48) : 9 * cin;
    L.w_off = woff;
    L.b_off = boff;
    woff += (size_t)co * L.kpad;
    boff += co;
    const size_t lds = conv_lds_bytes(L, bf16, nullptr, nullptr, nullptr, nullptr, nullptr);
    NSC_REQUIRE(lds <= kMaxLds, NSC_E_SHAPE,
                "conv layer %d needs %zu bytes of LDS (limit %zu)", l, lds, kMaxLds);
    if (pool) {
      h /= 2;
      w /= 2;
    }
    act = act > (size_t)h * w * co ? act : (size_t)h * w * co;
    cin = co;
  }
  c.feat_c = cin;
  c.feat_h = h;
  c.feat_w = w;
  c.flat = cin * h * w;
  c.dense = d->dense;
  c.act_elems = act;
  *cnn = c;
  return NSC_OK;
}

uint16_t host_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)(u >> 16);  // inf / nan
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

float host_bf16_value(float f) {
  const uint32_t u = (uint32_t)host_bf16(f) << 16;
  float v;
  memcpy(&v, &u, 4);
  return v;
}

// fp16 bits of v * 2^e, rounded to nearest even.
uint16_t host_f16_scaled(float v, int e) {
  const _Float16 h = (_Float16)ldexpf(v, e);
  uint16_t b;
  memcpy(&b, &h, 2);
  return b;
}

// Scale exponent of a weight array for the fp16 matrix cores: the largest
// magnitude times 2^e lies in [2^14, 2^15), so every bf16 value within 2^31
// of it (8 significant bits) is an fp16 value after scaling.  0 for all-zero
// weights.
int fp16_weight_exp(const float* w, size_t n) {
  float mx = 0.0f;
  for (size_t i = 0; i < n; ++i) {
    const float a = fabsf(host_bf16_value(w[i]));
    mx = a > mx ? a : mx;
  }
  if (mx == 0.0f) return 0;
  int e = 0;
  frexpf(mx, &e);  // mx = f 2^e, f in [0.5, 1): floor(log2 mx) = e - 1
  return 14 - (e - 1);
}

// Down-scale exponent (>= 0) of activations bounded by `bound` so that they
// stay below 2^15 in fp16 (whose largest finite value is 65504).
int fp16_act_exp(double bound) {
  int e = 0;
  while (bound * ldexp(1.0, -e) > 32768.0) ++e;
  return e;
}

// Frame skipping: the checked frames of a stream form a video of their own
// (every s-th frame, frames s * frame_stride bytes apart, delta / s checked
// frames back); the cascade runs on it unchanged.
int32_t stride_of(const nsc_cascade_cfg* c) { return c->check_stride > 1 ? c->check_stride : 1; }

nsc_cascade_cfg checked_cfg(const nsc_cascade_cfg* c) {
  nsc_cascade_cfg k = *c;
  const int32_t s = stride_of(c);
  k.frame_stride = c->frame_stride * s;
  if (c->ref_mode == NSC_REF_PREV) k.delta = c->delta / s;
  k.check_stride = 1;
  return k;
}

// Checked frames among [t0, t0 + n): absolute checked indices [k0, k0 + nc).
void checked_range(int64_t t0, int64_t n, int32_t s, int64_t* k0, int64_t* nc) {
  *k0 = (t0 + s - 1) / s;
  *nc = (t0 + n + s - 1) / s - *k0;
}

// Workspace layout of nsc_cascade_run (of the checked-frame cascade, plus the
// checked frames' outputs before they are spread over their skip blocks).
struct RunLayout {
  size_t sums, fire, dec, idx, count, tiles, tile_last, carry, logit, scratch, cnn, part;
  size_t sk_label, sk_defer, sk_fire, sk_score, sk_logit;
  int64_t part_units;  // units the partial-sum section holds
  size_t total;
};

// cnn_pass > 0 sizes the CNN's share for passes of at most that many
// survivors; a staged run (area sums written by earlier calls, detector in
// its own pass) reserves no partial sums.
RunLayout run_layout(const nsc_cascade_cfg* c0, const Cnn& cnn, int64_t n_frames,
                     int64_t cnn_pass = 0, bool staged = false) {
  RunLayout L{};
  const nsc_cascade_cfg kc = checked_cfg(c0);
  const nsc_cascade_cfg* c = &kc;
  const int32_t s = stride_of(c0);
  const int64_t n = s > 1 ? n_frames / s + 1 : n_frames;  // checked frames of any window
  const size_t cells = (size_t)c->dd_h * c->dd_w * 3;
  const ResolvePlan rp = make_resolve_plan(n, 0, c->ref_mode == NSC_REF_PREV ? c->delta : 1);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes, kAlign);
    return at;
  };
  L.sums = take(cells * 4 * (size_t)n);
  L.fire = take((size_t)n);
  L.dec = take((size_t)n);
  L.idx = take((size_t)n * 4);
  L.count = take(64);
  L.tiles = take((size_t)compact_tiles(n) * 4 + 4);
  L.tile_last = take((size_t)rp.tiles * rp.delta * 4);
  L.carry = take((size_t)rp.tiles * rp.delta * 4);
  L.logit = take((size_t)n * 4);
  const size_t dmax = c->ref_mode == NSC_REF_PREV ? (size_t)c->delta : 1;
  L.scratch = take(dmax * cells * 4 + dmax);
  if (s > 1) {
    L.sk_label = take((size_t)n);
    L.sk_defer = take((size_t)n);
    L.sk_fire = take((size_t)n);
    L.sk_score = take((size_t)n * 8);
    L.sk_logit = take((size_t)n * 4);
  }
  L.cnn = take(cnn_workspace_bytes(cnn, cnn_pass > 0 && cnn_pass < n ? cnn_pass : n));
  // detector fused into the area kernel: per-unit partial sums, bounded by
  // the plan's units at one output row per band (fixed reference), or by the
  // fused earlier-frame plan's count
  if (!staged && c->fuse_prev && c->ref_mode == NSC_REF_PREV && c->metric == NSC_METRIC_MSE) {
    AreaPlan ap;
    DiffArgs a{};
    a.ref_mode = c->ref_mode;
    a.metric = c->metric;
    a.delta = c->delta;
    a.grid_h = c->grid_h;
    a.grid_w = c->grid_w;
    PrevFusePlan fp;
    if (make_area_plan(c->in_h, c->in_w, c->frame_stride, reinterpret_cast<const void*>(kAlign),
                       c->dd_h, c->dd_w, n > 0 ? n : 1, &ap) == NSC_OK &&
        area_prev_plan(ap, a, n, &fp)) {
      L.part_units = fp.part_elems;
      L.part = take((size_t)L.part_units * sizeof(int64_t));
    }
  }
  if (!staged && c->ref_mode == NSC_REF_FIXED && c->grid_h * c->grid_w == 1) {
    AreaPlan ap;
    if (make_area_plan(c->in_h, c->in_w, c->frame_stride, reinterpret_cast<const void*>(kAlign),
                       c->dd_h, c->dd_w, n > 0 ? n : 1, &ap) == NSC_OK &&
        ap.wave) {
      L.part_units = (int64_t)n * c->dd_h * ap.wg.waves_per_frame;
      L.part = take((size_t)L.part_units * 3 * sizeof(int64_t));
    }
  }
  L.total = o;
  return L;
}

// State: sums and decisions of the last delta checked frames (PREV), then,
// with frame skipping, one byte with the last checked frame's decision.
size_t state_layout_bytes(const nsc_cascade_cfg* c0, size_t* sums_off, size_t* dec_off,
                          size_t* last_off = nullptr) {
  const nsc_cascade_cfg kc = checked_cfg(c0);
  const nsc_cascade_cfg* c = &kc;
  const size_t cells = (size_t)c->dd_h * c->dd_w * 3;
  const size_t d = c->ref_mode == NSC_REF_PREV ? (size_t)c->delta : 0;
  if (sums_off) *sums_off = 0;
  if (dec_off) *dec_off = align_up(d * cells * 4, kAlign);
  const size_t core = align_up(d * cells * 4, kAlign) + align_up(d > 0 ? d : 1, kAlign);
  if (last_off) *last_off = core;
  return core + (stride_of(c0) > 1 ? kAlign : 0);
}

}  // namespace
}  // namespace nsc

using namespace nsc;

struct nsc_cnn {
  Cnn c;
};

extern "C" {

const char* nsc_status_string(int s) {
  switch (s) {
    case NSC_OK: return "NSC_OK";
    case NSC_E_INVAL: return "NSC_E_INVAL";
    case NSC_E_SHAPE: return "NSC_E_SHAPE";
    case NSC_E_DTYPE: return "NSC_E_DTYPE";
    case NSC_E_WORKSPACE: return "NSC_E_WORKSPACE";
    case NSC_E_HIP: return "NSC_E_HIP";
    case NSC_E_NOMEM: return "NSC_E_NOMEM";
    case NSC_E_STATE: return "NSC_E_STATE";
    default: return "NSC_E_UNKNOWN";
  }
}

const char* nsc_last_error(void) { return g_err; }

int64_t nsc_area_den(int32_t in_h, int32_t in_w, int32_t out_h, int32_t out_w) {
  if (int rc = check_area(in_h, in_w, out_h, out_w)) return rc;
  return (int64_t)Axis::make(in_h, out_h).p * Axis::make(in_w, out_w).p;
}

int nsc_cfg_check(const nsc_cascade_cfg* cfg) {
  g_err[0] = 0;
  return check_cfg(cfg);
}

int nsc_cnn_check(const nsc_cnn_desc* desc) {
  g_err[0] = 0;
  Cnn c;
  return plan_cnn(desc, &c);
}

int64_t nsc_cnn_blob_floats(const nsc_cnn_desc* desc) {
  Cnn c;
  if (int rc = plan_cnn(desc, &c)) return rc;
  int64_t n = 0;
  for (int l = 0; l < c.n_layers; ++l)
    n += (int64_t)c.layers[l].cout * c.layers[l].cin * 9 + c.layers[l].cout;
  return n + (int64_t)c.dense * c.flat + 2 * c.dense + 1;
}

int nsc_cnn_create(const nsc_cnn_desc* desc, const float* hw, int64_t n_floats, nsc_cnn** out) {
  g_err[0] = 0;
  NSC_REQUIRE(out != nullptr && hw != nullptr, NSC_E_INVAL, "weights or out pointer is NULL");
  *out = nullptr;
  Cnn c;
  if (int rc = plan_cnn(desc, &c)) return rc;
  const int64_t need = nsc_cnn_blob_floats(desc);
  NSC_REQUIRE(n_floats == need, NSC_E_INVAL, "weight blob has %lld floats, the network needs %lld",
              (long long)n_floats, (long long)need);
  const size_t es = c.bf16 ? 2 : 4;
  // host packing
  size_t conv_elems = 0, bias_elems = 0;
  for (int l = 0; l < c.n_layers; ++l) {
    conv_elems += (size_t)c.layers[l].cout * c.layers[l].kpad;
    bias_elems += c.layers[l].cout;
  }
  std::vector<float> convw(conv_elems, 0.0f), convb(bias_elems, 0.0f);
  const float* p = hw;
  for (int l = 0; l < c.n_layers; ++l) {
    const CnnLayer& L = c.layers[l];
    for (int o = 0; o < L.cout; ++o)
      for (int ci = 0; ci < L.cin; ++ci)
        for (int t = 0; t < 9; ++t) {
          const float v = p[((size_t)o * L.cin + ci) * 9 + t];
          const size_t k = l == 0 ? (size_t)(t / 3) * 16 + (t % 3) * 4 + ci : (size_t)t * L.cin + ci;
          convw[L.w_off + (size_t)o * L.kpad + k] = v;
        }
    p += (size_t)L.cout * L.cin * 9;
    for (int o = 0; o < L.cout; ++o) convb[L.b_off + o] = p[o];
    p += L.cout;
  }
  std::vector<float> w1((size_t)c.dense * c.flat);
  for (int j = 0; j < c.dense; ++j)
    for (int ch = 0; ch < c.feat_c; ++ch)
      for (int y = 0; y < c.feat_h; ++y)
        for (int x = 0; x < c.feat_w; ++x)
          w1[(size_t)j * c.flat + ((size_t)y * c.feat_w + x) * c.feat_c + ch] =
              p[(size_t)j * c.flat + ((size_t)ch * c.feat_h + y) * c.feat_w + x];
  p += (size_t)c.dense * c.flat;
  std::vector<float> b1(p, p + c.dense);
  p += c.dense;
  std::vector<float> w2(p, p + c.dense);
  p += c.dense;
  c.b2 = *p;
  // bf16: the conv weights again in MFMA fragment order (see CnnLayer)
  std::vector<float> convwf(c.bf16 ? conv_elems : 0, 0.0f);
  if (c.bf16) {
    for (int l = 0; l < c.n_layers; ++l) {
      const CnnLayer& L = c.layers[l];
      const int nts = L.cout / 16, kst = L.kpad / 32;
      for (int ks = 0; ks < kst; ++ks)
        for (int nt = 0; nt < nts; ++nt)
          for (int lane = 0; lane < 64; ++lane)
            for (int e = 0; e < 8; ++e) {
              const int o = nt * 16 + (lane & 15), k = ks * 32 + (lane >> 4) * 8 + e;
              convwf[L.w_off + (((size_t)ks * nts + nt) * 64 + lane) * 8 + e] =
                  convw[L.w_off + (size_t)o * L.kpad + k];
            }
    }
  }
  // bf16: fp16 copies for the layers whose activations run through the fp16
  // matrix cores (see CnnLayer::wexp / aexp): fragment order like conv_wf,
  // each layer scaled by 2^wexp, and the dense weights likewise
  std::vector<uint16_t> convwh, w1h;
  if (c.bf16) {
    convwh.resize(conv_elems);
    w1h.resize(w1.size());
    double bound = 1.0;  // |input| <= 1 after pre-processing
    for (int l = 0; l < c.n_layers; ++l) {
      CnnLayer& L = c.layers[l];
      const size_t n = (size_t)L.cout * L.kpad;
      L.wexp = fp16_weight_exp(&convwf[L.w_off], n);
      L.aexp = fp16_act_exp(bound);
      for (size_t i = 0; i < n; ++i)
        convwh[L.w_off + i] = host_f16_scaled(host_bf16_value(convwf[L.w_off + i]), L.wexp);
      // the layer's output bound: max over channels of sum |w| x bound + |b|
      double nb = 0.0;
      for (int o = 0; o < L.cout; ++o) {
        double sw = 0.0;
        for (int k = 0; k < L.kpad; ++k)
          sw += fabs((double)host_bf16_value(convw[L.w_off + (size_t)o * L.kpad + k]));
        const double v = sw * bound + fabs((double)convb[L.b_off + o]);
        nb = v > nb ? v : nb;
      }
      bound = nb;
    }
    c.dense_wexp = fp16_weight_exp(w1.data(), w1.size());
    c.dense_aexp = fp16_act_exp(bound);
    for (size_t i = 0; i < w1.size(); ++i)
      w1h[i] = host_f16_scaled(host_bf16_value(w1[i]), c.dense_wexp);
  }
  // per layer (then the dense layer) the fp16 path's input and output scales
  std::vector<float> scales(2 * (size_t)(c.n_layers + 1), 1.0f);
  if (c.bf16) {
    for (int l = 0; l < c.n_layers; ++l) {
      scales[2 * l] = ldexpf(1.0f, -c.layers[l].aexp);
      scales[2 * l + 1] = ldexpf(1.0f, c.layers[l].aexp - c.layers[l].wexp);
    }
    scales[2 * c.n_layers] = ldexpf(1.0f, -c.dense_aexp);
    scales[2 * c.n_layers + 1] = ldexpf(1.0f, c.dense_aexp - c.dense_wexp);
  }
  // fp16 path with a 3-channel first layer (fused with the second by
  // k_pair64): the first layer's bf16 fragments multiplied by the second
  // layer's input scale 2^-aexp (exact), with the bias as two bf16 values
  // (hi, and the remainder lo) in the taps (0, 0) and (0, 1) of channel 3,
  // whose input is the constant 1: the matrix cores then produce the biased,
  // scaled pre-activation, and the epilogue only applies the ReLU
  std::vector<float> w0h;
  if (c.h16 && c.n_layers >= 2 && c.layers[0].cin == 3 && c.layers[0].kpad == 64) {
    const CnnLayer& L = c.layers[0];
    const float s1 = ldexpf(1.0f, -c.layers[1].aexp);
    const int nts = L.cout / 16;
    w0h.assign((size_t)L.cout * L.kpad, 0.0f);
    for (int ks = 0; ks < 2; ++ks)
      for (int nt = 0; nt < nts; ++nt)
        for (int lane = 0; lane < 64; ++lane)
          for (int e = 0; e < 8; ++e) {
            const int o = nt * 16 + (lane & 15), k = ks * 32 + (lane >> 4) * 8 + e;
            float v = host_bf16_value(convw[L.w_off + (size_t)o * L.kpad + k]) * s1;
            if (k == 3 || k == 7) {  // (dy, dx, c) = (0, 0, 3), (0, 1, 3): the bias
              const float b = convb[L.b_off + o] * s1;
              const float hi = host_bf16_value(b);
              v = k == 3 ? hi : host_bf16_value(b - hi);
            }
            w0h[(((size_t)ks * nts + nt) * 64 + lane) * 8 + e] = v;
          }
  }
  // fp16 path: the dense weights again in MFMA fragment order for
  // k_dense_tiles, K steps of 32 padded with zeros to whole chunks of
  // kDenseChunk steps: fragment (ks, nt), lane l = 16 g + m holds units
  // 16 nt + m, features 32 ks + 8 g .. + 7, so that a chunk is one contiguous
  // block of kDenseChunk x (D / 16) KB
  std::vector<uint16_t> w1f;
  if (c.bf16) {
    const int nts = c.dense / 16;
    const int nks = (c.flat + 31) / 32;
    const int nkc = (nks + kDenseChunk - 1) / kDenseChunk * kDenseChunk;
    w1f.assign((size_t)nkc * nts * 64 * 8, 0);
    for (int ks = 0; ks < nks; ++ks)
      for (int nt = 0; nt < nts; ++nt)
        for (int lane = 0; lane < 64; ++lane)
          for (int e = 0; e < 8; ++e) {
            const int u = nt * 16 + (lane & 15), k = ks * 32 + (lane >> 4) * 8 + e;
            if (k < c.flat)
              w1f[(((size_t)ks * nts + nt) * 64 + lane) * 8 + e] = w1h[(size_t)u * c.flat + k];
          }
  }
  // device image: [conv_w][conv_wf][conv_wh][conv_b][w1][w1h][b1][w2][scales][w0h][w1f]
  const size_t o_cw = 0;
  const size_t o_cwf = align_up(o_cw + conv_elems * es, kAlign);
  const size_t o_cwh = align_up(o_cwf + convwf.size() * es, kAlign);
  const size_t o_cb = align_up(o_cwh + convwh.size() * 2, kAlign);
  const size_t o_w1 = align_up(o_cb + bias_elems * 4, kAlign);
  const size_t o_w1h = align_up(o_w1 + w1.size() * es, kAlign);
  const size_t o_b1 = align_up(o_w1h + w1h.size() * 2, kAlign);
  const size_t o_w2 = align_up(o_b1 + (size_t)c.dense * 4, kAlign);
  const size_t o_sc = align_up(o_w2 + (size_t)c.dense * 4, kAlign);
  const size_t o_w0h = align_up(o_sc + scales.size() * 4, kAlign);
  const size_t o_w1f = align_up(o_w0h + w0h.size() * 2, kAlign);
  const size_t total = align_up(o_w1f + w1f.size() * 2, kAlign);
  std::vector<unsigned char> img(total, 0);
  auto put = [&](size_t off, const std::vector<float>& v, bool as_bf16) {
    if (as_bf16) {
      uint16_t* d = reinterpret_cast<uint16_t*>(img.data() + off);
      for (size_t i = 0; i < v.size(); ++i) d[i] = host_bf16(v[i]);
    } else {
      memcpy(img.data() + off, v.data(), v.size() * 4);
    }
  };
  put(o_cw, convw, c.bf16);
  if (c.bf16) put(o_cwf, convwf, true);
  put(o_cb, convb, false);
  put(o_w1, w1, c.bf16);
  if (c.bf16) {
    memcpy(img.data() + o_cwh, convwh.data(), convwh.size() * 2);
    memcpy(img.data() + o_w1h, w1h.data(), w1h.size() * 2);
  }
  put(o_b1, b1, false);
  put(o_w2, w2, false);
  put(o_sc, scales, false);
  if (!w0h.empty()) put(o_w0h, w0h, true);
  if (!w1f.empty()) memcpy(img.data() + o_w1f, w1f.data(), w1f.size() * 2);
  void* dev = nullptr;
  if (hipMalloc(&dev, total) != hipSuccess)
    return fail(NSC_E_NOMEM, "hipMalloc of %zu bytes for CNN weights failed", total);
  if (hipMemcpy(dev, img.data(), total, hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipFree(dev);
    return fail(NSC_E_HIP, "copying CNN weights to the device failed");
  }
  unsigned char* b = static_cast<unsigned char*>(dev);
  c.dev = dev;
  c.conv_w = b + o_cw;
  c.conv_wf = c.bf16 ? b + o_cwf : nullptr;
  c.conv_wh = c.bf16 ? b + o_cwh : nullptr;
  c.w1h = c.bf16 ? b + o_w1h : nullptr;
  c.conv_b = reinterpret_cast<float*>(b + o_cb);
  c.w1 = b + o_w1;
  c.b1 = reinterpret_cast<float*>(b + o_b1);
  c.w2 = reinterpret_cast<float*>(b + o_w2);
  c.scales = reinterpret_cast<float*>(b + o_sc);
  c.conv_w0h = w0h.empty() ? nullptr : b + o_w0h;
  c.w1f = w1f.empty() ? nullptr : b + o_w1f;
  nsc_cnn* h = new (std::nothrow) nsc_cnn;
  if (!h) {
    (void)hipFree(dev);
    return fail(NSC_E_NOMEM, "out of host memory");
  }
  h->c = c;
  *out = h;
  return NSC_OK;
}

int nsc_cnn_destroy(nsc_cnn* cnn) {
  if (!cnn) return NSC_OK;
  hipError_t e = hipFree(cnn->c.dev);
  delete cnn;
  return e == hipSuccess ? NSC_OK : fail(NSC_E_HIP, "hipFree failed: %s", hipGetErrorString(e));
}

int nsc_cascade_workspace_bytes(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn, int64_t max_frames,
                                size_t* bytes) {
  g_err[0] = 0;
  if (int rc = check_cfg(cfg)) return rc;
  NSC_REQUIRE(cnn != nullptr && bytes != nullptr, NSC_E_INVAL, "cnn or bytes is NULL");
  NSC_REQUIRE(max_frames >= 0 && max_frames <= kMaxFrames, NSC_E_INVAL, "max_frames %lld out of range",
              (long long)max_frames);
  *bytes = run_layout(cfg, cnn->c, max_frames).total;
  return NSC_OK;
}

int nsc_state_bytes(const nsc_cascade_cfg* cfg, size_t* bytes) {
  g_err[0] = 0;
  if (int rc = check_cfg(cfg)) return rc;
  NSC_REQUIRE(bytes != nullptr, NSC_E_INVAL, "bytes is NULL");
  *bytes = state_layout_bytes(cfg, nullptr, nullptr);
  return NSC_OK;
}

int nsc_compact_workspace_bytes(int64_t n, size_t* bytes) {
  g_err[0] = 0;
  NSC_REQUIRE(bytes != nullptr && n >= 0 && n <= kMaxFrames, NSC_E_INVAL, "bad arguments");
  *bytes = (size_t)compact_tiles(n) * 4 + 4;
  return NSC_OK;
}

int nsc_cnn_workspace_bytes(const nsc_cnn* cnn, int64_t max_count, size_t* bytes) {
  g_err[0] = 0;
  NSC_REQUIRE(cnn != nullptr && bytes != nullptr && max_count >= 0 && max_count <= kMaxFrames,
              NSC_E_INVAL, "bad arguments");
  *bytes = cnn_workspace_bytes(cnn->c, max_count);
  return NSC_OK;
}

int nsc_downsample(const uint8_t* frames, int64_t n, int32_t in_h, int32_t in_w,
                   int64_t frame_stride, int32_t out_h, int32_t out_w, int32_t* sums_out,
                   void* stream) {
  g_err[0] = 0;
  if (int rc = check_area(in_h, in_w, out_h, out_w)) return rc;
  NSC_REQUIRE(n >= 0 && n <= kMaxFrames, NSC_E_INVAL, "n = %lld out of range", (long long)n);
  NSC_REQUIRE(frame_stride >= (int64_t)in_h * in_w * 3, NSC_E_INVAL, "frame_stride too small");
  if (n == 0) return NSC_OK;
  NSC_REQUIRE(frames != nullptr && sums_out != nullptr, NSC_E_INVAL, "frames or sums_out is NULL");
  AreaPlan p;
  if (int rc = make_area_plan(in_h, in_w, frame_stride, frames, out_h, out_w, n, &p)) return rc;
  return launch_area_sums(p, frames, frame_stride, n, sums_out, (hipStream_t)stream);
}

int nsc_diff_detect(const nsc_cascade_cfg* cfg, const uint8_t* frames, int64_t n, int64_t t0,
                    const int32_t* prev_sums, int32_t* sums_out, double* score_out,
                    uint8_t* fire_out, void* stream) {
  g_err[0] = 0;
  if (int rc = check_cfg(cfg)) return rc;
  NSC_REQUIRE(n >= 0 && n <= kMaxFrames && t0 >= 0, NSC_E_INVAL, "n or t0 out of range");
  if (n == 0) return NSC_OK;
  NSC_REQUIRE(frames && sums_out && fire_out, NSC_E_INVAL, "frames, sums_out or fire_out is NULL");
  NSC_REQUIRE(!(cfg->ref_mode == NSC_REF_PREV && t0 > 0 && prev_sums == nullptr), NSC_E_STATE,
              "t0 > 0 in earlier-frame mode needs the sums of the previous delta frames");
  const hipStream_t st = (hipStream_t)stream;
  AreaPlan p;
  if (int rc = make_area_plan(cfg->in_h, cfg->in_w, cfg->frame_stride, frames, cfg->dd_h, cfg->dd_w,
                              n, &p))
    return rc;
  if (int rc = launch_area_sums(p, frames, cfg->frame_stride, n, sums_out, st)) return rc;
  const double den = (double)nsc_area_den(cfg->in_h, cfg->in_w, cfg->dd_h, cfg->dd_w);
  DiffArgs a{};
  a.sums = sums_out;
  a.prev_sums = prev_sums;
  a.ref_sums = cfg->ref_sums;
  a.lr_w = cfg->lr_w;
  a.lr_b = cfg->lr_b;
  a.delta_diff = cfg->delta_diff;
  a.den2 = den * den;
  a.den = den;
  a.metric = cfg->metric;
  a.n = n;
  a.t0 = t0;
  a.dd_h = cfg->dd_h;
  a.dd_w = cfg->dd_w;
  a.grid_h = cfg->grid_h;
  a.grid_w = cfg->grid_w;
  a.ref_mode = cfg->ref_mode;
  a.delta = cfg->ref_mode == NSC_REF_PREV ? cfg->delta : 0;
  a.score = score_out;
  a.fire = fire_out;
  return launch_diff(a, st);
}

int nsc_compact(const uint8_t* fire, int64_t n, int32_t* idx_out, int32_t* count_out, void* ws,
                size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  NSC_REQUIRE(n >= 0 && n <= kMaxFrames, NSC_E_INVAL, "n = %lld out of range", (long long)n);
  NSC_REQUIRE(count_out != nullptr, NSC_E_INVAL, "count_out is NULL");
  if (n > 0) {
    NSC_REQUIRE(fire && idx_out, NSC_E_INVAL, "fire or idx_out is NULL");
    const size_t need = (size_t)compact_tiles(n) * 4 + 4;
    NSC_REQUIRE(ws != nullptr && ws_bytes >= need && ((uintptr_t)ws & 3) == 0, NSC_E_WORKSPACE,
                "compaction needs %zu bytes of 4-byte aligned workspace", need);
  }
  return launch_compact(fire, n, idx_out, count_out, static_cast<int32_t*>(ws), (hipStream_t)stream);
}

int nsc_compact_noalloc(const uint8_t* fire, int64_t n, int32_t* idx_out, int32_t* count_out,
                        void* stream) {
  g_err[0] = 0;
  NSC_REQUIRE(n >= 0 && n <= kMaxFrames, NSC_E_INVAL, "n = %lld out of range", (long long)n);
  NSC_REQUIRE(n <= NSC_NOALLOC_MAX_FLAGS, NSC_E_WORKSPACE,
              "n = %lld exceeds the %lld flags the static scratch holds", (long long)n,
              (long long)NSC_NOALLOC_MAX_FLAGS);
  NSC_REQUIRE(count_out != nullptr, NSC_E_INVAL, "count_out is NULL");
  if (n > 0) NSC_REQUIRE(fire && idx_out, NSC_E_INVAL, "fire or idx_out is NULL");
  return launch_compact_noalloc(fire, n, idx_out, count_out, (hipStream_t)stream);
}

int nsc_specialized_cnn(const nsc_cnn* cnn, const int32_t* sums, int32_t sums_h, int32_t sums_w,
                        int64_t den, const int32_t* idx, const int32_t* count, int64_t max_count,
                        float* logit_out, float* prob_out, void* ws, size_t ws_bytes,
                        void* stream) {
  g_err[0] = 0;
  NSC_REQUIRE(cnn != nullptr, NSC_E_INVAL, "cnn is NULL");
  const Cnn& c = cnn->c;
  NSC_REQUIRE(max_count >= 0 && max_count <= kMaxFrames, NSC_E_INVAL, "max_count out of range");
  NSC_REQUIRE(sums_h >= c.desc.in_h && sums_w >= c.desc.in_w && sums_h % c.desc.in_h == 0 &&
                  sums_w % c.desc.in_w == 0,
              NSC_E_SHAPE, "sums grid %dx%d does not nest onto the CNN input %dx%d", sums_h, sums_w,
              c.desc.in_h, c.desc.in_w);
  NSC_REQUIRE(den >= 1, NSC_E_INVAL, "den must be positive");
  NSC_REQUIRE(255 * (double)den * (sums_h / c.desc.in_h) * (sums_w / c.desc.in_w) < 2147483648.0,
              NSC_E_SHAPE, "den %lld: the CNN input sums overflow 32 bits", (long long)den);
  if (max_count == 0) return NSC_OK;
  NSC_REQUIRE(sums && idx && count && logit_out, NSC_E_INVAL, "a required pointer is NULL");
  NSC_REQUIRE(ws != nullptr && ((uintptr_t)ws % kAlign) == 0, NSC_E_WORKSPACE,
              "workspace must be 256-byte aligned");
  CnnRunArgs r{};
  r.sums = sums;
  r.sums_h = sums_h;
  r.sums_w = sums_w;
  r.fy = sums_h / c.desc.in_h;
  r.fx = sums_w / c.desc.in_w;
  r.den_c = (double)den * r.fy * r.fx;
  r.idx = idx;
  r.count = count;
  r.max_count = max_count;
  r.logit = logit_out;
  r.prob = prob_out;
  return run_cnn(c, r, ws, ws_bytes, (hipStream_t)stream);
}

}  // extern "C"

namespace nsc {
namespace {

// Counts of a finished run, read back to the host (synchronizes the stream).
int run_stats(const uint8_t* label, const uint8_t* defer, const int32_t* count, int64_t n,
              hipStream_t st, nsc_run_stats* stats) {
  std::vector<uint8_t> hl(n), hd(n);
  int32_t hc = 0;
  NSC_TRY_HIP(hipMemcpyAsync(hl.data(), label, n, hipMemcpyDeviceToHost, st));
  NSC_TRY_HIP(hipMemcpyAsync(hd.data(), defer, n, hipMemcpyDeviceToHost, st));
  NSC_TRY_HIP(hipMemcpyAsync(&hc, count, 4, hipMemcpyDeviceToHost, st));
  NSC_TRY_HIP(hipStreamSynchronize(st));
  nsc_run_stats r{n, hc, 0, 0};
  for (int64_t i = 0; i < n; ++i) {
    r.positive += hl[i] && !hd[i];
    r.deferred += hd[i];
  }
  *stats = r;
  return NSC_OK;
}

// Steps 1-5 on frames [t0, t0 + n) of a configuration without frame skipping
// (the checked frames); records stage events 0..4 through `mark`.  With
// frames == nullptr step 1 is skipped: the area sums of the n frames are
// already in the workspace (staged by earlier calls).  cnn_pass > 0 runs the
// CNN in passes over at most that many compacted slots each.
template <class Mark>
int run_checked(const nsc_cascade_cfg* cfg, const Cnn& c, const uint8_t* frames, int64_t n,
                int64_t t0, void* state, unsigned char* w, const RunLayout& L, uint8_t* label_out,
                uint8_t* defer_out, double* score_out, uint8_t* fire_out, float* logit_out,
                int64_t cnn_pass, hipStream_t st, Mark&& mark) {
  const bool prev = cfg->ref_mode == NSC_REF_PREV;
  int32_t* sums = reinterpret_cast<int32_t*>(w + L.sums);
  uint8_t* fire = fire_out ? fire_out : w + L.fire;
  uint8_t* dec = w + L.dec;
  int32_t* idx = reinterpret_cast<int32_t*>(w + L.idx);
  int32_t* count = reinterpret_cast<int32_t*>(w + L.count);
  const int64_t cells = (int64_t)cfg->dd_h * cfg->dd_w * 3;
  size_t st_dec_off = 0;
  state_layout_bytes(cfg, nullptr, &st_dec_off);
  int32_t* st_sums = prev ? static_cast<int32_t*>(state) : nullptr;
  uint8_t* st_dec = prev ? static_cast<uint8_t*>(state) + st_dec_off : nullptr;

  // 1: area sums
  if (int rc = mark(0)) return rc;
  AreaPlan ap{};
  if (frames)
    if (int rc = make_area_plan(cfg->in_h, cfg->in_w, cfg->frame_stride, frames, cfg->dd_h,
                                cfg->dd_w, n, &ap))
      return rc;
  // 2: detector (against a fixed reference image fused into step 1, its
  // partial sums added up by a finishing kernel, when the plan allows)
  {
    const double den = (double)nsc_area_den(cfg->in_h, cfg->in_w, cfg->dd_h, cfg->dd_w);
    DiffArgs a{};
    a.sums = sums;
    a.prev_sums = t0 > 0 ? st_sums : nullptr;
    a.ref_sums = cfg->ref_sums;
    a.lr_w = cfg->lr_w;
    a.lr_b = cfg->lr_b;
    a.delta_diff = cfg->delta_diff;
    a.den2 = den * den;
    a.den = den;
    a.metric = cfg->metric;
    a.n = n;
    a.t0 = t0;
    a.dd_h = cfg->dd_h;
    a.dd_w = cfg->dd_w;
    a.grid_h = cfg->grid_h;
    a.grid_w = cfg->grid_w;
    a.ref_mode = cfg->ref_mode;
    a.delta = prev ? cfg->delta : 0;
    a.score = score_out;
    a.fire = fire;
    int64_t* part = reinterpret_cast<int64_t*>(w + L.part);
    const bool fused = frames && area_detect_fused(ap, a) && L.part_units > 0 &&
                       area_detect_part_count(ap, n) <= L.part_units;
    PrevFusePlan fp;
    const bool fused_prev = frames && cfg->fuse_prev && !fused && L.part_units > 0 &&
                            area_prev_plan(ap, a, n, &fp) && fp.part_elems <= L.part_units;
    if (!frames) {
      if (int rc = mark(1)) return rc;
      if (int rc = launch_diff(a, st)) return rc;
    } else if (fused_prev) {
      if (int rc = launch_area_prev(fp, frames, cfg->frame_stride, n, sums, a, part, st)) return rc;
      if (int rc = mark(1)) return rc;
      area_prev_diff_args(fp, part, &a);
      if (int rc = launch_diff(a, st)) return rc;
    } else if (fused) {
      if (int rc = launch_area_detect_fixed(ap, frames, cfg->frame_stride, n, sums, a, part, st))
        return rc;
      if (int rc = mark(1)) return rc;
    } else {
      if (int rc = launch_area_sums(ap, frames, cfg->frame_stride, n, sums, st)) return rc;
      if (int rc = mark(1)) return rc;
      if (int rc = launch_diff(a, st)) return rc;
    }
  }
  if (int rc = mark(2)) return rc;
  // 3: compaction
  if (int rc = launch_compact(fire, n, idx, count, reinterpret_cast<int32_t*>(w + L.tiles), st))
    return rc;
  if (int rc = mark(3)) return rc;
  // 4: CNN on survivors with decisions written at their frame positions
  if (logit_out)
    if (int rc = launch_fill_nan(logit_out, n, st)) return rc;
  CnnRunArgs r{};
  r.sums = sums;
  r.sums_h = cfg->dd_h;
  r.sums_w = cfg->dd_w;
  r.fy = cfg->dd_h / cfg->cnn_h;
  r.fx = cfg->dd_w / cfg->cnn_w;
  r.den_c = (double)nsc_area_den(cfg->in_h, cfg->in_w, cfg->dd_h, cfg->dd_w) * r.fy * r.fx;
  r.idx = idx;
  r.count = count;
  r.max_count = n;
  r.logit = reinterpret_cast<float*>(w + L.logit);
  r.prob = nullptr;
  r.dec = dec;
  r.c_low = cfg->c_low;
  r.c_high = cfg->c_high;
  r.frame_logit = logit_out;
  const int64_t pass = cnn_pass > 0 && cnn_pass < n ? cnn_pass : n;
  for (int64_t p0 = 0; p0 < n; p0 += pass) {
    if (pass < n) {
      // slots [p0, p0 + m) of the compacted list; the pass's count in count[1]
      const int64_t m = n - p0 < pass ? n - p0 : pass;
      if (int rc = launch_pass_count(count, p0, m, count + 1, st)) return rc;
      r.idx = idx + p0;
      r.count = count + 1;
      r.max_count = m;
      r.logit = reinterpret_cast<float*>(w + L.logit) + p0;
    }
    if (int rc = run_cnn(c, r, w + L.cnn, L.total - L.cnn, st)) return rc;
  }
  if (int rc = mark(4)) return rc;
  // 5: decisions of frames that did not fire
  const ResolvePlan rp = make_resolve_plan(n, t0, prev ? cfg->delta : 1);
  if (int rc = launch_resolve(rp, cfg->ref_mode, fire, dec, st_dec,
                              reinterpret_cast<int32_t*>(w + L.tile_last),
                              reinterpret_cast<int32_t*>(w + L.carry), label_out, defer_out, st))
    return rc;
  if (prev)
    if (int rc = launch_state_update(sums, label_out, defer_out, n, cfg->delta, cells, st_sums,
                                     st_dec, w + L.scratch, st))
      return rc;
  return NSC_OK;
}

}  // namespace
}  // namespace nsc

extern "C" {

int nsc_cascade_run(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn, const uint8_t* frames,
                    int64_t n, int64_t t0, void* state, void* ws, size_t ws_bytes,
                    uint8_t* label_out, uint8_t* defer_out, const nsc_frame_outputs* outs,
                    nsc_run_stats* stats, void* const* stage_events, void* stream) {
  g_err[0] = 0;
  if (int rc = check_cfg(cfg)) return rc;
  NSC_REQUIRE(cnn != nullptr, NSC_E_INVAL, "cnn is NULL");
  auto mark = [&](int k) -> int {
    if (stage_events && stage_events[k])
      NSC_TRY_HIP(hipEventRecord((hipEvent_t)stage_events[k], (hipStream_t)stream));
    return NSC_OK;
  };
  const Cnn& c = cnn->c;
  NSC_REQUIRE(c.desc.in_h == cfg->cnn_h && c.desc.in_w == cfg->cnn_w, NSC_E_SHAPE,
              "CNN input %dx%d differs from the configured %dx%d", c.desc.in_h, c.desc.in_w,
              cfg->cnn_h, cfg->cnn_w);
  NSC_REQUIRE(n >= 0 && n <= kMaxFrames && t0 >= 0, NSC_E_INVAL, "n or t0 out of range");
  const bool prev = cfg->ref_mode == NSC_REF_PREV;
  const int32_t s = stride_of(cfg);
  if (n == 0) {
    if (stats) *stats = nsc_run_stats{0, 0, 0, 0};
    return NSC_OK;
  }
  NSC_REQUIRE(frames && label_out && defer_out, NSC_E_INVAL, "frames, label_out or defer_out is NULL");
  NSC_REQUIRE(!(prev && state == nullptr), NSC_E_STATE, "earlier-frame mode needs a state buffer");
  NSC_REQUIRE(!(s > 1 && state == nullptr), NSC_E_STATE, "frame skipping needs a state buffer");
  const RunLayout L = run_layout(cfg, c, n);
  NSC_REQUIRE(ws != nullptr && ((uintptr_t)ws % kAlign) == 0 && ws_bytes >= L.total,
              NSC_E_WORKSPACE, "workspace needs %zu bytes (256-byte aligned), got %zu", L.total,
              ws_bytes);
  const hipStream_t st = (hipStream_t)stream;
  unsigned char* w = static_cast<unsigned char*>(ws);
  int32_t* count = reinterpret_cast<int32_t*>(w + L.count);
  size_t last_off = 0;
  state_layout_bytes(cfg, nullptr, nullptr, &last_off);

  if (s == 1) {
    if (int rc = run_checked(cfg, c, frames, n, t0, state, w, L, label_out, defer_out,
                             outs ? outs->score : nullptr, outs ? outs->fire : nullptr,
                             outs ? outs->logit : nullptr, 0, st, mark))
      return rc;
  } else {
    // the checked frames [k0, k0 + nc) as a video of their own, then every frame
    // takes the output of its checked frame
    const nsc_cascade_cfg kc = checked_cfg(cfg);
    int64_t k0, nc;
    checked_range(t0, n, s, &k0, &nc);
    uint8_t* k_label = w + L.sk_label;
    uint8_t* k_defer = w + L.sk_defer;
    uint8_t* k_fire = w + L.sk_fire;
    double* k_score = reinterpret_cast<double*>(w + L.sk_score);
    float* k_logit = reinterpret_cast<float*>(w + L.sk_logit);
    if (nc > 0) {
      const uint8_t* kf = frames + (k0 * s - t0) * cfg->frame_stride;
      if (int rc = run_checked(&kc, c, kf, nc, k0, state, w, L, k_label, k_defer, k_score, k_fire,
                               k_logit, 0, st, mark))
        return rc;
    } else {
      for (int k = 0; k < 5; ++k)
        if (int rc = mark(k)) return rc;
      if (int rc = launch_set_i32(count, 0, st)) return rc;
    }
    uint8_t* last = static_cast<uint8_t*>(state) + last_off;
    SkipExpand e{};
    e.n = n;
    e.t0 = t0;
    e.s = s;
    e.k0 = k0;
    e.nc = nc;
    e.k_label = k_label;
    e.k_defer = k_defer;
    e.k_score = k_score;
    e.k_fire = k_fire;
    e.k_logit = k_logit;
    e.last = last;
    e.label = label_out;
    e.defer = defer_out;
    e.score = outs ? outs->score : nullptr;
    e.fire = outs ? outs->fire : nullptr;
    e.logit = outs ? outs->logit : nullptr;
    if (int rc = launch_skip_expand(e, st)) return rc;
  }
  if (int rc = mark(5)) return rc;
  if (stats) return run_stats(label_out, defer_out, count, n, st, stats);
  return NSC_OK;
}

}  // extern "C"

// ------------------------------------------------- batches of staged chunks

namespace nsc {
namespace {

// Default bound on the survivors of one CNN pass in a staged batch.
constexpr int64_t kBatchCnnPass = 16384;

int64_t batch_cnn_pass(int64_t batch_frames, int64_t cnn_pass) {
  const int64_t p = cnn_pass > 0 ? cnn_pass : kBatchCnnPass;
  return p < batch_frames ? p : batch_frames;
}

int check_batch(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn, int64_t batch_frames,
                int64_t cnn_pass) {
  if (int rc = check_cfg(cfg)) return rc;
  NSC_REQUIRE(cnn != nullptr, NSC_E_INVAL, "cnn is NULL");
  NSC_REQUIRE(cnn->c.desc.in_h == cfg->cnn_h && cnn->c.desc.in_w == cfg->cnn_w, NSC_E_SHAPE,
              "CNN input %dx%d differs from the configured %dx%d", cnn->c.desc.in_h,
              cnn->c.desc.in_w, cfg->cnn_h, cfg->cnn_w);
  NSC_REQUIRE(stride_of(cfg) == 1, NSC_E_INVAL, "a staged batch needs check_stride 1, got %d",
              cfg->check_stride);
  NSC_REQUIRE(batch_frames > 0 && batch_frames <= kMaxFrames && cnn_pass >= 0, NSC_E_INVAL,
              "batch_frames %lld or cnn_pass %lld out of range", (long long)batch_frames,
              (long long)cnn_pass);
  return NSC_OK;
}

}  // namespace
}  // namespace nsc

extern "C" {

int nsc_batch_workspace_bytes(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn, int64_t batch_frames,
                              int64_t cnn_pass, size_t* bytes) {
  g_err[0] = 0;
  if (int rc = check_batch(cfg, cnn, batch_frames, cnn_pass)) return rc;
  NSC_REQUIRE(bytes != nullptr, NSC_E_INVAL, "bytes is NULL");
  *bytes = run_layout(cfg, cnn->c, batch_frames, batch_cnn_pass(batch_frames, cnn_pass), true).total;
  return NSC_OK;
}

int nsc_cascade_stage(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn, int64_t batch_frames,
                      int64_t cnn_pass, const uint8_t* frames, int64_t n, int64_t at, void* ws,
                      size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  if (int rc = check_batch(cfg, cnn, batch_frames, cnn_pass)) return rc;
  NSC_REQUIRE(n >= 0 && at >= 0 && at + n <= batch_frames, NSC_E_INVAL,
              "slots [%lld, %lld) outside the batch of %lld", (long long)at,
              (long long)(at + n), (long long)batch_frames);
  if (n == 0) return NSC_OK;
  NSC_REQUIRE(frames != nullptr, NSC_E_INVAL, "frames is NULL");
  const RunLayout L =
      run_layout(cfg, cnn->c, batch_frames, batch_cnn_pass(batch_frames, cnn_pass), true);
  NSC_REQUIRE(ws != nullptr && ((uintptr_t)ws % kAlign) == 0 && ws_bytes >= L.total,
              NSC_E_WORKSPACE, "workspace needs %zu bytes (256-byte aligned), got %zu", L.total,
              ws_bytes);
  AreaPlan ap;
  if (int rc = make_area_plan(cfg->in_h, cfg->in_w, cfg->frame_stride, frames, cfg->dd_h,
                              cfg->dd_w, n, &ap))
    return rc;
  const int64_t cells = (int64_t)cfg->dd_h * cfg->dd_w * 3;
  int32_t* sums = reinterpret_cast<int32_t*>(static_cast<unsigned char*>(ws) + L.sums) + at * cells;
  return launch_area_sums(ap, frames, cfg->frame_stride, n, sums, (hipStream_t)stream);
}

int nsc_cascade_finish(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn, int64_t batch_frames,
                       int64_t cnn_pass, int64_t n, int64_t t0, void* state, void* ws,
                       size_t ws_bytes, uint8_t* label_out, uint8_t* defer_out,
                       const nsc_frame_outputs* outs, nsc_run_stats* stats,
                       void* const* stage_events, void* stream) {
  g_err[0] = 0;
  if (int rc = check_batch(cfg, cnn, batch_frames, cnn_pass)) return rc;
  NSC_REQUIRE(n >= 0 && n <= batch_frames && t0 >= 0, NSC_E_INVAL,
              "n %lld (batch of %lld) or t0 out of range", (long long)n, (long long)batch_frames);
  auto mark = [&](int k) -> int {
    if (stage_events && stage_events[k])
      NSC_TRY_HIP(hipEventRecord((hipEvent_t)stage_events[k], (hipStream_t)stream));
    return NSC_OK;
  };
  if (n == 0) {
    if (stats) *stats = nsc_run_stats{0, 0, 0, 0};
    return NSC_OK;
  }
  NSC_REQUIRE(label_out && defer_out, NSC_E_INVAL, "label_out or defer_out is NULL");
  NSC_REQUIRE(!(cfg->ref_mode == NSC_REF_PREV && state == nullptr), NSC_E_STATE,
              "earlier-frame mode needs a state buffer");
  const int64_t pass = batch_cnn_pass(batch_frames, cnn_pass);
  const RunLayout L = run_layout(cfg, cnn->c, batch_frames, pass, true);
  NSC_REQUIRE(ws != nullptr && ((uintptr_t)ws % kAlign) == 0 && ws_bytes >= L.total,
              NSC_E_WORKSPACE, "workspace needs %zu bytes (256-byte aligned), got %zu", L.total,
              ws_bytes);
  const hipStream_t st = (hipStream_t)stream;
  unsigned char* w = static_cast<unsigned char*>(ws);
  if (int rc = run_checked(cfg, cnn->c, nullptr, n, t0, state, w, L, label_out, defer_out,
                           outs ? outs->score : nullptr, outs ? outs->fire : nullptr,
                           outs ? outs->logit : nullptr, pass, st, mark))
    return rc;
  if (int rc = mark(5)) return rc;
  if (stats)
    return run_stats(label_out, defer_out, reinterpret_cast<int32_t*>(w + L.count), n, st, stats);
  return NSC_OK;
}

}  // extern "C"

// ------------------------------------------------------------ camera groups

struct nsc_group {
  int32_t n_cams;
  nsc_cascade_cfg geo;   // camera 0's cfg: the shared geometry and metric
  const nsc_cnn* base;   // camera 0's network: kernel plans and base weights
  int32_t max_delta;     // largest delta of an earlier-frame camera (0: none)
  int32_t blocked;       // some camera scores a blocked grid
  int64_t slot;          // state bytes per camera
  void* dev;             // CamDiff[n_cams], then CamNet[n_cams]
  CamDiff* cams;
  CamNet* nets;
};

namespace nsc {
namespace {

// Workspace of a group run of n frames per camera.
struct GroupLayout {
  size_t sums, fire, dec, idx, count, tiles, logit, scratch, cnn, total;
};

GroupLayout group_layout(const nsc_group* g, int64_t n) {
  GroupLayout L{};
  const int64_t N = (int64_t)g->n_cams * n;
  const size_t cells = (size_t)g->geo.dd_h * g->geo.dd_w * 3;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes, kAlign);
    return at;
  };
  L.sums = take(cells * 4 * (size_t)N);
  L.fire = take((size_t)N);
  L.dec = take((size_t)N);
  L.idx = take((size_t)N * 4);
  L.count = take(64);
  L.tiles = take((size_t)compact_tiles(N) * 4 + 4);
  L.logit = take((size_t)N * 4);
  L.scratch = take(g->max_delta > 0 ? (size_t)g->n_cams * (size_t)g->slot : 0);
  L.cnn = take(cnn_workspace_bytes(g->base->c, N));
  L.total = o;
  return L;
}

bool same_desc(const nsc_cnn_desc& a, const nsc_cnn_desc& b) {
  if (a.n_conv != b.n_conv || a.pool_after_mask != b.pool_after_mask || a.dense != b.dense ||
      a.in_h != b.in_h || a.in_w != b.in_w || a.dtype != b.dtype)
    return false;
  for (int l = 0; l < a.n_conv; ++l)
    if (a.conv_out[l] != b.conv_out[l]) return false;
  return true;
}

}  // namespace
}  // namespace nsc

extern "C" {

int nsc_group_create(const nsc_cascade_cfg* cfgs, const nsc_cnn* const* cnns, int32_t n_cams,
                     nsc_group** out) {
  g_err[0] = 0;
  NSC_REQUIRE(out != nullptr && cfgs != nullptr && cnns != nullptr, NSC_E_INVAL,
              "cfgs, cnns or out is NULL");
  *out = nullptr;
  NSC_REQUIRE(n_cams >= 1 && n_cams <= NSC_MAX_CAMERAS, NSC_E_INVAL, "n_cams %d outside 1..%d",
              n_cams, NSC_MAX_CAMERAS);
  const nsc_cascade_cfg& g0 = cfgs[0];
  int32_t max_delta = 0;
  size_t slot = kAlign;
  for (int32_t c = 0; c < n_cams; ++c) {
    const nsc_cascade_cfg& k = cfgs[c];
    if (int rc = check_cfg(&k)) {
      char msg[512];
      snprintf(msg, sizeof msg, "%s", g_err);
      return fail(rc, "camera %d: %s", c, msg);
    }
    NSC_REQUIRE(k.in_h == g0.in_h && k.in_w == g0.in_w && k.frame_stride == g0.frame_stride &&
                    k.dd_h == g0.dd_h && k.dd_w == g0.dd_w && k.cnn_h == g0.cnn_h &&
                    k.cnn_w == g0.cnn_w,
                NSC_E_INVAL, "camera %d: frame, detector or CNN grid differs from camera 0's", c);
    NSC_REQUIRE(k.metric == g0.metric, NSC_E_INVAL,
                "camera %d: metric %d differs from camera 0's %d", c, k.metric, g0.metric);
    NSC_REQUIRE(k.check_stride <= 1, NSC_E_INVAL,
                "camera %d: frame skipping (check_stride %d) is not available in a group", c,
                k.check_stride);
    if (k.ref_mode == NSC_REF_PREV && k.delta > max_delta) max_delta = k.delta;
    const size_t sb = state_layout_bytes(&k, nullptr, nullptr);
    if (sb > slot) slot = sb;
  }
  slot = align_up(slot, kAlign);
  for (int32_t c = 0; c < n_cams; ++c) {
    NSC_REQUIRE(cnns[c] != nullptr, NSC_E_INVAL, "camera %d: network handle is NULL", c);
    NSC_REQUIRE(same_desc(cnns[c]->c.desc, cnns[0]->c.desc), NSC_E_SHAPE,
                "camera %d: network description differs from camera 0's", c);
  }
  NSC_REQUIRE(cnns[0]->c.desc.in_h == g0.cnn_h && cnns[0]->c.desc.in_w == g0.cnn_w, NSC_E_SHAPE,
              "CNN input %dx%d differs from the configured %dx%d", cnns[0]->c.desc.in_h,
              cnns[0]->c.desc.in_w, g0.cnn_h, g0.cnn_w);
  std::vector<CamDiff> hd((size_t)n_cams);
  std::vector<CamNet> hn((size_t)n_cams);
  for (int32_t c = 0; c < n_cams; ++c) {
    const nsc_cascade_cfg& k = cfgs[c];
    CamDiff d{};
    d.ref_sums = k.ref_sums;
    d.lr_w = k.lr_w;
    d.lr_b = k.lr_b;
    d.delta_diff = k.delta_diff;
    d.ref_mode = k.ref_mode;
    d.delta = k.ref_mode == NSC_REF_PREV ? k.delta : 0;
    d.grid_h = k.grid_h;
    d.grid_w = k.grid_w;
    size_t dec_off = 0;
    state_layout_bytes(&k, nullptr, &dec_off);
    d.dec_off = (int64_t)dec_off;
    hd[c] = d;
    CamNet t{};
    t.woff = static_cast<const unsigned char*>(cnns[c]->c.dev) -
             static_cast<const unsigned char*>(cnns[0]->c.dev);
    t.c_low = k.c_low;
    t.c_high = k.c_high;
    t.b2 = cnns[c]->c.b2;
    hn[c] = t;
  }
  const size_t diff_bytes = align_up(sizeof(CamDiff) * (size_t)n_cams, kAlign);
  const size_t total = diff_bytes + sizeof(CamNet) * (size_t)n_cams;
  void* dev = nullptr;
  if (hipMalloc(&dev, total) != hipSuccess)
    return fail(NSC_E_NOMEM, "hipMalloc of %zu bytes for the group tables failed", total);
  unsigned char* b = static_cast<unsigned char*>(dev);
  if (hipMemcpy(b, hd.data(), sizeof(CamDiff) * (size_t)n_cams, hipMemcpyHostToDevice) !=
          hipSuccess ||
      hipMemcpy(b + diff_bytes, hn.data(), sizeof(CamNet) * (size_t)n_cams,
                hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipFree(dev);
    return fail(NSC_E_HIP, "copying the group tables to the device failed");
  }
  nsc_group* g = new (std::nothrow) nsc_group{};
  if (!g) {
    (void)hipFree(dev);
    return fail(NSC_E_NOMEM, "host allocation of the group failed");
  }
  g->n_cams = n_cams;
  g->geo = g0;
  g->base = cnns[0];
  g->max_delta = max_delta;
  g->blocked = 0;
  for (int32_t c = 0; c < n_cams; ++c)
    if (cfgs[c].grid_h * cfgs[c].grid_w > 1) g->blocked = 1;
  g->slot = (int64_t)slot;
  g->dev = dev;
  g->cams = reinterpret_cast<CamDiff*>(b);
  g->nets = reinterpret_cast<CamNet*>(b + diff_bytes);
  *out = g;
  return NSC_OK;
}

int nsc_group_destroy(nsc_group* g) {
  g_err[0] = 0;
  if (!g) return NSC_OK;
  const hipError_t e = hipFree(g->dev);
  delete g;
  if (e != hipSuccess) return fail(NSC_E_HIP, "hipFree failed: %s", hipGetErrorString(e));
  return NSC_OK;
}

int nsc_group_state_bytes(const nsc_group* g, size_t* bytes, size_t* slot_bytes) {
  g_err[0] = 0;
  NSC_REQUIRE(g != nullptr && bytes != nullptr, NSC_E_INVAL, "group or bytes is NULL");
  *bytes = (size_t)g->n_cams * (size_t)g->slot;
  if (slot_bytes) *slot_bytes = (size_t)g->slot;
  return NSC_OK;
}

int nsc_group_workspace_bytes(const nsc_group* g, int64_t frames_per_cam, size_t* bytes) {
  g_err[0] = 0;
  NSC_REQUIRE(g != nullptr && bytes != nullptr, NSC_E_INVAL, "group or bytes is NULL");
  NSC_REQUIRE(frames_per_cam >= 0 && frames_per_cam <= kMaxFrames / g->n_cams, NSC_E_INVAL,
              "frames_per_cam %lld out of range for %d cameras", (long long)frames_per_cam,
              g->n_cams);
  *bytes = group_layout(g, frames_per_cam).total;
  return NSC_OK;
}

int nsc_group_run(const nsc_group* g, const uint8_t* frames, int64_t n, int64_t t0, void* state,
                  void* ws, size_t ws_bytes, uint8_t* label_out, uint8_t* defer_out,
                  const nsc_frame_outputs* outs, nsc_run_stats* stats, void* const* stage_events,
                  void* stream) {
  g_err[0] = 0;
  NSC_REQUIRE(g != nullptr, NSC_E_INVAL, "group is NULL");
  NSC_REQUIRE(n >= 0 && n <= kMaxFrames / g->n_cams && t0 >= 0, NSC_E_INVAL,
              "n or t0 out of range");
  auto mark = [&](int k) -> int {
    if (stage_events && stage_events[k])
      NSC_TRY_HIP(hipEventRecord((hipEvent_t)stage_events[k], (hipStream_t)stream));
    return NSC_OK;
  };
  const int64_t N = (int64_t)g->n_cams * n;
  if (n == 0) {
    if (stats) *stats = nsc_run_stats{0, 0, 0, 0};
    return NSC_OK;
  }
  NSC_REQUIRE(frames && label_out && defer_out, NSC_E_INVAL,
              "frames, label_out or defer_out is NULL");
  NSC_REQUIRE(!(g->max_delta > 0 && state == nullptr), NSC_E_STATE,
              "a camera compares with earlier frames: the group needs a state buffer");
  const GroupLayout L = group_layout(g, n);
  NSC_REQUIRE(ws != nullptr && ((uintptr_t)ws % kAlign) == 0 && ws_bytes >= L.total,
              NSC_E_WORKSPACE, "workspace needs %zu bytes (256-byte aligned), got %zu", L.total,
              ws_bytes);
  const nsc_cascade_cfg* cfg = &g->geo;
  const Cnn& c = g->base->c;
  const hipStream_t st = (hipStream_t)stream;
  unsigned char* w = static_cast<unsigned char*>(ws);
  int32_t* sums = reinterpret_cast<int32_t*>(w + L.sums);
  uint8_t* fire = outs && outs->fire ? outs->fire : w + L.fire;
  uint8_t* dec = w + L.dec;
  int32_t* idx = reinterpret_cast<int32_t*>(w + L.idx);
  int32_t* count = reinterpret_cast<int32_t*>(w + L.count);
  unsigned char* st_bytes = static_cast<unsigned char*>(state);
  const int64_t cells = (int64_t)cfg->dd_h * cfg->dd_w * 3;
  const double den = (double)nsc_area_den(cfg->in_h, cfg->in_w, cfg->dd_h, cfg->dd_w);

  // 1: area sums of every camera's frames (one video of n_cams * n frames)
  if (int rc = mark(0)) return rc;
  AreaPlan ap;
  if (int rc = make_area_plan(cfg->in_h, cfg->in_w, cfg->frame_stride, frames, cfg->dd_h,
                              cfg->dd_w, N, &ap))
    return rc;
  if (int rc = launch_area_sums(ap, frames, cfg->frame_stride, N, sums, st)) return rc;
  if (int rc = mark(1)) return rc;
  // 2: detector, each frame with its camera's settings
  {
    DiffArgs a{};
    a.sums = sums;
    a.den = den;
    a.den2 = den * den;
    a.metric = cfg->metric;
    a.n = N;
    a.t0 = t0;
    a.dd_h = cfg->dd_h;
    a.dd_w = cfg->dd_w;
    a.score = outs ? outs->score : nullptr;
    a.fire = fire;
    a.cams = g->cams;
    a.cams_blocked = g->blocked;
    a.per_cam = n;
    a.state = st_bytes;
    a.state_stride = g->slot;
    if (int rc = launch_diff(a, st)) return rc;
  }
  if (int rc = mark(2)) return rc;
  // 3: compaction over all cameras (survivors in camera-major frame order)
  if (int rc = launch_compact(fire, N, idx, count, reinterpret_cast<int32_t*>(w + L.tiles), st))
    return rc;
  if (int rc = mark(3)) return rc;
  // 4: CNN, every survivor with its camera's network and thresholds
  if (outs && outs->logit)
    if (int rc = launch_fill_nan(outs->logit, N, st)) return rc;
  CnnRunArgs r{};
  r.sums = sums;
  r.sums_h = cfg->dd_h;
  r.sums_w = cfg->dd_w;
  r.fy = cfg->dd_h / cfg->cnn_h;
  r.fx = cfg->dd_w / cfg->cnn_w;
  r.den_c = den * r.fy * r.fx;
  r.idx = idx;
  r.count = count;
  r.max_count = N;
  r.logit = reinterpret_cast<float*>(w + L.logit);
  r.prob = nullptr;
  r.dec = dec;
  r.frame_logit = outs ? outs->logit : nullptr;
  r.nets = g->nets;
  r.per_cam = n;
  r.n_nets = g->n_cams;
  if (int rc = run_cnn(c, r, w + L.cnn, L.total - L.cnn, st)) return rc;
  if (int rc = mark(4)) return rc;
  // 5: decisions of the frames that did not fire, then the cameras' state
  if (int rc = launch_group_resolve(g->cams, g->n_cams, fire, dec, n, t0, st_bytes, g->slot,
                                    label_out, defer_out, st))
    return rc;
  if (g->max_delta > 0)
    if (int rc = launch_group_state(g->cams, g->n_cams, g->max_delta, sums, label_out, defer_out,
                                    n, cells, st_bytes, g->slot, w + L.scratch, st))
      return rc;
  if (int rc = mark(5)) return rc;
  if (stats) {
    std::vector<uint8_t> hl(N), hdf(N);
    int32_t hc = 0;
    NSC_TRY_HIP(hipMemcpyAsync(hl.data(), label_out, N, hipMemcpyDeviceToHost, st));
    NSC_TRY_HIP(hipMemcpyAsync(hdf.data(), defer_out, N, hipMemcpyDeviceToHost, st));
    NSC_TRY_HIP(hipMemcpyAsync(&hc, count, 4, hipMemcpyDeviceToHost, st));
    NSC_TRY_HIP(hipStreamSynchronize(st));
    nsc_run_stats rs{N, hc, 0, 0};
    for (int64_t i = 0; i < N; ++i) {
      rs.positive += hl[i] && !hdf[i];
      rs.deferred += hdf[i];
    }
    *stats = rs;
  }
  return NSC_OK;
}

}  // extern "C"
