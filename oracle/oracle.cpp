// Oracle of the NoScope cascade filter: a plain, slow, single-threaded fp64
// CPU implementation, written from the paper.
//
// TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
// benchmark's CPU-baseline leg may load or call this library; the product
// path never does.  It shares no code, header or table with the HIP library.
//
// What it computes, step by step (paper section in brackets):
//   1. area sums: frames are resized before the models [Sec. 7]; read as the
//      exact area average of the piecewise-constant image, kept as integer
//      sums S with a common integer denominator den (value = S / den);
//   2. difference detector [Sec. 5]: MSE (or one of the alternatives the
//      paper names: SAD, NRMSE, PSNR) against the frame delta earlier or a
//      fixed reference image, over the whole image or per grid block weighed
//      by a logistic regression; it fires when the metric is higher than
//      delta_diff [Sec. 6.2];
//   3. the frames that fire, in ascending order [Sec. 7, batching];
//   4. specialized CNN [Sec. 4]: pre-processing to [-1, 1] [Sec. 7], conv3x3
//      + ReLU (+ 2x2 max-pool) layers, a ReLU dense layer and one output
//      logit, confidence c = sigmoid(logit);
//   5. decision [Sec. 3, Sec. 4]: c below c_low -> no object, above c_high
//      -> object, otherwise defer to the reference network; a frame on which
//      the earlier-frame detector does not fire reuses the compared frame's
//      output [Sec. 5].
//   6. threshold search of the cost-based optimizer [Sec. 6.2 cost model,
//      Sec. 6.3 step 3]: on logged per-frame detector scores, specialized-
//      CNN confidences and reference labels, the cheapest delta_diff /
//      c_low / c_high within false positive and false negative targets.
// Readings where the paper is silent (rounding points of bf16 networks,
// forced firing of the first delta frames, ties) are listed in the design
// notes; each is marked "reading" below.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <vector>

namespace {

int64_t gcd64(int64_t a, int64_t b) {
  while (b) {
    int64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

// Overlap of output cell o = [o*p, (o+1)*p) with input pixel i = [i*q, (i+1)*q),
// in units where one input pixel has length q = n_out/g and one output cell
// length p = n_in/g.
std::vector<int64_t> overlap_table(int n_in, int n_out) {
  int64_t g = gcd64(n_in, n_out);
  int64_t p = n_in / g, q = n_out / g;
  std::vector<int64_t> w((size_t)n_in * n_out, 0);
  for (int o = 0; o < n_out; ++o) {
    int64_t a0 = (int64_t)o * p, a1 = a0 + p;
    for (int i = 0; i < n_in; ++i) {
      int64_t b0 = (int64_t)i * q, b1 = b0 + q;
      int64_t lo = a0 > b0 ? a0 : b0;
      int64_t hi = a1 < b1 ? a1 : b1;
      w[(size_t)o * n_in + i] = hi > lo ? hi - lo : 0;
    }
  }
  return w;
}

// Round to the nearest bfloat16 value (8 significant bits), ties to even,
// from the definition: scale the significand to [128, 256) and round.
double round_bf16(double v) {
  if (v == 0.0 || !std::isfinite(v)) return v;
  int e;
  double m = std::frexp(v, &e);          // v = m * 2^e, 0.5 <= |m| < 1
  double r = std::nearbyint(m * 256.0);  // default rounding mode: ties to even
  return std::ldexp(r, e - 8);
}

struct Net {
  int n_conv;
  int cout[8];
  int pool[8];
  int dense;
  int in_h, in_w;
  bool bf16;
  // weights (fp64 copies of the fp32 blob)
  std::vector<std::vector<double>> cw, cb;
  std::vector<double> w1, b1, w2;
  double b2;
  int flat;
};

}  // namespace

extern "C" {

// ---------------------------------------------------------------- area sums

// Integer overlap weights w[o*n_in + i]; returns their per-row sum p.
int64_t oracle_area_weights(int32_t n_in, int32_t n_out, int64_t* w_out) {
  std::vector<int64_t> w = overlap_table(n_in, n_out);
  std::memcpy(w_out, w.data(), w.size() * sizeof(int64_t));
  int64_t s = 0;
  for (int i = 0; i < n_in; ++i) s += w[i];
  return s;
}

// Common denominator of the area sums: (row weight sum) * (column weight sum).
int64_t oracle_area_den(int32_t H, int32_t W, int32_t Ho, int32_t Wo) {
  std::vector<int64_t> wy = overlap_table(H, Ho), wx = overlap_table(W, Wo);
  int64_t sy = 0, sx = 0;
  for (int j = 0; j < H; ++j) sy += wy[j];
  for (int i = 0; i < W; ++i) sx += wx[i];
  return sy * sx;
}

// S[Y][X][c] = sum_j sum_i wy[Y][j] * wx[X][i] * F[j][i][c]   (frame: [H][W][3] uint8)
// The sum runs over the support of each output cell (the input indices whose
// overlap weight is non-zero), found by scanning the weight table.
void oracle_area_sums(const uint8_t* frame, int32_t H, int32_t W, int32_t Ho, int32_t Wo,
                      int64_t* S) {
  std::vector<int64_t> wy = overlap_table(H, Ho), wx = overlap_table(W, Wo);
  auto support = [](const std::vector<int64_t>& w, int n_in, int o, int* lo, int* hi) {
    *lo = n_in;
    *hi = 0;
    for (int i = 0; i < n_in; ++i)
      if (w[(size_t)o * n_in + i] != 0) {
        if (i < *lo) *lo = i;
        *hi = i + 1;
      }
  };
  for (int Y = 0; Y < Ho; ++Y) {
    int j0, j1;
    support(wy, H, Y, &j0, &j1);
    for (int X = 0; X < Wo; ++X) {
      int i0, i1;
      support(wx, W, X, &i0, &i1);
      for (int c = 0; c < 3; ++c) {
        int64_t s = 0;
        for (int j = j0; j < j1; ++j) {
          int64_t a = wy[(size_t)Y * H + j];
          for (int i = i0; i < i1; ++i) {
            int64_t b = wx[(size_t)X * W + i];
            s += a * b * (int64_t)frame[((size_t)j * W + i) * 3 + c];
          }
        }
        S[((size_t)Y * Wo + X) * 3 + c] = s;
      }
    }
  }
}

// ------------------------------------------------------- difference detector

}  // extern "C"

namespace {

// Distance between two area-sum images a (the frame) and b (the frame it is
// compared with), both holding N values with denominator den, i.e. a / den and
// b / den on the 0..255 scale.  Sec. 5 uses the MSE and names three
// alternatives that were tried: normalized root mean square error, peak
// signal-to-noise ratio and the sum of absolute differences.  Readings:
//   MSE   = sum ((a - b) / den)^2 / N;
//   SAD   = sum |a - b| / den, the sum over all N values;
//   NRMSE = sqrt(sum (a - b)^2 / sum b^2), the error's Euclidean norm relative
//           to the compared image's (den cancels): 0 when both sums are 0,
//           +inf when only the compared image is all zero;
//   PSNR  = 10 log10(255^2 / MSE), a similarity; the metric reported is its
//           negation, so that for every metric a larger value means "more
//           different" and the detector fires above delta_diff (with PSNR:
//           iff PSNR < -delta_diff); identical images give -inf.
// The integer sums are exact; each metric is one fp64 expression of them.
enum { METRIC_MSE = 0, METRIC_SAD = 1, METRIC_NRMSE = 2, METRIC_PSNR = 3 };

double metric_of(int32_t metric, const std::vector<int64_t>& a, const std::vector<int64_t>& b,
                 int64_t den, int64_t* E_out) {
  const int64_t N = (int64_t)a.size();
  int64_t E = 0, A = 0, R = 0;  // sum (a-b)^2, sum |a-b|, sum b^2
  for (int64_t k = 0; k < N; ++k) {
    const int64_t d = a[k] - b[k];
    E += d * d;
    A += d < 0 ? -d : d;
    R += b[k] * b[k];
  }
  if (E_out) *E_out = E;
  const double mse = (double)E / ((double)den * (double)den * (double)N);
  switch (metric) {
    case METRIC_MSE:
      return mse;
    case METRIC_SAD:
      return (double)A / (double)den;
    case METRIC_NRMSE:
      if (R == 0) return E == 0 ? 0.0 : std::numeric_limits<double>::infinity();
      return std::sqrt((double)E / (double)R);
    case METRIC_PSNR:
      return -(10.0 * std::log10(65025.0 / mse));
  }
  return std::numeric_limits<double>::quiet_NaN();
}

// The values of block k = by*Gw + bx of an [Ho][Wo][3] image: rows
// [floor(by*Ho/Gh), floor((by+1)*Ho/Gh)), columns likewise.
std::vector<int64_t> block_values(const int64_t* a, int32_t Ho, int32_t Wo, int32_t Gh, int32_t Gw,
                                  int by, int bx) {
  (void)Ho;
  const int y0 = (int)((int64_t)by * Ho / Gh), y1 = (int)((int64_t)(by + 1) * Ho / Gh);
  const int x0 = (int)((int64_t)bx * Wo / Gw), x1 = (int)((int64_t)(bx + 1) * Wo / Gw);
  std::vector<int64_t> v;
  for (int y = y0; y < y1; ++y)
    for (int x = x0; x < x1; ++x)
      for (int c = 0; c < 3; ++c) v.push_back(a[((size_t)y * Wo + x) * 3 + c]);
  return v;
}

}  // namespace

extern "C" {

// Whole-image metric (global detector, Sec. 5).  E_out (nullable) receives
// sum (a - b)^2 exactly.
double oracle_global_metric(int32_t metric, const int64_t* a, const int64_t* b, int32_t Ho,
                            int32_t Wo, int64_t den, int64_t* E_out) {
  const size_t N = (size_t)Ho * Wo * 3;
  return metric_of(metric, std::vector<int64_t>(a, a + N), std::vector<int64_t>(b, b + N), den,
                   E_out);
}

// Global MSE: mean over Ho*Wo*3 values of ((a - b) / den)^2 on the 0..255
// scale.  E_out receives sum (a - b)^2 exactly.
double oracle_global_mse(const int64_t* a, const int64_t* b, int32_t Ho, int32_t Wo, int64_t den,
                         int64_t* E_out) {
  return oracle_global_metric(METRIC_MSE, a, b, Ho, Wo, den, E_out);
}

// Blocked detector (Sec. 5): the metric m_k of every grid block k, weighed by
// a logistic regression: score = bias + sum_k w_k m_k, added in block order.
// Reading: with the PSNR metric an unchanged block has m_k = -inf and the sum
// is undefined, so the blocked detector takes MSE, SAD and NRMSE only (NaN
// returned for PSNR).
double oracle_blocked_metric(int32_t metric, const int64_t* a, const int64_t* b, int32_t Ho,
                             int32_t Wo, int64_t den, int32_t Gh, int32_t Gw, const float* w,
                             double bias, double* m_out) {
  if (metric == METRIC_PSNR) return std::numeric_limits<double>::quiet_NaN();
  double z = bias;
  for (int by = 0; by < Gh; ++by)
    for (int bx = 0; bx < Gw; ++bx) {
      const double m = metric_of(metric, block_values(a, Ho, Wo, Gh, Gw, by, bx),
                                 block_values(b, Ho, Wo, Gh, Gw, by, bx), den, nullptr);
      if (m_out) m_out[by * Gw + bx] = m;
      z += (double)w[by * Gw + bx] * m;
    }
  return z;
}

double oracle_blocked_score(const int64_t* a, const int64_t* b, int32_t Ho, int32_t Wo,
                            int64_t den, int32_t Gh, int32_t Gw, const float* w, double bias,
                            double* m_out) {
  return oracle_blocked_metric(METRIC_MSE, a, b, Ho, Wo, den, Gh, Gw, w, bias, m_out);
}

// ------------------------------------------------------------ specialized CNN

struct oracle_cnn_desc {
  int32_t n_conv;
  int32_t conv_out[8];
  int32_t pool_after[8];
  int32_t dense;
  int32_t in_h, in_w;
  int32_t bf16;
};

double oracle_round_bf16(double v) { return round_bf16(v); }

static bool load_net(const oracle_cnn_desc* d, const float* blob, Net* net) {
  if (d->n_conv < 1 || d->n_conv > 8) return false;
  net->n_conv = d->n_conv;
  net->dense = d->dense;
  net->in_h = d->in_h;
  net->in_w = d->in_w;
  net->bf16 = d->bf16 != 0;
  const float* p = blob;
  int cin = 3, h = d->in_h, w = d->in_w;
  for (int l = 0; l < d->n_conv; ++l) {
    net->cout[l] = d->conv_out[l];
    net->pool[l] = d->pool_after[l];
    size_t nw = (size_t)d->conv_out[l] * cin * 9;
    net->cw.emplace_back(p, p + nw);
    p += nw;
    net->cb.emplace_back(p, p + d->conv_out[l]);
    p += d->conv_out[l];
    cin = d->conv_out[l];
    if (d->pool_after[l]) {
      h /= 2;
      w /= 2;
    }
  }
  net->flat = cin * h * w;
  net->w1.assign(p, p + (size_t)d->dense * net->flat);
  p += (size_t)d->dense * net->flat;
  net->b1.assign(p, p + d->dense);
  p += d->dense;
  net->w2.assign(p, p + d->dense);
  p += d->dense;
  net->b2 = *p;
  return true;
}

// Number of floats in the canonical weight blob of a network.
int64_t oracle_cnn_blob_floats(const oracle_cnn_desc* d) {
  int64_t n = 0;
  int cin = 3, h = d->in_h, w = d->in_w;
  for (int l = 0; l < d->n_conv; ++l) {
    n += (int64_t)d->conv_out[l] * cin * 9 + d->conv_out[l];
    cin = d->conv_out[l];
    if (d->pool_after[l]) {
      h /= 2;
      w /= 2;
    }
  }
  int64_t flat = (int64_t)cin * h * w;
  return n + d->dense * flat + d->dense + d->dense + 1;
}

// Direct convolution, 3x3, stride 1, zero padding 1, input/output [C][H][W].
void oracle_conv3x3(const double* in, int32_t cin, int32_t h, int32_t w, const double* wt,
                    const double* bias, int32_t cout, double* out) {
  for (int o = 0; o < cout; ++o)
    for (int y = 0; y < h; ++y)
      for (int x = 0; x < w; ++x) {
        double s = bias[o];
        for (int c = 0; c < cin; ++c)
          for (int dy = 0; dy < 3; ++dy)
            for (int dx = 0; dx < 3; ++dx) {
              int yy = y + dy - 1, xx = x + dx - 1;
              if (yy < 0 || yy >= h || xx < 0 || xx >= w) continue;
              s += wt[(((size_t)o * cin + c) * 3 + dy) * 3 + dx] * in[((size_t)c * h + yy) * w + xx];
            }
        out[((size_t)o * h + y) * w + x] = s;
      }
}

// Evaluates the network on one frame's area sums S [in_h][in_w][3] with
// denominator den; returns the output logit.  For bf16 networks (reading: the
// weights are bf16 values and the pre-processed input is rounded to bf16; the
// activations of later layers are not rounded), everything after the input
// rounding is fp64 arithmetic on those values.  features_out (nullable)
// receives the flattened input of the dense layer in (c, y, x) order.
// scale_out (nullable) receives the logit's scale |b2| + sum_j |w2_j h_j|: the
// magnitude of the terms the output layer adds up, against which the logit's
// error is measured (a logit that is a small difference of large terms has no
// finer relative precision).
double oracle_cnn_logit(const oracle_cnn_desc* d, const float* blob, const int64_t* S, int64_t den,
                        double* features_out, double* scale_out) {
  Net net;
  if (!load_net(d, blob, &net)) return std::numeric_limits<double>::quiet_NaN();
  auto rnd_input = [&](double v) { return net.bf16 ? round_bf16(v) : v; };
  int c = 3, h = net.in_h, w = net.in_w;
  // pre-processing [Sec. 7]: area average in [0, 255] mapped to [-1, 1]
  std::vector<double> act((size_t)c * h * w);
  for (int ch = 0; ch < 3; ++ch)
    for (int y = 0; y < h; ++y)
      for (int x = 0; x < w; ++x) {
        double v = (double)S[((size_t)y * w + x) * 3 + ch] / (double)den;
        act[((size_t)ch * h + y) * w + x] = rnd_input(v / 127.5 - 1.0);
      }
  for (int l = 0; l < net.n_conv; ++l) {
    int co = net.cout[l];
    std::vector<double> out((size_t)co * h * w);
    oracle_conv3x3(act.data(), c, h, w, net.cw[l].data(), net.cb[l].data(), co, out.data());
    for (double& v : out) v = v > 0.0 ? v : 0.0;
    if (net.pool[l]) {
      int ph = h / 2, pw = w / 2;
      std::vector<double> pooled((size_t)co * ph * pw);
      for (int o = 0; o < co; ++o)
        for (int y = 0; y < ph; ++y)
          for (int x = 0; x < pw; ++x) {
            double m = out[((size_t)o * h + 2 * y) * w + 2 * x];
            for (int dy = 0; dy < 2; ++dy)
              for (int dx = 0; dx < 2; ++dx) {
                double v = out[((size_t)o * h + 2 * y + dy) * w + 2 * x + dx];
                if (v > m) m = v;
              }
            pooled[((size_t)o * ph + y) * pw + x] = m;
          }
      out.swap(pooled);
      h = ph;
      w = pw;
    }
    act.swap(out);
    c = co;
  }
  if (features_out) std::memcpy(features_out, act.data(), act.size() * sizeof(double));
  double z = net.b2;
  double scale = std::fabs(net.b2);
  for (int j = 0; j < net.dense; ++j) {
    double s = net.b1[j];
    for (int k = 0; k < net.flat; ++k) s += net.w1[(size_t)j * net.flat + k] * act[k];
    double hj = s > 0.0 ? s : 0.0;
    z += net.w2[j] * hj;
    scale += std::fabs(net.w2[j] * hj);
  }
  if (scale_out) *scale_out = scale;
  return z;
}

double oracle_sigmoid(double z) { return 1.0 / (1.0 + std::exp(-z)); }

// Decision on the specialized model's confidence p (Sec. 3, Sec. 4):
// p < c_low -> label 0; p > c_high -> label 1; otherwise defer (label 0).
// Returns label | (defer << 1).
int32_t oracle_decide(double p, double c_low, double c_high) {
  if (p < c_low) return 0;
  if (p > c_high) return 1;
  return 2;
}

// ---------------------------------------------------------------- cascade

struct oracle_cfg {
  int32_t H, W;           // raw frame size
  int32_t Ho, Wo;         // difference-detector grid
  int32_t Hc, Wc;         // CNN input grid
  int32_t ref_mode;       // 0: frame t - delta; 1: fixed reference image
  int32_t delta;
  int32_t Gh, Gw;         // 1x1: global MSE; otherwise blocked
  const float* lr_w;      // Gh*Gw logistic-regression weights (blocked)
  double lr_b;
  const int64_t* ref_sums;  // fixed reference image area sums, Ho*Wo*3 (mode 1)
  double delta_diff;
  double c_low, c_high;
  int32_t check_stride;   // frame skipping: check frames t with t mod s = 0 (0 or 1: all)
  int32_t metric;         // 0 MSE, 1 SAD, 2 NRMSE, 3 -PSNR (see metric_of)
};

// Number of earlier frames whose sums and decisions a chunked run carries:
// delta (mode 0) for the compared frame, s - 1 for the last checked frame.
int64_t oracle_history(const oracle_cfg* cfg) {
  const int64_t s = cfg->check_stride > 1 ? cfg->check_stride : 1;
  const int64_t d = cfg->ref_mode == 0 ? cfg->delta : 0;
  return d > s - 1 ? d : s - 1;
}

// Runs the cascade on frames [t0, t0 + n) (frames: n x H x W x 3 uint8).
// state_S / state_dec: area sums (Ho*Wo*3 each) and decisions of the
// oracle_history() frames before t0 (needed when t0 > 0 and the history is
// not empty); the same of the frames before t0 + n is written to state_S_out /
// state_dec_out (nullable).  Outputs per frame: score (+inf for a forced
// frame, NaN for a frame that is not checked), fire, logit, prob and the
// logit's scale (NaN where the CNN did not run), label, defer.
// Frame skipping (Sec. 5, the check interval t_skip, here s frames): only
// frames with t mod s = 0 run the difference detector (and, if it fires, the
// CNN).  Readings: a frame that is not checked keeps the output of the last
// checked frame, floor(t / s) * s; with the earlier-frame detector delta is a
// multiple of s, so the compared frame t - delta is a checked one.
// Reading: checked frames with absolute index t < delta have no frame
// t - delta and always fire.  Returns the number of frames that fired, or -1
// on bad input.
int64_t oracle_cascade(const oracle_cfg* cfg, const oracle_cnn_desc* net, const float* blob,
                       const uint8_t* frames, int64_t n, int64_t t0, const int64_t* state_S,
                       const uint8_t* state_dec, double* score, uint8_t* fire, double* logit,
                       double* prob, double* lscale, uint8_t* label, uint8_t* defer,
                       int64_t* state_S_out, uint8_t* state_dec_out) {
  if (!cfg || !net || n < 0 || t0 < 0) return -1;
  const int64_t cells = (int64_t)cfg->Ho * cfg->Wo * 3;
  const int64_t den = oracle_area_den(cfg->H, cfg->W, cfg->Ho, cfg->Wo);
  const int64_t den_c = oracle_area_den(cfg->H, cfg->W, cfg->Hc, cfg->Wc);
  const int64_t fb = (int64_t)cfg->H * cfg->W * 3;
  const int64_t s = cfg->check_stride > 1 ? cfg->check_stride : 1;
  if (cfg->check_stride < 0) return -1;
  if (cfg->ref_mode == 0 && cfg->delta < 1) return -1;
  if (cfg->ref_mode == 0 && cfg->delta % s != 0) return -1;
  if (cfg->metric < METRIC_MSE || cfg->metric > METRIC_PSNR) return -1;
  if (cfg->metric == METRIC_PSNR && cfg->Gh * cfg->Gw > 1) return -1;
  const int64_t D = oracle_history(cfg);  // history frames before t0
  if (D > 0 && t0 > 0 && (!state_S || !state_dec)) return -1;
  // area sums of every frame of the window (history first)
  std::vector<int64_t> S((size_t)(D + n) * cells);
  for (int64_t k = 0; k < D; ++k) {
    if (t0 > 0) std::memcpy(&S[(size_t)k * cells], state_S + k * cells, cells * sizeof(int64_t));
  }
  for (int64_t k = 0; k < n; ++k)
    oracle_area_sums(frames + k * fb, cfg->H, cfg->W, cfg->Ho, cfg->Wo, &S[(size_t)(D + k) * cells]);
  std::vector<uint8_t> dec((size_t)(D + n), 0);
  for (int64_t k = 0; k < D; ++k) dec[k] = (t0 > 0) ? state_dec[k] : 0;
  const bool blocked = cfg->Gh * cfg->Gw > 1;
  std::vector<int64_t> Sc((size_t)cfg->Hc * cfg->Wc * 3);
  int64_t fired = 0;
  const double nan = std::numeric_limits<double>::quiet_NaN();
  for (int64_t k = 0; k < n; ++k) {
    const int64_t t = t0 + k;
    if (t % s != 0) {  // not checked: the output of the last checked frame
      const uint8_t d = dec[(size_t)(D + k - t % s)];
      dec[(size_t)(D + k)] = d;
      if (score) score[k] = nan;
      if (fire) fire[k] = 0;
      if (logit) logit[k] = nan;
      if (prob) prob[k] = nan;
      if (lscale) lscale[k] = nan;
      if (label) label[k] = d & 1;
      if (defer) defer[k] = (d >> 1) & 1;
      continue;
    }
    const int64_t* cur = &S[(size_t)(D + k) * cells];
    double sc;
    const bool forced = cfg->ref_mode == 0 && t < cfg->delta;
    if (forced) {
      sc = std::numeric_limits<double>::infinity();
    } else {
      const int64_t* ref =
          cfg->ref_mode == 0 ? &S[(size_t)(D + k - cfg->delta) * cells] : cfg->ref_sums;
      sc = blocked ? oracle_blocked_metric(cfg->metric, cur, ref, cfg->Ho, cfg->Wo, den, cfg->Gh,
                                           cfg->Gw, cfg->lr_w, cfg->lr_b, nullptr)
                   : oracle_global_metric(cfg->metric, cur, ref, cfg->Ho, cfg->Wo, den, nullptr);
    }
    const bool f = forced || sc > cfg->delta_diff;
    if (score) score[k] = sc;
    if (fire) fire[k] = f ? 1 : 0;
    uint8_t d;
    if (f) {
      ++fired;
      oracle_area_sums(frames + k * fb, cfg->H, cfg->W, cfg->Hc, cfg->Wc, Sc.data());
      double sc_z = 0.0;
      double z = oracle_cnn_logit(net, blob, Sc.data(), den_c, nullptr, &sc_z);
      double p = oracle_sigmoid(z);
      if (logit) logit[k] = z;
      if (lscale) lscale[k] = sc_z;
      if (prob) prob[k] = p;
      d = (uint8_t)oracle_decide(p, cfg->c_low, cfg->c_high);
    } else {
      if (logit) logit[k] = std::numeric_limits<double>::quiet_NaN();
      if (prob) prob[k] = std::numeric_limits<double>::quiet_NaN();
      if (lscale) lscale[k] = std::numeric_limits<double>::quiet_NaN();
      d = cfg->ref_mode == 0 ? dec[(size_t)(D + k - cfg->delta)] : 0;  // the compared frame's output
    }
    dec[(size_t)(D + k)] = d;
    if (label) label[k] = d & 1;
    if (defer) defer[k] = (d >> 1) & 1;
  }
  for (int64_t k = 0; k < D; ++k) {
    if (state_S_out)
      std::memcpy(state_S_out + k * cells, &S[(size_t)(n + k) * cells], cells * sizeof(int64_t));
    if (state_dec_out) state_dec_out[k] = dec[(size_t)(n + k)];
  }
  return fired;
}


// Threshold search of the cost-based optimizer [Sec. 6.3, step 3] with its
// cost model [Sec. 6.2], on logged scores of every frame of an evaluation
// video: the detector score s[t] (+inf for a frame that always fires), the
// specialized CNN's confidence c[t], and the reference label y[t] (1 = the
// object is present).  For each candidate threshold delta[k]:
//   - the frames that fire are a prefix of the frames sorted by decreasing
//     score; a frame that does not fire takes the label of the frame it is
//     compared with (reading: its reference label, frame t - delta for the
//     earlier-frame detector, "no object" for a fixed reference image), so
//     the detector's false negatives / positives are the non-firing frames
//     whose own label is 1 / 0 and the copied label 0 / 1;
//   - on the fired frames sorted by confidence, c_low moves up until the
//     combined false negative rate would reach FN*, and c_high down until
//     the combined false positive rate would reach FP* (reading: rates are
//     counts over the frames with / without the object, and must stay
//     strictly below the targets; a frame at c_low or c_high is deferred,
//     and a deferred frame gets the reference label; c_high >= c_low);
//   - cost per frame = f_s T_MSE + f_s f_m T_SNN + f_s f_m f_c T_Full with
//     f_s = 1 (every frame checked), f_m = fired / n, f_c = deferred / fired.
// The candidate is feasible when the detector's errors alone stay below the
// targets.  Returns the index of the cheapest feasible candidate (the first
// on ties), or -1 when none is feasible or the input is invalid.
struct oracle_sweep_cfg {
  int32_t ref_mode;  // 0: earlier frame, 1: fixed reference image
  int32_t delta;     // frames back (earlier-frame detector)
  double fp_target, fn_target;
  double t_mse, t_snn, t_full;  // per-frame costs
};

struct oracle_sweep_row {
  double delta, c_low, c_high, f_m, f_c, cost;
  int64_t fired, deferred, fn_dd, fp_dd, fn_cnn, fp_cnn, positives, negatives;
  int32_t feasible, pad;
};

int32_t oracle_threshold_sweep(const oracle_sweep_cfg* cfg, const double* score, const float* conf,
                               const uint8_t* truth, int64_t n, const double* deltas, int32_t n_t,
                               oracle_sweep_row* rows) {
  if (!cfg || n < 1 || n_t < 1 || (cfg->ref_mode == 0 && cfg->delta < 1)) return -1;
  const double inf = std::numeric_limits<double>::infinity();
  int64_t positives = 0;
  for (int64_t t = 0; t < n; ++t) positives += truth[t] ? 1 : 0;
  const int64_t negatives = n - positives;
  // error budgets: count < target x (frames with / without the object); an
  // empty class leaves nothing to get wrong
  const double fn_budget = positives ? cfg->fn_target * (double)positives : inf;
  const double fp_budget = negatives ? cfg->fp_target * (double)negatives : inf;
  // L_D: frames in decreasing order of score (+inf first), and the detector
  // errors of each frame if it does not fire
  std::vector<int64_t> order((size_t)n);
  for (int64_t t = 0; t < n; ++t) order[(size_t)t] = t;
  std::stable_sort(order.begin(), order.end(),
                   [&](int64_t a, int64_t b) { return score[a] > score[b]; });
  std::vector<int64_t> fn_suffix((size_t)n + 1, 0), fp_suffix((size_t)n + 1, 0);
  for (int64_t i = n - 1; i >= 0; --i) {
    const int64_t t = order[(size_t)i];
    const int ref = cfg->ref_mode == 0 ? (t >= cfg->delta ? truth[t - cfg->delta] : 0) : 0;
    fn_suffix[(size_t)i] = fn_suffix[(size_t)i + 1] + (truth[t] && !ref ? 1 : 0);
    fp_suffix[(size_t)i] = fp_suffix[(size_t)i + 1] + (!truth[t] && ref ? 1 : 0);
  }
  int32_t best = -1;
  for (int32_t k = 0; k < n_t; ++k) {
    const double d = deltas[k];
    // prefix of L_D that fires: score above the threshold, or +inf (forced)
    int64_t fired = 0;
    while (fired < n && (score[order[(size_t)fired]] == inf || score[order[(size_t)fired]] > d))
      ++fired;
    oracle_sweep_row r{};
    r.delta = d;
    r.fired = fired;
    r.fn_dd = fn_suffix[(size_t)fired];
    r.fp_dd = fp_suffix[(size_t)fired];
    r.positives = positives;
    r.negatives = negatives;
    r.feasible = (double)r.fn_dd < fn_budget && (double)r.fp_dd < fp_budget ? 1 : 0;
    // the fired frames by confidence
    std::vector<int64_t> f(order.begin(), order.begin() + fired);
    std::stable_sort(f.begin(), f.end(), [&](int64_t a, int64_t b) { return conf[a] < conf[b]; });
    // c_low: up the list; the frames below c_low are labelled 0, and each with
    // the object is a false negative.  c_low stops at the first confidence
    // whose frames would bring the false negatives to the budget.
    double c_low = 1.0;
    {
      int64_t fn = r.fn_dd;
      for (size_t i = 0; i < f.size();) {
        size_t j = i;
        int64_t add = 0;
        while (j < f.size() && conf[f[j]] == conf[f[i]]) add += truth[f[j++]] ? 1 : 0;
        if ((double)(fn + add) >= fn_budget) {
          c_low = (double)conf[f[i]];
          break;
        }
        fn += add;
        i = j;
      }
      if (c_low > 1.0) c_low = 1.0;
    }
    // c_high: down the list; the frames above c_high are labelled 1
    double c_high = 0.0;
    {
      int64_t fp = r.fp_dd;
      for (size_t i = f.size(); i > 0;) {
        size_t j = i;
        int64_t add = 0;
        while (j > 0 && conf[f[j - 1]] == conf[f[i - 1]]) add += truth[f[--j]] ? 0 : 1;
        if ((double)(fp + add) >= fp_budget) {
          c_high = (double)conf[f[i - 1]];
          break;
        }
        fp += add;
        i = j;
      }
      if (c_high < c_low) c_high = c_low;
    }
    if (!r.feasible) {  // no thresholds meet the targets: report the extremes
      c_low = 0.0;
      c_high = 1.0;
    }
    r.c_low = c_low;
    r.c_high = c_high;
    for (int64_t t : f) {
      const double c = (double)conf[t];
      if (c < c_low) {
        r.fn_cnn += truth[t] ? 1 : 0;
      } else if (c > c_high) {
        r.fp_cnn += truth[t] ? 0 : 1;
      } else {
        ++r.deferred;
      }
    }
    r.f_m = (double)fired / (double)n;
    r.f_c = fired ? (double)r.deferred / (double)fired : 0.0;
    r.cost = cfg->t_mse + r.f_m * cfg->t_snn + (r.f_m * r.f_c) * cfg->t_full;
    rows[k] = r;
    if (r.feasible && (best < 0 || r.cost < rows[best].cost)) best = k;
  }
  return best;
}

}  // extern "C"
