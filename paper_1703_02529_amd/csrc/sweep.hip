// Threshold search of the cost-based optimizer (Sec. 6.3, step 3) with its
// cost model (Sec. 6.2), on logged per-frame scores: for each candidate
// delta_diff, the detector's errors on the frames that do not fire, the
// c_low / c_high that keep the combined false negative / positive rates below
// FN* / FP*, and the expected cost per frame
//   f_s T_MSE + f_s f_m T_SNN + f_s f_m f_c T_FullNN   (f_s = 1).
//
// One 1024-thread workgroup per candidate.  The paper sorts the fired frames
// by confidence and walks the list; here each threshold is found by a binary
// search over the bit patterns of the fp32 confidences (which order like the
// values for confidences in [0, 1]), each probe an exact count over all
// frames: c_low is the smallest confidence v with
//   fn_dd + #{fired, label 1, conf <= v} >= FN* x (frames with the object)
// (1 if none), c_high the largest v with
//   fp_dd + #{fired, label 0, conf >= v} >= FP* x (frames without it)
// (0 if none), raised to c_low.  Frames below c_low are labelled 0, above
// c_high 1, the others defer and get the reference label.  A frame that does
// not fire takes the reference label of the frame it is compared with (frame
// t - delta, or "no object" for a fixed reference image).  Counts are exact;
// the fp64 rates and the cost are evaluated in a fixed operation order with
// contraction off.
#include "nsc_internal.h"

#include <math.h>

namespace nsc {
namespace {

constexpr int kSweepThreads = 1024;
constexpr uint32_t kOneBits = 0x3F800000u;  // 1.0f

struct SweepArgs {
  const double* score;
  const float* conf;
  const uint8_t* truth;
  int64_t n;
  const double* deltas;
  int32_t n_t;
  int32_t ref_mode, delta;
  double fp_target, fn_target, t_mse, t_snn, t_full;
  nsc_sweep_row* rows;
  int32_t* best;
};

// Workgroup sum of two 64-bit counts (every thread gets the totals).
__device__ __forceinline__ void wg_sum2(int64_t& a, int64_t& b, int64_t* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    a += __shfl_xor(a, o, 64);
    b += __shfl_xor(b, o, 64);
  }
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();  // the previous use of red is finished
  if (lane == 0) {
    red[2 * wave] = a;
    red[2 * wave + 1] = b;
  }
  __syncthreads();
  a = b = 0;
  for (int w = 0; w < kSweepThreads / 64; ++w) {
    a += red[2 * w];
    b += red[2 * w + 1];
  }
}

__device__ __forceinline__ bool fires(double s, double d) {
  return s == INFINITY || s > d;
}

__global__ void __launch_bounds__(kSweepThreads) k_sweep(SweepArgs a) {
#pragma clang fp contract(off)
  __shared__ int64_t red[2 * kSweepThreads / 64];
  const int k = blockIdx.x;
  const double d = a.deltas[k];
  // frames with the object, fired frames and the detector's errors
  int64_t pos = 0, fired = 0, fn_dd = 0, fp_dd = 0;
  for (int64_t t = threadIdx.x; t < a.n; t += kSweepThreads) {
    const int y = a.truth[t] ? 1 : 0;
    pos += y;
    if (fires(a.score[t], d)) {
      ++fired;
    } else {
      const int ref = a.ref_mode == NSC_REF_PREV && t >= a.delta ? (a.truth[t - a.delta] ? 1 : 0) : 0;
      fn_dd += y && !ref ? 1 : 0;
      fp_dd += !y && ref ? 1 : 0;
    }
  }
  wg_sum2(pos, fired, red);
  wg_sum2(fn_dd, fp_dd, red);
  const int64_t neg = a.n - pos;
  const double fn_budget = pos ? a.fn_target * (double)pos : INFINITY;
  const double fp_budget = neg ? a.fp_target * (double)neg : INFINITY;
  const bool feasible = (double)fn_dd < fn_budget && (double)fp_dd < fp_budget;

  // counts over the fired frames with the given label and confidence bits in
  // [lo, hi]
  auto count = [&](int label, uint32_t lo, uint32_t hi) {
    int64_t c = 0, unused = 0;
    for (int64_t t = threadIdx.x; t < a.n; t += kSweepThreads) {
      if ((a.truth[t] ? 1 : 0) != label || !fires(a.score[t], d)) continue;
      const uint32_t u = __float_as_uint(a.conf[t] + 0.0f);  // -0 counts as +0
      c += u >= lo && u <= hi ? 1 : 0;
    }
    wg_sum2(c, unused, red);
    return c;
  };

  double c_low = 0.0, c_high = 1.0;
  if (feasible) {
    // c_low: the smallest u with fn_dd + #{label 1, bits <= u} >= budget
    if ((double)(fn_dd + count(1, 0u, kOneBits)) >= fn_budget) {
      uint32_t lo = 0, hi = kOneBits;  // the predicate holds at hi
      while (lo < hi) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if ((double)(fn_dd + count(1, 0u, mid)) >= fn_budget)
          hi = mid;
        else
          lo = mid + 1;
      }
      c_low = (double)__uint_as_float(lo);
    } else {
      c_low = 1.0;
    }
    // c_high: the largest u with fp_dd + #{label 0, bits >= u} >= budget
    if ((double)(fp_dd + count(0, 0u, kOneBits)) >= fp_budget) {
      uint32_t lo = 0, hi = kOneBits;  // the predicate holds at lo
      while (lo < hi) {
        const uint32_t mid = lo + (hi - lo + 1) / 2;
        if ((double)(fp_dd + count(0, mid, kOneBits)) >= fp_budget)
          lo = mid;
        else
          hi = mid - 1;
      }
      c_high = (double)__uint_as_float(lo);
    } else {
      c_high = 0.0;
    }
    if (c_high < c_low) c_high = c_low;
  }
  // the decisions these thresholds give
  int64_t fn_cnn = 0, fp_cnn = 0, deferred = 0, unused = 0;
  for (int64_t t = threadIdx.x; t < a.n; t += kSweepThreads) {
    if (!fires(a.score[t], d)) continue;
    const double c = (double)a.conf[t];
    const int y = a.truth[t] ? 1 : 0;
    if (c < c_low)
      fn_cnn += y;
    else if (c > c_high)
      fp_cnn += 1 - y;
    else
      ++deferred;
  }
  wg_sum2(fn_cnn, fp_cnn, red);
  wg_sum2(deferred, unused, red);
  if (threadIdx.x == 0) {
    nsc_sweep_row r{};
    r.delta = d;
    r.c_low = c_low;
    r.c_high = c_high;
    r.fired = fired;
    r.deferred = deferred;
    r.fn_dd = fn_dd;
    r.fp_dd = fp_dd;
    r.fn_cnn = fn_cnn;
    r.fp_cnn = fp_cnn;
    r.positives = pos;
    r.negatives = neg;
    r.feasible = feasible ? 1 : 0;
    r.f_m = (double)fired / (double)a.n;
    r.f_c = fired ? (double)deferred / (double)fired : 0.0;
    r.cost = a.t_mse + r.f_m * a.t_snn + (r.f_m * r.f_c) * a.t_full;
    a.rows[k] = r;
  }
}

// The cheapest feasible candidate (the first on ties), or -1.
__global__ void __launch_bounds__(64) k_sweep_best(const nsc_sweep_row* rows, int32_t n_t,
                                                    int32_t* best) {
  int32_t bi = -1;
  double bc = 0.0;
  for (int k = threadIdx.x; k < n_t; k += 64) {
    if (rows[k].feasible && (bi < 0 || rows[k].cost < bc)) {
      bi = k;
      bc = rows[k].cost;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const int32_t oi = __shfl_xor(bi, o, 64);
    const double oc = __shfl_xor(bc, o, 64);
    if (oi >= 0 && (bi < 0 || oc < bc || (oc == bc && oi < bi))) {
      bi = oi;
      bc = oc;
    }
  }
  if (threadIdx.x == 0) *best = bi;
}

}  // namespace
}  // namespace nsc

extern "C" int nsc_threshold_sweep(const nsc_sweep_cfg* cfg, const double* score, const float* conf,
                                   const uint8_t* truth, int64_t n, const double* deltas,
                                   int32_t n_t, nsc_sweep_row* rows, int32_t* best, void* stream) {
  using namespace nsc;
  if (!cfg || !score || !conf || !truth || !deltas || !rows || !best)
    return fail(NSC_E_INVAL, "a pointer argument is NULL");
  if (n < 1 || n > 0x7FFFFFFF) return fail(NSC_E_INVAL, "frame count %lld out of range", (long long)n);
  if (n_t < 1 || n_t > NSC_MAX_SWEEP)
    return fail(NSC_E_INVAL, "%d candidate thresholds outside 1..%d", n_t, NSC_MAX_SWEEP);
  if (cfg->ref_mode != NSC_REF_PREV && cfg->ref_mode != NSC_REF_FIXED)
    return fail(NSC_E_INVAL, "ref_mode %d is neither NSC_REF_PREV nor NSC_REF_FIXED", cfg->ref_mode);
  if (cfg->ref_mode == NSC_REF_PREV && (cfg->delta < 1 || cfg->delta > NSC_MAX_DELTA))
    return fail(NSC_E_INVAL, "delta %d outside 1..%d", cfg->delta, NSC_MAX_DELTA);
  if (!(cfg->fp_target >= 0.0 && cfg->fp_target <= 1.0 && cfg->fn_target >= 0.0 &&
        cfg->fn_target <= 1.0))
    return fail(NSC_E_INVAL, "targets must lie in [0, 1]");
  if (!(cfg->t_mse >= 0.0 && cfg->t_snn >= 0.0 && cfg->t_full >= 0.0 && isfinite(cfg->t_mse) &&
        isfinite(cfg->t_snn) && isfinite(cfg->t_full)))
    return fail(NSC_E_INVAL, "costs must be finite and non-negative");
  SweepArgs a{};
  a.score = score;
  a.conf = conf;
  a.truth = truth;
  a.n = n;
  a.deltas = deltas;
  a.n_t = n_t;
  a.ref_mode = cfg->ref_mode;
  a.delta = cfg->delta;
  a.fp_target = cfg->fp_target;
  a.fn_target = cfg->fn_target;
  a.t_mse = cfg->t_mse;
  a.t_snn = cfg->t_snn;
  a.t_full = cfg->t_full;
  a.rows = rows;
  a.best = best;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(k_sweep, dim3((unsigned)n_t), dim3(kSweepThreads), 0, st, a);
  NSC_CHECK_LAUNCH("k_sweep");
  hipLaunchKernelGGL(k_sweep_best, dim3(1), dim3(64), 0, st, rows, n_t, best);
  NSC_CHECK_LAUNCH("k_sweep_best");
  return NSC_OK;
}
