// Internal declarations shared by the translation units of libnsc.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "nsc.h"

namespace nsc {

// Records a formatted description for nsc_last_error() and returns `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

#define NSC_TRY_HIP(call)                                                          \
  do {                                                                             \
    hipError_t e_ = (call);                                                        \
    if (e_ != hipSuccess)                                                          \
      return ::nsc::fail(NSC_E_HIP, "%s failed: %s", #call, hipGetErrorString(e_)); \
  } while (0)

#define NSC_CHECK_LAUNCH(what)                                                       \
  do {                                                                               \
    hipError_t e_ = hipGetLastError();                                               \
    if (e_ != hipSuccess)                                                            \
      return ::nsc::fail(NSC_E_HIP, "launch of %s failed: %s", what, hipGetErrorString(e_)); \
  } while (0)

constexpr int kNumCU = 256;  // MI355X compute units (8 XCDs x 32)
constexpr int kNumXCD = 8;

// Logical index of workgroup b of a grid of nb: the hardware hands workgroup b
// to XCD b mod 8, so numbering each XCD's workgroups consecutively gives each
// XCD one contiguous range of the logical work (in its dispatch order), whose
// neighbouring items share that XCD's L2.  A bijection of [0, nb).
__device__ __forceinline__ int64_t xcd_block(int64_t b, int64_t nb) {
  const int64_t x = b % kNumXCD, slot = b / kNumXCD;
  const int64_t q = nb / kNumXCD, r = nb % kNumXCD;
  return x * q + (x < r ? x : r) + slot;
}

inline int64_t gcd64(int64_t a, int64_t b) {
  while (b) {
    int64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Exact area resampling of one axis: output cell o covers [o*p, (o+1)*p) and
// input pixel i covers [i*q, (i+1)*q), both in units of 1/q input pixel.
struct Axis {
  int32_t n_in, n_out, p, q;
  static Axis make(int32_t n_in, int32_t n_out) {
    int64_t g = gcd64(n_in, n_out);
    return Axis{n_in, n_out, (int32_t)(n_in / g), (int32_t)(n_out / g)};
  }
};

// Column strips of the wave-autonomous area kernel.
struct WaveGeom {
  int32_t chunk_bytes;      // bytes one lane reads per source row: 32 (two 16-byte loads), 16 or 4
  int32_t group_lanes;      // lanes of one group (whole periods of the column pattern)
  int32_t group_cols;       // output columns of one group
  int32_t groups_per_wave;  // groups in one wave's strip
  int32_t groups_per_row;   // groups across the frame
  int32_t waves_per_frame;  // strips across the frame
  int32_t waves_per_block;  // waves of a workgroup: whole rows of strips where they fit in 4
  int32_t bands;            // bands of output rows per frame (one wave each per strip)
  int32_t band_rows;        // at most this many output rows per band
  size_t lds_bytes;         // dynamic LDS of a workgroup
};

// Area-sum launch plan for one frame geometry.
struct AreaPlan {
  Axis ay, ax;
  int32_t chunk_bytes;   // bytes of a row one lane reads per load: 16, 4 or 1
  int32_t lanes;         // row chunks = in_w*3 / chunk_bytes
  int32_t threads;       // lanes rounded up to a multiple of 64
  int32_t bands;         // output-row bands per frame
  bool packed;           // 16-bit packed vertical accumulators are exact
  bool wave;             // wave-autonomous strips apply (else the per-row kernel)
  WaveGeom wg;
};
int make_area_plan(int32_t in_h, int32_t in_w, int64_t stride, const void* frames,
                   int32_t out_h, int32_t out_w, int64_t n, AreaPlan* plan);
int launch_area_sums(const AreaPlan& plan, const uint8_t* frames, int64_t stride, int64_t n,
                     int32_t* sums, hipStream_t stream);

// One camera's detector settings in a camera group (device table).
struct CamDiff {
  const int32_t* ref_sums;  // FIXED: reference area sums
  const float* lr_w;        // blocked: LR weights
  double lr_b, delta_diff;
  int32_t ref_mode, delta, grid_h, grid_w;
  int64_t dec_off;          // PREV: offset of the decisions in the camera's state slot
};

// Detector scoring of frames [t0, t0+n) whose area sums are in `sums`.  With
// a camera group (cams != null) the n frames are per_cam frames of each
// camera in turn, every camera with its own settings from cams[] and its
// earlier frames in its state slot (state + camera * state_stride); the
// per-stream fields below are then unused.
struct DiffArgs {
  const int32_t* sums;       // [n][cells]
  const int32_t* prev_sums;  // [delta][cells] frames t0-delta..t0-1 (PREV, t0 > 0)
  const int32_t* ref_sums;   // [cells] (FIXED)
  const float* lr_w;         // [grid_h*grid_w] (blocked)
  double lr_b, delta_diff, den, den2;  // den2 = den*den as a double
  int64_t n, t0;
  int32_t dd_h, dd_w, grid_h, grid_w, ref_mode, delta;
  int32_t metric;            // NSC_METRIC_*
  double* score;             // nullable
  uint8_t* fire;
  const CamDiff* cams;       // camera group (else null)
  int32_t cams_blocked;      // camera group: some camera scores a blocked grid
  int64_t per_cam;
  const unsigned char* state;
  int64_t state_stride;
  // earlier-frame global MSE detector fused into the area kernel
  // (k_area_prev_wave): frames whose index i has (i / delta) mod chain_r != 0
  // take their score from the partial sums (part_bands bands x part_strips
  // strips per frame); the others from the sums.  part == null: every frame
  // from the sums.
  const int64_t* part;
  int32_t chain_r, part_bands, part_strips;
};
int launch_diff(const DiffArgs& a, hipStream_t stream);
// The earlier-frame global MSE detector fused into the area kernel: whether
// it applies to a call of n frames, and then its plan, chain length and
// partial-sum count.
struct PrevFusePlan {
  AreaPlan ap;
  int32_t chain_r;
  int64_t part_elems;
};
bool area_prev_plan(const AreaPlan& p, const DiffArgs& a, int64_t n, PrevFusePlan* out);
// Launches the fused area kernel (sums and partial sums), then k_diff is
// launched with the fields area_prev_diff_args sets.
int launch_area_prev(const PrevFusePlan& fp, const uint8_t* frames, int64_t stride, int64_t n,
                     int32_t* sums, const DiffArgs& a, int64_t* part, hipStream_t stream);
void area_prev_diff_args(const PrevFusePlan& fp, const int64_t* part, DiffArgs* a);
// Area sums with the fixed-reference global detector fused in (when
// area_detect_fused): per-unit partial sums in `part` (area_detect_part_count
// units x 3 int64), then the scores and fire flags of `a`.
bool area_detect_fused(const AreaPlan& p, const DiffArgs& a);
int64_t area_detect_part_count(const AreaPlan& p, int64_t n);
int launch_area_detect_fixed(const AreaPlan& p, const uint8_t* frames, int64_t stride, int64_t n,
                             int32_t* sums, const DiffArgs& a, int64_t* part, hipStream_t stream);

// Compaction of fire flags into ascending indices.
int64_t compact_tiles(int64_t n);
int launch_compact(const uint8_t* fire, int64_t n, int32_t* idx, int32_t* count, int32_t* tile_counts,
                   hipStream_t stream);
// The same with the tile offsets in a static device array (no workspace).
int launch_compact_noalloc(const uint8_t* fire, int64_t n, int32_t* idx, int32_t* count,
                           hipStream_t stream);

// Label resolution (PREV: reuse the decision of frame t-delta; FIXED: 0).
struct ResolvePlan {
  int64_t n, t0;
  int32_t delta, rows_per_tile, tiles;
};
ResolvePlan make_resolve_plan(int64_t n, int64_t t0, int32_t delta);
int launch_resolve(const ResolvePlan& p, int32_t ref_mode, const uint8_t* fire, const uint8_t* dec,
                   const uint8_t* prev_dec, int32_t* tile_last, int32_t* carry, uint8_t* label,
                   uint8_t* defer, hipStream_t stream);
int launch_state_update(const int32_t* sums, const uint8_t* label, const uint8_t* defer, int64_t n,
                        int32_t delta, int64_t cells, int32_t* state_sums, uint8_t* state_dec,
                        void* scratch, hipStream_t stream);
int launch_fill_nan(float* p, int64_t n, hipStream_t stream);
// Camera groups: label resolution of n frames per camera, and the state slots
// (the last delta frames of every earlier-frame camera; scratch holds a copy
// of n_cams * state_stride bytes when n < max_delta).
int launch_group_resolve(const CamDiff* cams, int32_t n_cams, const uint8_t* fire,
                         const uint8_t* dec, int64_t n, int64_t t0, const unsigned char* state,
                         int64_t state_stride, uint8_t* label, uint8_t* defer,
                         hipStream_t stream);
int launch_group_state(const CamDiff* cams, int32_t n_cams, int32_t max_delta,
                       const int32_t* sums, const uint8_t* label, const uint8_t* defer, int64_t n,
                       int64_t cells, unsigned char* state, int64_t state_stride, void* scratch,
                       hipStream_t stream);
int launch_set_i32(int32_t* p, int32_t v, hipStream_t stream);
// *out = clamp(*count - off, 0, m): the survivors of the CNN pass over the
// compacted slots [off, off + m).
int launch_pass_count(const int32_t* count, int64_t off, int64_t m, int32_t* out,
                      hipStream_t stream);

// Frame skipping: frames [t0, t0+n) take the outputs of their checked frame
// floor(t / s) * s.  Checked frames [k0, k0+nc) (absolute checked indices)
// have their outputs in k_*; frames before the first of them take `last`
// (label | defer << 1 of the previous call's last checked frame), which is
// then replaced by this call's last checked decision.  Per-frame outputs
// (nullable) of frames between checks: score NaN, fire 0, logit NaN.
struct SkipExpand {
  int64_t n, t0, k0, nc;
  int32_t s;
  const uint8_t* k_label;
  const uint8_t* k_defer;
  const double* k_score;
  const uint8_t* k_fire;
  const float* k_logit;
  uint8_t* last;
  uint8_t* label;
  uint8_t* defer;
  double* score;
  uint8_t* fire;
  float* logit;
};
int launch_skip_expand(const SkipExpand& e, hipStream_t stream);
int launch_copy_u8(const uint8_t* src, uint8_t* dst, int64_t n, hipStream_t stream);

// Specialized CNN.
// K steps (of 32 features) per weight chunk of the tiled dense kernel.
constexpr int kDenseChunk = 4;

struct CnnLayer {
  int32_t cin, cout, h, w;  // input channels, output channels, input grid
  bool pool;
  int32_t kpad;             // padded reduction length of the packed weights
  size_t w_off, b_off;      // offsets (elements) into the packed weight/bias arrays
  // bf16 networks, fp16 path (layers after the first): the layer's weights
  // enter the fp16 matrix cores multiplied by 2^wexp (exact: every bf16
  // weight within 2^31 of the largest is an fp16 value after the scaling) and
  // its input activations multiplied by 2^-aexp (aexp >= 0, from the
  // worst-case bound of the input for inputs in [-1, 1], so that no fp16
  // value overflows); the accumulators are multiplied back by 2^(aexp - wexp)
  int32_t wexp, aexp;
};
// bf16 networks also hold every layer's weights in MFMA fragment order
// (conv_wf, same offsets w_off): for K step ks (32 values of the layer's K
// order) and output-channel block nt, lane l = 16 g + m holds the 8 values
// W[16 nt + m][32 ks + 8 g .. 32 ks + 8 g + 7], 16 bytes at element
// ((ks * (cout / 16) + nt) * 64 + l) * 8, so one wave's fragment is 1 KB of
// consecutive memory; conv_wh holds the same fragments as scaled fp16 values
// for the layers whose activations run through the fp16 matrix cores.
struct Cnn {
  nsc_cnn_desc desc;
  int32_t n_layers;
  CnnLayer layers[NSC_MAX_CONV];
  int32_t feat_c, feat_h, feat_w, flat, dense;
  bool bf16;
  void* dev;                // one allocation holding everything below
  void* conv_w;             // packed conv weights, bf16 or fp32
  void* conv_wf;            // bf16 networks: the same in fragment order (else null)
  void* conv_wh;            // bf16 networks: the same as fp16, each layer times 2^wexp
  void* w1h;                // bf16 networks: dense weights as fp16 times 2^dense_wexp
  void* conv_w0h;           // fp16 path: k_pair64's first layer, scaled, bias folded in (or null)
  void* w1f;                // fp16 path: w1h in fragment order, padded to whole chunks
  int32_t dense_wexp, dense_aexp;  // as CnnLayer::wexp / aexp, for the dense layer
  bool h16;                 // bf16 network whose banded layers and dense layer take the
                            // fp16 path (activations as fp16, one MFMA per product)
  float* conv_b;            // fp32 biases
  void* w1;                 // dense weights [D][flat] in (y, x, c) order
  float* b1;
  float* w2;                // output layer weights [D] (fp32)
  float* scales;            // [2 (n_layers + 1)]: per layer, then the dense layer, the fp16
                            // path's input scale 2^-aexp and output scale 2^(aexp - wexp)
  float b2;
  size_t act_elems;         // largest per-image activation (elements)
};
// One camera's network in a camera group: the group's networks share one
// description, so each camera's weights sit at the same offsets of its own
// allocation, `woff` bytes from the base network's; its output bias and
// decision thresholds.
struct CamNet {
  int64_t woff;
  double c_low, c_high;
  float b2;
  int32_t pad;
};

struct CnnRunArgs {
  const int32_t* sums;
  int32_t sums_h, sums_w, fy, fx;
  double den_c;             // denominator of the fy x fx cell sums
  const int32_t* idx;
  const int32_t* count;
  int64_t max_count;
  float* logit;             // per survivor slot
  float* prob;              // nullable
  // decisions: written when dec != nullptr, at dec[idx[i]]
  uint8_t* dec;
  double c_low, c_high;
  float* frame_logit;       // nullable: logit scattered to frame position idx[i]
  // camera group (nullable): survivor slot s is camera idx[s] / per_cam and
  // runs that camera's network, bias b2 and thresholds from nets[]
  const CamNet* nets;
  int64_t per_cam;
  int32_t n_nets;           // cameras of the group (0 without a group)
};
size_t cnn_workspace_bytes(const Cnn& cnn, int64_t max_count);
int run_cnn(const Cnn& cnn, const CnnRunArgs& a, void* ws, size_t ws_bytes, hipStream_t stream);

}  // namespace nsc
