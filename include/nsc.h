/*
 * nsc.h -- C ABI of the NoScope cascade filter on MI355X (gfx950).
 *
 * The cascade answers a binary presence query over fixed-camera video (Sec. 3
 * of Kang et al., "NoScope: Optimizing Neural Network Queries over Video at
 * Scale", VLDB 2017): for every frame it outputs a label (object present or
 * not) or defers the frame to the expensive reference network.  The target
 * object is implicit in the specialized model's weights (Sec. 4).
 *
 * Per frame the hot path is:
 *   1. downsample: exact area average onto a small grid (Sec. 7 resizes frames
 *      before the models); kept as integer area sums S with one denominator;
 *   2. difference detector (Sec. 5): MSE (or SAD, NRMSE, PSNR, the
 *      alternatives the paper names) against the frame `delta` earlier or
 *      against a fixed reference image, globally or per grid block weighed by
 *      logistic regression; fires when the metric exceeds delta_diff;
 *   3. compaction of the frames that fire (Sec. 7 batches frames for the GPU);
 *   4. specialized CNN on the survivors (Sec. 4), pre-processed to [-1, 1]
 *      (Sec. 7); confidence c = sigmoid(logit) against c_low / c_high;
 *   5. decision: c < c_low -> label 0, c > c_high -> label 1, otherwise defer;
 *      a frame on which the earlier-frame detector does not fire reuses the
 *      output of the frame it was compared with (Sec. 5); with a fixed
 *      reference image it is labelled "no object".
 *
 * Conventions for every entry point:
 *  - Pointers marked (device) are caller-owned device memory, (host) are host
 *    memory.  Frames are uint8 RGB, interleaved, row-major [H][W][3], one
 *    frame every `frame_stride` bytes.
 *  - All GPU work is enqueued on `stream` (a hipStream_t passed as void*;
 *    NULL is the default stream) and the call returns after enqueueing.
 *  - Arguments are validated on the host before any HIP call; the return
 *    value is NSC_OK (0) or a negative nsc_status, and nsc_last_error()
 *    returns a thread-local description.  Outputs are unspecified after an
 *    error.  Faults of already-enqueued work surface on a later HIP call.
 *  - The library owns only what its own *_create calls allocate (packed CNN
 *    weights) and one static 64 KB device array per GPU (the scratch of
 *    nsc_compact_noalloc); it allocates nothing else.  Scratch space is the
 *    caller's workspace, whose size the *_workspace_bytes calls report.
 *  - Calls that share a workspace or state buffer must be ordered on one
 *    stream by the caller.
 */
#ifndef NSC_H_
#define NSC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum nsc_status {
  NSC_OK = 0,
  NSC_E_INVAL = -1,     /* null pointer, NaN or out-of-range scalar        */
  NSC_E_SHAPE = -2,     /* shape outside the supported limits             */
  NSC_E_DTYPE = -3,     /* unknown element type                           */
  NSC_E_WORKSPACE = -4, /* workspace missing, too small or misaligned     */
  NSC_E_HIP = -5,       /* a HIP runtime call or kernel launch failed      */
  NSC_E_NOMEM = -6,     /* device allocation failed                       */
  NSC_E_STATE = -7      /* state does not hold the frames before t0       */
} nsc_status;

enum { NSC_REF_PREV = 0, NSC_REF_FIXED = 1 };
/* Difference metric of the detector (Sec. 5 uses the MSE and names NRMSE,
 * PSNR and SAD as alternatives it tried).  On the area-average values a
 * (frame) and b (compared frame), N values on the 0..255 scale:
 *   MSE   sum (a-b)^2 / N
 *   SAD   sum |a-b|
 *   NRMSE sqrt(sum (a-b)^2 / sum b^2)  (0 if both sums are 0, +inf if only
 *         sum b^2 is 0)
 *   PSNR  -10 log10(255^2 / MSE): the negated PSNR, so that for every metric
 *         the detector fires when the value exceeds delta_diff (PSNR below
 *         -delta_diff); identical images give -inf.
 * MSE, SAD and NRMSE are correctly rounded fp64 functions of exact integer
 * sums; PSNR goes through the device log10 (within a few ulp). */
enum { NSC_METRIC_MSE = 0, NSC_METRIC_SAD = 1, NSC_METRIC_NRMSE = 2, NSC_METRIC_PSNR = 3 };
/* Element types of a specialized CNN (its weights and activations):
 *   NSC_F32        fp32 weights and activations, fp32 matrix cores;
 *   NSC_BF16       bf16 weights; the pre-processed input rounded to bf16; the
 *                  64-input-channel layers and the dense layer run on the fp16
 *                  matrix cores with their activations rounded to fp16 (the
 *                  bf16 weights are scaled by powers of two, exactly, and the
 *                  activations by powers of two chosen from a worst-case bound
 *                  so that no fp16 value overflows), other layers as with
 *                  NSC_BF16_PAIRS; fp32 accumulation;
 *   NSC_BF16_PAIRS bf16 weights and input; every later activation enters the
 *                  bf16 matrix cores as a pair hi = bf16(a), lo = bf16(a - hi)
 *                  (two products per weight, about 2^-17 relative); fp32
 *                  accumulation. */
enum { NSC_F32 = 0, NSC_BF16 = 1, NSC_BF16_PAIRS = 2 };
enum { NSC_MAX_CONV = 8, NSC_MAX_DELTA = 256, NSC_MAX_BLOCKS = 1024, NSC_MAX_STRIDE = 4096,
       NSC_MAX_SWEEP = 65535 };
/* Largest n of nsc_compact_noalloc (16,384 tiles of 4,096 flags). */
#define NSC_NOALLOC_MAX_FLAGS 67108864LL

/* Stage boundaries at which nsc_cascade_run records optional events:
 * [0] start, [1] after the area sums, [2] after the detector, [3] after the
 * compaction, [4] after the CNN, [5] after label resolution (the end). */
enum { NSC_STAGE_EVENTS = 6 };

/* Difference-detector and decision settings of one video stream (Sec. 5, 6). */
typedef struct nsc_cascade_cfg {
  int32_t in_h, in_w;        /* raw frame size                                   */
  int64_t frame_stride;      /* bytes between frames, >= in_h*in_w*3             */
  int32_t dd_h, dd_w;        /* detector grid, 1 <= dd <= in (downsampling only)  */
  int32_t cnn_h, cnn_w;      /* CNN input grid; dd_h = fy*cnn_h, dd_w = fx*cnn_w  */
  int32_t ref_mode;          /* NSC_REF_PREV (frame t-delta) or NSC_REF_FIXED     */
  int32_t delta;             /* PREV: comparison offset, 1..NSC_MAX_DELTA frames  */
  int32_t grid_h, grid_w;    /* 1x1: global metric; otherwise blocked detector    */
  const float* lr_w;         /* (device) grid_h*grid_w LR weights, row-major;
                                blocked only                                     */
  double lr_b;               /* LR bias; blocked only                            */
  const int32_t* ref_sums;   /* (device) FIXED: reference image area sums on the
                                detector grid, [dd_h][dd_w][3], as produced by
                                nsc_downsample                                   */
  double delta_diff;         /* fire iff metric > delta_diff                      */
  double c_low, c_high;      /* 0 <= c_low <= c_high <= 1                         */
  int32_t check_stride;      /* frame skipping (Sec. 5, t_skip in frames): only
                                frames with absolute index t mod s = 0 are
                                checked; a frame in between keeps the output
                                of the last checked frame.  0 or 1: every frame;
                                at most NSC_MAX_STRIDE; PREV needs delta to be
                                a multiple of s (the compared frame is then a
                                checked one)                                   */
  int32_t metric;            /* NSC_METRIC_* (0 = MSE); the blocked detector
                                takes MSE, SAD or NRMSE per block              */
  int32_t fuse_prev;         /* 0 or 1.  1: PREV with the global MSE metric and
                                delta >= 2 runs the detector inside the area
                                kernel by temporal tiling (chains of frames
                                delta apart, partial sums) where the frame
                                geometry allows (16- or 4-byte lane chunks);
                                0: area sums, then the detector as its own
                                pass.  Same scores bit for bit; 0 measured
                                6-7 % faster on 640x480 frames.  Ignored by
                                camera groups and staged batches.              */
} nsc_cascade_cfg;

/* Shape of a specialized CNN (Sec. 4): n_conv x [conv3x3 'same' + bias + ReLU
 * (+ 2x2/2 max-pool, floor)], flatten, dense `dense` + ReLU, dense 1 -> logit. */
typedef struct nsc_cnn_desc {
  int32_t n_conv;                 /* 1..NSC_MAX_CONV                          */
  int32_t conv_out[NSC_MAX_CONV]; /* output channels per layer: multiples of 16;
                                     inner layers' inputs multiples of 32 (bf16)
                                     or 4 (f32)                               */
  uint32_t pool_after_mask;       /* bit l: max-pool after conv layer l        */
  int32_t dense;                  /* hidden units, multiple of 16             */
  int32_t in_h, in_w;             /* input grid (equal to cfg cnn_h, cnn_w)    */
  int32_t dtype;                  /* NSC_F32, NSC_BF16 or NSC_BF16_PAIRS       */
} nsc_cnn_desc;

typedef struct nsc_cnn nsc_cnn; /* opaque: packed device weights */

/* Optional per-frame outputs of nsc_cascade_run (each pointer nullable, device). */
typedef struct nsc_frame_outputs {
  double* score;  /* [n] detector metric (+inf for a frame forced to fire)   */
  uint8_t* fire;  /* [n] 1 if the detector fired                             */
  float* logit;   /* [n] CNN logit of fired frames, NaN elsewhere            */
} nsc_frame_outputs;

/* Host-side summary of a run; filling it synchronises `stream`. */
typedef struct nsc_run_stats {
  int64_t frames;   /* n                                  */
  int64_t fired;    /* frames the detector passed to the CNN */
  int64_t positive; /* frames labelled 1 without deferral */
  int64_t deferred; /* frames deferred to the reference network */
} nsc_run_stats;

/* ---------------------------------------------------------------- helpers */

/* Status name, e.g. "NSC_E_SHAPE".  Never NULL. */
const char* nsc_status_string(int status);
/* Description of the last error on the calling thread ("" if none). */
const char* nsc_last_error(void);

/* Denominator of the area sums from in_h x in_w onto out_h x out_w: an output
 * value is S / den.  den = (in_h/g_h) * (in_w/g_w) with g = gcd(in, out).
 * Returns a negative nsc_status on invalid sizes. */
int64_t nsc_area_den(int32_t in_h, int32_t in_w, int32_t out_h, int32_t out_w);

/* Validates a configuration without touching the GPU. */
int nsc_cfg_check(const nsc_cascade_cfg* cfg);
/* Validates a CNN description against an input grid without touching the GPU. */
int nsc_cnn_check(const nsc_cnn_desc* desc);

/* -------------------------------------------------------------- CNN handle */

/* Number of floats of the canonical weight blob of `desc`:
 *   per conv layer: weights [Cout][Cin][3][3] then bias [Cout];
 *   dense: weights [D][F] (F = C*h*w of the last pooled map, flattened in
 *   (c, y, x) order) then bias [D]; output: weights [D] then bias [1].
 * Returns a negative nsc_status on an invalid description. */
int64_t nsc_cnn_blob_floats(const nsc_cnn_desc* desc);

/* Packs a host fp32 weight blob (bf16 nets round each value to the
 * nearest bf16) into device memory owned by the returned handle.  Synchronous;
 * uses the current HIP device.  Errors: NSC_E_INVAL, NSC_E_SHAPE,
 * NSC_E_DTYPE, NSC_E_NOMEM, NSC_E_HIP. */
int nsc_cnn_create(const nsc_cnn_desc* desc, const float* host_weights, int64_t n_floats,
                   nsc_cnn** out);
/* Frees the handle's device memory (NULL is a no-op).  The caller must make
 * sure no enqueued work still uses it. */
int nsc_cnn_destroy(nsc_cnn* cnn);

/* ----------------------------------------------------------- workspace sizes */

/* Workspace of nsc_cascade_run for up to max_frames frames per call. */
int nsc_cascade_workspace_bytes(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn,
                                int64_t max_frames, size_t* bytes);
/* State carried between consecutive nsc_cascade_run calls on one stream
 * (PREV mode: area sums and decisions of the last `delta` frames, counted in
 * checked frames; with frame skipping also the last checked frame's output). */
int nsc_state_bytes(const nsc_cascade_cfg* cfg, size_t* bytes);
/* Workspace of nsc_compact for n flags. */
int nsc_compact_workspace_bytes(int64_t n, size_t* bytes);
/* Workspace of nsc_specialized_cnn for up to max_count images. */
int nsc_cnn_workspace_bytes(const nsc_cnn* cnn, int64_t max_count, size_t* bytes);

/* --------------------------------------------------------- hot-path calls */

/* Step 1 (Sec. 7, resize; exact area average).  For each of n frames:
 *   sums_out[f][Y][X][c] = sum_j sum_i wy[Y][j] * wx[X][i] * frame_f[j][i][c]
 * with integer overlap weights wy, wx (row sums in_h/g_h and in_w/g_w).
 * frames (device, n frames, frame_stride apart), sums_out (device,
 * n*out_h*out_w*3 int32).  Requires 1 <= out <= in, 255*den < 2^31.
 * Errors: NSC_E_INVAL, NSC_E_SHAPE, NSC_E_HIP. */
int nsc_downsample(const uint8_t* frames, int64_t n, int32_t in_h, int32_t in_w,
                   int64_t frame_stride, int32_t out_h, int32_t out_w, int32_t* sums_out,
                   void* stream);

/* Steps 1-2 (Sec. 5).  Downsamples frames [t0, t0+n) into sums_out (device,
 * n*dd_h*dd_w*3 int32) and scores each against its reference:
 *   global:  score = the metric of S_t / den against S_ref / den; with MSE
 *            sum (S_t - S_ref)^2 / (den^2 * dd_h*dd_w*3)
 *   blocked: score = lr_b + sum_k lr_w[k] * metric over block k, blocks being
 *            rows [floor(by*dd_h/grid_h), floor((by+1)*dd_h/grid_h)) x
 *            columns likewise, k = by*grid_w + bx;
 * S_ref is frame t-delta (PREV) or cfg->ref_sums (FIXED).  In PREV mode a
 * frame with absolute index t < delta has no reference: score = +inf and it
 * fires.  fire_out[i] = score > delta_diff (device, n bytes); score_out
 * (device, n doubles) is nullable.  prev_sums (device) holds the sums of
 * frames t0-delta .. t0-1 and is required iff PREV and t0 > 0.
 * Errors: NSC_E_INVAL, NSC_E_SHAPE, NSC_E_HIP. */
int nsc_diff_detect(const nsc_cascade_cfg* cfg, const uint8_t* frames, int64_t n, int64_t t0,
                    const int32_t* prev_sums, int32_t* sums_out, double* score_out,
                    uint8_t* fire_out, void* stream);

/* Step 3 (Sec. 7, batching).  idx_out (device, n int32) receives the
 * ascending indices i with fire[i] != 0 and count_out (device, one int32) their
 * number.  ws: nsc_compact_workspace_bytes(n).  Errors: NSC_E_INVAL,
 * NSC_E_WORKSPACE, NSC_E_HIP. */
int nsc_compact(const uint8_t* fire, int64_t n, int32_t* idx_out, int32_t* count_out, void* ws,
                size_t ws_bytes, void* stream);

/* Step 3 without a workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation).  Same outputs as nsc_compact: idx_out (device, n int32) gets
 * the ascending indices i with fire[i] != 0 and count_out (device, one int32)
 * their number.  The tile offsets live in a static device array inside the
 * library (64 KB, held by every GPU the library runs on until the process
 * ends), which limits n to NSC_NOALLOC_MAX_FLAGS; a larger n is rejected with
 * NSC_E_WORKSPACE before any GPU work.  The call allocates nothing.  Every
 * call on one GPU shares that array: calls that overlap on the same GPU (on
 * different streams or host threads) race and must be ordered by the caller.
 * The stream must belong to the current device.  Errors: NSC_E_INVAL,
 * NSC_E_WORKSPACE, NSC_E_HIP. */
int nsc_compact_noalloc(const uint8_t* fire, int64_t n, int32_t* idx_out, int32_t* count_out,
                        void* stream);

/* Step 4 (Sec. 4 model, Sec. 7 pre-processing).  For i < *count (device),
 * evaluates the network on frame idx[i]'s area sums: sums (device,
 * [*][sums_h][sums_w][3] int32 with denominator den) are summed over
 * fy x fx cells when sums_h = fy*in_h, sums_w = fx*in_w; the input is
 * x = (S/den')/127.5 - 1 (den' = den * fy * fx, with 255 den' < 2^31, the
 * sums being values of 0..255 times den).  Writes logit_out[i] (device, float) and, if
 * prob_out is not NULL, prob_out[i] = sigmoid(logit).  max_count bounds
 * *count (entries beyond max_count are not evaluated).  ws:
 * nsc_cnn_workspace_bytes(cnn, max_count).  Errors: NSC_E_INVAL,
 * NSC_E_SHAPE, NSC_E_WORKSPACE, NSC_E_HIP. */
int nsc_specialized_cnn(const nsc_cnn* cnn, const int32_t* sums, int32_t sums_h, int32_t sums_w,
                        int64_t den, const int32_t* idx, const int32_t* count, int64_t max_count,
                        float* logit_out, float* prob_out, void* ws, size_t ws_bytes,
                        void* stream);

/* Steps 1-5 on frames [t0, t0+n) of one stream.  Writes label_out and
 * defer_out (device, n bytes each; a deferred frame has label 0).  state
 * (device, nsc_state_bytes) carries the last delta frames between calls: with
 * t0 = 0 its content is ignored; with t0 > 0 it must hold what the previous
 * call (ending at frame t0) left.  With check_stride s > 1 only the checked
 * frames (t mod s = 0) are read and run through steps 1-4 (the cascade on the
 * subsampled video, delta / s checked frames back), and every frame then takes
 * its checked frame's output: frames between checks get score NaN, fire 0 and
 * logit NaN in `outs`; state is required (it holds the last checked output).  ws: nsc_cascade_workspace_bytes(cfg, cnn,
 * >= n).  outs (host struct of device pointers) and stats (host) are nullable;
 * stats synchronises the stream.  stage_events (host array of
 * NSC_STAGE_EVENTS hipEvent_t, nullable, entries nullable) are recorded on
 * `stream` at the stage boundaries, for timing.  Errors: NSC_E_INVAL,
 * NSC_E_SHAPE, NSC_E_WORKSPACE, NSC_E_STATE, NSC_E_HIP. */
int nsc_cascade_run(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn, const uint8_t* frames,
                    int64_t n, int64_t t0, void* state, void* ws, size_t ws_bytes,
                    uint8_t* label_out, uint8_t* defer_out, const nsc_frame_outputs* outs,
                    nsc_run_stats* stats, void* const* stage_events, void* stream);

/* ------------------------------------------------------------------------
 * Staged batches (Sec. 8: batching trades latency for throughput; Sec. 7:
 * frames are batched for the GPU).  Frames that arrive in chunks (a decoder's
 * or a generator's buffers) can be batched for steps 2-5 without keeping the
 * raw frames: nsc_cascade_stage runs step 1 of one chunk into the batch's
 * workspace, after which the chunk's frame buffer may be reused, and
 * nsc_cascade_finish runs steps 2-5 once over everything staged, so the CNN
 * sees the survivors of all the batch's chunks together.  Labels of a
 * staged chunk exist only once its batch is finished: the latency grows with
 * batch_frames.  The outputs equal those of nsc_cascade_run on the batch's
 * frames in one call, logits up to the rounding order of the dense layer's
 * sums (which depends on how many survivors share a pass).  The detector
 * runs as a pass of its own over the staged sums.  Frame skipping is not
 * available (check_stride 0 or 1).
 *
 * batch_frames (> 0) is the batch's capacity in frames; cnn_pass (>= 0)
 * bounds the survivors of one CNN pass (0: min(16384, batch_frames)): the
 * CNN runs ceil(batch_frames / pass) passes over the compacted list, each
 * sized on the device (empty passes cost their launches only), and the
 * workspace holds the CNN's buffers for one pass.  All three calls of one
 * batch take the same cfg, cnn, batch_frames and cnn_pass.  Errors of all
 * three: NSC_E_INVAL (a bad cfg or argument, frame skipping), NSC_E_SHAPE. */
/* Workspace of a staged batch: the area sums of batch_frames frames, the
 * detector, compaction and resolve buffers, and one CNN pass. */
int nsc_batch_workspace_bytes(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn, int64_t batch_frames,
                              int64_t cnn_pass, size_t* bytes);
/* Step 1 of n frames (device, frame i at frames + i * frame_stride) into
 * batch slots [at, at + n) (at + n <= batch_frames) of ws
 * (nsc_batch_workspace_bytes, 256-byte aligned).  Enqueued on `stream`; the
 * frames are not read after this call's work has run.  Errors also
 * NSC_E_WORKSPACE, NSC_E_HIP. */
int nsc_cascade_stage(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn, int64_t batch_frames,
                      int64_t cnn_pass, const uint8_t* frames, int64_t n, int64_t at, void* ws,
                      size_t ws_bytes, void* stream);
/* Steps 2-5 on the frames staged in slots [0, n) (n <= batch_frames), which
 * are frames [t0, t0 + n) of the stream: label_out, defer_out, outs, stats,
 * state and stage_events as for nsc_cascade_run (stage events 0 and 1 are
 * recorded together at the start: step 1 ran in the stage calls).  The
 * state continues across batches and plain nsc_cascade_run calls of the same
 * cfg.  Errors also NSC_E_WORKSPACE, NSC_E_STATE, NSC_E_HIP. */
int nsc_cascade_finish(const nsc_cascade_cfg* cfg, const nsc_cnn* cnn, int64_t batch_frames,
                       int64_t cnn_pass, int64_t n, int64_t t0, void* state, void* ws,
                       size_t ws_bytes, uint8_t* label_out, uint8_t* defer_out,
                       const nsc_frame_outputs* outs, nsc_run_stats* stats,
                       void* const* stage_events, void* stream);

/* ------------------------------------------------------------------------
 * Camera groups (Sec. 8: a system that watches many streams can batch frames
 * of different streams together, each stream with its own model).  A group of
 * n_cams fixed cameras shares the frame geometry (in_h, in_w, frame_stride,
 * dd_h, dd_w, cnn_h, cnn_w) and the detector metric; every camera keeps its
 * own reference (ref_mode, delta, ref_sums), block grid and LR weights,
 * thresholds (delta_diff, c_low, c_high) and specialized CNN (one network
 * description for the whole group, each camera with its own weights).  One
 * nsc_group_run call processes n frames of every camera, each stage as one
 * launch over all cameras' frames: the CNN runs every survivor with its
 * camera's weights (grouped GEMM).  Each camera's outputs are exactly those of
 * nsc_cascade_run on its own frames with its own cfg and network.  Frame
 * skipping is not available in a group (check_stride 0 or 1). */
enum { NSC_MAX_CAMERAS = 65535 };

typedef struct nsc_group nsc_group; /* opaque: per-camera device tables */

/* cfgs: host array of n_cams configurations (1 .. NSC_MAX_CAMERAS); cnns:
 * host array of n_cams network handles.  The device buffers the cfgs point to
 * (lr_w, ref_sums) and the networks must outlive the group.  Allocates the
 * group's device tables (synchronous, current device).  Errors: NSC_E_INVAL
 * (a bad cfg, geometry or metric differing from camera 0's, frame skipping,
 * a NULL handle), NSC_E_SHAPE (a network description differing from camera
 * 0's, or not matching the CNN grid), NSC_E_NOMEM, NSC_E_HIP. */
int nsc_group_create(const nsc_cascade_cfg* cfgs, const nsc_cnn* const* cnns, int32_t n_cams,
                     nsc_group** out);
/* Frees the group's tables (NULL is a no-op); no enqueued work may use it. */
int nsc_group_destroy(nsc_group* group);
/* State carried between consecutive nsc_group_run calls: camera c's slot
 * (laid out as nsc_cascade_run's state of its cfg) at c * slot_bytes;
 * bytes = n_cams * slot_bytes.  slot_bytes is nullable. */
int nsc_group_state_bytes(const nsc_group* group, size_t* bytes, size_t* slot_bytes);
/* Workspace of nsc_group_run for up to frames_per_cam frames per camera. */
int nsc_group_workspace_bytes(const nsc_group* group, int64_t frames_per_cam, size_t* bytes);
/* Steps 1-5 on frames [t0, t0+n) of every camera.  frames (device): camera
 * c's frame t0 + j at frames + (c * n + j) * frame_stride.  label_out,
 * defer_out (device, n_cams * n bytes) and the per-frame outputs of `outs`
 * use the same order (camera-major).  state (device, nsc_group_state_bytes)
 * is required when a camera compares with earlier frames; with t0 = 0 its
 * content is ignored.  ws: nsc_group_workspace_bytes(group, >= n).  stats
 * (host, nullable) sums over all cameras and synchronises the stream;
 * stage_events as for nsc_cascade_run.  Errors: NSC_E_INVAL, NSC_E_SHAPE,
 * NSC_E_WORKSPACE, NSC_E_STATE, NSC_E_HIP. */
int nsc_group_run(const nsc_group* group, const uint8_t* frames, int64_t n, int64_t t0,
                  void* state, void* ws, size_t ws_bytes, uint8_t* label_out, uint8_t* defer_out,
                  const nsc_frame_outputs* outs, nsc_run_stats* stats,
                  void* const* stage_events, void* stream);

/* ------------------------------------------------------------------------
 * Threshold search of the cost-based optimizer (Sec. 6.3, step 3) with its
 * cost model (Sec. 6.2), on logged scores of every frame of an evaluation
 * video.  For each candidate delta_diff[k]:
 *   - a frame fires when its detector score is +inf (no compared frame) or
 *     above delta_diff; a frame that does not fire takes the reference label
 *     of the frame it is compared with (frame t - delta, or "no object" with
 *     a fixed reference image): fn_dd / fp_dd count those with label 1 / 0
 *     whose copied label is 0 / 1;
 *   - c_low is the smallest confidence v of a fired frame with
 *     fn_dd + #{fired, label 1, conf <= v} >= fn_target x positives (1 if
 *     none), c_high the largest v with fp_dd + #{fired, label 0, conf >= v}
 *     >= fp_target x negatives (0 if none), raised to c_low: the loosest
 *     thresholds whose false negative / positive rates stay strictly below
 *     the targets, frames below c_low labelled 0, above c_high 1, the others
 *     deferred to the reference network (counted as right);
 *   - cost = t_mse + f_m t_snn + f_m f_c t_full per frame, with f_m = fired
 *     / n, f_c = deferred / fired (every frame checked: f_s = 1).
 * A candidate is feasible when fn_dd and fp_dd alone stay below the
 * targets; an infeasible one reports c_low = 0, c_high = 1. */
typedef struct nsc_sweep_cfg {
  int32_t ref_mode;          /* NSC_REF_PREV or NSC_REF_FIXED                    */
  int32_t delta;             /* PREV: frames back, 1..NSC_MAX_DELTA              */
  double fp_target, fn_target; /* FP*, FN*: rates in [0, 1] (FP / frames without
                                the object, FN / frames with it)                 */
  double t_mse, t_snn, t_full; /* per-frame costs of the detector, the specialized
                                CNN and the reference network (finite, >= 0)     */
} nsc_sweep_cfg;

typedef struct nsc_sweep_row {  /* one per candidate, 120 bytes                  */
  double delta, c_low, c_high, f_m, f_c, cost;
  int64_t fired, deferred, fn_dd, fp_dd, fn_cnn, fp_cnn, positives, negatives;
  int32_t feasible, pad;
} nsc_sweep_row;

/* score: device, n doubles (the detector score of every frame, +inf for a
 * frame without a compared frame, as nsc_diff_detect writes them; no NaN);
 * conf: device, n floats in [0, 1] (the specialized CNN's confidence of every
 * frame); truth: device, n bytes (nonzero: the reference label says the
 * object is present); deltas: device, n_t candidate thresholds (1 ..
 * NSC_MAX_SWEEP); rows: device, n_t rows (written); best: device int32, the
 * index of the cheapest feasible candidate (the first on ties) or -1.  All
 * buffers are the caller's.  Enqueued on `stream`; the arguments are checked
 * on the host (NSC_E_INVAL), launch failures give NSC_E_HIP. */
int nsc_threshold_sweep(const nsc_sweep_cfg* cfg, const double* score, const float* conf,
                        const uint8_t* truth, int64_t n, const double* deltas, int32_t n_t,
                        nsc_sweep_row* rows, int32_t* best, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* NSC_H_ */
