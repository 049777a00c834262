// Stream compaction of fired frames and label resolution (gfx950).
//
// Compaction (frames batched for the GPU model, Sec. 7): tiles of 4096 flags.
// A first kernel counts each tile with wave ballots; one workgroup turns the
// counts into exclusive tile offsets (a single scan, linear in the number of
// tiles) and writes the total; a third kernel scans each tile's four waves'
// counts in LDS and writes the ascending indices at the tile's offset with
// ballot + lane-mask popcounts, so the output order is the frame order.
//
// Resolution (Sec. 5: a frame on which the earlier-frame detector does not
// fire reuses the compared frame's output): frame u copies frame u - delta,
// so the decision of u is that of the last fired frame of its residue chain
// u, u - delta, u - 2 delta, ...; that is a running max of fired indices per
// residue class.  Frames are viewed as rows of `delta` columns, cut into
// tiles of rows: per-tile last fired index per column, an exclusive max-scan
// across tiles per column, and a per-tile sequential walk down each column.
#include "nsc_internal.h"

#include <mutex>

namespace nsc {
namespace {

constexpr int kTile = 4096;   // flags per compaction tile
constexpr int kTileThreads = 256;

__device__ __forceinline__ uint64_t lanemask_lt(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

__global__ void __launch_bounds__(kTileThreads) k_tile_count(const uint8_t* __restrict__ fire,
                                                             int64_t n,
                                                             int32_t* __restrict__ tile_counts) {
  __shared__ int32_t wsum[kTileThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)wave * (kTile / 4);
  int32_t c = 0;
  for (int s = 0; s < kTile / 4 / 64; ++s) {
    const int64_t u = base + s * 64 + lane;
    const bool f = u < n && fire[u] != 0;
    c += __popcll(__ballot(f));
  }
  if (lane == 0) wsum[wave] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t t = 0;
    for (int w = 0; w < kTileThreads / 64; ++w) t += wsum[w];
    tile_counts[blockIdx.x] = t;
  }
}

// Exclusive scan of the tile counts in place (tile offsets) and the total
// into *count; one workgroup walks the tiles 1024 at a time.
constexpr int kScanThreads = 1024;

__global__ void __launch_bounds__(kScanThreads) k_tile_scan(int32_t* __restrict__ tile_counts,
                                                            int64_t tiles,
                                                            int32_t* __restrict__ count) {
  __shared__ int32_t wsum[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int32_t carry = 0;  // the same in every thread
  for (int64_t b0 = 0; b0 < tiles; b0 += kScanThreads) {
    const int64_t b = b0 + tid;
    const int32_t v = b < tiles ? tile_counts[b] : 0;
    int32_t x = v;  // inclusive scan within the wave
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int32_t y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int32_t before = 0, total = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) {
      before += w < wave ? wsum[w] : 0;
      total += wsum[w];
    }
    if (b < tiles) tile_counts[b] = carry + before + x - v;
    carry += total;
    __syncthreads();  // wsum is rewritten by the next round
  }
  if (tid == 0) *count = carry;
}

__global__ void __launch_bounds__(kTileThreads) k_tile_scatter(const uint8_t* __restrict__ fire,
                                                               int64_t n,
                                                               const int32_t* __restrict__ tile_off,
                                                               int32_t* __restrict__ idx) {
  __shared__ int32_t wcount[kTileThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)wave * (kTile / 4);
  // pass 1: this wave's count
  int32_t c = 0;
  for (int st = 0; st < kTile / 4 / 64; ++st) {
    const int64_t u = base + st * 64 + lane;
    c += __popcll(__ballot(u < n && fire[u] != 0));
  }
  if (lane == 0) wcount[wave] = c;
  __syncthreads();
  int64_t off = tile_off[blockIdx.x];
  for (int w = 0; w < wave; ++w) off += wcount[w];
  // pass 2: write ascending indices
  for (int st = 0; st < kTile / 4 / 64; ++st) {
    const int64_t u = base + st * 64 + lane;
    const bool f = u < n && fire[u] != 0;
    const uint64_t m = __ballot(f);
    if (f) idx[off + __popcll(m & lanemask_lt(lane))] = (int32_t)u;
    off += __popcll(m);
  }
}

__global__ void k_set_i32(int32_t* p, int32_t v) { *p = v; }

// Survivors of one CNN pass: the slots [off, off + m) of the compacted list
// that exist, i.e. clamp(*count - off, 0, m).
__global__ void k_pass_count(const int32_t* __restrict__ count, int64_t off, int64_t m,
                             int32_t* __restrict__ out) {
  const int64_t left = (int64_t)*count - off;
  *out = (int32_t)(left < 0 ? 0 : left < m ? left : m);
}

// Per-tile last fired local index per residue column (or -1).
__global__ void __launch_bounds__(256) k_resolve_tile_last(const uint8_t* __restrict__ fire,
                                                           int64_t n, int32_t delta,
                                                           int32_t rows_per_tile,
                                                           int32_t* __restrict__ tile_last) {
  __shared__ int32_t last[NSC_MAX_DELTA];
  for (int r = threadIdx.x; r < delta; r += blockDim.x) last[r] = -1;
  __syncthreads();
  const int64_t u0 = (int64_t)blockIdx.x * rows_per_tile * delta;
  const int64_t span = (int64_t)rows_per_tile * delta;
  for (int64_t k = threadIdx.x; k < span; k += blockDim.x) {
    const int64_t u = u0 + k;
    if (u < n && fire[u]) atomicMax(&last[(int)(u % delta)], (int32_t)u);
  }
  __syncthreads();
  for (int r = threadIdx.x; r < delta; r += blockDim.x)
    tile_last[(int64_t)blockIdx.x * delta + r] = last[r];
}

// carry[b][r] = max over tiles b' < b of tile_last[b'][r]; one block per column.
__global__ void __launch_bounds__(1024) k_resolve_carry(const int32_t* __restrict__ tile_last,
                                                        int32_t tiles, int32_t delta,
                                                        int32_t* __restrict__ carry) {
  __shared__ int32_t v[1024];
  const int r = blockIdx.x, b = threadIdx.x;
  v[b] = b < tiles ? tile_last[(int64_t)b * delta + r] : -1;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    const int32_t x = b >= o ? v[b - o] : -1;
    __syncthreads();
    if (x > v[b]) v[b] = x;
    __syncthreads();
  }
  if (b < tiles) carry[(int64_t)b * delta + r] = b > 0 ? v[b - 1] : -1;
}

// Walks each residue column of a tile and writes label / defer.
__global__ void __launch_bounds__(256) k_resolve_apply(const uint8_t* __restrict__ fire,
                                                       const uint8_t* __restrict__ dec,
                                                       const uint8_t* __restrict__ prev_dec,
                                                       int64_t n, int32_t delta,
                                                       int32_t rows_per_tile,
                                                       const int32_t* __restrict__ carry,
                                                       uint8_t* __restrict__ label,
                                                       uint8_t* __restrict__ defer) {
  for (int r = threadIdx.x; r < delta; r += blockDim.x) {
    int32_t cur = carry[(int64_t)blockIdx.x * delta + r];
    const int64_t row0 = (int64_t)blockIdx.x * rows_per_tile;
    for (int q = 0; q < rows_per_tile; ++q) {
      const int64_t u = (row0 + q) * delta + r;
      if (u >= n) break;
      if (fire[u]) cur = (int32_t)u;
      // no fired frame of this chain in the call: continue the carried state
      const uint8_t d = cur >= 0 ? dec[cur] : (prev_dec ? prev_dec[r] : (uint8_t)0);
      label[u] = d & 1;
      defer[u] = (d >> 1) & 1;
    }
  }
}

// Fixed reference image: a frame that does not fire is labelled "no object".
__global__ void __launch_bounds__(256) k_resolve_fixed(const uint8_t* __restrict__ fire,
                                                       const uint8_t* __restrict__ dec, int64_t n,
                                                       uint8_t* __restrict__ label,
                                                       uint8_t* __restrict__ defer) {
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < n;
       u += (int64_t)gridDim.x * blockDim.x) {
    const uint8_t d = fire[u] ? dec[u] : (uint8_t)0;
    label[u] = d & 1;
    defer[u] = (d >> 1) & 1;
  }
}

// State of the last `delta` frames after a call of n frames.  When n < delta
// the old state is read from `old_*` (a copy), otherwise only from this call.
__global__ void __launch_bounds__(256) k_state_update(const int32_t* __restrict__ sums,
                                                      const uint8_t* __restrict__ label,
                                                      const uint8_t* __restrict__ defer, int64_t n,
                                                      int32_t delta, int64_t cells,
                                                      const int32_t* __restrict__ old_sums,
                                                      const uint8_t* __restrict__ old_dec,
                                                      int32_t* __restrict__ st_sums,
                                                      uint8_t* __restrict__ st_dec) {
  const int64_t total = (int64_t)delta * cells;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = e / cells, c = e - k * cells;
    const int64_t src = n - delta + k;  // local index of the frame kept in slot k
    st_sums[e] = src >= 0 ? sums[src * cells + c] : old_sums[(k + n) * cells + c];
    if (c == 0)
      st_dec[k] = src >= 0 ? (uint8_t)(label[src] | (defer[src] << 1)) : old_dec[k + n];
  }
}

// Camera group: one workgroup per camera resolves its n frames (frames
// cam * n .. cam * n + n - 1 of the batch).  Earlier-frame cameras walk each
// residue column down its chain (the decision of the last fired frame, else
// the state slot's); fixed-reference cameras label non-firing frames 0.
__global__ void __launch_bounds__(256) k_group_resolve(const CamDiff* __restrict__ cams,
                                                       const uint8_t* __restrict__ fire,
                                                       const uint8_t* __restrict__ dec, int64_t n,
                                                       int64_t t0,
                                                       const unsigned char* __restrict__ state,
                                                       int64_t state_stride,
                                                       uint8_t* __restrict__ label,
                                                       uint8_t* __restrict__ defer) {
  const int64_t cam = blockIdx.x;
  const CamDiff cd = cams[cam];
  const int64_t base = cam * n;
  if (cd.ref_mode == NSC_REF_FIXED) {
    for (int64_t u = threadIdx.x; u < n; u += blockDim.x) {
      const uint8_t d = fire[base + u] ? dec[base + u] : (uint8_t)0;
      label[base + u] = d & 1;
      defer[base + u] = (d >> 1) & 1;
    }
    return;
  }
  const uint8_t* st_dec = state + cam * state_stride + cd.dec_off;
  for (int r = threadIdx.x; r < cd.delta; r += blockDim.x) {
    // frames of the chain before the call: slot r holds frame t0 - delta + r
    // (frames t < delta always fire, so t0 = 0 never reads it)
    uint8_t d = t0 > 0 ? st_dec[r] : (uint8_t)0;
    for (int64_t u = r; u < n; u += cd.delta) {
      if (fire[base + u]) d = dec[base + u];
      label[base + u] = d & 1;
      defer[base + u] = (d >> 1) & 1;
    }
  }
}

// Camera group state after a call of n frames per camera: every earlier-frame
// camera keeps the sums and decisions of its last delta frames in its slot.
// `old` is a copy of the state before the call, read where n < delta.
__global__ void __launch_bounds__(256) k_group_state(const CamDiff* __restrict__ cams,
                                                     const int32_t* __restrict__ sums,
                                                     const uint8_t* __restrict__ label,
                                                     const uint8_t* __restrict__ defer, int64_t n,
                                                     int64_t cells,
                                                     const unsigned char* __restrict__ old,
                                                     unsigned char* __restrict__ state,
                                                     int64_t state_stride) {
  const int64_t cam = blockIdx.y;
  const CamDiff cd = cams[cam];
  if (cd.ref_mode != NSC_REF_PREV) return;
  const int64_t total = (int64_t)cd.delta * cells;
  int32_t* st_sums = reinterpret_cast<int32_t*>(state + cam * state_stride);
  uint8_t* st_dec = state + cam * state_stride + cd.dec_off;
  const int32_t* o_sums = reinterpret_cast<const int32_t*>(old + cam * state_stride);
  const uint8_t* o_dec = old + cam * state_stride + cd.dec_off;
  const int64_t base = cam * n;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = e / cells, c = e - k * cells;
    const int64_t src = n - cd.delta + k;  // local index of the frame kept in slot k
    st_sums[e] = src >= 0 ? sums[(base + src) * cells + c] : o_sums[(k + n) * cells + c];
    if (c == 0)
      st_dec[k] = src >= 0 ? (uint8_t)(label[base + src] | (defer[base + src] << 1))
                           : o_dec[k + n];
  }
}

// Frame skipping (Sec. 5): each frame takes its checked frame's output.
__global__ void __launch_bounds__(256) k_skip_expand(SkipExpand e) {
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < e.n;
       u += (int64_t)gridDim.x * blockDim.x) {
    const int64_t t = e.t0 + u;
    const int64_t k = t / e.s;
    const bool checked = k * e.s == t;  // then k >= k0
    uint8_t l, d;
    if (k >= e.k0) {
      l = e.k_label[k - e.k0];
      d = e.k_defer[k - e.k0];
    } else {
      const uint8_t v = *e.last;
      l = v & 1;
      d = (v >> 1) & 1;
    }
    e.label[u] = l;
    e.defer[u] = d;
    if (e.score) e.score[u] = checked ? e.k_score[k - e.k0] : __builtin_nan("");
    if (e.fire) e.fire[u] = checked ? e.k_fire[k - e.k0] : 0;
    if (e.logit) e.logit[u] = checked ? e.k_logit[k - e.k0] : __builtin_nanf("");
  }
}

__global__ void k_skip_last(const uint8_t* __restrict__ label, const uint8_t* __restrict__ defer,
                            int64_t nc, uint8_t* __restrict__ last) {
  if (threadIdx.x == 0) *last = (uint8_t)(label[nc - 1] | (defer[nc - 1] << 1));
}

__global__ void __launch_bounds__(256) k_copy_u8(const uint8_t* __restrict__ s,
                                                 uint8_t* __restrict__ d, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    d[i] = s[i];
}

__global__ void __launch_bounds__(256) k_fill_nan(float* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = __builtin_nanf("");
}

unsigned grid_for(int64_t n, int per_block) {
  int64_t b = (n + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > kNumCU * 16) b = kNumCU * 16;
  return (unsigned)b;
}

}  // namespace

int64_t compact_tiles(int64_t n) { return (n + kTile - 1) / kTile; }

int launch_compact(const uint8_t* fire, int64_t n, int32_t* idx, int32_t* count,
                   int32_t* tile_counts, hipStream_t stream) {
  if (n <= 0) {
    hipLaunchKernelGGL(k_set_i32, dim3(1), dim3(1), 0, stream, count, 0);
    NSC_CHECK_LAUNCH("k_set_i32");
    return NSC_OK;
  }
  const int64_t tiles = compact_tiles(n);
  hipLaunchKernelGGL(k_tile_count, dim3((unsigned)tiles), dim3(kTileThreads), 0, stream, fire, n,
                     tile_counts);
  NSC_CHECK_LAUNCH("k_tile_count");
  hipLaunchKernelGGL(k_tile_scan, dim3(1), dim3(kScanThreads), 0, stream, tile_counts, tiles,
                     count);
  NSC_CHECK_LAUNCH("k_tile_scan");
  hipLaunchKernelGGL(k_tile_scatter, dim3((unsigned)tiles), dim3(kTileThreads), 0, stream, fire, n,
                     tile_counts, idx);
  NSC_CHECK_LAUNCH("k_tile_scatter");
  return NSC_OK;
}

// Compaction without a caller workspace, for callers that cannot allocate:
// the tile offsets live in this file-scope device array (every GPU holds its
// own copy until the process ends), so at most NSC_NOALLOC_MAX_FLAGS flags
// (kNoAllocTiles tiles) per call.  Every call on one GPU shares the array:
// calls that overlap on a GPU race.  Nothing in it has to start at zero
// (each call writes every tile count it reads).
constexpr int64_t kNoAllocTiles = NSC_NOALLOC_MAX_FLAGS / kTile;
static_assert(NSC_NOALLOC_MAX_FLAGS % kTile == 0, "the flag limit is whole tiles");
static __device__ __align__(256) int32_t scratch[kNoAllocTiles];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int32_t* g_scratch[kMaxDevices] = {};
}  // namespace

// Device address of the current device's copy of `scratch`, looked up once per
// device (the array's name in host code is not a device address).
int noalloc_scratch(int32_t** out) {
  int dev = -1;
  NSC_TRY_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(NSC_E_HIP, "device %d beyond the %d devices the static scratch tracks", dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(NSC_E_HIP, "hipGetSymbolAddress of the compaction scratch failed on device %d: %s",
                  dev, hipGetErrorString(e));
    g_scratch[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch[dev];
  return NSC_OK;
}

int launch_compact_noalloc(const uint8_t* fire, int64_t n, int32_t* idx, int32_t* count,
                           hipStream_t stream) {
  if (compact_tiles(n) > kNoAllocTiles)
    return fail(NSC_E_WORKSPACE, "%lld flags exceed the static scratch's %lld", (long long)n,
                (long long)NSC_NOALLOC_MAX_FLAGS);
  int32_t* tiles = nullptr;
  if (int rc = noalloc_scratch(&tiles)) return rc;
  return launch_compact(fire, n, idx, count, tiles, stream);
}

ResolvePlan make_resolve_plan(int64_t n, int64_t t0, int32_t delta) {
  ResolvePlan p{};
  p.n = n;
  p.t0 = t0;
  p.delta = delta < 1 ? 1 : delta;
  const int64_t rows = (n + p.delta - 1) / p.delta;
  int64_t rpt = (rows + 1023) / 1024;
  if (rpt < 1) rpt = 1;
  p.rows_per_tile = (int32_t)rpt;
  p.tiles = (int32_t)((rows + rpt - 1) / rpt);
  if (p.tiles < 1) p.tiles = 1;
  return p;
}

int launch_resolve(const ResolvePlan& p, int32_t ref_mode, const uint8_t* fire, const uint8_t* dec,
                   const uint8_t* prev_dec, int32_t* tile_last, int32_t* carry, uint8_t* label,
                   uint8_t* defer, hipStream_t stream) {
  if (p.n <= 0) return NSC_OK;
  if (ref_mode == NSC_REF_FIXED) {
    hipLaunchKernelGGL(k_resolve_fixed, dim3(grid_for(p.n, 256)), dim3(256), 0, stream, fire, dec,
                       p.n, label, defer);
    NSC_CHECK_LAUNCH("k_resolve_fixed");
    return NSC_OK;
  }
  hipLaunchKernelGGL(k_resolve_tile_last, dim3(p.tiles), dim3(256), 0, stream, fire, p.n, p.delta,
                     p.rows_per_tile, tile_last);
  NSC_CHECK_LAUNCH("k_resolve_tile_last");
  hipLaunchKernelGGL(k_resolve_carry, dim3(p.delta), dim3(1024), 0, stream, tile_last, p.tiles,
                     p.delta, carry);
  NSC_CHECK_LAUNCH("k_resolve_carry");
  hipLaunchKernelGGL(k_resolve_apply, dim3(p.tiles), dim3(256), 0, stream, fire, dec,
                     p.t0 > 0 ? prev_dec : nullptr, p.n, p.delta, p.rows_per_tile, carry, label,
                     defer);
  NSC_CHECK_LAUNCH("k_resolve_apply");
  return NSC_OK;
}

int launch_state_update(const int32_t* sums, const uint8_t* label, const uint8_t* defer, int64_t n,
                        int32_t delta, int64_t cells, int32_t* state_sums, uint8_t* state_dec,
                        void* scratch, hipStream_t stream) {
  if (n <= 0) return NSC_OK;
  const int32_t* old_sums = state_sums;
  const uint8_t* old_dec = state_dec;
  if (n < delta) {
    // slots k < delta - n keep frames of the previous state: copy it first
    uint8_t* s = static_cast<uint8_t*>(scratch);
    const int64_t sb = (int64_t)delta * cells * 4;
    hipLaunchKernelGGL(k_copy_u8, dim3(grid_for(sb, 256)), dim3(256), 0, stream,
                       reinterpret_cast<const uint8_t*>(state_sums), s, sb);
    NSC_CHECK_LAUNCH("k_copy_u8");
    hipLaunchKernelGGL(k_copy_u8, dim3(1), dim3(256), 0, stream, state_dec, s + sb, (int64_t)delta);
    NSC_CHECK_LAUNCH("k_copy_u8");
    old_sums = reinterpret_cast<const int32_t*>(s);
    old_dec = s + sb;
  }
  hipLaunchKernelGGL(k_state_update, dim3(grid_for((int64_t)delta * cells, 256)), dim3(256), 0,
                     stream, sums, label, defer, n, delta, cells, old_sums, old_dec, state_sums,
                     state_dec);
  NSC_CHECK_LAUNCH("k_state_update");
  return NSC_OK;
}

int launch_group_resolve(const CamDiff* cams, int32_t n_cams, const uint8_t* fire,
                         const uint8_t* dec, int64_t n, int64_t t0, const unsigned char* state,
                         int64_t state_stride, uint8_t* label, uint8_t* defer,
                         hipStream_t stream) {
  if (n <= 0 || n_cams <= 0) return NSC_OK;
  hipLaunchKernelGGL(k_group_resolve, dim3((unsigned)n_cams), dim3(256), 0, stream, cams, fire,
                     dec, n, t0, state, state_stride, label, defer);
  NSC_CHECK_LAUNCH("k_group_resolve");
  return NSC_OK;
}

int launch_group_state(const CamDiff* cams, int32_t n_cams, int32_t max_delta,
                       const int32_t* sums, const uint8_t* label, const uint8_t* defer, int64_t n,
                       int64_t cells, unsigned char* state, int64_t state_stride, void* scratch,
                       hipStream_t stream) {
  if (n <= 0 || n_cams <= 0 || max_delta <= 0) return NSC_OK;
  const unsigned char* old = state;
  if (n < max_delta) {
    // slots k < delta - n keep frames of the previous state: copy it first
    unsigned char* cp = static_cast<unsigned char*>(scratch);
    const int64_t bytes = (int64_t)n_cams * state_stride;
    hipLaunchKernelGGL(k_copy_u8, dim3(grid_for(bytes, 256)), dim3(256), 0, stream, state, cp,
                       bytes);
    NSC_CHECK_LAUNCH("k_copy_u8");
    old = cp;
  }
  const unsigned gx = grid_for((int64_t)max_delta * cells, 256);
  hipLaunchKernelGGL(k_group_state, dim3(gx, (unsigned)n_cams), dim3(256), 0, stream, cams, sums,
                     label, defer, n, cells, old, state, state_stride);
  NSC_CHECK_LAUNCH("k_group_state");
  return NSC_OK;
}

int launch_pass_count(const int32_t* count, int64_t off, int64_t m, int32_t* out,
                      hipStream_t stream) {
  hipLaunchKernelGGL(k_pass_count, dim3(1), dim3(1), 0, stream, count, off, m, out);
  NSC_CHECK_LAUNCH("k_pass_count");
  return NSC_OK;
}

int launch_set_i32(int32_t* p, int32_t v, hipStream_t stream) {
  hipLaunchKernelGGL(k_set_i32, dim3(1), dim3(1), 0, stream, p, v);
  NSC_CHECK_LAUNCH("k_set_i32");
  return NSC_OK;
}

int launch_skip_expand(const SkipExpand& e, hipStream_t stream) {
  if (e.n <= 0) return NSC_OK;
  hipLaunchKernelGGL(k_skip_expand, dim3(grid_for(e.n, 256)), dim3(256), 0, stream, e);
  NSC_CHECK_LAUNCH("k_skip_expand");
  if (e.nc > 0) {  // after every reader of the previous value
    hipLaunchKernelGGL(k_skip_last, dim3(1), dim3(64), 0, stream, e.k_label, e.k_defer, e.nc,
                       e.last);
    NSC_CHECK_LAUNCH("k_skip_last");
  }
  return NSC_OK;
}

int launch_fill_nan(float* p, int64_t n, hipStream_t stream) {
  if (n <= 0) return NSC_OK;
  hipLaunchKernelGGL(k_fill_nan, dim3(grid_for(n, 256)), dim3(256), 0, stream, p, n);
  NSC_CHECK_LAUNCH("k_fill_nan");
  return NSC_OK;
}

int launch_copy_u8(const uint8_t* src, uint8_t* dst, int64_t n, hipStream_t stream) {
  if (n <= 0) return NSC_OK;
  hipLaunchKernelGGL(k_copy_u8, dim3(grid_for(n, 256)), dim3(256), 0, stream, src, dst, n);
  NSC_CHECK_LAUNCH("k_copy_u8");
  return NSC_OK;
}

}  // namespace nsc
