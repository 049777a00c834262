// Device renderer of the synthetic fixed-camera video.
//
// Input infrastructure shared by tests and the benchmark, not part of the
// cascade: it computes, per byte, exactly the integer rule that the host
// renderer in synth/__init__.py computes, from the same host-built tables.
//   base  = colour of the last active rectangle covering (x, y), else bg
//   noise = T[(splitmix64(key + (pix + 1) * GOLDEN) >> 16c) & 0xFFFF]
//   value = clamp(base + drift[t] + noise, 0, 255)
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kMix1 = 0xBF58476D1CE4E5B9ull;
constexpr uint64_t kMix2 = 0x94D049BB133111EBull;
constexpr int kRectFields = 8;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * kMix1;
  z = (z ^ (z >> 27)) * kMix2;
  return z ^ (z >> 31);
}

constexpr int kNoiseEntries = 65536;
constexpr int kMaxRects = 32;

// One workgroup per CU holds the 128 KB noise table in LDS (the per-byte
// lookups are random, so from L2 they would bound the rate) and loops over work
// items: a frame, or a segment of a frame's 16-byte chunks when there are few
// frames.  One thread renders 16 consecutive bytes of one frame; the pixel's
// hash, colour and rectangle cover are computed once per pixel (3 bytes).
// Frame-uniform values (the rectangle table row, the drift) are read once per
// item; the rectangle row goes to LDS, and each thread keeps a bit mask of the
// rectangles that cover its row so that a pixel tests only those.
__global__ void __launch_bounds__(1024) render_frames(uint8_t* __restrict__ out, int64_t t0,
                                                      int64_t n, int32_t segs, int32_t H, int32_t W,
                                                      uint64_t key, const uint8_t* __restrict__ bg,
                                                      const int16_t* __restrict__ noise,
                                                      const int8_t* __restrict__ drift,
                                                      const int32_t* __restrict__ rects, int32_t K) {
  extern __shared__ __align__(16) int16_t tab[];
  __shared__ int32_t rt[kMaxRects * kRectFields];
  for (int i = threadIdx.x; i < kNoiseEntries / 8; i += blockDim.x)
    reinterpret_cast<uint4*>(tab)[i] = reinterpret_cast<const uint4*>(noise)[i];
  __syncthreads();
  const int32_t fb = H * W * 3;
  const int32_t chunks = (fb + 15) / 16;
  const int32_t per_seg = (chunks + segs - 1) / segs;
  const bool aligned = (fb & 15) == 0;
  for (int64_t item = blockIdx.x; item < n * segs; item += gridDim.x) {
    const int64_t f = item / segs;
    const int32_t seg = (int32_t)(item - f * segs);
    const int64_t t = t0 + f;
    const int32_t* R = rects + t * K * kRectFields;
    __syncthreads();  // the previous item's readers of rt are done
    for (int i = threadIdx.x; i < K * kRectFields; i += blockDim.x) rt[i] = R[i];
    __syncthreads();
    const int dr = drift[t];
    auto row_mask = [&](int yy) {
      uint32_t m = 0;
      for (int j = 0; j < K; ++j) {
        const int32_t* r = rt + j * kRectFields;
        if (r[7] && yy >= r[1] && yy < r[3]) m |= 1u << j;
      }
      return m;
    };
    uint8_t* fo = out + f * (int64_t)fb;
    const int32_t c1 = min(chunks, (seg + 1) * per_seg);
    for (int32_t ch = seg * per_seg + threadIdx.x; ch < c1; ch += blockDim.x) {
      const int32_t b = ch * 16;
      int32_t pix = b / 3;
      int c = b - pix * 3;
      int y = pix / W;
      int x = pix - y * W;
      uint8_t vals[16];
      int base[3] = {0, 0, 0};
      uint64_t h = 0;
      uint32_t rows = row_mask(y);
      for (int k = 0; k < 16; ++k) {
        if (b + k >= fb) {
          vals[k] = 0;
          continue;
        }
        if (k == 0 || c == 0) {  // entering a pixel
          const uint64_t gp = ((uint64_t)t * (uint64_t)H + (uint64_t)y) * (uint64_t)W + (uint64_t)x;
          h = mix64(key + (gp + 1ull) * kGolden);
          const uint8_t* bp = bg + ((int64_t)y * W + x) * 3;
          base[0] = bp[0];
          base[1] = bp[1];
          base[2] = bp[2];
          for (uint32_t mm = rows; mm; mm &= mm - 1) {  // ascending: the last cover wins
            const int32_t* r = rt + (__builtin_ctz(mm)) * kRectFields;
            if (x >= r[0] && x < r[2]) {
              base[0] = r[4];
              base[1] = r[5];
              base[2] = r[6];
            }
          }
        }
        const int v = base[c] + dr + (int)tab[(h >> (16 * c)) & 0xFFFFull];
        vals[k] = (uint8_t)(v < 0 ? 0 : (v > 255 ? 255 : v));
        if (++c == 3) {
          c = 0;
          if (++x == W) {
            x = 0;
            ++y;
            if (y < H) rows = row_mask(y);
          }
        }
      }
      if (aligned && b + 16 <= fb) {
        uint4 v;
        v.x = vals[0] | (vals[1] << 8) | (vals[2] << 16) | ((uint32_t)vals[3] << 24);
        v.y = vals[4] | (vals[5] << 8) | (vals[6] << 16) | ((uint32_t)vals[7] << 24);
        v.z = vals[8] | (vals[9] << 8) | (vals[10] << 16) | ((uint32_t)vals[11] << 24);
        v.w = vals[12] | (vals[13] << 8) | (vals[14] << 16) | ((uint32_t)vals[15] << 24);
        *reinterpret_cast<uint4*>(fo + b) = v;
      } else {
        for (int k = 0; k < 16 && b + k < fb; ++k) fo[b + k] = vals[k];
      }
    }
  }
}

// The same rule for frames of a whole number of 16-pixel groups (H*W a
// multiple of 16, so every group starts 16-byte aligned): a thread renders
// one group, 48 bytes written as three 16-byte stores.  Byte positions are
// compile-time constants (the background's 48 bytes are read as three
// 16-byte loads), the hash input of consecutive pixels advances by GOLDEN,
// and the rectangle masks are recomputed only when a group crosses a row.
__global__ void __launch_bounds__(1024) render_groups(uint8_t* __restrict__ out, int64_t t0,
                                                      int64_t n, int32_t segs, int32_t H, int32_t W,
                                                      uint64_t key, const uint8_t* __restrict__ bg,
                                                      const int16_t* __restrict__ noise,
                                                      const int8_t* __restrict__ drift,
                                                      const int32_t* __restrict__ rects, int32_t K) {
  extern __shared__ __align__(16) int16_t tab[];
  __shared__ int32_t rt[kMaxRects * kRectFields];
  for (int i = threadIdx.x; i < kNoiseEntries / 8; i += blockDim.x)
    reinterpret_cast<uint4*>(tab)[i] = reinterpret_cast<const uint4*>(noise)[i];
  __syncthreads();
  const int32_t groups = H * W / 16;
  const int32_t per_seg = (groups + segs - 1) / segs;
  for (int64_t item = blockIdx.x; item < n * segs; item += gridDim.x) {
    const int64_t f = item / segs;
    const int32_t seg = (int32_t)(item - f * segs);
    const int64_t t = t0 + f;
    const int32_t* R = rects + t * K * kRectFields;
    __syncthreads();  // the previous item's readers of rt are done
    for (int i = threadIdx.x; i < K * kRectFields; i += blockDim.x) rt[i] = R[i];
    __syncthreads();
    int live = 0;  // rectangles active in this frame (uniform)
    for (int j = 0; j < K; ++j) live |= rt[j * kRectFields + 7];
    const int dr = drift[t];
    auto row_mask = [&](int yy) {
      uint32_t m = 0;
      for (int j = 0; j < K; ++j) {
        const int32_t* r = rt + j * kRectFields;
        if (r[7] && yy >= r[1] && yy < r[3]) m |= 1u << j;
      }
      return m;
    };
    uint8_t* fo = out + f * (int64_t)H * W * 3;
    const int32_t g1 = min(groups, (seg + 1) * per_seg);
    for (int32_t gi = seg * per_seg + (int32_t)threadIdx.x; gi < g1; gi += blockDim.x) {
      const int32_t p0 = gi * 16;
      int y = p0 / W;
      int x = p0 - y * W;
      uint64_t hin = key + ((uint64_t)t * (uint64_t)H * (uint64_t)W + (uint64_t)p0 + 1ull) * kGolden;
      const uint4* bq = reinterpret_cast<const uint4*>(bg + (int64_t)p0 * 3);
      const uint4 q0 = bq[0], q1 = bq[1], q2 = bq[2];
      const uint32_t bw[12] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w,
                               q2.x, q2.y, q2.z, q2.w};
      uint32_t ow[12] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
      uint32_t rows = live ? row_mask(y) : 0u;
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const uint64_t h = mix64(hin);
        hin += kGolden;
        int b[3];
#pragma unroll
        for (int c = 0; c < 3; ++c) b[c] = (bw[(3 * k + c) >> 2] >> (8 * ((3 * k + c) & 3))) & 0xFF;
        for (uint32_t mm = rows; mm; mm &= mm - 1) {  // ascending: the last cover wins
          const int32_t* r = rt + (__builtin_ctz(mm)) * kRectFields;
          if (x >= r[0] && x < r[2]) {
            b[0] = r[4];
            b[1] = r[5];
            b[2] = r[6];
          }
        }
#pragma unroll
        for (int c = 0; c < 3; ++c) {
          int v = b[c] + dr + (int)tab[(uint32_t)(h >> (16 * c)) & 0xFFFFu];
          v = v < 0 ? 0 : (v > 255 ? 255 : v);
          ow[(3 * k + c) >> 2] |= (uint32_t)v << (8 * ((3 * k + c) & 3));
        }
        if (++x == W) {
          x = 0;
          ++y;
          if (live && y < H) rows = row_mask(y);
        }
      }
      uint4* o = reinterpret_cast<uint4*>(fo + (int64_t)p0 * 3);
      o[0] = make_uint4(ow[0], ow[1], ow[2], ow[3]);
      o[1] = make_uint4(ow[4], ow[5], ow[6], ow[7]);
      o[2] = make_uint4(ow[8], ow[9], ow[10], ow[11]);
    }
  }
}

}  // namespace

// Renders frames [t0, t0 + n) of the video into `out` (device, n*H*W*3 bytes,
// 16-byte aligned; frames of a whole number of 16-pixel groups take
// render_groups, other sizes render_frames, which writes a frame that is not
// a multiple of 16 bytes byte by byte).  Tables are device pointers: bg [H][W][3] uint8, noise
// [65536] int16, drift [n_total] int8, rects [n_total][K][8] int32 with K <= 32.
// Returns 0 or the HIP error code of the launch.
extern "C" int synth_render(void* out, int64_t t0, int64_t n, int32_t H, int32_t W, uint64_t key,
                            const void* bg, const void* noise, const void* drift,
                            const void* rects, int32_t K, void* stream) {
  if (n <= 0) return 0;
  if (((uintptr_t)out & 15) != 0) return (int)hipErrorInvalidValue;
  if ((int64_t)H * W * 3 > 0x7FFFFFF0 || K < 0 || K > kMaxRects) return (int)hipErrorInvalidValue;
  const int64_t chunks = ((int64_t)H * W * 3 + 15) / 16;
  // enough work items for 4 per workgroup, segments of at least 1024 chunks
  constexpr int64_t kBlocks = 256;
  int64_t segs = (4 * kBlocks + n - 1) / n;
  const int64_t max_segs = (chunks + 1023) / 1024;
  if (segs > max_segs) segs = max_segs;
  if (segs < 1) segs = 1;
  if (((int64_t)H * W) % 16 == 0 && ((uintptr_t)bg & 15) == 0) {
    const int64_t groups = (int64_t)H * W / 16;
    int64_t gsegs = (4 * kBlocks + n - 1) / n;
    const int64_t max_gsegs = (groups + 1023) / 1024;
    if (gsegs > max_gsegs) gsegs = max_gsegs;
    if (gsegs < 1) gsegs = 1;
    hipLaunchKernelGGL(render_groups, dim3((unsigned)kBlocks), dim3(1024),
                       kNoiseEntries * sizeof(int16_t), (hipStream_t)stream, (uint8_t*)out, t0, n,
                       (int32_t)gsegs, H, W, key, (const uint8_t*)bg, (const int16_t*)noise,
                       (const int8_t*)drift, (const int32_t*)rects, K);
    return (int)hipGetLastError();
  }
  hipLaunchKernelGGL(render_frames, dim3((unsigned)kBlocks), dim3(1024),
                     kNoiseEntries * sizeof(int16_t), (hipStream_t)stream, (uint8_t*)out, t0, n,
                     (int32_t)segs, H, W, key, (const uint8_t*)bg, (const int16_t*)noise,
                     (const int8_t*)drift, (const int32_t*)rects, K);
  return (int)hipGetLastError();
}
