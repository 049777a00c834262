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

// One thread renders 16 consecutive bytes of the [n][H][W][3] chunk.
__global__ void __launch_bounds__(256) render16(uint8_t* __restrict__ out, int64_t t0,
                                                int64_t total_bytes, int32_t H, int32_t W,
                                                uint64_t key, const uint8_t* __restrict__ bg,
                                                const int16_t* __restrict__ noise,
                                                const int8_t* __restrict__ drift,
                                                const int32_t* __restrict__ rects, int32_t K) {
  const int64_t frame_bytes = (int64_t)H * W * 3;
  for (int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; chunk * 16 < total_bytes;
       chunk += (int64_t)gridDim.x * blockDim.x) {
    int64_t b = chunk * 16;
    int64_t lt = b / frame_bytes;
    int64_t rem = b - lt * frame_bytes;
    int64_t pix_in_frame = rem / 3;
    int c = (int)(rem - pix_in_frame * 3);
    int y = (int)(pix_in_frame / W);
    int x = (int)(pix_in_frame - (int64_t)y * W);
    int64_t t = t0 + lt;
    uint8_t vals[16];
    uint64_t h = 0;
    bool have_h = false;
    for (int k = 0; k < 16; ++k) {
      if (b + k >= total_bytes) {
        vals[k] = 0;
        continue;
      }
      if (!have_h) {
        uint64_t pix = ((uint64_t)t * (uint64_t)H + (uint64_t)y) * (uint64_t)W + (uint64_t)x;
        h = mix64(key + (pix + 1ull) * kGolden);
        have_h = true;
      }
      int base = bg[((int64_t)y * W + x) * 3 + c];
      const int32_t* r = rects + (t * K) * kRectFields;
      for (int j = 0; j < K; ++j, r += kRectFields) {
        if (r[7] && x >= r[0] && x < r[2] && y >= r[1] && y < r[3]) base = r[4 + c];
      }
      int v = base + (int)drift[t] + (int)noise[(h >> (16 * c)) & 0xFFFFull];
      vals[k] = (uint8_t)(v < 0 ? 0 : (v > 255 ? 255 : v));
      // advance to the next byte
      if (++c == 3) {
        c = 0;
        have_h = false;
        if (++x == W) {
          x = 0;
          if (++y == H) {
            y = 0;
            ++t;
          }
        }
      }
    }
    if (b + 16 <= total_bytes) {
      uint4 v;
      v.x = vals[0] | (vals[1] << 8) | (vals[2] << 16) | ((uint32_t)vals[3] << 24);
      v.y = vals[4] | (vals[5] << 8) | (vals[6] << 16) | ((uint32_t)vals[7] << 24);
      v.z = vals[8] | (vals[9] << 8) | (vals[10] << 16) | ((uint32_t)vals[11] << 24);
      v.w = vals[12] | (vals[13] << 8) | (vals[14] << 16) | ((uint32_t)vals[15] << 24);
      *reinterpret_cast<uint4*>(out + b) = v;
    } else {
      for (int k = 0; b + k < total_bytes; ++k) out[b + k] = vals[k];
    }
  }
}

}  // namespace

// Renders frames [t0, t0 + n) of the video into `out` (device, n*H*W*3 bytes,
// 16-byte aligned).  Tables are device pointers: bg [H][W][3] uint8, noise
// [65536] int16, drift [n_total] int8, rects [n_total][K][8] int32.
// Returns 0 or the HIP error code of the launch.
extern "C" int synth_render(void* out, int64_t t0, int64_t n, int32_t H, int32_t W, uint64_t key,
                            const void* bg, const void* noise, const void* drift,
                            const void* rects, int32_t K, void* stream) {
  if (n <= 0) return 0;
  if (((uintptr_t)out & 15) != 0) return (int)hipErrorInvalidValue;
  int64_t total = n * (int64_t)H * W * 3;
  int64_t chunks = (total + 15) / 16;
  int64_t blocks = (chunks + 255) / 256;
  if (blocks > 65536 * 8) blocks = 65536 * 8;
  hipLaunchKernelGGL(render16, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                     (uint8_t*)out, t0, total, H, W, key, (const uint8_t*)bg,
                     (const int16_t*)noise, (const int8_t*)drift, (const int32_t*)rects, K);
  return (int)hipGetLastError();
}
