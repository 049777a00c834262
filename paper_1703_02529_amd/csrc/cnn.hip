// Specialized CNN on the survivors (Sec. 4 model, Sec. 7 pre-processing), gfx950.
//
// Conv layers run as implicit GEMM on 16x16 MFMA tiles: M = 16 output pixels
// of a 4x4 tile, N = 16 output channels, K = 9 taps x input channels.  The
// 16 pixels are ordered so that each lane's four accumulator rows form one
// 2x2 pooling window, so bias + ReLU + 2x2 max-pool happen in registers in
// the epilogue.  A workgroup stages the layer's packed weights in
// LDS once and then loops over (image, tile-row) work items, staging the
// input band (4 output rows + halo, zero padded) in LDS per item.  The first
// layer's staging gathers the survivor's area sums, sums nested cells and
// applies the [-1, 1] pre-processing.  bf16 layers use
// v_mfma_f32_16x16x32_bf16, fp32 layers v_mfma_f32_16x16x4_f32; both
// accumulate in fp32.
//
// Activations between layers are fp32 in the workspace.  A bf16 network has
// bf16 weights and a bf16-rounded input; each later activation a enters the
// bf16 matrix cores as the pair hi = bf16(a), lo = bf16(a - hi) (the
// difference is exact in fp32), multiplied by the same weights into a second
// accumulator.  a is then carried to about 2^-17 of itself, so the result is a
// continuous function of the fp32 accumulation error instead of flipping
// bf16 roundings of intermediate values.
//
// The dense layer is a GEMM over 16-survivor tiles (M) x hidden units (N) x
// features (K) on the same MFMA shapes; its epilogue adds the bias, applies
// ReLU, folds the 1-unit output layer in with a 16-lane
// shuffle reduction, and writes the logit, the sigmoid confidence and the
// c_low / c_high decision of each frame.
#include "nsc_internal.h"

#include <math.h>

namespace nsc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- numerics

// Round an fp32 value to bf16 (nearest, ties to even); finite inputs.
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}
// Round an fp64 value straight to bf16 (nearest, ties to even; finite, normal
// range): keep 8 significant bits of the 53.
__device__ __forceinline__ uint16_t f64_to_bf16_bits(double d) {
  uint64_t u = (uint64_t)__double_as_longlong(d);
  u += 0x0FFFFFFFFFFFull + ((u >> 45) & 1ull);
  u &= ~0x1FFFFFFFFFFFull;
  return (uint16_t)(__float_as_uint((float)__longlong_as_double((long long)u)) >> 16);
}

// Element-type traits: E = elements per lane per MFMA, KS = K per MFMA.
template <typename T> struct Elt;
template <> struct Elt<uint16_t> {  // bf16 stored as raw bits
  static constexpr int E = 8, KS = 32;
  typedef bf16x8 frag;
  static __device__ __forceinline__ uint16_t from_f32(float v) { return f32_to_bf16_bits(v); }
  static __device__ __forceinline__ uint16_t from_f64(double v) { return f64_to_bf16_bits(v); }
  static __device__ __forceinline__ float to_f32(uint16_t v) { return bf16_bits_to_f32(v); }
  static __device__ __forceinline__ f32x4 mma(const frag& a, const frag& b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag load(const uint16_t* p) {  // 16-byte aligned
    return *reinterpret_cast<const frag*>(p);
  }
  static __device__ __forceinline__ frag load8(const uint16_t* p) {  // 8-byte aligned
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    const bf16x4 lo = *reinterpret_cast<const bf16x4*>(p);
    const bf16x4 hi = *reinterpret_cast<const bf16x4*>(p + 4);
    return frag{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  }
  static __device__ __forceinline__ frag zero() {
    frag z;
#pragma unroll
    for (int e = 0; e < 8; ++e) z[e] = (__bf16)0.0f;
    return z;
  }
  static __device__ __forceinline__ void set(frag& f, int e, uint16_t v) {
    f[e] = __builtin_bit_cast(__bf16, v);
  }
  // Activations enter as hi + lo pairs (see the top of this file).
  static constexpr bool SPLIT = true;
  static __device__ __forceinline__ void split1(float v, uint16_t& hi, uint16_t& lo) {
    hi = f32_to_bf16_bits(v);
    lo = f32_to_bf16_bits(v - bf16_bits_to_f32(hi));
  }
  // 4 fp32 values -> 4 hi and 4 lo bf16 values, packed pairwise in uint2
  static __device__ __forceinline__ void split4(const float4& v, uint2& hi, uint2& lo) {
    uint16_t h[4], l[4];
    split1(v.x, h[0], l[0]);
    split1(v.y, h[1], l[1]);
    split1(v.z, h[2], l[2]);
    split1(v.w, h[3], l[3]);
    hi = make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
    lo = make_uint2((uint32_t)l[0] | ((uint32_t)l[1] << 16), (uint32_t)l[2] | ((uint32_t)l[3] << 16));
  }
  // A fragment pair from 8 consecutive fp32 values (16-byte aligned)
  static __device__ __forceinline__ void split8(const float* p, frag& hi, frag& lo) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint16_t h, l;
      split1(v[e], h, l);
      set(hi, e, h);
      set(lo, e, l);
    }
  }
};
template <> struct Elt<float> {
  static constexpr int E = 1, KS = 4;
  typedef float frag;
  static __device__ __forceinline__ float from_f32(float v) { return v; }
  static __device__ __forceinline__ float from_f64(double v) { return (float)v; }
  static __device__ __forceinline__ float to_f32(float v) { return v; }
  static __device__ __forceinline__ f32x4 mma(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ float load(const float* p) { return *p; }
  static __device__ __forceinline__ float load8(const float* p) { return *p; }
  static __device__ __forceinline__ float zero() { return 0.0f; }
  static __device__ __forceinline__ void set(float& f, int, float v) { f = v; }
  static constexpr bool SPLIT = false;
};

// ------------------------------------------------------------------- conv

struct ConvArgs {
  // input: the first layer reads area sums of frame idx[s]; others read act_in[s]
  const int32_t* sums;
  const int32_t* idx;
  int32_t sums_h, sums_w, fy, fx;
  int64_t den255;           // 255 * den_c: pre-processing x = (2 S - den255) / den255
  const float* act_in;      // [slot][h][w][cin] fp32
  float* act_out;           // [slot][ho][wo][cout] fp32
  const void* wts;          // packed [cout][kpad]
  const float* bias;        // [cout]
  const int32_t* count;
  int64_t max_count;
  int32_t cin, cout, h, w, kpad;
  int32_t pool;
  int32_t tiles_y, tiles_x;
  int32_t band_tiles;       // tile rows per work item
  int32_t seg_tiles;        // tile columns per work item
  int32_t cin_lds;          // channel stride of a staged pixel (elements)
  int32_t w_lds;            // row stride of staged weights (elements)
  int32_t band_w;           // staged columns of a segment (halo and tail zero-filled)
  int32_t lo_plane;         // elements from a staged hi value to its lo value (split layers)
};

// Pixel (py, px) of M row m inside a 4x4 tile: m = 4 * window + j, the four
// windows being the 2x2 pooling windows of the tile.
__device__ __forceinline__ void tile_pixel(int m, int& py, int& px) {
  const int wi = m >> 2, j = m & 3;
  py = 2 * (wi >> 1) + (j >> 1);
  px = 2 * (wi & 1) + (j & 1);
}

template <typename T>
__device__ __forceinline__ void stage_weights(const ConvArgs& a, T* wl) {
  const T* src = reinterpret_cast<const T*>(a.wts);
  for (int e = threadIdx.x; e < a.cout * a.kpad; e += blockDim.x) {
    const int o = e / a.kpad, k = e - o * a.kpad;
    wl[o * a.w_lds + k] = src[e];
  }
}

// Bias, ReLU, optional 2x2 max-pool and fp32 NHWC store of one 4x4 tile.
// Lane (m, g) holds rows 4g..4g+3 (one pooling window) of output channel m.
template <int NT>
__device__ __forceinline__ void conv_epilogue(const ConvArgs& a, const f32x4 (&acc)[NT], float* out,
                                              int ty, int tx, int ho, int wo, int m, int g) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = nt * 16 + m;
    const float b = a.bias[n];
    const int wy = g >> 1, wx = g & 1;
    if (a.pool) {
      float v = 0.0f;  // ReLU floor
#pragma unroll
      for (int r = 0; r < 4; ++r) v = fmaxf(v, acc[nt][r] + b);
      const int oy = 2 * ty + wy, ox = 2 * tx + wx;
      if (oy < ho && ox < wo) out[((int64_t)oy * wo + ox) * a.cout + n] = v;
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int oy = 4 * ty + 2 * wy + (r >> 1), ox = 4 * tx + 2 * wx + (r & 1);
        if (oy < ho && ox < wo)
          out[((int64_t)oy * wo + ox) * a.cout + n] = fmaxf(acc[nt][r] + b, 0.0f);
      }
    }
  }
}

// First layer (3 input channels).  The survivor's area sums are gathered
// (fy x fx nested cells summed) and pre-processed into a zero-padded band in
// LDS, 4 channels per pixel (the fourth is 0).  K is ordered (dy, dx, c) with
// dx padded to 4 and c to 4 (zero weights), so the 8 K values of a lane group
// are the 4 channels of two horizontally adjacent pixels: one 16-byte LDS read
// per MFMA for bf16.  K = 48, run as 2 steps of 32 (bf16) or 12 of 4 (fp32).
template <typename T, int NT>
__global__ void __launch_bounds__(256) k_conv_first(ConvArgs a) {
  using X = Elt<T>;
  constexpr int E = X::E, KS = X::KS;
  extern __shared__ __align__(16) unsigned char lds_raw[];
  T* wl = reinterpret_cast<T*>(lds_raw);
  T* in = wl + (size_t)a.cout * a.w_lds;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nwaves = blockDim.x >> 6;
  stage_weights(a, wl);
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int bands = (a.tiles_y + a.band_tiles - 1) / a.band_tiles;
  const int segs = (a.tiles_x + a.seg_tiles - 1) / a.seg_tiles;
  const int64_t items = cnt * bands * segs;
  const int band_w = a.band_w;
  const int ho = a.pool ? a.h / 2 : a.h, wo = a.pool ? a.w / 2 : a.w;
  const int m = lane & 15, g = lane >> 4;
  int py, px;
  tile_pixel(m, py, px);

  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int64_t s = item / (bands * segs);
    const int bs = (int)(item - s * (bands * segs));
    const int band = bs / segs, seg = bs - band * segs;
    const int ty0 = band * a.band_tiles, tx0 = seg * a.seg_tiles;
    const int nty = min(a.band_tiles, a.tiles_y - ty0);
    const int ntx = min(a.seg_tiles, a.tiles_x - tx0);
    const int rows = 4 * nty + 2;
    const int y_top = 4 * ty0 - 1;  // input row of band row 0
    __syncthreads();  // previous item's readers are done with `in` (and weights staged)
    {
      const int32_t* S = a.sums + (int64_t)a.idx[s] * a.sums_h * a.sums_w * 3;
      for (int e = tid; e < rows * band_w * 4; e += blockDim.x) {
        const int c = e & 3, pix = e >> 2;
        const int br = pix / band_w, bc = pix - br * band_w;
        const int y = y_top + br, x = 4 * tx0 + bc - 1;
        T v = X::from_f32(0.0f);
        if (c < 3 && y >= 0 && y < a.h && x >= 0 && x < a.w) {
          int64_t acc = 0;
          for (int dy = 0; dy < a.fy; ++dy)
            for (int dx = 0; dx < a.fx; ++dx)
              acc += S[((int64_t)(y * a.fy + dy) * a.sums_w + (x * a.fx + dx)) * 3 + c];
          // (S / den) / 127.5 - 1 as one correctly rounded division of integers:
          // bf16 rounding of it matches the exact value's (exact ties included)
          v = X::from_f64((double)(2 * acc - a.den255) / (double)a.den255);
        }
        in[pix * 4 + c] = v;
      }
    }
    __syncthreads();
    float* out = a.act_out + s * (int64_t)ho * wo * a.cout;
    for (int t = wave; t < nty * ntx; t += nwaves) {
      const int tyl = t / ntx, txl = t - tyl * ntx;
      f32x4 acc[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int row0 = 4 * tyl + py, col0 = 4 * txl + px;  // band coordinates of tap (0, 0)
#pragma unroll
      for (int k0 = 0; k0 < 48; k0 += KS) {
        const int k = k0 + g * E;  // first K value of this lane group
        typename X::frag av = X::zero();
        if (k < 48) {
          const int dy = k >> 4, dx = (k >> 2) & 3, c = k & 3;
          av = X::load8(in + ((row0 + dy) * band_w + col0 + dx) * 4 + c);
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const typename X::frag bv = X::load(wl + (nt * 16 + m) * a.w_lds + k);
          acc[nt] = X::mma(av, bv, acc[nt]);
        }
      }
      conv_epilogue<NT>(a, acc, out, ty0 + tyl, tx0 + txl, ho, wo, m, g);
    }
  }
}

// Inner layers (input channels a multiple of KS): K = 9 taps x cin, tap-major.
// The fp32 input band is staged as fp32 (fp32 nets) or as hi and lo bf16
// planes lo_plane elements apart (bf16 nets); the lo plane is multiplied by the
// same weight fragments into a second set of accumulators.
template <typename T, int NT>
__global__ void __launch_bounds__(256) k_conv(ConvArgs a) {
  using X = Elt<T>;
  constexpr int E = X::E, KS = X::KS;
  constexpr bool SPLIT = X::SPLIT;
  extern __shared__ __align__(16) unsigned char lds_raw[];
  T* wl = reinterpret_cast<T*>(lds_raw);
  T* in = wl + (size_t)a.cout * a.w_lds;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nwaves = blockDim.x >> 6;
  stage_weights(a, wl);
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int bands = (a.tiles_y + a.band_tiles - 1) / a.band_tiles;
  const int segs = (a.tiles_x + a.seg_tiles - 1) / a.seg_tiles;
  const int64_t items = cnt * bands * segs;
  const int band_w = a.band_w;
  const int ho = a.pool ? a.h / 2 : a.h, wo = a.pool ? a.w / 2 : a.w;
  const int m = lane & 15, g = lane >> 4;
  int py, px;
  tile_pixel(m, py, px);
  const int vec_per_pix = a.cin / 4;  // float4 vectors per input pixel
  const int chunks = a.cin / KS;

  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int64_t s = item / (bands * segs);
    const int bs = (int)(item - s * (bands * segs));
    const int band = bs / segs, seg = bs - band * segs;
    const int ty0 = band * a.band_tiles, tx0 = seg * a.seg_tiles;
    const int nty = min(a.band_tiles, a.tiles_y - ty0);
    const int ntx = min(a.seg_tiles, a.tiles_x - tx0);
    const int rows = 4 * nty + 2;
    const int y_top = 4 * ty0 - 1;
    __syncthreads();  // previous item's readers are done with `in` (and weights staged)
    {
      const float* src = a.act_in + s * (int64_t)a.h * a.w * a.cin;
      for (int e = tid; e < rows * band_w * vec_per_pix; e += blockDim.x) {
        const int pix = e / vec_per_pix, cv = e - pix * vec_per_pix;
        const int br = pix / band_w, bc = pix - br * band_w;
        const int y = y_top + br, x = 4 * tx0 + bc - 1;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (y >= 0 && y < a.h && x >= 0 && x < a.w)
          v = *reinterpret_cast<const float4*>(src + ((int64_t)y * a.w + x) * a.cin + cv * 4);
        T* dst = in + pix * a.cin_lds + cv * 4;
        if constexpr (SPLIT) {
          uint2 hi, lo;
          X::split4(v, hi, lo);
          *reinterpret_cast<uint2*>(dst) = hi;
          *reinterpret_cast<uint2*>(dst + a.lo_plane) = lo;
        } else {
          *reinterpret_cast<float4*>(dst) = v;
        }
      }
    }
    __syncthreads();
    float* out = a.act_out + s * (int64_t)ho * wo * a.cout;
    for (int t = wave; t < nty * ntx; t += nwaves) {
      const int tyl = t / ntx, txl = t - tyl * ntx;
      f32x4 acc[NT], acc_lo[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        acc_lo[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
      const int row0 = 4 * tyl + py, col0 = 4 * txl + px;
      for (int tap = 0; tap < 9; ++tap) {
        const int dy = tap / 3, dx = tap - 3 * dy;
        const T* arow = in + ((row0 + dy) * band_w + col0 + dx) * a.cin_lds + g * E;
        const T* brow = wl + m * a.w_lds + tap * a.cin + g * E;
        for (int ch = 0; ch < chunks; ++ch) {
          const typename X::frag av = X::load(arow + ch * KS);
          typename X::frag av_lo;
          if constexpr (SPLIT) av_lo = X::load(arow + a.lo_plane + ch * KS);
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const typename X::frag bv = X::load(brow + nt * 16 * a.w_lds + ch * KS);
            acc[nt] = X::mma(av, bv, acc[nt]);
            if constexpr (SPLIT) acc_lo[nt] = X::mma(av_lo, bv, acc_lo[nt]);
          }
        }
      }
      if constexpr (SPLIT) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[nt] += acc_lo[nt];
      }
      conv_epilogue<NT>(a, acc, out, ty0 + tyl, tx0 + txl, ho, wo, m, g);
    }
  }
}

// ------------------------------------------------------------------ dense

struct DenseArgs {
  const float* feat;        // [slot][flat] fp32 in (y, x, c) order
  const void* w1;           // [D][flat]
  const float* b1;
  const float* w2;
  float b2;
  int32_t flat;
  const int32_t* count;
  int64_t max_count;
  const int32_t* idx;
  float* logit;
  float* prob;
  uint8_t* dec;
  float* frame_logit;
  double c_low, c_high;
};

template <typename T, int NT>
__global__ void __launch_bounds__(256) k_dense(DenseArgs a) {
  using X = Elt<T>;
  constexpr int E = X::E, KS = X::KS;
  constexpr bool SPLIT = X::SPLIT;
  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int64_t groups = (cnt + 15) / 16;
  const int64_t wave_id = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t nwaves = (int64_t)gridDim.x * (blockDim.x >> 6);
  const T* w1 = reinterpret_cast<const T*>(a.w1);
  for (int64_t grp = wave_id; grp < groups; grp += nwaves) {
    const int64_t s = grp * 16 + m;
    const bool valid = s < cnt;
    const float* arow = a.feat + (valid ? s : 0) * (int64_t)a.flat + g * E;
    f32x4 acc[NT], acc_lo[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      acc_lo[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    for (int k0 = 0; k0 < a.flat; k0 += KS) {
      typename X::frag av = X::zero(), av_lo = X::zero();
      if constexpr (SPLIT) {
        if (valid) X::split8(arow + k0, av, av_lo);
      } else {
        if (valid) av = arow[k0];
      }
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const typename X::frag bv = X::load(w1 + (int64_t)(nt * 16 + m) * a.flat + k0 + g * E);
        acc[nt] = X::mma(av, bv, acc[nt]);
        if constexpr (SPLIT) acc_lo[nt] = X::mma(av_lo, bv, acc_lo[nt]);
      }
    }
    if constexpr (SPLIT) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[nt] += acc_lo[nt];
    }
    // hidden = ReLU(acc + b1); z = b2 + sum_n w2[n] * hidden[n]
    float part[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = nt * 16 + m;
      const float b = a.b1[n], w = a.w2[n];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float hval = fmaxf(acc[nt][r] + b, 0.0f);
        part[r] += w * hval;
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) part[r] += __shfl_xor(part[r], o, 64);
    }
    if (m == 0) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t slot = grp * 16 + 4 * g + r;
        if (slot < cnt) {
          const float z = part[r] + a.b2;
          const double p = 1.0 / (1.0 + exp(-(double)z));
          a.logit[slot] = z;
          if (a.prob) a.prob[slot] = (float)p;
          if (a.dec || a.frame_logit) {
            const int32_t f = a.idx[slot];
            if (a.dec) a.dec[f] = p < a.c_low ? 0 : (p > a.c_high ? 1 : 2);
            if (a.frame_logit) a.frame_logit[f] = z;
          }
        }
      }
    }
  }
}

template <typename T, bool FIRST>
int launch_conv_nt(int nt, const ConvArgs& a, unsigned grid, size_t lds, hipStream_t st) {
#define NSC_CONV_CASE(N)                                                                       \
  case N:                                                                                      \
    if (FIRST)                                                                                 \
      hipLaunchKernelGGL((k_conv_first<T, N>), dim3(grid), dim3(256), lds, st, a);             \
    else                                                                                       \
      hipLaunchKernelGGL((k_conv<T, N>), dim3(grid), dim3(256), lds, st, a);                   \
    break;
  switch (nt) {
    NSC_CONV_CASE(1)
    NSC_CONV_CASE(2)
    NSC_CONV_CASE(3)
    NSC_CONV_CASE(4)
    NSC_CONV_CASE(6)
    NSC_CONV_CASE(8)
    NSC_CONV_CASE(16)
    default:
      return fail(NSC_E_SHAPE, "conv with %d output channels is not supported", nt * 16);
  }
#undef NSC_CONV_CASE
  NSC_CHECK_LAUNCH("k_conv");
  return NSC_OK;
}

template <typename T>
int launch_dense_nt(int nt, const DenseArgs& a, unsigned grid, hipStream_t st) {
#define NSC_DENSE_CASE(N)                                                          \
  case N:                                                                          \
    hipLaunchKernelGGL((k_dense<T, N>), dim3(grid), dim3(256), 0, st, a);           \
    break;
  switch (nt) {
    NSC_DENSE_CASE(1)
    NSC_DENSE_CASE(2)
    NSC_DENSE_CASE(4)
    NSC_DENSE_CASE(8)
    NSC_DENSE_CASE(16)
    default:
      return fail(NSC_E_SHAPE, "dense layer of %d units is not supported", nt * 16);
  }
#undef NSC_DENSE_CASE
  NSC_CHECK_LAUNCH("k_dense");
  return NSC_OK;
}

}  // namespace

// LDS bytes of one conv layer's workgroup (weights + input band).
// Output tiles of a layer: 4x4 pixels; a pooled layer only needs the pixels
// of whole pooling windows.
void conv_tiles(const CnnLayer& L, int32_t* tiles_y, int32_t* tiles_x) {
  const int hn = L.pool ? (L.h / 2) * 2 : L.h, wn = L.pool ? (L.w / 2) * 2 : L.w;
  *tiles_y = (hn + 3) / 4;
  *tiles_x = (wn + 3) / 4;
}

// LDS of one conv layer's workgroup: staged weights plus an input band of
// band_tiles tile rows (4 output rows each + 2 halo rows) by seg_tiles tile
// columns (+ halo), in two planes (hi, lo) for the inner layers of a bf16
// network.  A band spans the full width unless that does not fit 128 KB (then
// the width is halved until it does); it is as tall as fits a budget of about
// 48 KB (the whole image when possible), at least one tile row.
size_t conv_lds_bytes(const CnnLayer& L, bool bf16, int32_t* cin_lds, int32_t* w_lds,
                      int32_t* band_w, int32_t* band_tiles, int32_t* seg_tiles) {
  const size_t es = bf16 ? 2 : 4;
  const int32_t vec = (int32_t)(16 / es);
  const bool first = L.cin == 3;
  const int32_t cl = first ? 4 : L.cin + vec;          // inner layers: pad pixels by 16 bytes
  const int32_t wr = L.kpad + vec;                     // pad weight rows by 16 bytes
  int32_t ty, tx;
  conv_tiles(L, &ty, &tx);
  const size_t planes = bf16 && !first ? 2 : 1;
  const size_t wbytes = (size_t)L.cout * wr * es;
  // staged columns of st tile columns; the first layer also reads tap dx = 3 (weight 0)
  auto cols = [&](int32_t st) { return 4 * st + (first ? 3 : 2); };
  int32_t st = tx;
  while (st > 1 && wbytes + (size_t)6 * cols(st) * cl * es * planes > 128 * 1024) st = (st + 1) / 2;
  const int32_t bw = cols(st);
  const size_t row_bytes = (size_t)bw * cl * es * planes;
  int32_t bt = 1;
  while (bt < ty && wbytes + (size_t)(4 * (bt + 1) + 2) * row_bytes <= 48 * 1024) ++bt;
  if (cin_lds) *cin_lds = cl;
  if (w_lds) *w_lds = wr;
  if (band_w) *band_w = bw;
  if (band_tiles) *band_tiles = bt;
  if (seg_tiles) *seg_tiles = st;
  return wbytes + (size_t)(4 * bt + 2) * row_bytes;
}

// Two ping-pong buffers of fp32 activations per image.
size_t cnn_workspace_bytes(const Cnn& cnn, int64_t max_count) {
  const size_t per = align_up(cnn.act_elems * sizeof(float), 256);
  return 2 * per * (size_t)(max_count > 0 ? max_count : 0) + 256;
}

int run_cnn(const Cnn& cnn, const CnnRunArgs& r, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (r.max_count <= 0) return NSC_OK;
  const size_t es = cnn.bf16 ? 2 : 4;  // weight element bytes
  const size_t per = align_up(cnn.act_elems * sizeof(float), 256);
  if (ws_bytes < cnn_workspace_bytes(cnn, r.max_count))
    return fail(NSC_E_WORKSPACE, "CNN workspace of %zu bytes is below the %zu required", ws_bytes,
                cnn_workspace_bytes(cnn, r.max_count));
  float* buf[2] = {static_cast<float*>(ws),
                   reinterpret_cast<float*>(static_cast<unsigned char*>(ws) + per * (size_t)r.max_count)};
  for (int l = 0; l < cnn.n_layers; ++l) {
    const CnnLayer& L = cnn.layers[l];
    ConvArgs a{};
    a.sums = r.sums;
    a.idx = r.idx;
    a.sums_h = r.sums_h;
    a.sums_w = r.sums_w;
    a.fy = r.fy;
    a.fx = r.fx;
    a.den255 = (int64_t)(255.0 * r.den_c);
    a.act_in = l > 0 ? buf[(l - 1) & 1] : nullptr;
    a.act_out = buf[l & 1];
    a.wts = static_cast<const unsigned char*>(cnn.conv_w) + L.w_off * es;
    a.bias = cnn.conv_b + L.b_off;
    a.count = r.count;
    a.max_count = r.max_count;
    a.cin = L.cin;
    a.cout = L.cout;
    a.h = L.h;
    a.w = L.w;
    a.kpad = L.kpad;
    a.pool = L.pool ? 1 : 0;
    conv_tiles(L, &a.tiles_y, &a.tiles_x);
    const size_t lds =
        conv_lds_bytes(L, cnn.bf16, &a.cin_lds, &a.w_lds, &a.band_w, &a.band_tiles, &a.seg_tiles);
    a.lo_plane = (4 * a.band_tiles + 2) * a.band_w * a.cin_lds;
    int per_cu = (int)((160 * 1024) / (lds + 1024));
    if (per_cu > 8) per_cu = 8;
    if (per_cu < 1) per_cu = 1;
    int64_t items = r.max_count * ((a.tiles_y + a.band_tiles - 1) / a.band_tiles) *
                    ((a.tiles_x + a.seg_tiles - 1) / a.seg_tiles);
    int64_t grid = (int64_t)kNumCU * per_cu;
    if (grid > items) grid = items;
    if (grid < 1) grid = 1;
    int rc;
    const int nt = L.cout / 16;
    if (cnn.bf16)
      rc = l == 0 ? launch_conv_nt<uint16_t, true>(nt, a, (unsigned)grid, lds, stream)
                  : launch_conv_nt<uint16_t, false>(nt, a, (unsigned)grid, lds, stream);
    else
      rc = l == 0 ? launch_conv_nt<float, true>(nt, a, (unsigned)grid, lds, stream)
                  : launch_conv_nt<float, false>(nt, a, (unsigned)grid, lds, stream);
    if (rc) return rc;
  }
  DenseArgs d{};
  d.feat = buf[(cnn.n_layers - 1) & 1];
  d.w1 = cnn.w1;
  d.b1 = cnn.b1;
  d.w2 = cnn.w2;
  d.b2 = cnn.b2;
  d.flat = cnn.flat;
  d.count = r.count;
  d.max_count = r.max_count;
  d.idx = r.idx;
  d.logit = r.logit;
  d.prob = r.prob;
  d.dec = r.dec;
  d.frame_logit = r.frame_logit;
  d.c_low = r.c_low;
  d.c_high = r.c_high;
  int64_t groups = (r.max_count + 15) / 16;
  int64_t grid = (groups + 3) / 4;
  if (grid > kNumCU * 8) grid = kNumCU * 8;
  if (grid < 1) grid = 1;
  const int nt = cnn.dense / 16;
  return cnn.bf16 ? launch_dense_nt<uint16_t>(nt, d, (unsigned)grid, stream)
                  : launch_dense_nt<float>(nt, d, (unsigned)grid, stream);
}

}  // namespace nsc
