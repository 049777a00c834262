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
// A bf16 network has bf16 weights and a bf16-rounded input.  Its later
// activations enter the matrix cores in one of two ways:
//  - NSC_BF16: the 64-input-channel (banded) layers and the dense layer run on
//    the fp16 matrix cores, activations rounded to fp16 once (2^-12 of
//    themselves), one product per weight.  The bf16 weights are scaled by 2^wexp
//    per layer so that each is an fp16 value, the activations by 2^-aexp (from
//    a worst-case bound of the layer's input, so that none overflows), and the
//    accumulators are multiplied back in the epilogue; activations passed
//    between two such layers (or into the dense layer) are stored as fp16,
//    already scaled for the next layer.  The other layers use the pairs below.
//  - NSC_BF16_PAIRS: each later activation a enters the bf16 matrix cores as
//    the pair hi = bf16(a), lo = bf16(a - hi) (the difference is exact in
//    fp32), multiplied by the same weights into the same accumulator: a is
//    carried to about 2^-17 of itself, at two products per weight.
// Either way the result is a continuous function of the activations' rounding
// and of the fp32 accumulation error; activations are fp32 in the workspace
// otherwise.
//
// The dense layer is a GEMM over 16-survivor tiles (M) x hidden units (N) x
// features (K) on the same MFMA shapes, one workgroup per tile whose waves
// split K and add their partial sums through LDS; its epilogue adds the bias,
// applies ReLU, folds the 1-unit output layer in with a 16-lane shuffle
// reduction, and writes the logit, the sigmoid confidence and the c_low /
// c_high decision of each frame.
#include "nsc_internal.h"

#include <math.h>

namespace nsc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// fp16 matrix cores (the fp16 path of a bf16 network's later layers).
__device__ __forceinline__ f32x4 mma_f16(const f16x8& a, const f16x8& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
// Two fp32 values times sc (a power of two) rounded to fp16 (nearest even),
// packed.
__device__ __forceinline__ uint32_t f16x2_bits(float a, float b, float sc) {
  return __builtin_bit_cast(uint32_t, f16x2{(_Float16)(a * sc), (_Float16)(b * sc)});
}
__device__ __forceinline__ uint2 f16x4_bits(float a, float b, float c, float d, float sc) {
  return make_uint2(f16x2_bits(a, b, sc), f16x2_bits(c, d, sc));
}
__device__ __forceinline__ uint4 f16x8_bits(const float4& a, const float4& b, float sc) {
  return make_uint4(f16x2_bits(a.x, a.y, sc), f16x2_bits(a.z, a.w, sc), f16x2_bits(b.x, b.y, sc),
                    f16x2_bits(b.z, b.w, sc));
}

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

// bf16 (nearest, ties to even) of the exact quotient N / D for 0 < D < 2^24,
// |N| <= D.  Both are exact in fp32 and the fp32 division is correctly
// rounded, so rounding its result to bf16 can only differ from rounding the
// exact quotient when the fp32 result is itself a bf16 midpoint m; then the
// side of m the quotient lies on (N - m D, exact in fp64 as m has 9
// significant bits) decides, and an exact tie stays a tie.
__device__ __forceinline__ uint16_t div_to_bf16_bits(int32_t N, int32_t D) {
  const float r = (float)N / (float)D;
  uint32_t u = __float_as_uint(r);
  if ((u & 0xFFFFu) == 0x8000u) {  // r != 0: step one fp32 ulp toward the quotient
    const double diff = (double)N - (double)r * (double)D;
    const bool up_in_magnitude = r > 0.0f ? diff > 0.0 : diff < 0.0;
    if (diff != 0.0) u = up_in_magnitude ? u + 1 : u - 1;
  }
  return f32_to_bf16_bits(__uint_as_float(u));
}

// The same from the product with inv = fp32(1 / D): N * inv is within 2 fp32
// ulps of N / D (two roundings of 2^-24 each), so unless it lies within 2
// ulps of a bf16 midpoint (low 16 bits 0x7FFE .. 0x8002) it rounds to bf16
// like the exact quotient; those rare values take the division above.
__device__ __forceinline__ uint16_t div_to_bf16_bits_fast(int32_t N, int32_t D, float inv) {
  const float r = (float)N * inv;
  const uint32_t low = __float_as_uint(r) & 0xFFFFu;
  if (low - 0x7FFEu <= 4u) return div_to_bf16_bits(N, D);
  return f32_to_bf16_bits(r);
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
  // Activations enter as hi + lo pairs (see the top of this file); the
  // conversions are the hardware's packed round-to-nearest-even.
  static constexpr bool SPLIT = true;
  static constexpr bool CVT = false;
  // two fp32 values -> (hi0, hi1) and (lo0, lo1), packed as bf16 pairs
  // (one packed conversion for the hi pair; its fp32 values are the pair's
  // bits moved into the upper halves)
  static __device__ __forceinline__ void split2(float v0, float v1, uint32_t& hi, uint32_t& lo) {
    hi = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)v0, (__bf16)v1});
    const float h0 = __uint_as_float(hi << 16), h1 = __uint_as_float(hi & 0xFFFF0000u);
    lo = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)(v0 - h0), (__bf16)(v1 - h1)});
  }
  static __device__ __forceinline__ void split2(float v0, float v1, bf16x2& hi, bf16x2& lo) {
    uint32_t h, l;
    split2(v0, v1, h, l);
    hi = __builtin_bit_cast(bf16x2, h);
    lo = __builtin_bit_cast(bf16x2, l);
  }
  // 4 fp32 values -> 4 hi and 4 lo bf16 values, packed pairwise in uint2
  static __device__ __forceinline__ void split4(const float4& v, uint2& hi, uint2& lo) {
    split2(v.x, v.y, hi.x, lo.x);
    split2(v.z, v.w, hi.y, lo.y);
  }
  // A fragment pair from 8 consecutive fp32 values (16-byte aligned)
  static __device__ __forceinline__ void split8(const float* p, frag& hi, frag& lo) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      bf16x2 h, l;
      split2(v[e], v[e + 1], h, l);
      hi[e] = h[0];
      hi[e + 1] = h[1];
      lo[e] = l[0];
      lo[e + 1] = l[1];
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
  static constexpr bool CVT = false;
};
// fp16 path of a bf16 network's dense layer: scaled fp16 weights, fp32
// activations converted to fp16 (times a power-of-two input scale) as they are
// loaded, one MFMA per product.
template <> struct Elt<_Float16> {
  static constexpr int E = 8, KS = 32;
  typedef f16x8 frag;
  static __device__ __forceinline__ f32x4 mma(const frag& a, const frag& b, f32x4 c) {
    return mma_f16(a, b, c);
  }
  static __device__ __forceinline__ frag load(const _Float16* p) {  // 16-byte aligned
    return *reinterpret_cast<const frag*>(p);
  }
  static __device__ __forceinline__ frag zero() {
    frag z;
#pragma unroll
    for (int e = 0; e < 8; ++e) z[e] = (_Float16)0.0f;
    return z;
  }
  // 8 consecutive fp32 values (16-byte aligned) times sc
  static __device__ __forceinline__ frag cvt8(const float* p, float sc) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    return __builtin_bit_cast(frag, f16x8_bits(a, b, sc));
  }
  static constexpr bool SPLIT = false;
  static constexpr bool CVT = true;
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
  const float* scl;         // fp16 path: the layer's (input scale 2^-aexp, output scale
                            // 2^(aexp - wexp)) in the network's weight image, followed by
                            // the next layer's (or the dense layer's) pair
  int32_t in_f16;           // act_in holds fp16 values already times the input scale
  int32_t out_f16;          // act_out gets fp16 values times the next layer's input scale
  const CamNet* nets;       // camera group: per-camera weight offsets (else null)
  int64_t per_cam;          // frames per camera of a group
};

// Byte offset of survivor slot s's network from the base network's weights
// in a camera group; s is uniform across the wave, and so is the result
// (moved to scalar registers).
__device__ __forceinline__ int64_t slot_woff(const CamNet* nets, int64_t per_cam,
                                             const int32_t* idx, int64_t s) {
  const uint64_t off = (uint64_t)nets[idx[s] / per_cam].woff;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)off);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(off >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
template <typename P>
__device__ __forceinline__ const P* at_off(const P* p, int64_t off) {
  return reinterpret_cast<const P*>(reinterpret_cast<const unsigned char*>(p) + off);
}

// Pixel (py, px) of M row m inside a 4x4 tile: m = 4 * window + j, the four
// windows being the 2x2 pooling windows of the tile.
__device__ __forceinline__ void tile_pixel(int m, int& py, int& px) {
  const int wi = m >> 2, j = m & 3;
  py = 2 * (wi >> 1) + (j >> 1);
  px = 2 * (wi & 1) + (j & 1);
}

template <typename T>
__device__ __forceinline__ void stage_weights(const ConvArgs& a, T* wl, int64_t off = 0) {
  const T* src = at_off(reinterpret_cast<const T*>(a.wts), off);
  for (int e = threadIdx.x; e < a.cout * a.kpad; e += blockDim.x) {
    const int o = e / a.kpad, k = e - o * a.kpad;
    wl[o * a.w_lds + k] = src[e];
  }
}

// The lane's bias of output channel nt * 16 + m, for each nt.
template <int NT>
__device__ __forceinline__ void load_bias(const float* bias, int m, float (&b)[NT]) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) b[nt] = bias[nt * 16 + m];
}

// Bias, ReLU, optional 2x2 max-pool and NHWC store of one 4x4 tile: fp32,
// or with st16 != 0 fp16 values times st16 (the next layer's input scale on
// the fp16 path).  Lane (m, g) holds rows 4g..4g+3 (one pooling window) of
// output channel m.
template <int NT>
__device__ __forceinline__ void conv_epilogue(const ConvArgs& a, const f32x4 (&acc)[NT],
                                              const float (&bias)[NT], void* out, int ty, int tx,
                                              int ho, int wo, int m, int g, float st16 = 0.0f) {
  auto store = [&](int64_t e, float v) {
    if (st16 != 0.0f)
      static_cast<_Float16*>(out)[e] = (_Float16)(v * st16);
    else
      static_cast<float*>(out)[e] = v;
  };
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = nt * 16 + m;
    const float b = bias[nt];
    const int wy = g >> 1, wx = g & 1;
    if (a.pool) {
      float v = 0.0f;  // ReLU floor
#pragma unroll
      for (int r = 0; r < 4; ++r) v = fmaxf(v, acc[nt][r] + b);
      const int oy = 2 * ty + wy, ox = 2 * tx + wx;
      if (oy < ho && ox < wo) store(((int64_t)oy * wo + ox) * a.cout + n, v);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int oy = 4 * ty + 2 * wy + (r >> 1), ox = 4 * tx + 2 * wx + (r & 1);
        if (oy < ho && ox < wo) store(((int64_t)oy * wo + ox) * a.cout + n, fmaxf(acc[nt][r] + b, 0.0f));
      }
    }
  }
}

// The pooled epilogue with the lane's output address precomputed: o is the
// lane's channel m of its pooled pixel, inside when that pixel is stored.
template <int NT>
__device__ __forceinline__ void pool_epilogue_at(const f32x4 (&acc)[NT], const float (&bias)[NT],
                                                 float* o, bool inside) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float v = 0.0f;  // ReLU floor
#pragma unroll
    for (int r = 0; r < 4; ++r) v = fmaxf(v, acc[nt][r] + bias[nt]);
    if (inside) o[nt * 16] = v;
  }
}

// First layer (3 input channels).  The survivor's area sums are gathered
// (fy x fx nested cells summed) and pre-processed into a zero-padded band in
// LDS, 4 channels per pixel (the fourth is 0).  K is ordered (dy, dx, c) with
// dx padded to 4 and c to 4 (zero weights), so the 8 K values of a lane group
// are the 4 channels of two horizontally adjacent pixels: one 16-byte LDS read
// per MFMA for bf16.  K = 48, run as 2 steps of 32 (bf16) or 12 of 4 (fp32).

// Sums over the fy x fx cells of input pixel (y, x) of one frame's area sums
// S (3 channels per cell); below 255 * den_c < 2^31 (checked on the host).
// With two cells per row (fx = 2), an even row length and an 8-byte-aligned
// frame, the two cells of a row are 24 consecutive 8-byte-aligned bytes:
// three 8-byte loads instead of six 4-byte ones.
__device__ __forceinline__ void cell_sums(const ConvArgs& a, const int32_t* __restrict__ S, int y,
                                          int x, int32_t (&acc)[3]) {
  if (a.fy == 1 && a.fx == 1) {  // the area sums are at the CNN's grid
    const int32_t* q = S + ((int64_t)y * a.sums_w + x) * 3;
    acc[0] = q[0];
    acc[1] = q[1];
    acc[2] = q[2];
    return;
  }
  acc[0] = acc[1] = acc[2] = 0;
  if (a.fx == 2 && (a.sums_w & 1) == 0 && ((uintptr_t)S & 7) == 0) {
    for (int dy = 0; dy < a.fy; ++dy) {
      const int2* q =
          reinterpret_cast<const int2*>(S + ((int64_t)(y * a.fy + dy) * a.sums_w + 2 * x) * 3);
      const int2 u = q[0], v = q[1], w = q[2];  // cell 2x: u.x u.y v.x, cell 2x + 1: v.y w.x w.y
      acc[0] += u.x + v.y;
      acc[1] += u.y + w.x;
      acc[2] += v.x + w.y;
    }
    return;
  }
  for (int dy = 0; dy < a.fy; ++dy)
    for (int dx = 0; dx < a.fx; ++dx) {
      const int32_t* q = S + ((int64_t)(y * a.fy + dy) * a.sums_w + (x * a.fx + dx)) * 3;
      acc[0] += q[0];
      acc[1] += q[1];
      acc[2] += q[2];
    }
}

// Stages rows x band_w pixels starting at input (y_top, x_left) of frame
// idx[s], one pixel (3 channels + a zero, one 8- or 16-byte LDS store) per
// thread and step, by the nthreads threads from thread tid0 on.
template <typename T>
__device__ __forceinline__ void stage_first(const ConvArgs& a, T* in, int64_t s, int y_top,
                                            int x_left, int rows, int band_w, int tid0,
                                            int nthreads) {
  using X = Elt<T>;
  if ((int)threadIdx.x < tid0) return;
  const int32_t* S = a.sums + (int64_t)a.idx[s] * a.sums_h * a.sums_w * 3;
  const int npix = rows * band_w;
  const bool f32div = a.den255 < (1 << 24);  // the fp32 quotient path is exact
  const float inv = 1.0f / (float)a.den255;
#pragma unroll 2
  for (int p = threadIdx.x - tid0; p < npix; p += nthreads) {
    const int br = p / band_w, bc = p - br * band_w;
    const int y = y_top + br, x = x_left + bc;
    T v[4] = {X::from_f32(0.0f), X::from_f32(0.0f), X::from_f32(0.0f), X::from_f32(0.0f)};
    if (y >= 0 && y < a.h && x >= 0 && x < a.w) {
      int32_t acc[3];
      cell_sums(a, S, y, x, acc);
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        // (S / den) / 127.5 - 1 = (2 S - den255) / den255, rounded once (exact ties included)
        const int64_t num = 2 * (int64_t)acc[c] - a.den255;
        if constexpr (X::SPLIT) {
          v[c] = f32div ? div_to_bf16_bits_fast((int32_t)num, (int32_t)a.den255, inv)
                        : X::from_f64((double)num / (double)a.den255);
        } else {
          v[c] = X::from_f64((double)num / (double)a.den255);
        }
      }
    }
    if constexpr (sizeof(T) == 2) {
      *reinterpret_cast<uint2*>(in + p * 4) =
          make_uint2((uint32_t)v[0] | ((uint32_t)v[1] << 16), (uint32_t)v[2] | ((uint32_t)v[3] << 16));
    } else {
      *reinterpret_cast<float4*>(in + p * 4) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

// MFMA accumulation of one first-layer 4x4 tile whose tap (0, 0) of the
// lane's pixel is band pixel (row0, col0).
template <typename T, int NT>
__device__ __forceinline__ void first_tile(const T* in, const T* wl, int w_lds, int band_w,
                                           int row0, int col0, int m, int g, f32x4 (&acc)[NT]) {
  using X = Elt<T>;
  constexpr int E = X::E, KS = X::KS;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
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
      const typename X::frag bv = X::load(wl + (nt * 16 + m) * w_lds + k);
      acc[nt] = X::mma(av, bv, acc[nt]);
    }
  }
}

// The same with the weight fragments already in registers (bf16: K = 64 in two
// steps of 32, fragment [step][nt]).
template <int NT>
__device__ __forceinline__ void first_tile_b(const uint16_t* in, const bf16x8 (&bw)[2][NT],
                                             int band_w, int row0, int col0, int g,
                                             f32x4 (&acc)[NT]) {
  using X = Elt<uint16_t>;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const int k = ks * 32 + g * 8;
    bf16x8 av = X::zero();
    if (k < 48) {
      const int dy = k >> 4, dx = (k >> 2) & 3;
      av = X::load8(in + ((row0 + dy) * band_w + col0 + dx) * 4);
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = X::mma(av, bw[ks][nt], acc[nt]);
  }
}

template <typename T, int NT, bool G>
__global__ void __launch_bounds__(256) k_conv_first(ConvArgs a) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  T* wl = reinterpret_cast<T*>(lds_raw);
  T* in = wl + (size_t)a.cout * a.w_lds;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwaves = blockDim.x >> 6;
  // a camera group stages each item's network (when it changes) in the loop
  if constexpr (!G) stage_weights(a, wl);
  int64_t staged = 0;
  bool have = !G;
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int bands = (a.tiles_y + a.band_tiles - 1) / a.band_tiles;
  const int segs = (a.tiles_x + a.seg_tiles - 1) / a.seg_tiles;
  const int64_t items = cnt * bands * segs;
  const int ho = a.pool ? a.h / 2 : a.h, wo = a.pool ? a.w / 2 : a.w;
  const int m = lane & 15, g = lane >> 4;
  int py, px;
  tile_pixel(m, py, px);
  float bias[NT];
  if constexpr (!G) load_bias(a.bias, m, bias);

  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int64_t s = item / (bands * segs);
    const int bs = (int)(item - s * (bands * segs));
    const int band = bs / segs, seg = bs - band * segs;
    const int ty0 = band * a.band_tiles, tx0 = seg * a.seg_tiles;
    const int nty = min(a.band_tiles, a.tiles_y - ty0);
    const int ntx = min(a.seg_tiles, a.tiles_x - tx0);
    __syncthreads();  // previous item's readers are done with `in` (and weights staged)
    if constexpr (G) {
      const int64_t off = slot_woff(a.nets, a.per_cam, a.idx, s);
      if (!have || off != staged) {  // uniform: the item's camera
        stage_weights(a, wl, off);
        load_bias(at_off(a.bias, off), m, bias);
        staged = off;
        have = true;
      }
    }
    stage_first(a, in, s, 4 * ty0 - 1, 4 * tx0 - 1, 4 * nty + 2, a.band_w, 0, (int)blockDim.x);
    __syncthreads();
    // fp16 output (the next layer on the fp16 path): times its input scale
    const float st16 = a.out_f16 ? at_off(a.scl, G ? slot_woff(a.nets, a.per_cam, a.idx, s) : 0)[2]
                                 : 0.0f;
    const int64_t out_e = s * (int64_t)ho * wo * a.cout;
    void* out = a.out_f16 ? static_cast<void*>(reinterpret_cast<_Float16*>(a.act_out) + out_e)
                          : static_cast<void*>(a.act_out + out_e);
    for (int t = wave; t < nty * ntx; t += nwaves) {
      const int tyl = t / ntx, txl = t - tyl * ntx;
      f32x4 acc[NT];
      first_tile<T, NT>(in, wl, a.w_lds, a.band_w, 4 * tyl + py, 4 * txl + px, m, g, acc);
      conv_epilogue<NT>(a, acc, bias, out, ty0 + tyl, tx0 + txl, ho, wo, m, g, st16);
    }
  }
}

// Inner layers (input channels a multiple of KS): K = 9 taps x cin, tap-major.
// The fp32 input band is staged as fp32 (fp32 nets) or as hi and lo bf16
// planes lo_plane elements apart (bf16 nets); the lo plane is multiplied by the
// same weight fragments into a second set of accumulators.

// Stages rows x band_w pixels starting at input (y_top, x_left) of image s's
// fp32 activations; every thread of the workgroup takes part.
template <typename T>
__device__ __forceinline__ void stage_inner(const ConvArgs& a, T* in, int64_t s, int y_top,
                                            int x_left, int rows, int band_w) {
  using X = Elt<T>;
  const float* src = a.act_in + s * (int64_t)a.h * a.w * a.cin;
  const int vec_per_pix = a.cin / 4;  // float4 vectors per input pixel
  const int total = rows * band_w * vec_per_pix;
#pragma unroll 4
  for (int e = threadIdx.x; e < total; e += blockDim.x) {
    const int pix = e / vec_per_pix, cv = e - pix * vec_per_pix;
    const int br = pix / band_w, bc = pix - br * band_w;
    const int y = y_top + br, x = x_left + bc;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (y >= 0 && y < a.h && x >= 0 && x < a.w)
      v = *reinterpret_cast<const float4*>(src + ((int64_t)y * a.w + x) * a.cin + cv * 4);
    T* dst = in + pix * a.cin_lds + cv * 4;
    if constexpr (X::SPLIT) {
      uint2 hi, lo;
      X::split4(v, hi, lo);
      *reinterpret_cast<uint2*>(dst) = hi;
      *reinterpret_cast<uint2*>(dst + a.lo_plane) = lo;
    } else {
      *reinterpret_cast<float4*>(dst) = v;
    }
  }
}

// MFMA accumulation of one inner-layer 4x4 tile from a band with pixel stride
// cin_lds (and, for bf16, its lo plane lo_plane elements further).
template <typename T, int NT>
__device__ __forceinline__ void inner_tile(const T* in, const T* wl, int w_lds, int cin,
                                           int cin_lds, int lo_plane, int band_w, int row0,
                                           int col0, int m, int g, f32x4 (&acc)[NT]) {
  using X = Elt<T>;
  constexpr int E = X::E, KS = X::KS;
  constexpr bool SPLIT = X::SPLIT;
  f32x4 acc_lo[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc_lo[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int chunks = cin / KS;
  for (int tap = 0; tap < 9; ++tap) {
    const int dy = tap / 3, dx = tap - 3 * dy;
    const T* arow = in + ((row0 + dy) * band_w + col0 + dx) * cin_lds + g * E;
    const T* brow = wl + m * w_lds + tap * cin + g * E;
    for (int ch = 0; ch < chunks; ++ch) {
      const typename X::frag av = X::load(arow + ch * KS);
      typename X::frag av_lo;
      if constexpr (SPLIT) av_lo = X::load(arow + lo_plane + ch * KS);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const typename X::frag bv = X::load(brow + nt * 16 * w_lds + ch * KS);
        acc[nt] = X::mma(av, bv, acc[nt]);
        if constexpr (SPLIT) acc_lo[nt] = X::mma(av_lo, bv, acc_lo[nt]);
      }
    }
  }
  if constexpr (SPLIT) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] += acc_lo[nt];
  }
}

// bf16 inner layer with 32 input channels (one K step per tap) and the weight
// fragments of all 9 taps in registers ([tap][nt]); the hi and lo products go
// into the same accumulators (registers are the limit here).
// The LDS reads of tap t + 1 are issued before the MFMAs of tap t (two
// register pairs; scheduling fences keep them there).
template <int NT>
__device__ __forceinline__ void inner_tile32_b(const uint16_t* in, const bf16x8 (&bw)[9][NT],
                                               int cin_lds, int lo_plane, int band_w, int row0,
                                               int col0, int g, f32x4 (&acc)[NT]);

// The same from the lane's address of tap (0, 0) (hi plane, its K chunk).
template <int NT>
__device__ __forceinline__ void inner_tile32_b_at(const uint16_t* base, const bf16x8 (&bw)[9][NT],
                                                  int cin_lds, int lo_plane, int band_w,
                                                  f32x4 (&acc)[NT]) {
  using X = Elt<uint16_t>;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 av[2], av_lo[2];
  av[0] = X::load(base);
  av_lo[0] = X::load(base + lo_plane);
#pragma unroll
  for (int tap = 0; tap < 9; ++tap) {
    const int cur = tap & 1, nxt = cur ^ 1;
    if (tap + 1 < 9) {
      const int dy = (tap + 1) / 3, dx = (tap + 1) - 3 * dy;
      const uint16_t* arow = base + (dy * band_w + dx) * cin_lds;
      av[nxt] = X::load(arow);
      av_lo[nxt] = X::load(arow + lo_plane);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = X::mma(av[cur], bw[tap][nt], acc[nt]);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = X::mma(av_lo[cur], bw[tap][nt], acc[nt]);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int NT>
__device__ __forceinline__ void inner_tile32_b(const uint16_t* in, const bf16x8 (&bw)[9][NT],
                                               int cin_lds, int lo_plane, int band_w, int row0,
                                               int col0, int g, f32x4 (&acc)[NT]) {
  inner_tile32_b_at<NT>(in + (row0 * band_w + col0) * cin_lds + g * 8, bw, cin_lds, lo_plane,
                        band_w, acc);
}

template <typename T, int NT, bool G>
__global__ void __launch_bounds__(256) k_conv(ConvArgs a) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  T* wl = reinterpret_cast<T*>(lds_raw);
  T* in = wl + (size_t)a.cout * a.w_lds;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwaves = blockDim.x >> 6;
  // a camera group stages each item's network (when it changes) in the loop
  if constexpr (!G) stage_weights(a, wl);
  int64_t staged = 0;
  bool have = !G;
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int bands = (a.tiles_y + a.band_tiles - 1) / a.band_tiles;
  const int segs = (a.tiles_x + a.seg_tiles - 1) / a.seg_tiles;
  const int64_t items = cnt * bands * segs;
  const int ho = a.pool ? a.h / 2 : a.h, wo = a.pool ? a.w / 2 : a.w;
  const int m = lane & 15, g = lane >> 4;
  int py, px;
  tile_pixel(m, py, px);
  float bias[NT];
  if constexpr (!G) load_bias(a.bias, m, bias);

  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int64_t s = item / (bands * segs);
    const int bs = (int)(item - s * (bands * segs));
    const int band = bs / segs, seg = bs - band * segs;
    const int ty0 = band * a.band_tiles, tx0 = seg * a.seg_tiles;
    const int nty = min(a.band_tiles, a.tiles_y - ty0);
    const int ntx = min(a.seg_tiles, a.tiles_x - tx0);
    __syncthreads();  // previous item's readers are done with `in` (and weights staged)
    if constexpr (G) {
      const int64_t off = slot_woff(a.nets, a.per_cam, a.idx, s);
      if (!have || off != staged) {  // uniform: the item's camera
        stage_weights(a, wl, off);
        load_bias(at_off(a.bias, off), m, bias);
        staged = off;
        have = true;
      }
    }
    stage_inner(a, in, s, 4 * ty0 - 1, 4 * tx0 - 1, 4 * nty + 2, a.band_w);
    __syncthreads();
    float* out = a.act_out + s * (int64_t)ho * wo * a.cout;
    for (int t = wave; t < nty * ntx; t += nwaves) {
      const int tyl = t / ntx, txl = t - tyl * ntx;
      f32x4 acc[NT];
      inner_tile<T, NT>(in, wl, a.w_lds, a.cin, a.cin_lds, a.lo_plane, a.band_w, 4 * tyl + py,
                        4 * txl + px, m, g, acc);
      conv_epilogue<NT>(a, acc, bias, out, ty0 + tyl, tx0 + txl, ho, wo, m, g);
    }
  }
}

// The first two layers of a bf16 network fused per image, when the pooled
// output of the first fits in LDS beside both layers' weights: a workgroup
// (one per CU, 16 waves) stages the first layer's whole input, runs it into
// the second layer's hi / lo input band in LDS (halo and tail kept zero), and
// runs the second layer from there into the fp32 workspace.  The first
// layer's input of the next image is staged while the second layer runs.
struct PairArgs {
  int32_t off_w1, off_in0, off_in1;  // LDS offsets (bf16 elements) of w1, in0, in1
};

// The value of lane l + 1 of each 16-lane row (DPP row shift; the last lane
// of a row gets 0).
__device__ __forceinline__ float row_next(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x101, 0xF, 0xF, false));
}

// The same epilogue with the lane's store address precomputed: p is the lane's
// channel m at the tile's pooled pixel in the hi plane.
template <int NT>
__device__ __forceinline__ void pair_epilogue_at(const f32x4 (&acc)[NT], const float (&bias)[NT],
                                                 uint16_t* p, bool store, int lo_plane) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float v = 0.0f;  // ReLU floor
#pragma unroll
    for (int r = 0; r < 4; ++r) v = fmaxf(v, acc[nt][r] + bias[nt]);
    // even lanes store channels n, n + 1 (the odd neighbour's value) as dwords
    const float v1 = row_next(v);
    uint32_t hi, lo;
    Elt<uint16_t>::split2(v, v1, hi, lo);
    if (store) {
      *reinterpret_cast<uint32_t*>(p + nt * 16) = hi;
      *reinterpret_cast<uint32_t*>(p + nt * 16 + lo_plane) = lo;
    }
  }
}

// Bias, ReLU and 2x2 max-pool of one first-layer tile, stored as hi / lo bf16
// at (oy + 1, ox + 1) of the second layer's band (row / column 0 are halo).
template <int NT>
__device__ __forceinline__ void pair_epilogue(const ConvArgs& a1, const f32x4 (&acc)[NT],
                                              const float (&bias)[NT], uint16_t* in1, int ty,
                                              int tx, int ho, int wo, int m, int g) {
  const int oy = 2 * ty + (g >> 1), ox = 2 * tx + (g & 1);
  const bool store = oy < ho && ox < wo && (m & 1) == 0;
  uint16_t* p = in1 + ((oy + 1) * a1.band_w + ox + 1) * a1.cin_lds;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = nt * 16 + m;
    float v = 0.0f;  // ReLU floor
#pragma unroll
    for (int r = 0; r < 4; ++r) v = fmaxf(v, acc[nt][r] + bias[nt]);
    // even lanes store channels n, n + 1 (the odd neighbour's value) as dwords
    const float v1 = __shfl_down(v, 1, 16);
    uint32_t hi, lo;
    Elt<uint16_t>::split2(v, v1, hi, lo);
    if (store) {
      *reinterpret_cast<uint32_t*>(p + n) = hi;
      *reinterpret_cast<uint32_t*>(p + n + a1.lo_plane) = lo;
    }
  }
}

template <int NT0, int NT1, bool B1REG, bool G>
__global__ void __launch_bounds__(1024) k_conv_pair(ConvArgs a0, ConvArgs a1, PairArgs pa) {
  using T = uint16_t;
  using X = Elt<T>;
  extern __shared__ __align__(16) unsigned char lds_raw[];
  T* lds = reinterpret_cast<T*>(lds_raw);
  T* w0 = lds;
  T* w1 = lds + pa.off_w1;
  T* in0 = lds + pa.off_in0;
  T* in1 = lds + pa.off_in1;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwaves = blockDim.x >> 6;
  // a camera group stages each image's networks (when they change) in the loop
  if constexpr (!G) {
    stage_weights(a0, w0);
    stage_weights(a1, w1);
  }
  int64_t staged = 0;
  bool have = !G;
  for (int i = threadIdx.x; i < 2 * a1.lo_plane; i += blockDim.x) in1[i] = 0;
  int64_t cnt = *a0.count;
  if (cnt > a0.max_count) cnt = a0.max_count;
  const int ho0 = a0.h / 2, wo0 = a0.w / 2;  // the first layer pools
  const int ho1 = a1.pool ? a1.h / 2 : a1.h, wo1 = a1.pool ? a1.w / 2 : a1.w;
  const int rows0 = 4 * a0.tiles_y + 2;
  const int m = lane & 15, g = lane >> 4;
  int py, px;
  tile_pixel(m, py, px);
  float bias0[NT0], bias1[NT1];
  if constexpr (!G) {
    load_bias(a0.bias, m, bias0);
    load_bias(a1.bias, m, bias1);
  }
  // the next image is staged by the waves that run one second-layer tile fewer
  const int tiles1 = a1.tiles_y * a1.tiles_x;
  const int extra = tiles1 % nwaves;
  const int stage_tid0 = extra ? extra * 64 : 0;
  int64_t s = blockIdx.x;
  if (s < cnt) stage_first(a0, in0, s, -1, -1, rows0, a0.band_w, 0, (int)blockDim.x);
  for (; s < cnt; s += gridDim.x) {
    __syncthreads();  // in0 staged; the previous image's second layer is done with in1
    if constexpr (G) {
      const int64_t off = slot_woff(a0.nets, a0.per_cam, a0.idx, s);
      if (!have || off != staged) {  // uniform: the image's camera
        stage_weights(a0, w0, off);
        stage_weights(a1, w1, off);
        load_bias(at_off(a0.bias, off), m, bias0);
        load_bias(at_off(a1.bias, off), m, bias1);
        staged = off;
        have = true;
        __syncthreads();  // weights staged before the first layer reads them
      }
    }
    if constexpr (NT0 <= 2) {
      // each wave keeps the first layer's weight fragments in registers
      bf16x8 bw0[2][NT0];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int nt = 0; nt < NT0; ++nt)
          bw0[ks][nt] = X::load(w0 + (nt * 16 + m) * a0.w_lds + ks * 32 + g * 8);
      // per-lane parts of the addresses; a tile adds wave-uniform offsets.
      // K steps 0 and 1 of lane group g start at K = 8 g and 32 + 8 g, i.e.
      // at tap (dy, dx) = (k / 16, k / 4 mod 4) of the lane's pixel (py, px);
      // step 1 is past K = 48 (zero weights) for lane groups 2 and 3.
      const int k1 = 32 + g * 8;
      const int in_l0 = ((py + (g >> 1)) * a0.band_w + px + 2 * (g & 1)) * 4;
      const int in_l1 = ((py + (k1 >> 4)) * a0.band_w + px + ((k1 >> 2) & 3)) * 4;
      const bool use1 = k1 < 48;
      const int out_l = (((g >> 1) + 1) * a1.band_w + (g & 1) + 1) * a1.cin_lds + m;
      for (int t = wave; t < a0.tiles_y * a0.tiles_x; t += nwaves) {
        const int ty = t / a0.tiles_x, tx = t - ty * a0.tiles_x;
        const uint16_t* tin = in0 + (4 * ty * a0.band_w + 4 * tx) * 4;
        const bf16x8 x0 = X::load8(tin + in_l0);
        const bf16x8 x1 = use1 ? X::load8(tin + in_l1) : X::zero();
        f32x4 acc[NT0];
#pragma unroll
        for (int nt = 0; nt < NT0; ++nt) {
          acc[nt] = X::mma(x0, bw0[0][nt], f32x4{0.f, 0.f, 0.f, 0.f});
          acc[nt] = X::mma(x1, bw0[1][nt], acc[nt]);
        }
        const int oy = 2 * ty + (g >> 1), ox = 2 * tx + (g & 1);
        const bool store = oy < ho0 && ox < wo0 && (m & 1) == 0;
        pair_epilogue_at<NT0>(acc, bias0, in1 + (2 * ty * a1.band_w + 2 * tx) * a1.cin_lds + out_l,
                              store, a1.lo_plane);
      }
    } else {
      for (int t = wave; t < a0.tiles_y * a0.tiles_x; t += nwaves) {
        const int ty = t / a0.tiles_x, tx = t - ty * a0.tiles_x;
        f32x4 acc[NT0];
        first_tile<T, NT0>(in0, w0, a0.w_lds, a0.band_w, 4 * ty + py, 4 * tx + px, m, g, acc);
        pair_epilogue<NT0>(a1, acc, bias0, in1, ty, tx, ho0, wo0, m, g);
      }
    }
    __syncthreads();  // in1 complete; in0 free
    float* out = a1.act_out + s * (int64_t)ho1 * wo1 * a1.cout;
    if constexpr (B1REG) {  // 32 input channels: all 9 taps' fragments in registers
      bf16x8 bw1[9][NT1];
#pragma unroll
      for (int tap = 0; tap < 9; ++tap)
#pragma unroll
        for (int nt = 0; nt < NT1; ++nt)
          bw1[tap][nt] = X::load(w1 + (nt * 16 + m) * a1.w_lds + tap * 32 + g * 8);
      const int in_l = (py * a1.band_w + px) * a1.cin_lds + g * 8;  // per-lane address parts
      const int out_l = ((g >> 1) * wo1 + (g & 1)) * a1.cout + m;
      for (int t = wave; t < a1.tiles_y * a1.tiles_x; t += nwaves) {
        const int ty = t / a1.tiles_x, tx = t - ty * a1.tiles_x;
        f32x4 acc[NT1];
        inner_tile32_b_at<NT1>(in1 + (4 * ty * a1.band_w + 4 * tx) * a1.cin_lds + in_l, bw1,
                               a1.cin_lds, a1.lo_plane, a1.band_w, acc);
        if (a1.pool) {
          const bool inside = 2 * ty + (g >> 1) < ho1 && 2 * tx + (g & 1) < wo1;
          pool_epilogue_at<NT1>(acc, bias1, out + (2 * ty * wo1 + 2 * tx) * a1.cout + out_l,
                                inside);
        } else {
          conv_epilogue<NT1>(a1, acc, bias1, out, ty, tx, ho1, wo1, m, g);
        }
      }
    } else {
      for (int t = wave; t < a1.tiles_y * a1.tiles_x; t += nwaves) {
        const int ty = t / a1.tiles_x, tx = t - ty * a1.tiles_x;
        f32x4 acc[NT1];
        inner_tile<T, NT1>(in1, w1, a1.w_lds, a1.cin, a1.cin_lds, a1.lo_plane, a1.band_w,
                           4 * ty + py, 4 * tx + px, m, g, acc);
        conv_epilogue<NT1>(a1, acc, bias1, out, ty, tx, ho1, wo1, m, g);
      }
    }
    if (s + gridDim.x < cnt)
      stage_first(a0, in0, s + gridDim.x, -1, -1, rows0, a0.band_w, stage_tid0,
                  (int)blockDim.x - stage_tid0);
  }
}

// ------------------------------------------- 64-input-channel bf16 layers
//
// A layer with 64 input channels (bf16 network) keeps its weights in global
// memory in fragment order (L2-resident, shared by every CU) and loads them
// straight into registers, one K step ahead of their use; the LDS holds only
// a band of the layer's input: band_tiles tile rows (4 output rows each) plus
// a halo row above and below, as bf16 hi and lo planes.  Without weights in
// LDS two workgroups fit on a CU, and one stages while the other computes.
//
// Band layout: band row r is image row y0 + r, band column cb is image column
// cb - 1; row stride wb >= w + 2 with wb = 4 (mod 8).  Each pixel's 64
// channels are 8 chunks of 8 bf16, stored chunk-major: chunk c of band pixel
// p = r * wb + cb is the 16 bytes at (c * cp + p) * 16 of the hi plane (and
// lo_bytes further in the lo plane), with cp = rows * wb + 1 = 1 (mod 8).
// The 16-byte index c * cp + p is then (c + p) mod 8 on the 8 LDS bank
// groups, so the 8 pixels of two rows by four columns that a lane group
// reads, and the 8 chunks of one pixel that staging writes, all fall on
// distinct bank groups.  Image column -1, columns >= w and rows outside the
// image hold zeros, so a tap needs no bounds test: its address is the tile's
// address plus (dy * wb + dx) * 16.  A tile that overhangs column w reads up
// to two pixels into the next row for outputs that are never stored.
//
// The MFMA runs transposed: A = 16 output channels x 32 K of the weights,
// B = 32 K x the 16 pixels of a 4x4 tile.  Lane (m, g) then holds channels
// 16 nt + 4 g .. 16 nt + 4 g + 3 of pixel m, so a pooled output is a max over
// the four lanes of one quad (DPP) and every store is 16 bytes.

constexpr int kBandWaves = 4;  // waves per workgroup of the banded kernels
constexpr int kBandMaxTilesH = 7;  // tiles per wave and round on the fp16 path (4 with hi / lo)

struct Band64 {
  int32_t w, h;      // layer input grid
  int32_t rows;      // staged rows of a band: 4 * band_tiles + 2
  int32_t wb;        // pixels per band row
  int32_t cp;        // pixels per chunk plane: rows * wb + 1
  int32_t lo_bytes;  // bytes of one plane (from the hi plane to the lo plane): 8 * cp * 16
  int32_t planes;    // 2: bf16 hi and lo planes; 1: one fp16 plane
};

// Bytes of the planes plus 32 bytes for the overhanging reads.
__host__ __device__ inline size_t band64_bytes(const Band64& b) {
  return (size_t)b.planes * b.lo_bytes + 32;
}

// Work item -> (image, band).  Workgroup i of a grid that is a multiple of 8
// runs on XCD i mod 8 and takes items i, i + grid, ...; all bands of one
// image get the same residue mod 8, so their shared halo rows stay in one
// XCD's L2.  Images past cnt (padding to a multiple of 8) are skipped.
__device__ __forceinline__ void band_item(int64_t item, int bands, int64_t* s, int* band) {
  const int64_t q = item >> 3;
  const int64_t blk = q / bands;
  *band = (int)(q - blk * bands);
  *s = blk * 8 + (item & 7);
}

__device__ __forceinline__ void band64_clear(unsigned char* lds, const Band64& b) {
  const int n = (int)(band64_bytes(b) / 16);
  for (int i = threadIdx.x; i < n; i += blockDim.x)
    *reinterpret_cast<uint4*>(lds + (size_t)i * 16) = make_uint4(0u, 0u, 0u, 0u);
}

// floor(pix / w) for a band pixel index, without an integer division.  A
// band's pixels fit the LDS (pix < rows * wb <= 1280), so the exact quotient
// (pix + 1/2) / w lies at least 1 / (2 w) >= 3.9e-4 from an integer, while the
// two fp32 roundings move it by at most 2^-23 of itself (< 1.6e-4).
__device__ __forceinline__ int band_row(int pix, float inv_w) {
  return (int)(((float)pix + 0.5f) * inv_w);
}

// Stages band rows [0, rows_used), columns 1..w: image rows y0 + r inside the
// image from one image's fp32 NHWC 64-channel activations, split into hi / lo
// bf16 (H = false) or as fp16 times in_scale (H), zeros for rows outside.
// Eight consecutive threads read one pixel's 256 bytes.  Each thread issues
// the loads of kStageBatch units before it stores any, so that their
// latencies overlap.
constexpr int kStageBatch = 8;

template <bool H>
__device__ __forceinline__ void stage_band64(const float* __restrict__ src, const Band64& b,
                                             unsigned char* lds, int y0, int rows_used,
                                             float in_scale) {
  const int units = rows_used * b.w * 8;
  const float inv_w = 1.0f / (float)b.w;
  for (int u0 = threadIdx.x; u0 < units; u0 += kStageBatch * blockDim.x) {
    float4 v[kStageBatch][2];
    int addr[kStageBatch];
#pragma unroll
    for (int j = 0; j < kStageBatch; ++j) {
      const int u = u0 + j * blockDim.x;
      const int pix = u >> 3, c = u & 7;
      const int r = band_row(pix, inv_w), x = pix - r * b.w;
      const int y = y0 + r;
      addr[j] = u < units ? (c * b.cp + r * b.wb + x + 1) * 16 : -1;
      v[j][0] = v[j][1] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (u < units && (unsigned)y < (unsigned)b.h) {
        const float* p = src + ((int64_t)y * b.w + x) * 64 + c * 8;
        v[j][0] = *reinterpret_cast<const float4*>(p);
        v[j][1] = *reinterpret_cast<const float4*>(p + 4);
      }
    }
#pragma unroll
    for (int j = 0; j < kStageBatch; ++j) {
      if (addr[j] < 0) continue;
      if constexpr (H) {
        *reinterpret_cast<uint4*>(lds + addr[j]) = f16x8_bits(v[j][0], v[j][1], in_scale);
      } else {
        uint2 h0, l0, h1, l1;
        Elt<uint16_t>::split4(v[j][0], h0, l0);
        Elt<uint16_t>::split4(v[j][1], h1, l1);
        *reinterpret_cast<uint4*>(lds + addr[j]) = make_uint4(h0.x, h0.y, h1.x, h1.y);
        *reinterpret_cast<uint4*>(lds + b.lo_bytes + addr[j]) = make_uint4(l0.x, l0.y, l1.x, l1.y);
      }
    }
  }
}

// The same from fp16 activations already scaled by the producing layer: a
// 16-byte copy per chunk.
__device__ __forceinline__ void stage_band64_f16(const _Float16* __restrict__ src, const Band64& b,
                                                 unsigned char* lds, int y0, int rows_used) {
  const int units = rows_used * b.w * 8;
  const float inv_w = 1.0f / (float)b.w;
  for (int u0 = threadIdx.x; u0 < units; u0 += kStageBatch * blockDim.x) {
    uint4 v[kStageBatch];
    int addr[kStageBatch];
#pragma unroll
    for (int j = 0; j < kStageBatch; ++j) {
      const int u = u0 + j * blockDim.x;
      const int pix = u >> 3, c = u & 7;
      const int r = band_row(pix, inv_w), x = pix - r * b.w;
      const int y = y0 + r;
      addr[j] = u < units ? (c * b.cp + r * b.wb + x + 1) * 16 : -1;
      v[j] = make_uint4(0u, 0u, 0u, 0u);
      if (u < units && (unsigned)y < (unsigned)b.h)
        v[j] = *reinterpret_cast<const uint4*>(src + ((int64_t)y * b.w + x) * 64 + c * 8);
    }
#pragma unroll
    for (int j = 0; j < kStageBatch; ++j)
      if (addr[j] >= 0) *reinterpret_cast<uint4*>(lds + addr[j]) = v[j];
  }
}

// MFMA accumulation of MT 4x4 output tiles from a staged band; tile i sits at
// band tile row tr[i], tile column tc[i].  K is tap-major: 9 taps x 2 steps
// of 32 channels (chunks 0-3, then 4-7).  Software pipeline: the weight and
// activation fragments of the next step are issued before the MFMAs of the
// current one, in two register sets (steps A and B of a tap), and scheduling
// fences keep the compiler from sinking those loads to their first use.  The
// hi products of all tiles are issued before the lo products.
// H: fp16 fragments (one plane, fp16 weights), else bf16 hi / lo pairs.
// Tiles of a band of a banded layer: 16 output pixels of the band in raster
// order, or on a pooling layer 4 of its 2x2 windows in raster order (the four
// pixels of a window in a quad of lanes, for the pooling in the epilogue), so
// that no tile overhangs the map (a 25 x 25 map in 4 x 4 tiles computes 784
// pixels for 625).  rows (even when pooling) and wn (the computed columns:
// the width, even when pooling) bound the band.
__host__ __device__ inline int band64_ntile(bool pool, int rows, int wn) {
  return pool ? ((rows >> 1) * (wn >> 1) + 3) >> 2 : (rows * wn + 15) >> 4;
}

// Band-local output pixel (r, x) of lane m in tile t; false (and (0, 0))
// past the band's last pixel or window.
__device__ __forceinline__ bool band_pixel(int t, int m, int pool, int rows, int wn, int& r,
                                           int& x) {
  r = 0;
  x = 0;
  if (pool) {
    const int wc = wn >> 1;  // windows per row
    const int wi = 4 * t + (m >> 2), j = m & 3;
    if (wi >= (rows >> 1) * wc) return false;
    const int wr = wi / wc;
    r = 2 * wr + (j >> 1);
    x = 2 * (wi - wr * wc) + (j & 1);
    return true;
  }
  const int q = 16 * t + m;
  if (q >= rows * wn) return false;
  r = q / wn;
  x = q - r * wn;
  return true;
}

template <bool H> struct Band64Frag { typedef bf16x8 type; };
template <> struct Band64Frag<true> { typedef f16x8 type; };

template <int MT, int NT, bool H>
struct Band64Step {
  typedef typename Band64Frag<H>::type frag;
  frag w[NT];
  frag xh[MT], xl[H ? 1 : MT];
};

template <int MT, int NT, bool H>
__device__ __forceinline__ void band64_load(const unsigned char* lds,
                                            const typename Band64Frag<H>::type* __restrict__ wp,
                                            int ks, const uint32_t (&base)[MT],
                                            const uint32_t (&base_lo)[MT], uint32_t off,
                                            Band64Step<MT, NT, H>& st) {
  typedef typename Band64Frag<H>::type frag;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) st.w[nt] = wp[(ks * NT + nt) * 64];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    st.xh[i] = *reinterpret_cast<const frag*>(lds + base[i] + off);
    if constexpr (!H) st.xl[i] = *reinterpret_cast<const frag*>(lds + base_lo[i] + off);
  }
}

template <int MT, int NT, bool H>
__device__ __forceinline__ void band64_mma(const Band64Step<MT, NT, H>& st, f32x4 (&acc)[MT][NT]) {
  if constexpr (H) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[i][nt] = mma_f16(st.w[nt], st.xh[i], acc[i][nt]);
  } else {
    using X = Elt<uint16_t>;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[i][nt] = X::mma(st.w[nt], st.xh[i], acc[i][nt]);
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[i][nt] = X::mma(st.w[nt], st.xl[i], acc[i][nt]);
  }
}

template <int MT, int NT, bool H>
__device__ __forceinline__ void band64_tiles(const unsigned char* lds, const Band64& b,
                                             const typename Band64Frag<H>::type* __restrict__ wf,
                                             const int (&pix)[MT], int g, int lane,
                                             f32x4 (&acc)[MT][NT]) {
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[i][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint32_t base[MT], base_lo[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    base[i] = (uint32_t)(g * b.cp + pix[i]) * 16u;
    base_lo[i] = base[i] + (uint32_t)b.lo_bytes;
  }
  const uint32_t step2 = (uint32_t)b.cp * 64u;  // chunks 4..7: 4 chunk planes on
  const typename Band64Frag<H>::type* wp = wf + lane;
  if constexpr (H) {
    // fp16: the weight fragments (from L2) and the activation fragments (LDS)
    // of the next K step are loaded while the current one computes, in two
    // register sets (steps 2 j and 2 j + 1), so that up to 7 tiles fit
    constexpr int KSTEPS = 18;  // 9 taps x 2 steps of 32 channels
    f16x8 wa[NT], wb[NT], xa[MT], xb[MT];
    auto ldw = [&](int j, f16x8 (&d)[NT]) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) d[nt] = wp[(j * NT + nt) * 64];
    };
    auto ldx = [&](int j, f16x8 (&d)[MT]) {
      const int tap = j >> 1, dy = tap / 3, dx = tap - 3 * dy;
      const uint32_t off = (uint32_t)(dy * b.wb + dx) * 16u + ((j & 1) ? step2 : 0u);
#pragma unroll
      for (int i = 0; i < MT; ++i) d[i] = *reinterpret_cast<const f16x8*>(lds + base[i] + off);
    };
    auto mma = [&](const f16x8 (&wv)[NT], const f16x8 (&xv)[MT]) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[i][nt] = mma_f16(wv[nt], xv[i], acc[i][nt]);
    };
    ldw(0, wa);
    ldx(0, xa);
#pragma unroll 1
    for (int j = 0; j < KSTEPS; j += 2) {
      ldw(j + 1, wb);
      ldx(j + 1, xb);
      __builtin_amdgcn_sched_barrier(0);
      mma(wa, xa);
      __builtin_amdgcn_sched_barrier(0);
      const int jn = j + 2 < KSTEPS ? j + 2 : j + 1;  // the last step reloads its own, unused
      ldw(jn, wa);
      ldx(jn, xa);
      __builtin_amdgcn_sched_barrier(0);
      mma(wb, xb);
      __builtin_amdgcn_sched_barrier(0);
    }
    return;
  }
  Band64Step<MT, NT, H> sa, sb;
  band64_load<MT, NT, H>(lds, wp, 0, base, base_lo, 0u, sa);
#pragma unroll 1
  for (int tap = 0; tap < 9; ++tap) {
    const int dy = tap / 3, dx = tap - 3 * dy;
    const uint32_t toff = (uint32_t)(dy * b.wb + dx) * 16u;
    // step B of this tap in flight while step A computes
    band64_load<MT, NT, H>(lds, wp, 2 * tap + 1, base, base_lo, toff + step2, sb);
    __builtin_amdgcn_sched_barrier(0);
    band64_mma<MT, NT, H>(sa, acc);
    __builtin_amdgcn_sched_barrier(0);
    // step A of the next tap (the last tap reloads its own, unused)
    const int tn = tap < 8 ? tap + 1 : tap;
    const int dyn = tn / 3, dxn = tn - 3 * dyn;
    band64_load<MT, NT, H>(lds, wp, 2 * tn, base, base_lo, (uint32_t)(dyn * b.wb + dxn) * 16u, sa);
    __builtin_amdgcn_sched_barrier(0);
    band64_mma<MT, NT, H>(sb, acc);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Lane permutation within quads of lanes (DPP quad_perm).
template <int CTRL>
__device__ __forceinline__ float quad_perm(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kQuadXor1 = 0xB1;  // [1, 0, 3, 2]
constexpr int kQuadXor2 = 0x4E;  // [2, 3, 0, 1]

// Bias, ReLU, optional 2x2 max-pool and NHWC stores of one transposed tile;
// (oy, ox) is this lane's pixel in the layer's input grid.  Each value is
// max(acc * k + bb, 0) in one fused multiply-add: on the fp16 path k is the
// accumulator scale times the output scale s and bb the bias times s (s the
// next layer's input scale when the output is fp16, else 1; all scales are
// powers of two, so this equals scaling after the bias and the ReLU, bit for
// bit); otherwise k = 1 and bb is the bias.  The output is fp32 (16-byte
// stores), or with f16out fp16 (8-byte stores).
template <int NT>
__device__ __forceinline__ void band64_epilogue(const f32x4 (&acc)[NT], const float* __restrict__ bp,
                                                float s, float k, void* out, int cout, int oy,
                                                int ox, int h, int w, int pool, int m, bool f16out) {
  auto store = [&](int64_t e, const float (&v)[4]) {  // element offset e, 4 channels
    if (f16out)
      *reinterpret_cast<uint2*>(static_cast<_Float16*>(out) + e) =
          make_uint2(__builtin_bit_cast(uint32_t, f16x2{(_Float16)v[0], (_Float16)v[1]}),
                     __builtin_bit_cast(uint32_t, f16x2{(_Float16)v[2], (_Float16)v[3]}));
    else
      *reinterpret_cast<float4*>(static_cast<float*>(out) + e) = make_float4(v[0], v[1], v[2], v[3]);
  };
  const int qy = oy >> 1, qx = ox >> 1;
  const bool st = pool ? ((m & 3) == 0 && qy < (h >> 1) && qx < (w >> 1)) : (oy < h && ox < w);
  const int64_t e0 = pool ? ((int64_t)qy * (w >> 1) + qx) * cout : ((int64_t)oy * w + ox) * cout;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const f32x4 t = acc[nt];
    const float4 bb = *reinterpret_cast<const float4*>(bp + nt * 16);
    float v[4] = {fmaxf(fmaf(t[0], k, bb.x * s), 0.f), fmaxf(fmaf(t[1], k, bb.y * s), 0.f),
                  fmaxf(fmaf(t[2], k, bb.z * s), 0.f), fmaxf(fmaf(t[3], k, bb.w * s), 0.f)};
    if (pool) {
      // the four pixels of a pooling window are the four lanes of a quad; the
      // values are >= 0 (or -0) after the ReLU, so their maximum is the
      // signed-integer maximum of their bits (which needs no NaN quieting of
      // the permuted operands, and takes the permutation as a DPP operand)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        int iv = __float_as_int(v[r]);
        iv = max(iv, __builtin_amdgcn_update_dpp(0, iv, kQuadXor1, 0xF, 0xF, false));
        iv = max(iv, __builtin_amdgcn_update_dpp(0, iv, kQuadXor2, 0xF, 0xF, false));
        v[r] = __int_as_float(iv);
      }
    }
    if (st) store(e0 + nt * 16, v);
  }
}

// MT tiles of a band: tiles first, first + 4, ... (band-local tile index, see
// band_pixel), through the epilogue.  out already points at this lane's
// channel group (4 g).
template <int MT, int NT, bool H>
__device__ __forceinline__ void band64_run(const unsigned char* lds, const Band64& b, int ty0,
                                           const typename Band64Frag<H>::type* __restrict__ wf,
                                           const float* __restrict__ bp, float s, float k,
                                           void* out, int cout, int pool, int rows, int wn,
                                           int first, int m, int g, int lane, bool f16out) {
  int pix[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    int r, x;
    band_pixel(first + kBandWaves * i, m, pool, rows, wn, r, x);
    pix[i] = r * b.wb + x;  // (0, 0) past the band's last pixel: in bounds
  }
  f32x4 acc[MT][NT];
  band64_tiles<MT, NT, H>(lds, b, wf, pix, g, lane, acc);
  // the pixels again, computed only now (an opaque copy of `first` after the
  // tiles' loads) so that they take no registers through the tiles
  int first2 = first;
  asm volatile("" : "+s"(first2) : : "memory");
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    int r, x;
    const bool in = band_pixel(first2 + kBandWaves * i, m, pool, rows, wn, r, x);
    band64_epilogue<NT>(acc[i], bp, s, k, out, cout, in ? 4 * ty0 + r : b.h, x, b.h, b.w, pool, m,
                        f16out);  // no store past the band's last pixel
  }
}

// One band's work of a 64-input-channel layer: the band's output rows 4 ty0
// .. 4 (ty0 + nty) - 1 (those the layer computes) as band64_ntile tiles over
// the 4 waves, at most MTMAX per wave per round.  sc is the accumulator scale
// (fp16 path, else 1) and st16 the next layer's input scale when the output
// is fp16 (else 0).
template <int NT, bool H>
__device__ __forceinline__ void band64_layer(const unsigned char* lds, const Band64& b, int ty0,
                                             int nty,
                                             const typename Band64Frag<H>::type* __restrict__ wf,
                                             const float* __restrict__ bias, void* out, int cout,
                                             int pool, int wave, int m, int g, int lane, float sc,
                                             float st16) {
  const int hn = pool ? (b.h / 2) * 2 : b.h, wn = pool ? (b.w / 2) * 2 : b.w;
  const int rows = min(4 * nty, hn - 4 * ty0);
  const int ntile = band64_ntile(pool != 0, rows, wn);
  const bool f16out = st16 != 0.0f;
  const float s = f16out ? st16 : 1.0f;
  const float k = H ? sc * s : 1.0f;
  const float* bp = bias + 4 * g;  // this lane's channel group
  out = f16out ? static_cast<void*>(static_cast<_Float16*>(out) + 4 * g)
               : static_cast<void*>(static_cast<float*>(out) + 4 * g);
  constexpr int MTMAX = H ? kBandMaxTilesH : 4;
  for (int base = 0; base < ntile; base += MTMAX * kBandWaves) {
    const int first = base + wave;
    const int mt = first >= ntile ? 0 : min(MTMAX, (ntile - first + kBandWaves - 1) / kBandWaves);
    if constexpr (H) {
      switch (mt) {
        case 7:
          band64_run<7, NT, H>(lds, b, ty0, wf, bp, s, k, out, cout, pool, rows, wn, first, m, g,
                               lane, f16out);
          continue;
        case 6:
          band64_run<6, NT, H>(lds, b, ty0, wf, bp, s, k, out, cout, pool, rows, wn, first, m, g,
                               lane, f16out);
          continue;
        case 5:
          band64_run<5, NT, H>(lds, b, ty0, wf, bp, s, k, out, cout, pool, rows, wn, first, m, g,
                               lane, f16out);
          continue;
        default:
          break;
      }
    }
    switch (mt) {
      case 4:
        band64_run<4, NT, H>(lds, b, ty0, wf, bp, s, k, out, cout, pool, rows, wn, first, m, g,
                             lane, f16out);
        break;
      case 3:
        band64_run<3, NT, H>(lds, b, ty0, wf, bp, s, k, out, cout, pool, rows, wn, first, m, g,
                             lane, f16out);
        break;
      case 2:
        band64_run<2, NT, H>(lds, b, ty0, wf, bp, s, k, out, cout, pool, rows, wn, first, m, g,
                             lane, f16out);
        break;
      case 1:
        band64_run<1, NT, H>(lds, b, ty0, wf, bp, s, k, out, cout, pool, rows, wn, first, m, g,
                             lane, f16out);
        break;
      default:
        break;
    }
  }
}

// One 64-input-channel layer over bands of fp32 activations (H: through the
// fp16 matrix cores, weights a.wts in scaled fp16 fragments).
template <int NT, bool G, bool H>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_band64(ConvArgs a, Band64 b) {
  typedef typename Band64Frag<H>::type frag;
  extern __shared__ __align__(16) unsigned char lds[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m = lane & 15, g = lane >> 4;
  const frag* wf = reinterpret_cast<const frag*>(a.wts);
  band64_clear(lds, b);
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int bands = (a.tiles_y + a.band_tiles - 1) / a.band_tiles;
  const int64_t items = (cnt + 7) / 8 * 8 * bands;
  const int ho = a.pool ? a.h / 2 : a.h, wo = a.pool ? a.w / 2 : a.w;
  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    int64_t s;
    int bi;
    band_item(item, bands, &s, &bi);
    if (s >= cnt) continue;  // workgroup-uniform
    const int ty0 = bi * a.band_tiles;
    const int nty = min(a.band_tiles, a.tiles_y - ty0);
    const int64_t off = G ? slot_woff(a.nets, a.per_cam, a.idx, s) : 0;  // camera group
    float in_scale = 1.0f, out_scale = 1.0f, st16 = 0.0f;
    if constexpr (H) {
      const float* sc = at_off(a.scl, off);
      in_scale = sc[0];
      out_scale = sc[1];
      if (a.out_f16) st16 = sc[2];
    }
    const int64_t in_e = s * (int64_t)a.h * a.w * 64, out_e = s * (int64_t)ho * wo * a.cout;
    __syncthreads();  // the previous band's readers are done (and the clear)
    if (H && a.in_f16)
      stage_band64_f16(reinterpret_cast<const _Float16*>(a.act_in) + in_e, b, lds, 4 * ty0 - 1,
                       4 * nty + 2);
    else
      stage_band64<H>(a.act_in + in_e, b, lds, 4 * ty0 - 1, 4 * nty + 2, in_scale);
    __syncthreads();
    void* out = st16 != 0.0f ? static_cast<void*>(reinterpret_cast<_Float16*>(a.act_out) + out_e)
                             : static_cast<void*>(a.act_out + out_e);
    band64_layer<NT, H>(lds, b, ty0, nty, at_off(wf, off), at_off(a.bias, off), out, a.cout,
                        a.pool, wave, m, g, lane, out_scale, st16);
  }
}

// Channel 3 of the pre-processed input is the constant 1 (bf16 bits 0x3F80 in
// the upper half of the pixel's second word), also on the zero border: the
// fp16 path's first-layer weights carry the bias there; elsewhere its
// weights are 0.
constexpr uint32_t kOneBf16Hi = 0x3F800000u;

// The pre-processed bf16 input of one first-layer pixel: channels 0-2 of
// (S / den) / 127.5 - 1 from the fy x fx cell sums of image pixel (y, x) of
// frame idx[s], correctly rounded, and channel 3 = 1.
__device__ __forceinline__ uint2 first_input_bf16(const ConvArgs& a, int64_t s, int y, int x) {
  const int32_t* S = a.sums + (int64_t)a.idx[s] * a.sums_h * a.sums_w * 3;
  int32_t acc[3];
  cell_sums(a, S, y, x, acc);
  uint16_t v[3];
  const bool f32div = a.den255 < (1 << 24);
  const float inv = 1.0f / (float)a.den255;
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    const int64_t num = 2 * (int64_t)acc[c] - a.den255;
    v[c] = f32div ? div_to_bf16_bits_fast((int32_t)num, (int32_t)a.den255, inv)
                  : f64_to_bf16_bits((double)num / (double)a.den255);
  }
  return make_uint2((uint32_t)v[0] | ((uint32_t)v[1] << 16), (uint32_t)v[2] | kOneBf16Hi);
}

// Pre-processed bf16 input of every survivor for k_pair64, zero-bordered
// (channel 3 = 1 everywhere): xin[slot][xr][xw] pixels of 4 bf16, image pixel
// (y, x) at (y + 2, x + 1).
__global__ void __launch_bounds__(256) k_prep_input(ConvArgs a, uint2* xin, int32_t xr, int32_t xw) {
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int64_t per = (int64_t)xr * xw;
  const int64_t total = cnt * per;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t s = i / per;
    const int q = (int)(i - s * per);
    const int row = q / xw, col = q - row * xw;
    const int y = row - 2, x = col - 1;
    uint2 v = make_uint2(0u, kOneBf16Hi);
    if ((unsigned)y < (unsigned)a.h && (unsigned)x < (unsigned)a.w) v = first_input_bf16(a, s, y, x);
    xin[i] = v;
  }
}

// The first two layers of a bf16 network fused per band, when the first
// (3 -> 64 channels) does not pool: the first layer computes the band's rows
// (with the halo rows) from the pre-processed input (k_prep_input) straight
// into the hi / lo planes, then the second layer runs from them.  First-layer
// tiles are 2 rows x 8 columns; its K is (dy, dx of 4, c of 4) = 48 of 64.
// A wave issues the input loads of up to kPairL1Batch of its first-layer tiles
// of a band before computing the first of them.

constexpr int kPairL1Batch = 7;  // first-layer tiles per wave whose loads are issued together

template <int NT, bool G, bool H>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_pair64(ConvArgs a0, ConvArgs a1, Band64 b, const uint2* __restrict__ xin, int32_t xr,
         int32_t xw) {
  using X = Elt<uint16_t>;
  typedef typename Band64Frag<H>::type frag1;
  extern __shared__ __align__(16) unsigned char lds[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m = lane & 15, g = lane >> 4;
  const bf16x8* wf0 = reinterpret_cast<const bf16x8*>(a0.wts);
  const frag1* wf1 = reinterpret_cast<const frag1*>(a1.wts);
  band64_clear(lds, b);
  int64_t cnt = *a0.count;
  if (cnt > a0.max_count) cnt = a0.max_count;
  const int bands = (a1.tiles_y + a1.band_tiles - 1) / a1.band_tiles;
  const int ho = a1.pool ? a1.h / 2 : a1.h, wo = a1.pool ? a1.w / 2 : a1.w;
  const int tx0 = (b.w + 7) / 8;      // first-layer tile columns
  const int qy = m >> 3, qx = m & 7;  // first-layer lane pixel in a 2 x 8 tile
  // this lane's K chunks of the first layer: pixels (dy, dx) and (dy, dx + 1)
  // of steps 0 and 1 (step 1 only for lane groups 0 and 1: K = 48)
  const int k0 = g * 8, k1 = 32 + g * 8;
  const int off0 = (k0 >> 4) * xw + ((k0 >> 2) & 3);
  const int off1 = (k1 >> 4) * xw + ((k1 >> 2) & 3);
  const bool use1 = k1 < 48;

  // the two K chunks of first-layer tile t of a band (band row 0 = image row y0)
  auto l1_load = [&](const uint2* xs, int y0, int t, uint4 (&x)[2]) {
    const int ti = t / tx0, tj = t - ti * tx0;
    const int y = y0 + 2 * ti + qy, col = 8 * tj + qx;
    // input pixel (y + dy - 1, col + dx - 1) is xin (y + dy + 1, col + dx)
    const uint2* p = xs + (int64_t)(y + 1) * xw + col;
    const uint2 p00 = p[off0], p01 = p[off0 + 1];
    uint2 p10 = make_uint2(0u, 0u), p11 = p10;
    if (use1) {
      p10 = p[off1];
      p11 = p[off1 + 1];
    }
    x[0] = make_uint4(p00.x, p00.y, p01.x, p01.y);
    x[1] = make_uint4(p10.x, p10.y, p11.x, p11.y);
  };
  // first-layer tile t: 8 MFMAs, then into the planes: on the fp16 path the
  // ReLU of the (biased, scaled) result as fp16, else bias, ReLU and the hi /
  // lo split
  const float* bias0 = a0.bias;  // the item's network (camera group)
  float out_scale1 = 1.0f, st16 = 0.0f;  // fp16 path: the second layer's scales
  auto l1_tile = [&](const bf16x8 (&w0)[2][4], int y0, int t, const uint4 (&x)[2]) {
    const int ti = t / tx0, tj = t - ti * tx0;
    const int r = 2 * ti + qy, col = 8 * tj + qx;
    const int y = y0 + r;
    const bf16x8 x0 = __builtin_bit_cast(bf16x8, x[0]);
    const bf16x8 x1 = __builtin_bit_cast(bf16x8, x[1]);
    f32x4 acc[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      acc[nt] = X::mma(w0[0][nt], x0, f32x4{0.f, 0.f, 0.f, 0.f});
      acc[nt] = X::mma(w0[1][nt], x1, acc[nt]);
    }
    if (col < b.w) {
      const bool inside = (unsigned)y < (unsigned)b.h;  // rows outside are zero
      const int addr = ((g >> 1) * b.cp + r * b.wb + col + 1) * 16 + (g & 1) * 8;
      if constexpr (H) {
        // the weights carry the bias and the second layer's input scale:
        // fp16 of the ReLU (the conversion is monotonic and keeps 0)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          const f16x2 z = {(_Float16)0.0f, (_Float16)0.0f};
          const f16x2 p0 = __builtin_elementwise_max(
              f16x2{(_Float16)acc[nt][0], (_Float16)acc[nt][1]}, z);
          const f16x2 p1 = __builtin_elementwise_max(
              f16x2{(_Float16)acc[nt][2], (_Float16)acc[nt][3]}, z);
          *reinterpret_cast<uint2*>(lds + addr + 2 * nt * b.cp * 16) =
              inside ? make_uint2(__builtin_bit_cast(uint32_t, p0), __builtin_bit_cast(uint32_t, p1))
                     : make_uint2(0u, 0u);
        }
        return;
      }
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const float4 bb = *reinterpret_cast<const float4*>(bias0 + nt * 16 + 4 * g);
        const float v0 = inside ? fmaxf(acc[nt][0] + bb.x, 0.f) : 0.f;
        const float v1 = inside ? fmaxf(acc[nt][1] + bb.y, 0.f) : 0.f;
        const float v2 = inside ? fmaxf(acc[nt][2] + bb.z, 0.f) : 0.f;
        const float v3 = inside ? fmaxf(acc[nt][3] + bb.w, 0.f) : 0.f;
        const int ad = addr + 2 * nt * b.cp * 16;  // chunk 2 nt + g / 2
        uint32_t h01, l01, h23, l23;
        X::split2(v0, v1, h01, l01);
        X::split2(v2, v3, h23, l23);
        *reinterpret_cast<uint2*>(lds + ad) = make_uint2(h01, h23);
        *reinterpret_cast<uint2*>(lds + b.lo_bytes + ad) = make_uint2(l01, l23);
      }
    }
  };

  // The first layer of band (ty0, nty) of image s into the planes, rows
  // 2 tfirst_row .. 4 nty + 1 (rows 0-1 taken from the previous band when
  // tfirst_row is 1), then the second layer from them.
  const int bt = a1.band_tiles;
  auto band = [&](int64_t s, int ty0, int nty, int prev_rows) {
    const uint2* xs = xin + s * (int64_t)xr * xw;
    const int64_t off = G ? slot_woff(a0.nets, a0.per_cam, a0.idx, s) : 0;  // camera group
    bias0 = at_off(a0.bias, off);
    if constexpr (H) {
      const float* sc = at_off(a1.scl, off);
      out_scale1 = sc[1];
      if (a1.out_f16) st16 = sc[2];
    }
    const int y0 = 4 * ty0 - 1;
    const int t0n = (2 * nty + 1) * tx0;     // first-layer tiles: rows 4 nty + 2
    const int tfirst = prev_rows ? tx0 : 0;  // rows 0-1 copied after an image's first band
    // this wave's first-layer tiles of the band (up to kPairL1Batch at once):
    // all their input loads are issued before the first is used
    uint4 xb[kPairL1Batch][2];
    auto load_batch = [&](int tb) {
#pragma unroll
      for (int i = 0; i < kPairL1Batch; ++i)
        if (tb + kBandWaves * i < t0n) l1_load(xs, y0, tb + kBandWaves * i, xb[i]);
    };
    load_batch(tfirst + wave);
    // first-layer weights for this band's first-layer phase only: an opaque
    // zero keeps the compiler from hoisting them out of the band loop (which
    // would hold 32 registers through the second layer)
    int opaque = 0;
    asm volatile("" : "+s"(opaque));
    const bf16x8* w0p = at_off(wf0, off) + opaque + lane;
    bf16x8 w0[2][4];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) w0[ks][nt] = w0p[(ks * 4 + nt) * 64];
    __syncthreads();  // the previous band's second layer is done with the planes
    if (prev_rows) {
      // rows prev_rows - 2, prev_rows - 1 -> rows 0, 1 of every chunk plane
      const int per = 2 * b.wb;
      for (int u = threadIdx.x; u < 8 * b.planes * per; u += blockDim.x) {
        const int pc = u / per, e = u - pc * per;  // plane x chunk, unit in the two rows
        const int base = ((pc >> 3) * 8 * b.cp + (pc & 7) * b.cp) * 16;
        const uint4 v = *reinterpret_cast<const uint4*>(lds + base + ((prev_rows - 2) * b.wb + e) * 16);
        *reinterpret_cast<uint4*>(lds + base + e * 16) = v;
      }
      __syncthreads();  // copied before the first layer overwrites the source rows
    }
    for (int tb = tfirst + wave; tb < t0n; tb += kBandWaves * kPairL1Batch) {
      if (tb != tfirst + wave) load_batch(tb);
#pragma unroll
      for (int i = 0; i < kPairL1Batch; ++i)
        if (tb + kBandWaves * i < t0n) l1_tile(w0, y0, tb + kBandWaves * i, xb[i]);
    }
    __syncthreads();  // planes complete
    const int64_t out_e = s * (int64_t)ho * wo * a1.cout;
    void* out = st16 != 0.0f ? static_cast<void*>(reinterpret_cast<_Float16*>(a1.act_out) + out_e)
                             : static_cast<void*>(a1.act_out + out_e);
    band64_layer<NT, H>(lds, b, ty0, nty, at_off(wf1, off), at_off(a1.bias, off), out, a1.cout,
                        a1.pool, wave, m, g, lane, out_scale1, st16);
  };
  // Rounds of work either way: image-major (a band there skips recomputing
  // two of its first-layer rows, counted as a tenth of its cost) or one band
  // per item.
  const int64_t items = (cnt + 7) / 8 * 8 * bands;
  const int64_t im_rounds = (cnt + gridDim.x - 1) / gridDim.x * bands;
  const int64_t bp_rounds = (items + gridDim.x - 1) / gridDim.x;
  if (10 * im_rounds <= 11 * bp_rounds) {
    // a workgroup runs the bands of an image in order (workgroup i, and so
    // one XCD, takes images i, i + grid, ...), copying the two halo rows a
    // band shares with the previous one
    for (int64_t s = blockIdx.x; s < cnt; s += gridDim.x) {
      int prev_rows = 0;
      for (int bi = 0; bi < bands; ++bi) {
        const int ty0 = bi * bt, nty = min(bt, a1.tiles_y - ty0);
        band(s, ty0, nty, prev_rows);
        prev_rows = 4 * nty + 2;
      }
    }
  } else {
    // few images: every (image, band) is a work item of its own (all bands of
    // an image on one XCD, see band_item), each band computing its halo rows
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
      int64_t s;
      int bi;
      band_item(it, bands, &s, &bi);
      if (s >= cnt) continue;  // workgroup-uniform
      const int ty0 = bi * bt;
      band(s, ty0, min(bt, a1.tiles_y - ty0), 0);
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
  const float* scl;         // fp16 path: (input scale, output scale) in the weight image
  int32_t feat_f16;         // fp16 path: feat holds fp16 values already times the input scale
  int32_t tiled;            // the partial blocks come from k_dense_tiles (its K parts)
  const CamNet* nets;       // camera group (else null)
  int64_t per_cam;
};

// The output of one 16-survivor tile from its hidden pre-activations t (lane
// (m, g): rows row0 + 4 g + r, units 16 nt + m): hidden = ReLU(t + b1),
// z = b2 + sum_n w2[n] hidden[n] (a 16-lane shuffle reduction), then the
// logit, the sigmoid and the decision at the frame's position, for the rows
// of camera cam (every row without a camera group).
template <int NT, bool G>
__device__ __forceinline__ void dense_out(const DenseArgs& a, const f32x4 (&t)[NT],
                                          const float* b1, const float* w2, float b2,
                                          double c_low, double c_high, int64_t row0,
                                          int64_t cnt, int64_t cam, int m, int g) {
  float sum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = nt * 16 + m;
    const float b = b1[n], w = w2[n];
#pragma unroll
    for (int r = 0; r < 4; ++r) sum[r] += w * fmaxf(t[nt][r] + b, 0.0f);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) sum[r] += __shfl_xor(sum[r], o, 64);
  }
  if (m == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t slot = row0 + 4 * g + r;
      if (slot < cnt && (!G || a.idx[slot] / a.per_cam == cam)) {
        const float z = sum[r] + b2;
        const double p = 1.0 / (1.0 + exp(-(double)z));
        a.logit[slot] = z;
        if (a.prob) a.prob[slot] = (float)p;
        if (a.dec || a.frame_logit) {
          const int32_t f = a.idx[slot];
          if (a.dec) a.dec[f] = p < c_low ? 0 : (p > c_high ? 1 : 2);
          if (a.frame_logit) a.frame_logit[f] = z;
        }
      }
    }
  }
}

// Dense workgroups for large batches (kDenseBig survivors and more): NW
// waves split K (so that a group is a short dependence chain per wave), and
// each wave keeps MT tiles of 16 survivors, so that every weight fragment it
// loads serves MT x 16 survivors.  The partial sums meet in LDS
// (NW x MT x NT x 1 KB, at most 64 KB).  Smaller batches take
// k_dense_part / k_dense_finish below.
template <int NT>
constexpr int dense_mt() {
  return NT >= 16 ? 1 : (NT >= 8 ? 2 : 4);
}
constexpr int kDenseWaves = 4;
constexpr int64_t kDenseBig = 16384;  // max_count from which k_dense is used

template <typename T, int NT, bool G>
__global__ void __launch_bounds__(64 * kDenseWaves) k_dense(DenseArgs a) {
  using X = Elt<T>;
  constexpr int E = X::E, KS = X::KS;
  constexpr bool SPLIT = X::SPLIT;
  constexpr int NW = kDenseWaves, MT = dense_mt<NT>(), R = 16 * MT;  // rows of a group
  // per wave, row tile and output tile, each lane's 4 partial sums
  __shared__ f32x4 part[NW][MT][NT][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m = lane & 15, g = lane >> 4;
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int64_t groups = (cnt + R - 1) / R;
  const int nks = (a.flat + KS - 1) / KS;  // K steps
  const int ks0 = wave * nks / NW, ks1 = (wave + 1) * nks / NW;
  // camera of survivor slot u of a camera group (slots are in frame order, so
  // a group's cameras are non-decreasing)
  auto cam_of = [&](int64_t u) -> int64_t { return a.idx[u] / a.per_cam; };
  for (int64_t grp = blockIdx.x; grp < groups; grp += gridDim.x) {
    // A group runs once per camera among its rows (once without a camera
    // group), each pass with that camera's weights over its own rows.
    int64_t cam = G ? cam_of(grp * R) : 0;
    for (;;) {
      int64_t off = 0;
      float b2 = a.b2;
      double c_low = a.c_low, c_high = a.c_high;
      if constexpr (G) {
        const CamNet& cn = a.nets[cam];
        off = cn.woff;
        b2 = cn.b2;
        c_low = cn.c_low;
        c_high = cn.c_high;
      }
      const T* w1 = at_off(reinterpret_cast<const T*>(a.w1), off);
      const float* b1 = at_off(a.b1, off);
      const float* w2 = at_off(a.w2, off);
      float in_scale = 1.0f, out_scale = 1.0f;
      if constexpr (X::CVT) {
        const float* sc = at_off(a.scl, off);
        in_scale = sc[0];
        out_scale = sc[1];
      }
      bool valid[MT];
      const float* arow[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int64_t s = grp * R + mt * 16 + m;
        valid[mt] = s < cnt && (!G || cam_of(s) == cam);
        arow[mt] = a.feat + (valid[mt] ? s : 0) * (int64_t)a.flat + g * E;
      }
      f32x4 acc[MT][NT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      // flat is a multiple of 16 (and of E): a lane group's E values of the last,
      // partial K step are either all inside or all past the end (zero); the
      // hi and lo products of a bf16 network share the accumulators
      for (int ks = ks0; ks < ks1; ++ks) {
        const int k0 = ks * KS;
        const bool kin = k0 + g * E < a.flat;
        typename X::frag bv[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          bv[nt] = X::zero();
          if (kin) bv[nt] = X::load(w1 + (int64_t)(nt * 16 + m) * a.flat + k0 + g * E);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          typename X::frag av = X::zero(), av_lo = X::zero();
          if constexpr (SPLIT) {
            if (valid[mt] && kin) X::split8(arow[mt] + k0, av, av_lo);
          } else if constexpr (X::CVT) {
            if (valid[mt] && kin)
              av = a.feat_f16 ? X::load(reinterpret_cast<const _Float16*>(a.feat) + (arow[mt] - a.feat) + k0)
                              : X::cvt8(arow[mt] + k0, in_scale);
          } else {
            if (valid[mt] && kin) av = arow[mt][k0];
          }
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            acc[mt][nt] = X::mma(av, bv[nt], acc[mt][nt]);
            if constexpr (SPLIT) acc[mt][nt] = X::mma(av_lo, bv[nt], acc[mt][nt]);
          }
        }
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) part[wave][mt][nt][lane] = acc[mt][nt];
      __syncthreads();
      // wave w finishes row tiles w, w + NW, ...
      for (int mt = wave; mt < MT; mt += NW) {
        f32x4 t[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          t[nt] = part[0][mt][nt][lane];
#pragma unroll
          for (int w = 1; w < NW; ++w) t[nt] += part[w][mt][nt][lane];
          if constexpr (X::CVT) t[nt] *= out_scale;
        }
        dense_out<NT, G>(a, t, b1, w2, b2, c_low, c_high, grp * R + mt * 16, cnt, cam, m, g);
      }
      __syncthreads();  // the partial sums are read before the next pass writes them
      if constexpr (!G) break;
      // the next camera among the group's rows (uniform)
      int64_t next = -1;
      for (int r = 0; r < R && next < 0; ++r) {
        const int64_t u = grp * R + r;
        if (u < cnt && cam_of(u) > cam) next = cam_of(u);
      }
      if (next < 0) break;
      cam = next;
    }
  }
}

// Small batches (a stream's chunk with a few hundred survivors): the K
// range is split over workgroups as well, so that the few 16-survivor tiles
// still spread over the chip and every wave's dependence chain is short.
// k_dense_part: a (tile, K part) item per workgroup, whose 8 waves split the
// part and add their sums through LDS into the item's partial block
// (NT x 1 KB, lane layout of the accumulators); in a camera group each
// camera among the tile's rows is a pass with its own weights over its own
// rows, all passes into the same accumulators.  k_dense_finish: a wave per
// tile adds its parts in order and applies dense_out.  Deterministic.
constexpr int kDenseSplitItems = 1024;  // most (tile, K part) items, so the partial blocks' bound
constexpr int kDenseSplitWaves = 8;

// K parts per tile: enough items to fill the chip, at least one K step per wave.
__device__ __forceinline__ int dense_kparts(int64_t tiles, int nks) {
  int64_t k = kDenseSplitItems / (tiles > 0 ? tiles : 1);
  const int64_t kmax = nks / kDenseSplitWaves > 0 ? nks / kDenseSplitWaves : 1;
  if (k > kmax) k = kmax;
  return k < 1 ? 1 : (int)k;
}

template <typename T, int NT, bool G>
__global__ void __launch_bounds__(64 * kDenseSplitWaves) k_dense_part(DenseArgs a,
                                                                      f32x4* __restrict__ part) {
  using X = Elt<T>;
  constexpr int E = X::E, KS = X::KS;
  constexpr bool SPLIT = X::SPLIT;
  constexpr int NW = kDenseSplitWaves;
  __shared__ f32x4 red[NW][NT][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m = lane & 15, g = lane >> 4;
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int64_t tiles = (cnt + 15) / 16;
  const int nks = (a.flat + KS - 1) / KS;
  const int kparts = dense_kparts(tiles, nks);
  const int64_t items = tiles * kparts;
  auto cam_of = [&](int64_t u) -> int64_t { return a.idx[u] / a.per_cam; };
  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int64_t tile = item / kparts;
    const int kp = (int)(item - tile * kparts);
    const int kb = (int)((int64_t)kp * nks / kparts), ke = (int)((int64_t)(kp + 1) * nks / kparts);
    const int ks0 = kb + wave * (ke - kb) / NW, ks1 = kb + (wave + 1) * (ke - kb) / NW;
    const int64_t s = tile * 16 + m;  // this lane's row (survivor slot)
    f32x4 acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    int64_t cam = G ? cam_of(tile * 16) : 0;
    for (;;) {
      const int64_t off = G ? (int64_t)a.nets[cam].woff : 0;
      const T* w1 = at_off(reinterpret_cast<const T*>(a.w1), off);
      const float in_scale = X::CVT ? at_off(a.scl, off)[0] : 1.0f;
      const bool valid = s < cnt && (!G || cam_of(s) == cam);
      const float* arow = a.feat + (valid ? s : 0) * (int64_t)a.flat + g * E;
      // as in k_dense: a lane group's E values of the last K step are all
      // inside or all past the end; hi and lo products share the accumulators
      for (int ks = ks0; ks < ks1; ++ks) {
        const int k0 = ks * KS;
        const bool kin = k0 + g * E < a.flat;
        typename X::frag bv[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          bv[nt] = X::zero();
          if (kin) bv[nt] = X::load(w1 + (int64_t)(nt * 16 + m) * a.flat + k0 + g * E);
        }
        typename X::frag av = X::zero(), av_lo = X::zero();
        if constexpr (SPLIT) {
          if (valid && kin) X::split8(arow + k0, av, av_lo);
        } else if constexpr (X::CVT) {
          if (valid && kin)
            av = a.feat_f16 ? X::load(reinterpret_cast<const _Float16*>(a.feat) + (arow - a.feat) + k0)
                            : X::cvt8(arow + k0, in_scale);
        } else {
          if (valid && kin) av = arow[k0];
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          acc[nt] = X::mma(av, bv[nt], acc[nt]);
          if constexpr (SPLIT) acc[nt] = X::mma(av_lo, bv[nt], acc[nt]);
        }
      }
      if constexpr (!G) break;
      // the next camera among the tile's rows (uniform)
      int64_t next = -1;
      for (int r = 0; r < 16 && next < 0; ++r) {
        const int64_t u = tile * 16 + r;
        if (u < cnt && cam_of(u) > cam) next = cam_of(u);
      }
      if (next < 0) break;
      cam = next;
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) red[wave][nt][lane] = acc[nt];
    __syncthreads();
    for (int nt = wave; nt < NT; nt += NW) {
      f32x4 t = red[0][nt][lane];
#pragma unroll
      for (int w = 1; w < NW; ++w) t += red[w][nt][lane];
      part[(item * NT + nt) * 64 + lane] = t;
    }
    __syncthreads();  // red is read before the next item writes it
  }
}

// Tiled dense layer (fp16 path): an item is a block of
// kDenseTileRows survivors and a K part; its 4 waves take 32 survivors each
// (two 16-row tiles) and walk the part's K range together in chunks of
// kDenseChunk K steps, whose weight fragments the workgroup stages in LDS
// (one contiguous block of the fragment-ordered copy), so that each weight is
// read from memory once per 128 survivors.  The activation fragments of the
// next K step are loaded while the current one computes.  Each item writes
// one partial block per 16-row tile and NT; k_dense_finish adds the parts.
constexpr int kDenseTileRows = 128;
constexpr int kDenseTileItems = 512;  // K parts are chosen for about this many items

__device__ __forceinline__ int dense_tile_kparts(int64_t cnt, int nks) {
  const int64_t blocks = (cnt + kDenseTileRows - 1) / kDenseTileRows;
  const int nch = (nks + kDenseChunk - 1) / kDenseChunk;
  int64_t k = kDenseTileItems / (blocks > 0 ? blocks : 1);
  if (k > nch) k = nch;
  return k < 1 ? 1 : (int)k;
}

template <int NT, bool G>
__global__ void __launch_bounds__(256) k_dense_tiles(DenseArgs a, f32x4* __restrict__ part) {
  constexpr int MT = 2;
  __shared__ __align__(16) f16x8 wl[kDenseChunk][NT][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m = lane & 15, g = lane >> 4;
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int nks = (a.flat + 31) / 32;
  const int nch = (nks + kDenseChunk - 1) / kDenseChunk;
  const int kparts = dense_tile_kparts(cnt, nks);
  const int64_t blocks = (cnt + kDenseTileRows - 1) / kDenseTileRows;
  const int64_t items = blocks * kparts;
  auto cam_of = [&](int64_t u) -> int64_t { return a.idx[u] / a.per_cam; };
  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int64_t blk = item / kparts;
    const int kp = (int)(item - blk * kparts);
    const int c0 = (int)((int64_t)kp * nch / kparts), c1 = (int)((int64_t)(kp + 1) * nch / kparts);
    const int64_t tile0 = blk * (kDenseTileRows / 16) + wave * MT;  // this wave's 16-row tiles
    f32x4 acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[i][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    // In a camera group the block runs once per camera among its rows, each
    // pass with that camera's weights over its own rows (the other rows add
    // zero products, which leave their sums unchanged).
    int64_t cam = G ? cam_of(blk * kDenseTileRows) : 0;
    for (;;) {
      const int64_t off = G ? (int64_t)a.nets[cam].woff : 0;
      const float in_scale = at_off(a.scl, off)[0];
      const f16x8* wsrc = at_off(reinterpret_cast<const f16x8*>(a.w1), off);
      bool valid[MT];
      int64_t row[MT];
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const int64_t s = (tile0 + i) * 16 + m;
        valid[i] = s < cnt && (!G || cam_of(s) == cam);
        row[i] = (valid[i] ? s : 0) * (int64_t)a.flat + g * 8;
      }
      // the activation fragment of K step ks for tile i (zero past the end)
      auto ldx = [&](int ks, f16x8 (&x)[MT]) {
        const int k0 = ks * 32;
        const bool kin = k0 + g * 8 < a.flat;
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          x[i] = Elt<_Float16>::zero();
          if (valid[i] && kin)
            x[i] = a.feat_f16 ? *reinterpret_cast<const f16x8*>(
                                    reinterpret_cast<const _Float16*>(a.feat) + row[i] + k0)
                              : Elt<_Float16>::cvt8(a.feat + row[i] + k0, in_scale);
        }
      };
      f16x8 xc[MT], xn[MT];
      ldx(c0 * kDenseChunk, xc);
#pragma unroll
      for (int i = 0; i < MT; ++i) xn[i] = xc[i];
      for (int c = c0; c < c1; ++c) {
        __syncthreads();  // the previous chunk's fragments are read
        {
          const f16x8* src = wsrc + (size_t)c * kDenseChunk * NT * 64;
          f16x8* dst = &wl[0][0][0];
          for (int i = threadIdx.x; i < kDenseChunk * NT * 64; i += 256) dst[i] = src[i];
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kDenseChunk; ++j) {
          const int ks = c * kDenseChunk + j;
          if (ks + 1 < c1 * kDenseChunk) ldx(ks + 1, xn);
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const f16x8 w = wl[j][nt][lane];
#pragma unroll
            for (int i = 0; i < MT; ++i) acc[i][nt] = mma_f16(xc[i], w, acc[i][nt]);
          }
#pragma unroll
          for (int i = 0; i < MT; ++i) xc[i] = xn[i];
        }
      }
      if constexpr (!G) break;
      // the next camera among the block's rows (uniform)
      int64_t next = -1;
      for (int r = 0; r < kDenseTileRows && next < 0; ++r) {
        const int64_t u = blk * kDenseTileRows + r;
        if (u < cnt && cam_of(u) > cam) next = cam_of(u);
      }
      if (next < 0) break;
      cam = next;
    }
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        part[(((tile0 + i) * kparts + kp) * NT + nt) * 64 + lane] = acc[i][nt];
  }
}

// k_dense_finish: a workgroup per 16-survivor tile; its kDenseFinWaves waves
// add interleaved subsets of the tile's K parts (wave w: parts w, w + 4, ...),
// wave 0 adds the waves' sums in wave order and applies dense_out.
constexpr int kDenseFinWaves = 4;

template <typename T, int NT, bool G>
__global__ void __launch_bounds__(64 * kDenseFinWaves) k_dense_finish(DenseArgs a,
                                                                     const f32x4* __restrict__ part) {
  constexpr int KS = Elt<T>::KS;
  __shared__ f32x4 red[kDenseFinWaves][NT][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m = lane & 15, g = lane >> 4;
  int64_t cnt = *a.count;
  if (cnt > a.max_count) cnt = a.max_count;
  const int64_t tiles = (cnt + 15) / 16;
  const int kparts = a.tiled ? dense_tile_kparts(cnt, (a.flat + 31) / 32)
                             : dense_kparts(tiles, (a.flat + KS - 1) / KS);
  for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    f32x4 t[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) t[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int kp = wave; kp < kparts; kp += kDenseFinWaves) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) t[nt] += part[((tile * kparts + kp) * NT + nt) * 64 + lane];
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) red[wave][nt][lane] = t[nt];
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        t[nt] = red[0][nt][lane];
#pragma unroll
        for (int w = 1; w < kDenseFinWaves; ++w) t[nt] += red[w][nt][lane];
      }
      int64_t cam = G ? a.idx[tile * 16] / a.per_cam : 0;
      for (;;) {
        int64_t off = 0;
        float b2 = a.b2;
        double c_low = a.c_low, c_high = a.c_high;
        if constexpr (G) {
          const CamNet& cn = a.nets[cam];
          off = cn.woff;
          b2 = cn.b2;
          c_low = cn.c_low;
          c_high = cn.c_high;
        }
        if constexpr (Elt<T>::CVT) {
          // the camera's output scale (a row's partial sums hold only its own
          // camera's products, and this pass writes only that camera's rows)
          f32x4 u[NT];
          const float sc = at_off(a.scl, off)[1];
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) u[nt] = t[nt] * sc;
          dense_out<NT, G>(a, u, at_off(a.b1, off), at_off(a.w2, off), b2, c_low, c_high,
                           tile * 16, cnt, cam, m, g);
        } else {
          dense_out<NT, G>(a, t, at_off(a.b1, off), at_off(a.w2, off), b2, c_low, c_high,
                           tile * 16, cnt, cam, m, g);
        }
        if constexpr (!G) break;
        int64_t next = -1;
        for (int r = 0; r < 16 && next < 0; ++r) {
          const int64_t u = tile * 16 + r;
          if (u < cnt && a.idx[u] / a.per_cam > cam) next = a.idx[u] / a.per_cam;
        }
        if (next < 0) break;
        cam = next;
      }
    }  // wave 0
    __syncthreads();  // red is read before the next tile writes it
  }
}

template <typename T, bool FIRST>
int launch_conv_nt(int nt, const ConvArgs& a, unsigned grid, size_t lds, hipStream_t st) {
#define NSC_CONV_CASE(N)                                                                       \
  case N:                                                                                      \
    if (FIRST && a.nets)                                                                       \
      hipLaunchKernelGGL((k_conv_first<T, N, true>), dim3(grid), dim3(256), lds, st, a);       \
    else if (FIRST)                                                                            \
      hipLaunchKernelGGL((k_conv_first<T, N, false>), dim3(grid), dim3(256), lds, st, a);      \
    else if (a.nets)                                                                           \
      hipLaunchKernelGGL((k_conv<T, N, true>), dim3(grid), dim3(256), lds, st, a);             \
    else                                                                                       \
      hipLaunchKernelGGL((k_conv<T, N, false>), dim3(grid), dim3(256), lds, st, a);            \
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
int launch_dense_split_nt(int nt, const DenseArgs& a, f32x4* part, unsigned grid_part,
                          unsigned grid_fin, hipStream_t st) {
#define NSC_SPLIT_LAUNCH(N, G)                                                                  \
  hipLaunchKernelGGL((k_dense_part<T, N, G>), dim3(grid_part), dim3(64 * kDenseSplitWaves), 0, \
                     st, a, part);                                                              \
  hipLaunchKernelGGL((k_dense_finish<T, N, G>), dim3(grid_fin), dim3(64 * kDenseFinWaves), 0,  \
                     st, a, (const f32x4*)part)
#define NSC_SPLIT_CASE(N)                                                                       \
  case N:                                                                                       \
    if (a.nets) {                                                                               \
      NSC_SPLIT_LAUNCH(N, true);                                                                \
    } else {                                                                                    \
      NSC_SPLIT_LAUNCH(N, false);                                                               \
    }                                                                                           \
    break;
  switch (nt) {
    NSC_SPLIT_CASE(1)
    NSC_SPLIT_CASE(2)
    NSC_SPLIT_CASE(4)
    NSC_SPLIT_CASE(8)
    NSC_SPLIT_CASE(16)
    default:
      return fail(NSC_E_SHAPE, "dense layer of %d units is not supported", nt * 16);
  }
#undef NSC_SPLIT_CASE
#undef NSC_SPLIT_LAUNCH
  NSC_CHECK_LAUNCH("k_dense_part / k_dense_finish");
  return NSC_OK;
}

int launch_dense_tiles_nt(int nt, const DenseArgs& a, f32x4* part, unsigned grid,
                          unsigned grid_fin, hipStream_t st) {
#define NSC_TILES_LAUNCH(N, G)                                                                  \
  hipLaunchKernelGGL((k_dense_tiles<N, G>), dim3(grid), dim3(256), 0, st, a, part);            \
  hipLaunchKernelGGL((k_dense_finish<_Float16, N, G>), dim3(grid_fin),                         \
                     dim3(64 * kDenseFinWaves), 0, st, a, (const f32x4*)part)
#define NSC_TILES_CASE(N)                                                                       \
  case N:                                                                                       \
    if (a.nets) {                                                                               \
      NSC_TILES_LAUNCH(N, true);                                                                \
    } else {                                                                                    \
      NSC_TILES_LAUNCH(N, false);                                                               \
    }                                                                                           \
    break;
  switch (nt) {
    NSC_TILES_CASE(1)
    NSC_TILES_CASE(2)
    NSC_TILES_CASE(4)
    NSC_TILES_CASE(8)
    NSC_TILES_CASE(16)
    default:
      return fail(NSC_E_SHAPE, "dense layer of %d units is not supported", nt * 16);
  }
#undef NSC_TILES_CASE
#undef NSC_TILES_LAUNCH
  NSC_CHECK_LAUNCH("k_dense_tiles / k_dense_finish");
  return NSC_OK;
}

template <typename T>
int launch_dense_nt(int nt, const DenseArgs& a, unsigned grid, hipStream_t st) {
#define NSC_DENSE_LAUNCH(N, G)                                                                 \
  hipLaunchKernelGGL((k_dense<T, N, G>), dim3(grid), dim3(64 * kDenseWaves), 0, st, a)
#define NSC_DENSE_CASE(N)                                                                      \
  case N:                                                                                      \
    if (a.nets) NSC_DENSE_LAUNCH(N, true); else NSC_DENSE_LAUNCH(N, false);                    \
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
#undef NSC_DENSE_LAUNCH
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

// Smallest n' >= n with n' = 12 (mod 16).
int32_t pad_row_pixels(int32_t n) {
  int32_t p = (n + 3) / 16 * 16 + 12;
  return p - 16 >= n ? p - 16 : p;
}

// LDS of one conv layer's workgroup: staged weights plus an input band of
// band_tiles tile rows (4 output rows each + 2 halo rows) by seg_tiles tile
// columns (+ halo), in two planes (hi, lo) for the inner layers of a bf16
// network.  A band spans the full width unless that does not fit 128 KB (then
// the width is halved until it does); it is as tall as fits a budget of about
// 48 KB (the whole image when possible), at least one tile row, and at most
// max_bt tile rows when max_bt > 0.
size_t conv_lds_bytes(const CnnLayer& L, bool bf16, int32_t* cin_lds, int32_t* w_lds,
                      int32_t* band_w, int32_t* band_tiles, int32_t* seg_tiles, int32_t max_bt) {
  const size_t es = bf16 ? 2 : 4;
  const int32_t vec = (int32_t)(16 / es);
  const bool first = L.cin == 3;
  const int32_t cl = first ? 4 : L.cin + vec;          // inner layers: pad pixels by 16 bytes
  const int32_t wr = L.kpad + vec;                     // pad weight rows by 16 bytes
  int32_t ty, tx;
  conv_tiles(L, &ty, &tx);
  const size_t planes = bf16 && !first ? 2 : 1;
  const size_t wbytes = (size_t)L.cout * wr * es;
  // staged columns of st tile columns (the first layer also reads tap dx = 3,
  // weight 0), padded to 12 (mod 16) pixels: the 16 pixels of a 4x4 tile then
  // fall on distinct LDS banks (pixel strides of 8 bytes, or an odd number of
  // 16 bytes).  Without the padding when only that fits the LDS.
  int32_t st = tx, bw = 0, bt = 1;
  size_t row_bytes = 0;
  for (int pad = 1; pad >= 0; --pad) {
    auto cols = [&](int32_t n) {
      const int32_t c = 4 * n + (first ? 3 : 2);
      return pad ? pad_row_pixels(c) : c;
    };
    st = tx;
    while (st > 1 && wbytes + (size_t)6 * cols(st) * cl * es * planes > 128 * 1024)
      st = (st + 1) / 2;
    bw = cols(st);
    row_bytes = (size_t)bw * cl * es * planes;
    bt = 1;
    while (bt < ty && (max_bt <= 0 || bt < max_bt) &&
           wbytes + (size_t)(4 * (bt + 1) + 2) * row_bytes <= 48 * 1024)
      ++bt;
    if (wbytes + (size_t)(4 * bt + 2) * row_bytes <= 160 * 1024) break;
  }
  if (cin_lds) *cin_lds = cl;
  if (w_lds) *w_lds = wr;
  if (band_w) *band_w = bw;
  if (band_tiles) *band_tiles = bt;
  if (seg_tiles) *seg_tiles = st;
  return wbytes + (size_t)(4 * bt + 2) * row_bytes;
}

// Whether the first two layers run fused (k_conv_pair): a bf16 network whose
// first layer pools, with output channel counts the kernel is built for, and
// whose weights, first-layer input and second-layer hi / lo band fit the LDS
// of one CU.  Fills the whole-image geometry of both layers and the LDS
// offsets.
bool pair_plan(const Cnn& cnn, ConvArgs* a0, ConvArgs* a1, PairArgs* pa, size_t* lds_bytes) {
  const CnnLayer& L0 = cnn.layers[0];
  const CnnLayer& L1 = cnn.layers[1];
  auto nt_ok = [](int c) { return c == 16 || c == 32 || c == 64; };
  if (!cnn.bf16 || !L0.pool || !nt_ok(L0.cout) || !nt_ok(L1.cout)) return false;
  if (L0.cout == 64 && L1.cout == 64) return false;  // register pressure: run layered
  auto al8 = [](int64_t e) { return (e + 7) / 8 * 8; };  // 16-byte alignment of bf16 arrays
  a0->cin_lds = 4;
  a0->w_lds = L0.kpad + 8;
  a0->band_tiles = a0->tiles_y;
  a0->seg_tiles = a0->tiles_x;
  a0->band_w = 4 * a0->tiles_x + 3;
  a0->lo_plane = 0;
  a1->cin_lds = L1.cin + 8;
  a1->w_lds = L1.kpad + 8;
  a1->band_tiles = a1->tiles_y;
  a1->seg_tiles = a1->tiles_x;
  // row stride of the band padded to 12 (mod 16) pixels: with the 80-byte
  // pixel stride (odd in 16-byte units) the 16 pixels of a 4x4 tile then fall
  // on distinct 16-byte bank groups
  a1->band_w = pad_row_pixels(4 * a1->tiles_x + 2);
  const int64_t plane = al8((int64_t)(4 * a1->tiles_y + 2) * a1->band_w * a1->cin_lds);
  a1->lo_plane = (int32_t)plane;
  const int64_t w0 = al8((int64_t)L0.cout * a0->w_lds);
  const int64_t w1 = al8((int64_t)L1.cout * a1->w_lds);
  const int64_t in0 = al8((int64_t)(4 * a0->tiles_y + 2) * a0->band_w * 4);
  const int64_t total = w0 + w1 + in0 + 2 * plane;
  if (total * 2 > 160 * 1024) return false;
  pa->off_w1 = (int32_t)w0;
  pa->off_in0 = (int32_t)(w0 + w1);
  pa->off_in1 = (int32_t)(w0 + w1 + in0);
  *lds_bytes = (size_t)total * 2;
  return true;
}

namespace {
int launch_pair(int nt0, int nt1, const ConvArgs& a0, const ConvArgs& a1, const PairArgs& pa,
                unsigned grid, size_t lds, hipStream_t st) {
  // second-layer weights in registers when they are 9 taps x 32 channels x <= 32 outputs
  const bool breg = a1.cin == 32 && nt1 <= 2;
#define NSC_PAIR_LAUNCH(A, B, R, G)                                                            \
  hipLaunchKernelGGL((k_conv_pair<A, B, R, G>), dim3(grid), dim3(1024), lds, st, a0, a1, pa)
#define NSC_PAIR_CASE(A, B)                                                                    \
  if (nt0 == A && nt1 == B) {                                                                  \
    constexpr bool R = A <= 2 && B <= 2;                                                       \
    if (breg && R) {                                                                           \
      if (a0.nets) NSC_PAIR_LAUNCH(A, B, R, true); else NSC_PAIR_LAUNCH(A, B, R, false);       \
    } else {                                                                                   \
      if (a0.nets) NSC_PAIR_LAUNCH(A, B, false, true); else NSC_PAIR_LAUNCH(A, B, false, false); \
    }                                                                                          \
    NSC_CHECK_LAUNCH("k_conv_pair");                                                           \
    return NSC_OK;                                                                             \
  }
  NSC_PAIR_CASE(1, 1)
  NSC_PAIR_CASE(1, 2)
  NSC_PAIR_CASE(1, 4)
  NSC_PAIR_CASE(2, 1)
  NSC_PAIR_CASE(2, 2)
  NSC_PAIR_CASE(2, 4)
  NSC_PAIR_CASE(4, 1)
  NSC_PAIR_CASE(4, 2)
#undef NSC_PAIR_CASE
#undef NSC_PAIR_LAUNCH
  return fail(NSC_E_SHAPE, "fused conv pair with %d and %d output channels", nt0 * 16, nt1 * 16);
}
}  // namespace

// Band plan of a 64-input-channel bf16 layer (k_band64 / k_pair64): among
// the band heights of at most 16 tiles or two tile rows whose planes (one
// fp16 plane with h16, else the bf16 hi and lo planes) fit 80 KB, so that two
// workgroups share a CU, the one with
// the least work per image for the busiest wave: per band the most tiles any
// of the 4 waves computes, plus half a tile for the band's staging and
// barriers; else one band row in up to 160 KB.  False when the layer does not
// qualify or no band fits.
bool band64_plan(const CnnLayer& L, bool h16, Band64* b, int32_t* band_tiles, size_t* lds) {
  if (L.cin != 64 || (L.cout != 64 && L.cout != 32)) return false;
  int32_t ty, tx;
  conv_tiles(L, &ty, &tx);
  int32_t wb = L.w + 2;
  wb += ((4 - wb) % 8 + 8) % 8;  // = 4 (mod 8)
  auto plan = [&](int32_t bt) {
    Band64 p{};
    p.w = L.w;
    p.h = L.h;
    p.rows = 4 * bt + 2;
    p.wb = wb;
    p.cp = p.rows * wb + 1;
    p.lo_bytes = 8 * p.cp * 16;
    p.planes = h16 ? 1 : 2;
    return p;
  };
  int32_t bt = 1;
  int64_t best = INT64_MAX;
  // at most one round of tiles (4 per wave with hi / lo planes, 7 on the
  // fp16 path) or two tile rows per band: taller bands with two rounds
  // measured slower (4 tile rows of a 25 x 25 map with 4 tiles per wave and
  // round: 523 against 459 us per 8,192 images).  Every band costs about as
  // much as the one with the most tiles per wave (a wave streams the layer's
  // weights once per band whatever its tile count), so the plan minimises
  // bands x the largest band's tiles per wave, and takes the taller band on
  // a tie (less halo staging).  Measured per 8,192 images, fp16 path: 25 x 25
  // map, 7 x 7 tiles: 4 tile rows 587 us, 3 rows 590, 2 rows 683; pooled
  // 25 x 25 map, 6 x 6 tiles: 4 rows (6 and 3 tiles per wave) 447 us, 3 rows
  // 407, 2 rows 403.
  const int32_t per_round = (h16 ? kBandMaxTilesH : 4) * kBandWaves;
  const int32_t hn = L.pool ? (L.h / 2) * 2 : L.h, wn = L.pool ? (L.w / 2) * 2 : L.w;
  for (int32_t c = 1; c <= ty; ++c) {
    if (c > 2 && band64_ntile(L.pool, std::min(4 * c, hn), wn) > per_round) break;
    if (band64_bytes(plan(c)) > 80 * 1024) break;
    const int64_t bands = (ty + c - 1) / c;
    int64_t per_wave = 0;  // the fullest band's tiles per wave
    for (int32_t y0 = 0; y0 < ty; y0 += c) {
      const int64_t t = band64_ntile(L.pool, std::min(4 * c, hn - 4 * y0), wn);
      per_wave = std::max(per_wave, (t + kBandWaves - 1) / kBandWaves);
    }
    if (bands * per_wave <= best) {
      best = bands * per_wave;
      bt = c;
    }
  }
  if (band64_bytes(plan(bt)) > 160 * 1024) return false;
  *b = plan(bt);
  *band_tiles = bt;
  *lds = band64_bytes(*b);
  return true;
}

// The fused k_pair64 plan of a network (first layer 3 -> 64 without pooling,
// second with 64 input channels), with the size of the pre-processed input
// per image (xr rows x xw pixels of 8 bytes).
bool pair64_plan(const Cnn& cnn, Band64* b, int32_t* band_tiles, size_t* lds, int32_t* xr,
                 int32_t* xw) {
  if (!cnn.bf16 || cnn.n_layers < 2 || cnn.layers[0].cout != 64 || cnn.layers[0].pool) return false;
  if (!band64_plan(cnn.layers[1], cnn.h16, b, band_tiles, lds)) return false;
  int32_t ty, tx;
  conv_tiles(cnn.layers[1], &ty, &tx);
  *xr = 4 * ty + 4;
  *xw = 8 * ((cnn.layers[1].w + 7) / 8) + 3;
  return true;
}

namespace {
int launch_band64(bool pair, int nt, const ConvArgs& a0, const ConvArgs& a1, const Band64& b,
                  const uint2* xin, int32_t xr, int32_t xw, size_t lds, int64_t max_count,
                  hipStream_t st) {
  const int64_t bands = (a1.tiles_y + a1.band_tiles - 1) / a1.band_tiles;
  const int64_t items = (max_count + 7) / 8 * 8 * bands;
  const int64_t per_cu = lds <= 80 * 1024 ? 2 : 1;
  int64_t grid = kNumCU * per_cu;  // a multiple of 8 (see band_item)
  if (grid > items) grid = items;
  if (grid < 1) grid = 1;
#define NSC_BAND_LAUNCH2(N, G, H)                                                               \
  if (pair)                                                                                     \
    hipLaunchKernelGGL((k_pair64<N, G, H>), dim3((unsigned)grid), dim3(64 * kBandWaves), lds,   \
                       st, a0, a1, b, xin, xr, xw);                                             \
  else                                                                                          \
    hipLaunchKernelGGL((k_band64<N, G, H>), dim3((unsigned)grid), dim3(64 * kBandWaves), lds,   \
                       st, a1, b)
#define NSC_BAND_LAUNCH(N, G)                                                                   \
  if (b.planes == 1) {                                                                          \
    NSC_BAND_LAUNCH2(N, G, true);                                                               \
  } else {                                                                                      \
    NSC_BAND_LAUNCH2(N, G, false);                                                              \
  }
#define NSC_BAND_CASE(N)                                                                        \
  case N:                                                                                       \
    if (a1.nets) {                                                                              \
      NSC_BAND_LAUNCH(N, true);                                                                 \
    } else {                                                                                    \
      NSC_BAND_LAUNCH(N, false);                                                                \
    }                                                                                           \
    break;
  switch (nt) {
    NSC_BAND_CASE(2)
    NSC_BAND_CASE(4)
    default:
      return fail(NSC_E_SHAPE, "banded layer with %d output channels", nt * 16);
  }
#undef NSC_BAND_CASE
#undef NSC_BAND_LAUNCH
#undef NSC_BAND_LAUNCH2
  NSC_CHECK_LAUNCH(pair ? "k_pair64" : "k_band64");
  return NSC_OK;
}
}  // namespace

// Two ping-pong buffers of fp32 activations per image, then (fused 64-channel
// first pair) the pre-processed bf16 input of every image.
size_t cnn_xin_bytes(const Cnn& cnn, int64_t max_count) {
  Band64 b{};
  int32_t bt = 0, xr = 0, xw = 0;
  size_t lds = 0;
  if (!pair64_plan(cnn, &b, &bt, &lds, &xr, &xw)) return 0;
  return align_up((size_t)xr * xw * 8 * (size_t)(max_count > 0 ? max_count : 0), 256);
}

// The dense layer's partial blocks when it splits K over workgroups: one
// NT x 1 KB block per (16-row tile, K part), for k_dense_tiles (fp16 path:
// its 128-row blocks times their K parts, at most the
// larger of kDenseTileItems x 8 and the tiles of max_count) or k_dense_part
// (fewer than kDenseBig survivors otherwise); room for both.
size_t cnn_dense_part_bytes(const Cnn& cnn, int64_t max_count) {
  if (max_count <= 0) return 0;
  const size_t blk = (size_t)(cnn.dense / 16) * 64 * sizeof(f32x4);
  size_t n = max_count < kDenseBig ? (size_t)kDenseSplitItems * blk : 0;
  if (cnn.h16 && cnn.w1f) {
    const int64_t t8 = (max_count + kDenseTileRows - 1) / kDenseTileRows * 8;
    const int64_t blocks = t8 > (int64_t)kDenseTileItems * 8 ? t8 : (int64_t)kDenseTileItems * 8;
    if ((size_t)blocks * blk > n) n = (size_t)blocks * blk;
  }
  return n;
}

size_t cnn_workspace_bytes(const Cnn& cnn, int64_t max_count) {
  const size_t per = align_up(cnn.act_elems * sizeof(float), 256);
  return 2 * per * (size_t)(max_count > 0 ? max_count : 0) + 256 + cnn_xin_bytes(cnn, max_count) +
         cnn_dense_part_bytes(cnn, max_count);
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
  auto layer_args = [&](int l) {
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
    a.scl = cnn.scales + 2 * l;
    a.nets = r.nets;
    a.per_cam = r.per_cam;
    return a;
  };
  // weights in fragment order for the banded kernels (bf16; scaled fp16 for
  // the layers on the fp16 path)
  auto frag_weights = [&](int l, bool h16) {
    return static_cast<const void*>(static_cast<const unsigned char*>(h16 ? cnn.conv_wh : cnn.conv_wf) +
                                    cnn.layers[l].w_off * 2);
  };
  // Which layers run on the fp16 band path (k_pair64's second layer,
  // k_band64), and where activations between two such layers (or into the
  // fp16 dense layer) are stored as fp16: the producer writes them scaled for
  // the consumer, which stages them as they are.
  bool band[NSC_MAX_CONV] = {};
  bool out16[NSC_MAX_CONV] = {};
  {
    Band64 pb{};
    int32_t pbt = 0, pxr = 0, pxw = 0;
    size_t plds = 0;
    const bool p64 = pair64_plan(cnn, &pb, &pbt, &plds, &pxr, &pxw);
    bool pair = false;
    if (!p64 && cnn.n_layers >= 2) {
      ConvArgs t0 = layer_args(0), t1 = layer_args(1);
      PairArgs tp{};
      size_t tl = 0;
      pair = pair_plan(cnn, &t0, &t1, &tp, &tl);
    }
    for (int l = 1; l < cnn.n_layers; ++l) {
      Band64 b{};
      int32_t bt = 0;
      size_t lds = 0;
      if (l == 1 && (p64 || pair))
        band[l] = p64 && cnn.h16;
      else
        band[l] = cnn.h16 && band64_plan(cnn.layers[l], true, &b, &bt, &lds);
    }
    for (int l = 0; l < cnn.n_layers; ++l)
      out16[l] = band[l] && (l + 1 < cnn.n_layers ? band[l + 1] : cnn.h16);
    // a first layer run alone (k_conv_first) writes fp16 for a banded fp16
    // second layer
    if (!p64 && !pair && cnn.n_layers > 1) out16[0] = band[1];
  }
  auto set_formats = [&](ConvArgs& a, int l) {
    a.in_f16 = l > 0 && out16[l - 1];
    a.out_f16 = out16[l];
  };
  int first_layered = 0;
  {
    Band64 b{};
    int32_t bt = 0, xr = 0, xw = 0;
    size_t lds = 0;
    if (pair64_plan(cnn, &b, &bt, &lds, &xr, &xw)) {
      ConvArgs a0 = layer_args(0), a1 = layer_args(1);
      set_formats(a1, 1);
      a0.wts = cnn.h16 && cnn.conv_w0h ? cnn.conv_w0h : frag_weights(0, false);
      a1.wts = frag_weights(1, cnn.h16);
      a1.band_tiles = bt;
      uint2* xin = reinterpret_cast<uint2*>(static_cast<unsigned char*>(ws) +
                                            2 * per * (size_t)r.max_count + 256);
      int64_t pgrid = (r.max_count * xr * xw + 255) / 256;
      if (pgrid > kNumCU * 8) pgrid = kNumCU * 8;
      if (pgrid < 1) pgrid = 1;
      hipLaunchKernelGGL(k_prep_input, dim3((unsigned)pgrid), dim3(256), 0, stream, a0, xin, xr,
                         xw);
      NSC_CHECK_LAUNCH("k_prep_input");
      const int rc = launch_band64(true, cnn.layers[1].cout / 16, a0, a1, b, xin, xr, xw, lds,
                                   r.max_count, stream);
      if (rc) return rc;
      first_layered = 2;
    }
  }
  if (first_layered == 0) {
    ConvArgs a0 = layer_args(0);
    ConvArgs a1{};
    PairArgs pa{};
    size_t lds = 0;
    if (cnn.n_layers >= 2) a1 = layer_args(1);
    if (cnn.n_layers >= 2 && pair_plan(cnn, &a0, &a1, &pa, &lds)) {
      int64_t grid = r.max_count < kNumCU ? r.max_count : kNumCU;
      const int rc = launch_pair(cnn.layers[0].cout / 16, cnn.layers[1].cout / 16, a0, a1, pa,
                                 (unsigned)grid, lds, stream);
      if (rc) return rc;
      first_layered = 2;
    }
  }
  for (int l = first_layered; l < cnn.n_layers; ++l) {
    const CnnLayer& L = cnn.layers[l];
    ConvArgs a = layer_args(l);
    set_formats(a, l);
    if (cnn.bf16 && l > 0) {
      Band64 b{};
      int32_t bt = 0;
      size_t lds = 0;
      if (band64_plan(L, cnn.h16, &b, &bt, &lds)) {
        a.wts = frag_weights(l, cnn.h16);
        a.band_tiles = bt;
        const int rc =
            launch_band64(false, L.cout / 16, a, a, b, nullptr, 0, 0, lds, r.max_count, stream);
        if (rc) return rc;
        continue;
      }
    }
    // few images (a small call): bands short enough for about 32 work items
    // per CU, since a workgroup works through its band's tiles one after
    // another (1,000 frames of 100x100, 204 survivors: 0.224 -> 0.203 ms per
    // call with one tile row per band)
    int32_t ty = 0, tx = 0;
    conv_tiles(L, &ty, &tx);
    const int64_t want = 32 * (int64_t)kNumCU;
    const int64_t min_bands = r.max_count > 0 ? (want + r.max_count - 1) / r.max_count : 1;
    const int32_t max_bt = min_bands <= 1 ? 0 : (int32_t)std::max<int64_t>(1, ty / min_bands);
    const size_t lds = conv_lds_bytes(L, cnn.bf16, &a.cin_lds, &a.w_lds, &a.band_w, &a.band_tiles,
                                      &a.seg_tiles, max_bt);
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
  d.w1 = cnn.h16 ? cnn.w1h : cnn.w1;
  d.scl = cnn.scales + 2 * cnn.n_layers;
  d.feat_f16 = out16[cnn.n_layers - 1];
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
  d.nets = r.nets;
  d.per_cam = r.per_cam;
  const int nt = cnn.dense / 16;
  f32x4* part = reinterpret_cast<f32x4*>(static_cast<unsigned char*>(ws) +
                                         2 * per * (size_t)r.max_count + 256 +
                                         cnn_xin_bytes(cnn, r.max_count));
  // the tiled kernel for one network (also a one-camera group, which then
  // gives nsc_cascade_run's results bit for bit); a group of several cameras
  // runs a block's 128 rows once per camera among them, slower than the
  // 16-row tiles below (0.19 against 0.09 ms for 100 cameras' 500 survivors)
  if (cnn.h16 && cnn.w1f && (!r.nets || r.n_nets == 1)) {
    d.w1 = cnn.w1f;
    d.tiled = 1;
    const int64_t grid = kDenseTileItems;  // the kernel loops over its items
    int64_t grid_fin = (r.max_count + 15) / 16;
    if (grid_fin > kNumCU * 4) grid_fin = kNumCU * 4;
    if (grid_fin < 1) grid_fin = 1;
    return launch_dense_tiles_nt(nt, d, part, (unsigned)grid, (unsigned)grid_fin, stream);
  }
  if (r.max_count < kDenseBig) {
    // items: up to kDenseSplitItems; finishing: a wave per 16-survivor tile
    const int64_t tiles = (r.max_count + 15) / 16;
    int64_t grid_part = kDenseSplitItems;
    if (grid_part > kNumCU * 4) grid_part = kNumCU * 4;
    int64_t grid_fin = tiles;  // a workgroup per tile
    if (grid_fin > kNumCU * 4) grid_fin = kNumCU * 4;
    if (grid_fin < 1) grid_fin = 1;
    if (cnn.h16)
      return launch_dense_split_nt<_Float16>(nt, d, part, (unsigned)grid_part, (unsigned)grid_fin,
                                             stream);
    return cnn.bf16 ? launch_dense_split_nt<uint16_t>(nt, d, part, (unsigned)grid_part,
                                                      (unsigned)grid_fin, stream)
                    : launch_dense_split_nt<float>(nt, d, part, (unsigned)grid_part,
                                                   (unsigned)grid_fin, stream);
  }
  const int64_t rows = nt >= 16 ? 16 : (nt >= 8 ? 32 : 64);  // 16 x dense_mt
  int64_t groups = (r.max_count + rows - 1) / rows;  // one workgroup per group of rows
  int64_t grid = groups;
  if (grid > kNumCU * 2) grid = kNumCU * 2;
  if (grid < 1) grid = 1;
  if (cnn.h16) return launch_dense_nt<_Float16>(nt, d, (unsigned)grid, stream);
  return cnn.bf16 ? launch_dense_nt<uint16_t>(nt, d, (unsigned)grid, stream)
                  : launch_dense_nt<float>(nt, d, (unsigned)grid, stream);
}

}  // namespace nsc
