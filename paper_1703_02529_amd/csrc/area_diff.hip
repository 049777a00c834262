// Area downsample and difference detector kernels (gfx950).
//
// Area sums (exact area average kept as integers, value = S / den): one
// workgroup walks one frame's band of output rows.  Each lane owns a fixed
// 16/4/1-byte column chunk of the raw RGB row and reads it from HBM exactly
// once per source row with coalesced loads; it first accumulates vertically
// (weights uniform across the workgroup), two bytes per 32-bit register when
// the sums fit in 16 bits, then the workgroup reduces horizontally through a
// double-buffered LDS row, one output cell per thread.
//
// Detector (Sec. 5): one wavefront per frame reduces the squared differences
// of its area sums against the reference with 64-bit shuffle reductions; the
// blocked variant reduces per grid block and applies the logistic-regression
// weights in fp64 in block order.
#include "nsc_internal.h"

#include <math.h>

namespace nsc {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Vertical pass over the source rows of output row Y for one lane's chunk.
// Returns the per-byte weighted column sums in out[CB].
template <int CB, bool PACKED>
__device__ __forceinline__ void vertical_sums(const uint8_t* __restrict__ col, int64_t row_bytes,
                                              int64_t a0, int64_t a1, int32_t q, int j0, int j1,
                                              int32_t out[CB]) {
  if constexpr (CB == 1) {
    int32_t acc = 0;
    for (int j = j0; j < j1; ++j) {
      int64_t r0 = (int64_t)j * q;
      int32_t w = (int32_t)(min(a1, r0 + q) - max(a0, r0));
      acc += w * (int32_t)col[(int64_t)j * row_bytes];
    }
    out[0] = acc;
  } else {
    constexpr int ND = CB / 4;
    uint32_t lo[ND], hi[ND];
#pragma unroll
    for (int d = 0; d < ND; ++d) lo[d] = hi[d] = 0;
    for (int j = j0; j < j1; j += 4) {
      uint32_t v[4][ND];
      uint32_t w[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int jj = j + k;
        w[k] = 0;
#pragma unroll
        for (int d = 0; d < ND; ++d) v[k][d] = 0;
        if (jj < j1) {
          const int64_t r0 = (int64_t)jj * q;
          w[k] = (uint32_t)(min(a1, r0 + q) - max(a0, r0));
          const uint8_t* p = col + (int64_t)jj * row_bytes;
          if constexpr (CB == 16) {
            const u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
            v[k][0] = x[0];
            v[k][1] = x[1];
            v[k][2] = x[2];
            v[k][3] = x[3];
          } else {
            v[k][0] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p));
          }
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
#pragma unroll
        for (int d = 0; d < ND; ++d) {
          if constexpr (PACKED) {
            lo[d] += w[k] * (v[k][d] & 0x00FF00FFu);
            hi[d] += w[k] * ((v[k][d] >> 8) & 0x00FF00FFu);
          } else {
            // unpacked: lo/hi hold bytes 0,1 and bytes 2,3 would overflow; use 4 sums
            // (stored in out directly below)
            out[4 * d + 0] += (int32_t)(w[k] * (v[k][d] & 0xFFu));
            out[4 * d + 1] += (int32_t)(w[k] * ((v[k][d] >> 8) & 0xFFu));
            out[4 * d + 2] += (int32_t)(w[k] * ((v[k][d] >> 16) & 0xFFu));
            out[4 * d + 3] += (int32_t)(w[k] * (v[k][d] >> 24));
          }
        }
      }
    }
    if constexpr (PACKED) {
#pragma unroll
      for (int d = 0; d < ND; ++d) {
        out[4 * d + 0] = (int32_t)(lo[d] & 0xFFFFu);
        out[4 * d + 1] = (int32_t)(hi[d] & 0xFFFFu);
        out[4 * d + 2] = (int32_t)(lo[d] >> 16);
        out[4 * d + 3] = (int32_t)(hi[d] >> 16);
      }
    }
  }
}

template <int CB, bool PACKED>
__global__ void __launch_bounds__(1024) k_area_sums(const uint8_t* __restrict__ frames,
                                                    int64_t stride, Axis ay, Axis ax,
                                                    int32_t lanes, int32_t bands,
                                                    int32_t* __restrict__ sums) {
  extern __shared__ int32_t rowbuf[];  // 2 x (in_w * 3) int32, double buffered
  const int64_t f = blockIdx.x / bands;
  const int band = blockIdx.x - (int)(f * bands);
  const int Ho = ay.n_out, Wo = ax.n_out;
  const int Y0 = (int)((int64_t)band * Ho / bands);
  const int Y1 = (int)((int64_t)(band + 1) * Ho / bands);
  const int64_t row_bytes = (int64_t)ax.n_in * 3;
  const int tid = threadIdx.x;
  const uint8_t* col = frames + f * stride + (int64_t)tid * CB;
  int32_t* out = sums + f * (int64_t)Ho * Wo * 3;
  for (int Y = Y0; Y < Y1; ++Y) {
    const int64_t a0 = (int64_t)Y * ay.p, a1 = a0 + ay.p;
    const int j0 = (int)(a0 / ay.q), j1 = (int)((a1 + ay.q - 1) / ay.q);
    int32_t* buf = rowbuf + (Y & 1) * row_bytes;
    if (tid < lanes) {
      int32_t v[CB];
#pragma unroll
      for (int b = 0; b < CB; ++b) v[b] = 0;
      vertical_sums<CB, PACKED>(col, row_bytes, a0, a1, ay.q, j0, j1, v);
      if constexpr (CB == 16) {
        int4* dst = reinterpret_cast<int4*>(buf + tid * 16);
        dst[0] = make_int4(v[0], v[1], v[2], v[3]);
        dst[1] = make_int4(v[4], v[5], v[6], v[7]);
        dst[2] = make_int4(v[8], v[9], v[10], v[11]);
        dst[3] = make_int4(v[12], v[13], v[14], v[15]);
      } else {
#pragma unroll
        for (int b = 0; b < CB; ++b) buf[tid * CB + b] = v[b];
      }
    }
    __syncthreads();
    // Horizontal pass: thread t owns output cell (X, c) = (t / 3, t % 3).
    for (int t = tid; t < Wo * 3; t += blockDim.x) {
      const int X = t / 3, c = t - 3 * (t / 3);
      const int64_t b0 = (int64_t)X * ax.p, b1 = b0 + ax.p;
      const int i0 = (int)(b0 / ax.q), i1 = (int)((b1 + ax.q - 1) / ax.q);
      int32_t s = 0;
      for (int i = i0; i < i1; ++i) {
        const int64_t c0 = (int64_t)i * ax.q;
        const int32_t w = (int32_t)(min(b1, c0 + ax.q) - max(b0, c0));
        s += w * buf[3 * i + c];
      }
      out[((int64_t)Y * Wo + X) * 3 + c] = s;
    }
    // The next row writes the other buffer; its readers (row Y-1) all passed
    // this row's barrier, so no second barrier is needed.
  }
}

// ------------------------------------------------------------- detector

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ void __launch_bounds__(256) k_diff(DiffArgs a) {
  // the blocked score is summed with separate multiplies and adds, in block
  // order, so it is reproducible bit for bit
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= a.n) return;
  const int64_t t = a.t0 + i;
  const int64_t cells = (int64_t)a.dd_h * a.dd_w * 3;
  const bool forced = a.ref_mode == NSC_REF_PREV && t < a.delta;
  double score = INFINITY;
  if (!forced) {
    const int32_t* cur = a.sums + i * cells;
    const int32_t* ref;
    if (a.ref_mode == NSC_REF_FIXED)
      ref = a.ref_sums;
    else if (i >= a.delta)
      ref = a.sums + (i - a.delta) * cells;
    else
      ref = a.prev_sums + i * cells;  // frame t - delta = t0 - delta + i
    if (a.grid_h * a.grid_w == 1) {
      int64_t e = 0;
      if ((cells & 3) == 0 && (((uintptr_t)cur | (uintptr_t)ref) & 15) == 0) {
        const int4* c4 = reinterpret_cast<const int4*>(cur);
        const int4* r4 = reinterpret_cast<const int4*>(ref);
        for (int64_t k = lane; k < cells / 4; k += 64) {
          const int4 x = c4[k], y = r4[k];
          const int64_t d0 = x.x - y.x, d1 = x.y - y.y, d2 = x.z - y.z, d3 = x.w - y.w;
          e += d0 * d0 + d1 * d1 + d2 * d2 + d3 * d3;
        }
      } else {
        for (int64_t k = lane; k < cells; k += 64) {
          const int64_t d = cur[k] - ref[k];
          e += d * d;
        }
      }
      e = wave_sum_i64(e);
      score = (double)e / (a.den2 * (double)cells);
    } else {
      double z = a.lr_b;
      for (int by = 0; by < a.grid_h; ++by) {
        const int y0 = (int)((int64_t)by * a.dd_h / a.grid_h);
        const int y1 = (int)((int64_t)(by + 1) * a.dd_h / a.grid_h);
        for (int bx = 0; bx < a.grid_w; ++bx) {
          const int x0 = (int)((int64_t)bx * a.dd_w / a.grid_w);
          const int x1 = (int)((int64_t)(bx + 1) * a.dd_w / a.grid_w);
          const int rl = (x1 - x0) * 3;
          const int total = (y1 - y0) * rl;
          int64_t e = 0;
          for (int k = lane; k < total; k += 64) {
            const int r = k / rl, cc = k - r * rl;
            const int64_t off = ((int64_t)(y0 + r) * a.dd_w + x0) * 3 + cc;
            const int64_t d = cur[off] - ref[off];
            e += d * d;
          }
          e = wave_sum_i64(e);
          const double ncell = ((double)(y1 - y0) * (double)(x1 - x0)) * 3.0;
          const double m = (double)e / (a.den2 * ncell);
          z = z + (double)a.lr_w[by * a.grid_w + bx] * m;
        }
      }
      score = z;
    }
  }
  if (lane == 0) {
    a.fire[i] = (forced || score > a.delta_diff) ? 1 : 0;
    if (a.score) a.score[i] = score;
  }
}

}  // namespace

int make_area_plan(int32_t in_h, int32_t in_w, int64_t stride, const void* frames, int32_t out_h,
                   int32_t out_w, int64_t n, AreaPlan* plan) {
  AreaPlan p{};
  p.ay = Axis::make(in_h, out_h);
  p.ax = Axis::make(in_w, out_w);
  const int64_t row_bytes = (int64_t)in_w * 3;
  const uintptr_t addr = (uintptr_t)frames;
  if (row_bytes % 16 == 0 && stride % 16 == 0 && addr % 16 == 0)
    p.chunk_bytes = 16;
  else if (row_bytes % 4 == 0 && stride % 4 == 0 && addr % 4 == 0)
    p.chunk_bytes = 4;
  else
    p.chunk_bytes = 1;
  p.lanes = (int32_t)(row_bytes / p.chunk_bytes);
  if (p.lanes > 1024)
    return fail(NSC_E_SHAPE, "frame rows of %lld bytes need %d lanes (> 1024) at %d-byte chunks",
                (long long)row_bytes, p.lanes, p.chunk_bytes);
  p.threads = (p.lanes + 63) / 64 * 64;
  if (p.threads < 64) p.threads = 64;
  // vertical column sums reach 255 * p_y; 16-bit packing is exact below 65536
  p.packed = 255LL * p.ay.p < 65536;
  int64_t bands = (4096 + n - 1) / (n > 0 ? n : 1);
  if (bands < 1) bands = 1;
  if (bands > out_h) bands = out_h;
  p.bands = (int32_t)bands;
  *plan = p;
  return NSC_OK;
}

int launch_area_sums(const AreaPlan& p, const uint8_t* frames, int64_t stride, int64_t n,
                     int32_t* sums, hipStream_t stream) {
  if (n <= 0) return NSC_OK;
  const int64_t blocks = n * p.bands;
  if (blocks > 0x7FFFFFFF) return fail(NSC_E_SHAPE, "too many frames in one call");
  const size_t lds = 2 * (size_t)p.ax.n_in * 3 * sizeof(int32_t);
  dim3 grid((unsigned)blocks), block(p.threads);
#define NSC_AREA_LAUNCH(CB, PK)                                                          \
  hipLaunchKernelGGL((k_area_sums<CB, PK>), grid, block, lds, stream, frames, stride, p.ay, \
                     p.ax, p.lanes, p.bands, sums)
  if (p.chunk_bytes == 16) {
    if (p.packed) NSC_AREA_LAUNCH(16, true); else NSC_AREA_LAUNCH(16, false);
  } else if (p.chunk_bytes == 4) {
    if (p.packed) NSC_AREA_LAUNCH(4, true); else NSC_AREA_LAUNCH(4, false);
  } else {
    NSC_AREA_LAUNCH(1, false);
  }
#undef NSC_AREA_LAUNCH
  NSC_CHECK_LAUNCH("k_area_sums");
  return NSC_OK;
}

int launch_diff(const DiffArgs& a, hipStream_t stream) {
  if (a.n <= 0) return NSC_OK;
  const int64_t blocks = (a.n + 3) / 4;
  hipLaunchKernelGGL(k_diff, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  NSC_CHECK_LAUNCH("k_diff");
  return NSC_OK;
}

}  // namespace nsc
