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
// Detector (Sec. 5): one wavefront per frame reduces the squared (or
// absolute) differences of its area sums against the reference with 64-bit
// shuffle reductions and turns them into the metric (MSE, or SAD, NRMSE,
// -PSNR); the blocked variant reduces per grid block and applies the
// logistic-regression weights in fp64 in block order.
#include "nsc_internal.h"

#include <math.h>

#include <type_traits>

namespace nsc {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#ifndef NSC_ROWS_BATCH
#define NSC_ROWS_BATCH 12
#endif

// One lane's 4 bytes split into two words of two 16-bit fields:
// e0 = (b0, b2), e1 = (b1, b3).
__device__ __forceinline__ uint32_t bytes02(uint32_t x) { return x & 0x00FF00FFu; }
__device__ __forceinline__ uint32_t bytes13(uint32_t x) {
  return __builtin_amdgcn_perm(0u, x, 0x0C030C01u);  // (x.b1, 0, x.b3, 0)
}

// A lane's CB bytes of one row; a 32-byte chunk is two 16-byte halves `split`
// bytes apart (the halves of all lanes of a strip are two contiguous runs, so
// that each load instruction of the wave reads consecutive bytes).
template <int CB>
__device__ __forceinline__ void load_chunk(const uint8_t* p, uint32_t (&v)[CB >= 4 ? CB / 4 : 1],
                                           int split = 16) {
  if constexpr (CB == 32) {
    const u32x4 x = *reinterpret_cast<const u32x4*>(p);
    const u32x4 y = *reinterpret_cast<const u32x4*>(p + split);
    v[0] = x[0];
    v[1] = x[1];
    v[2] = x[2];
    v[3] = x[3];
    v[4] = y[0];
    v[5] = y[1];
    v[6] = y[2];
    v[7] = y[3];
  } else if constexpr (CB == 16) {
    const u32x4 x = *reinterpret_cast<const u32x4*>(p);
    v[0] = x[0];
    v[1] = x[1];
    v[2] = x[2];
    v[3] = x[3];
  } else if constexpr (CB == 4) {
    v[0] = *reinterpret_cast<const uint32_t*>(p);
  } else {
    v[0] = *p;
  }
}

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// The sums one metric needs over a set of values: squared differences e,
// absolute differences s, squared reference values r.  All exact in int64.
template <int M>
struct DiffSums {
  int64_t e = 0, s = 0, r = 0;
  __device__ __forceinline__ void add(int32_t x, int32_t y) {
    const int64_t d = (int64_t)x - y;
    if constexpr (M != NSC_METRIC_SAD) e += d * d;
    if constexpr (M == NSC_METRIC_SAD) s += d < 0 ? -d : d;
    if constexpr (M == NSC_METRIC_NRMSE) r += (int64_t)y * y;
  }
  __device__ __forceinline__ void reduce() {
    if constexpr (M != NSC_METRIC_SAD) e = wave_sum_i64(e);
    if constexpr (M == NSC_METRIC_SAD) s = wave_sum_i64(s);
    if constexpr (M == NSC_METRIC_NRMSE) r = wave_sum_i64(r);
  }
  // The metric over `count` values (Sec. 5 and the alternatives it names):
  // each is one fp64 expression of the exact sums, in a fixed operation order.
  __device__ __forceinline__ double value(const DiffArgs& a, double count) const {
    if constexpr (M == NSC_METRIC_MSE) {
      return (double)e / (a.den2 * count);
    } else if constexpr (M == NSC_METRIC_SAD) {
      return (double)s / a.den;
    } else if constexpr (M == NSC_METRIC_NRMSE) {
      if (r == 0) return e == 0 ? 0.0 : INFINITY;
      return sqrt((double)e / (double)r);
    } else {  // the negated PSNR, -10 log10(255^2 / MSE); -inf for identical images
      const double mse = (double)e / (a.den2 * count);
      return -(10.0 * log10(65025.0 / mse));
    }
  }
};

// Vertical pass of one output row for one lane's chunk of CB bytes: the
// output row covers source rows j0..j1-1; the first and last may be partial
// (weights wf, wl), every row in between has the full weight q.  Each row is
// added with its weight by a 24-bit multiply-add; PACKED keeps two 16-bit
// fields per 32-bit register (exact while 255 * p < 65536: the weights of an
// output row add up to p).  The rows are loaded in batches of up to RB, all
// loads of a batch issued before any add, so that an output row's loads are
// in flight together (an output row spans 7 to 16 source rows at the frame
// sizes here).  All control flow is uniform across the wave.
template <int CB, bool PACKED, int RB = NSC_ROWS_BATCH>
__device__ __forceinline__ void vertical_sums(const uint8_t* __restrict__ col, int64_t row_bytes,
                                              int a0, int a1, int q, int j0, int j1,
                                              int32_t out[CB], int split = 16) {
  constexpr int ND = CB >= 4 ? CB / 4 : 1;
  constexpr int NA = CB == 1 ? 1 : (PACKED ? 2 * ND : CB);
  const int nrows = j1 - j0;
  const uint32_t wf = nrows > 1 ? (uint32_t)(min(a1, (j0 + 1) * q) - a0) : (uint32_t)(a1 - a0);
  const uint32_t wl = (uint32_t)(a1 - max(a0, (j1 - 1) * q));
  uint32_t A[NA];
#pragma unroll
  for (int k = 0; k < NA; ++k) A[k] = 0;
  const uint8_t* p = col + (int64_t)j0 * row_bytes;
  for (int jb = 0; jb < nrows; jb += RB, p += RB * row_bytes) {
    const int cnt = min(RB, nrows - jb);
    uint32_t v[RB][ND];
#pragma unroll
    for (int k = 0; k < RB; ++k)
      if (k < cnt) load_chunk<CB>(p + k * row_bytes, v[k], split);
#pragma unroll
    for (int k = 0; k < RB; ++k) {
      if (k < cnt) {
        const int r = jb + k;  // row j0 + r
        const uint32_t w = r == 0 ? wf : (r == nrows - 1 ? wl : (uint32_t)q);
#pragma unroll
        for (int d = 0; d < ND; ++d) {
          if constexpr (CB == 1) {
            A[0] += __umul24(w, v[k][0]);
          } else if constexpr (PACKED) {
            A[d] += __umul24(w, bytes02(v[k][d]));
            A[ND + d] += __umul24(w, bytes13(v[k][d]));
          } else {
#pragma unroll
            for (int bb = 0; bb < 4; ++bb) A[4 * d + bb] += __umul24(w, __builtin_amdgcn_ubfe(v[k][d], 8 * bb, 8));
          }
        }
      }
    }
  }
  if constexpr (CB == 1) {
    out[0] = (int32_t)A[0];
  } else if constexpr (PACKED) {
#pragma unroll
    for (int d = 0; d < ND; ++d) {
      out[4 * d + 0] = (int32_t)(A[d] & 0xFFFFu);
      out[4 * d + 1] = (int32_t)(A[ND + d] & 0xFFFFu);
      out[4 * d + 2] = (int32_t)(A[d] >> 16);
      out[4 * d + 3] = (int32_t)(A[ND + d] >> 16);
    }
  } else {
#pragma unroll
    for (int k = 0; k < CB; ++k) out[k] = (int32_t)A[k];
  }
}

// Per-output-row kernel (any chunk width): for each output row, the lanes
// load its source rows in batches of four and accumulate vertically; the
// column sums go to a double-buffered LDS row (16-bit when exact) and, after
// one barrier, one thread per output cell applies the column weights.
template <int CB, bool PACKED>
__global__ void __launch_bounds__(1024) k_area_sums_rows(const uint8_t* __restrict__ frames,
                                                         int64_t stride, Axis ay, Axis ax,
                                                         int32_t lanes, int32_t bands,
                                                         int32_t* __restrict__ sums) {
  using cell_t = typename std::conditional<PACKED, uint16_t, int32_t>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  const int row_bytes = ax.n_in * 3;
  cell_t* rowbuf = reinterpret_cast<cell_t*>(smem);  // 2 x row_bytes, double buffered
  const int64_t f = blockIdx.x / bands;
  const int band = blockIdx.x - (int)(f * bands);
  const int Ho = ay.n_out, Wo = ax.n_out;
  const int Y0 = (int)((int64_t)band * Ho / bands);
  const int Y1 = (int)((int64_t)(band + 1) * Ho / bands);
  const int px = ax.p, qx = ax.q;
  const int tid = threadIdx.x;
  const bool active = tid < lanes;
  const uint8_t* col = frames + f * stride + (int64_t)(active ? tid : 0) * CB;
  int32_t* out = sums + f * (int64_t)Ho * Wo * 3;
  // Output column X covers source pixels i0..il: interior pixels have weight
  // qx, the end pixels the partial overlaps wf, wl.
  size_t xoff = (2 * (size_t)row_bytes * sizeof(cell_t) + 15) / 16 * 16;
  int4* xtab = reinterpret_cast<int4*>(smem + xoff);
  for (int X = tid; X < Wo; X += blockDim.x) {
    const int b0 = X * px, b1 = b0 + px;
    const int i0 = b0 / qx, il = (b1 - 1) / qx;
    xtab[X] = make_int4(i0, il - i0, il == i0 ? px : (i0 + 1) * qx - b0, b1 - il * qx);
  }
  for (int Y = Y0; Y < Y1; ++Y) {
    // uniform row bounds (divisions run on the vector unit; move them to scalars)
    const int a0 = Y * ay.p, a1 = a0 + ay.p;
    const int j0 = __builtin_amdgcn_readfirstlane(a0 / ay.q);
    const int j1 = __builtin_amdgcn_readfirstlane((a1 + ay.q - 1) / ay.q);
    cell_t* buf = rowbuf + (Y & 1) * row_bytes;
    int32_t v[CB];
    vertical_sums<CB, PACKED>(col, row_bytes, a0, a1, ay.q, j0, j1, v);
    if (active) {
#pragma unroll
      for (int b = 0; b < CB; ++b) buf[tid * CB + b] = (cell_t)v[b];
    }
    __syncthreads();
    int32_t* orow = out + (int64_t)Y * Wo * 3;
    for (int t = tid; t < Wo * 3; t += blockDim.x) {
      const int X = t / 3, c = t - 3 * X;
      const int4 e = xtab[X];  // i0, number of pixels after the first, wf, wl
      const cell_t* bp = buf + 3 * e.x + c;
      int32_t mid = 0;
      int i = 1;
      for (; i + 8 <= e.y; i += 8) {  // eight independent LDS reads per step
        int32_t m8 = 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) m8 += (int32_t)bp[3 * (i + u)];
        mid += m8;
      }
      for (; i < e.y; ++i) mid += (int32_t)bp[3 * i];
      int32_t s;
      if constexpr (PACKED) {  // all factors below 2^24
        s = (int32_t)(__umul24((uint32_t)e.z, bp[0]) + __umul24((uint32_t)qx, (uint32_t)mid));
        if (e.y > 0) s += (int32_t)__umul24((uint32_t)e.w, bp[3 * e.y]);
      } else {
        s = e.z * (int32_t)bp[0] + qx * mid;
        if (e.y > 0) s += e.w * (int32_t)bp[3 * e.y];
      }
      orow[t] = s;
    }
    // The next row writes the other buffer; its readers (row Y-1) all passed
    // this row's barrier, so no second barrier is needed.
  }
}

// Area sums of one wave's strip for output rows Y0..Y1-1: per output row, the
// vertical pass into the wave's LDS column sums buf, then the horizontal
// pass; value t of band row r (cell (t / 3) of the strip, channel t mod 3)
// with sum s is handed to cell(t, r, s).  Lane l handles the values t = l,
// l + 64, ... of every row.  The nl active lanes read the strip's CB x nl
// bytes: 16 or 4 bytes at col = strip + CB l, or with CB = 32 the 16-byte
// pieces l and nl + l (col = strip + 16 l).
// With MAXS > 0 (at most 64 MAXS values per row) the loop over a lane's
// values is unrolled and cell(k, t, r, s) also gets the slot k (t = l + 64 k).
template <int CB, bool PACKED, int RB, int MAXS = 0, class Cell, class Buf>
__device__ __forceinline__ void strip_band_sums(const uint8_t* __restrict__ col, int64_t row_bytes,
                                                const Axis& ay, int qx, int Y0, int Y1, int lane,
                                                int nl, Buf* buf, const int4* xtab, int ncells,
                                                Cell&& cell) {
  using cell_t = Buf;
  const bool active = lane < nl;
  const int split = 16 * nl;  // CB = 32: bytes from a lane's first piece to its second
  // LDS position (cells) of the lane's c-th 16-byte piece (c = 0, 1 for CB = 32)
  auto piece = [&](int c) { return CB == 32 ? (c * nl + lane) * 16 : lane * CB; };
  for (int Y = Y0; Y < Y1; ++Y) {
    // uniform row bounds (divisions run on the vector unit; move them to scalars)
    const int a0 = Y * ay.p, a1 = a0 + ay.p;
    const int j0 = __builtin_amdgcn_readfirstlane(a0 / ay.q);
    const int j1 = __builtin_amdgcn_readfirstlane((a1 + ay.q - 1) / ay.q);
    int32_t v[CB];
    vertical_sums<CB, PACKED, RB>(col, row_bytes, a0, a1, ay.q, j0, j1, v, split);
    if (active) {
      if constexpr (PACKED && CB % 8 == 0) {  // 2 CB bytes per lane as 16-byte stores
#pragma unroll
        for (int q = 0; q < CB / 8; ++q) {
          uint4* d = reinterpret_cast<uint4*>(buf + piece(q / 2)) + (q & 1);
          *d = make_uint4(v[8 * q] | (v[8 * q + 1] << 16), v[8 * q + 2] | (v[8 * q + 3] << 16),
                          v[8 * q + 4] | (v[8 * q + 5] << 16), v[8 * q + 6] | (v[8 * q + 7] << 16));
        }
      } else {
#pragma unroll
        for (int b = 0; b < CB; ++b) buf[piece(b / 16) + (b & 15)] = (cell_t)v[b];
      }
    }
    __syncwarp();
    auto horizontal = [&](int t) -> int32_t {
      const int x = t / 3, c = t - 3 * x;
      const int4 e = xtab[x];
      const cell_t* bp = buf + 3 * e.x + c;
      int32_t mid = 0;
      int i = 1;
      for (; i + 8 <= e.y; i += 8) {
        int32_t m8 = 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) m8 += (int32_t)bp[3 * (i + u)];
        mid += m8;
      }
      for (; i < e.y; ++i) mid += (int32_t)bp[3 * i];
      int32_t s;
      if constexpr (PACKED) {  // all factors below 2^24
        s = (int32_t)(__umul24((uint32_t)e.z, bp[0]) + __umul24((uint32_t)qx, (uint32_t)mid));
        if (e.y > 0) s += (int32_t)__umul24((uint32_t)e.w, bp[3 * e.y]);
      } else {
        s = e.z * (int32_t)bp[0] + qx * mid;
        if (e.y > 0) s += e.w * (int32_t)bp[3 * e.y];
      }
      return s;
    };
    if constexpr (MAXS > 0) {
#pragma unroll
      for (int k = 0; k < MAXS; ++k) {
        const int t = lane + 64 * k;
        if (t < ncells) cell(k, t, Y - Y0, horizontal(t));
      }
    } else {
      for (int t = lane; t < ncells; t += 64) cell(t, Y - Y0, horizontal(t));
    }
    __syncwarp();  // reads of this row's strip precede the next row's writes
  }
}

// Wave-autonomous kernel: no workgroup barriers, and no global stores until
// the end of a wave's work.  The horizontal resampling pattern repeats every
// p_x source pixels (q_x output columns); a "group" is the smallest whole
// number of periods whose bytes split into 16/4-byte lane chunks.  Each wave
// owns a strip of whole groups of one band of output rows of one frame, so
// the horizontal reduction stays inside the wave: lanes write their vertical
// sums to a wave-private LDS strip, __syncwarp() orders the writes before the
// reads, and the same lanes produce the strip's output cells into a
// wave-private LDS block of the band's sums.  That block is written to HBM
// once, after the last source row: on this architecture a store makes the
// wave wait for it before it may consume later loads, so stores interleaved
// with the row stream would stall it.
//
// FM >= 0 fuses the difference detector against a fixed reference image
// (global metric FM): as the wave stores its band's sums it also adds up the
// metric's exact integer sums of its cells against the reference sums (read
// once per wave from L2, where the small reference image stays resident) and
// writes them as the unit's partial sums, part[unit][3] = (sum of squared
// differences, of absolute differences, of squared reference values);
// k_diff_fixed_finish adds a frame's partials and applies the metric.
template <int CB, bool PACKED, int RB = NSC_ROWS_BATCH, int FM = -1>
__global__ void __launch_bounds__(256) k_area_sums_wave(const uint8_t* __restrict__ frames,
                                                        int64_t stride, Axis ay, Axis ax,
                                                        WaveGeom g, int32_t bands, int64_t n,
                                                        int32_t* __restrict__ sums,
                                                        const int32_t* __restrict__ ref,
                                                        int64_t* __restrict__ part) {
  using cell_t = typename std::conditional<PACKED, uint16_t, int32_t>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  // the wave index is uniform across the wave; say so, so that everything
  // derived from it (frame, strip, rows) lives in scalar registers
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int Ho = ay.n_out, Wo = ax.n_out;
  const int px = ax.p, qx = ax.q;
  const int scols = g.groups_per_wave * g.group_cols;  // output columns of a full strip
  // per-column table of a strip (identical for every strip): first pixel,
  // pixels after the first, partial weights of the first and last pixel
  int4* xtab = reinterpret_cast<int4*>(smem);
  for (int x = threadIdx.x; x < scols; x += blockDim.x) {
    const int b0 = x * px, b1 = b0 + px;
    const int i0 = b0 / qx, il = (b1 - 1) / qx;
    xtab[x] = make_int4(i0, il - i0, il == i0 ? px : (i0 + 1) * qx - b0, b1 - il * qx);
  }
  __syncthreads();  // the only workgroup barrier
  // each wave's region starts 16-byte aligned (the column sums are stored as uint4)
  const size_t per_wave =
      ((size_t)64 * CB * sizeof(cell_t) + (size_t)g.band_rows * scols * 3 * 4 + 15) & ~(size_t)15;
  unsigned char* wbase = smem + (size_t)scols * 16 + (size_t)wv * per_wave;
  cell_t* buf = reinterpret_cast<cell_t*>(wbase);                              // column sums
  int32_t* sbuf = reinterpret_cast<int32_t*>(wbase + (size_t)64 * CB * sizeof(cell_t));  // band sums

  // each XCD walks a contiguous range of frames, so the source rows that two
  // bands of a frame share are fetched into one L2
  const int64_t unit = xcd_block(blockIdx.x, gridDim.x) * (blockDim.x >> 6) + wv;
  const int64_t per_frame = (int64_t)bands * g.waves_per_frame;
  if (unit >= n * per_frame) return;
  const int64_t f = unit / per_frame;
  const int rem = (int)(unit - f * per_frame);
  const int band = rem / g.waves_per_frame, strip = rem - band * g.waves_per_frame;
  const int group0 = strip * g.groups_per_wave;
  const int ngroups = min(g.groups_per_wave, g.groups_per_row - group0);
  const int nl = ngroups * g.group_lanes;  // active lanes
  const int ncells = ngroups * g.group_cols * 3;
  const int X0 = group0 * g.group_cols;
  const int Y0 = (int)((int64_t)band * Ho / bands);
  const int Y1 = (int)((int64_t)(band + 1) * Ho / bands);
  const int64_t row_bytes = (int64_t)ax.n_in * 3;
  const uint8_t* col = frames + f * stride + (int64_t)group0 * g.group_lanes * CB +
                       (int64_t)(lane < nl ? lane : 0) * (CB == 32 ? 16 : CB);
  strip_band_sums<CB, PACKED, RB>(col, row_bytes, ay, qx, Y0, Y1, lane, nl, buf, xtab, ncells,
                                  [&](int t, int r, int32_t s) { sbuf[r * ncells + t] = s; });
  // the band's sums, one output row segment after another
  int32_t* out = sums + (f * (int64_t)Ho * Wo + X0) * 3;
  DiffSums<FM < 0 ? NSC_METRIC_MSE : FM> acc;
  for (int Y = Y0; Y < Y1; ++Y) {
    const int32_t* srow = sbuf + (Y - Y0) * ncells;
    int32_t* orow = out + (int64_t)Y * Wo * 3;
    for (int t = lane; t < ncells; t += 64) {
      const int32_t v = srow[t];
      orow[t] = v;
      if constexpr (FM >= 0) acc.add(v, ref[((int64_t)Y * Wo + X0) * 3 + t]);
    }
  }
  if constexpr (FM >= 0) {
    acc.reduce();
    if (lane == 0) {
      int64_t* pp = part + (f * per_frame + rem) * 3;
      pp[0] = acc.e;
      pp[1] = acc.s;
      pp[2] = acc.r;
    }
  }
}

// The earlier-frame global MSE detector fused into the area kernel by
// temporal tiling along the reuse distance delta: a wave owns one (band,
// strip) of the R frames f_i = r + delta (sg R + i), i = 0 .. R-1, of chain
// (sg, r), so that while it forms the sums of f_i its LDS block still holds
// those of f_(i-1) = f_i - delta, and each value's squared difference is
// added as the new value replaces the old one.  For every chain frame after
// the first the wave writes its partial sum of squared differences (exact
// int64) at part[(f * bands + band) * strips + strip].  The first frame of a
// chain, whose frame f - delta is another wave's (or in the state), is scored
// from the sums by k_diff afterwards, which also adds up the partials of the
// other frames.  Sums stores and the LDS layout are those of
// k_area_sums_wave.
constexpr int kPrevSlots = 4;  // values per lane and row (at most 256 per strip row)

template <int CB, bool PACKED, int RB>
__global__ void __launch_bounds__(256) k_area_prev_wave(const uint8_t* __restrict__ frames,
                                                        int64_t stride, Axis ay, Axis ax,
                                                        WaveGeom g, int64_t n, int32_t delta,
                                                        int32_t R, int32_t* __restrict__ sums,
                                                        int64_t* __restrict__ part) {
  using cell_t = typename std::conditional<PACKED, uint16_t, int32_t>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int Ho = ay.n_out, Wo = ax.n_out;
  const int qx = ax.q;
  const int scols = g.groups_per_wave * g.group_cols;
  int4* xtab = reinterpret_cast<int4*>(smem);
  for (int x = threadIdx.x; x < scols; x += blockDim.x) {
    const int b0 = x * ax.p, b1 = b0 + ax.p;
    const int i0 = b0 / qx, il = (b1 - 1) / qx;
    xtab[x] = make_int4(i0, il - i0, il == i0 ? ax.p : (i0 + 1) * qx - b0, b1 - il * qx);
  }
  __syncthreads();  // the only workgroup barrier
  const size_t per_wave =
      ((size_t)64 * CB * sizeof(cell_t) + (size_t)g.band_rows * scols * 3 * 4 + 15) & ~(size_t)15;
  unsigned char* wbase = smem + (size_t)scols * 16 + (size_t)wv * per_wave;
  cell_t* buf = reinterpret_cast<cell_t*>(wbase);
  int32_t* sbuf = reinterpret_cast<int32_t*>(wbase + (size_t)64 * CB * sizeof(cell_t));

  const int bands = g.bands, strips = g.waves_per_frame;
  const int64_t unit = xcd_block(blockIdx.x, gridDim.x) * (blockDim.x >> 6) + wv;
  const int64_t per_chain = (int64_t)bands * strips;
  const int64_t chain = unit / per_chain;
  const int rem = (int)(unit - chain * per_chain);
  const int band = rem / strips, strip = rem - band * strips;
  const int64_t sg = chain / delta;
  const int r = (int)(chain - sg * delta);
  if (sg * R * delta + r >= n) return;  // no frames (uniform)
  const int group0 = strip * g.groups_per_wave;
  const int ngroups = min(g.groups_per_wave, g.groups_per_row - group0);
  const int nl = ngroups * g.group_lanes;  // active lanes
  const int ncells = ngroups * g.group_cols * 3;
  const int X0 = group0 * g.group_cols;
  const int Y0 = (int)((int64_t)band * Ho / bands);
  const int Y1 = (int)((int64_t)(band + 1) * Ho / bands);
  const int64_t row_bytes = (int64_t)ax.n_in * 3;
  for (int i = 0; i < R; ++i) {
    const int64_t f = (sg * R + i) * delta + r;
    if (f >= n) break;
    const uint8_t* col = frames + f * stride + (int64_t)group0 * g.group_lanes * CB +
                         (int64_t)(lane < nl ? lane : 0) * (CB == 32 ? 16 : CB);
    int64_t e[kPrevSlots];
#pragma unroll
    for (int k = 0; k < kPrevSlots; ++k) e[k] = 0;
    const bool diff = i > 0;
    strip_band_sums<CB, PACKED, RB, kPrevSlots>(
        col, row_bytes, ay, qx, Y0, Y1, lane, nl, buf, xtab, ncells,
        [&](int k, int t, int rr, int32_t s) {
          int32_t* q = sbuf + rr * ncells + t;
          if (diff) {
            const int64_t d = (int64_t)s - *q;
            e[k] += d * d;
          }
          *q = s;
        });
    int32_t* out = sums + (f * (int64_t)Ho * Wo + X0) * 3;
    for (int Y = Y0; Y < Y1; ++Y) {
      const int32_t* srow = sbuf + (Y - Y0) * ncells;
      int32_t* orow = out + (int64_t)Y * Wo * 3;
      for (int t = lane; t < ncells; t += 64) orow[t] = srow[t];
    }
    if (!diff) continue;
    int64_t v = 0;
#pragma unroll
    for (int k = 0; k < kPrevSlots; ++k) v += e[k];
    v = wave_sum_i64(v);
    if (lane == 0) part[(f * bands + band) * strips + strip] = v;
  }
}

// ------------------------------------------------------------- detector

// Blocked score by rows: a wave streams the frame row by row, lane l taking
// values l + 64 j of each row (coalesced), whose block column is fixed; the
// lane keeps one partial sum per slot j over a block row's rows, and at the
// end of the block row the slots are added into per-block LDS sums (64-bit
// LDS atomics, exact), from which lane bx computes block bx's metric.  Rows
// of up to 64 x kDiffSlots values and up to 64 block columns.
constexpr int kDiffSlots = 6;

struct BlockRowSums {  // one wave's sums of the block row in progress
  unsigned long long e[64], s[64], r[64];
};

template <int M, int J>  // J = slots per lane: rows of 64 (J - 1) + 1 .. 64 J values
__device__ __forceinline__ double blocked_score_rows(const int32_t* __restrict__ cur,
                                                     const int32_t* __restrict__ ref,
                                                     const DiffArgs& a, int32_t grid_h,
                                                     int32_t grid_w, const float* lr_w,
                                                     double lr_b, int lane, BlockRowSums* bs) {
#pragma clang fp contract(off)
  const int rl = a.dd_w * 3;  // values per row
  // every lane loads all J slots (from value 0 where a slot is past the row,
  // counted as no difference) so that the loads of a row issue together
  int bxs[J], off[J];         // block column (-1: none) and offset of each slot's value
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = lane + 64 * j;
    bxs[j] = c < rl ? ((c / 3 + 1) * grid_w - 1) / a.dd_w : -1;
    off[j] = c < rl ? c : 0;
  }
  double z = lr_b;
  for (int by = 0; by < grid_h; ++by) {
    const int y0 = (int)((int64_t)by * a.dd_h / grid_h);
    const int y1 = (int)((int64_t)(by + 1) * a.dd_h / grid_h);
    DiffSums<M> acc[J];
#pragma unroll 2
    for (int y = y0; y < y1; ++y) {
      const int32_t* cr = cur + (int64_t)y * rl;
      const int32_t* rr = ref + (int64_t)y * rl;
      int32_t xv[J], yv[J];
#pragma unroll
      for (int j = 0; j < J; ++j) {
        xv[j] = cr[off[j]];
        yv[j] = rr[off[j]];
      }
#pragma unroll
      for (int j = 0; j < J; ++j) acc[j].add(bxs[j] >= 0 ? xv[j] : 0, bxs[j] >= 0 ? yv[j] : 0);
    }
    if (lane < grid_w) {
      bs->e[lane] = 0;
      bs->s[lane] = 0;
      bs->r[lane] = 0;
    }
    __syncwarp();  // cleared before the adds
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if (bxs[j] < 0) continue;
      if constexpr (M != NSC_METRIC_SAD) atomicAdd(&bs->e[bxs[j]], (unsigned long long)acc[j].e);
      if constexpr (M == NSC_METRIC_SAD) atomicAdd(&bs->s[bxs[j]], (unsigned long long)acc[j].s);
      if constexpr (M == NSC_METRIC_NRMSE)
        atomicAdd(&bs->r[bxs[j]], (unsigned long long)acc[j].r);
    }
    __syncwarp();  // block sums complete
    double m = 0.0;
    if (lane < grid_w) {
      DiffSums<M> b;
      b.e = (int64_t)bs->e[lane];
      b.s = (int64_t)bs->s[lane];
      b.r = (int64_t)bs->r[lane];
      const int x0 = (int)((int64_t)lane * a.dd_w / grid_w);
      const int x1 = (int)((int64_t)(lane + 1) * a.dd_w / grid_w);
      const double ncell = ((double)(y1 - y0) * (double)(x1 - x0)) * 3.0;
      m = b.value(a, ncell);
    }
    __syncwarp();  // sums read before the next block row clears them
    // in block order, as separate multiplies and adds
    for (int bx = 0; bx < grid_w; ++bx) z = z + (double)lr_w[by * grid_w + bx] * __shfl(m, bx, 64);
  }
  return z;
}

// The detector score of one frame (area sums `cur`) against its reference
// `ref`, by one wave: the metric over the whole grid, or the logistic score of
// the per-block metrics (blocks in row-major order, weights lr_w).
template <int M, bool BLK>  // BLK: blocked grids possible (else grid_h = grid_w = 1)
__device__ __forceinline__ double frame_score(const int32_t* cur, const int32_t* ref,
                                              const DiffArgs& a, int32_t grid_h, int32_t grid_w,
                                              const float* lr_w, double lr_b, int lane,
                                              BlockRowSums* bs) {
  // the blocked score is summed with separate multiplies and adds, in block
  // order, so it is reproducible bit for bit
#pragma clang fp contract(off)
  const int64_t cells = (int64_t)a.dd_h * a.dd_w * 3;
  if (!BLK || grid_h * grid_w == 1) {
    DiffSums<M> acc;
    if ((cells & 3) == 0 && (((uintptr_t)cur | (uintptr_t)ref) & 15) == 0) {
      const int4* c4 = reinterpret_cast<const int4*>(cur);
      const int4* r4 = reinterpret_cast<const int4*>(ref);
      for (int64_t k = lane; k < cells / 4; k += 64) {
        const int4 x = c4[k], y = r4[k];
        acc.add(x.x, y.x);
        acc.add(x.y, y.y);
        acc.add(x.z, y.z);
        acc.add(x.w, y.w);
      }
    } else {
      for (int64_t k = lane; k < cells; k += 64) acc.add(cur[k], ref[k]);
    }
    acc.reduce();
    return acc.value(a, (double)cells);
  }
  if constexpr (!BLK) return 0.0;
  if (grid_w <= 64 && a.dd_w * 3 <= 64 * kDiffSlots) {
    switch ((a.dd_w * 3 + 63) / 64) {
#define NSC_ROWS_CASE(J) \
  case J:                \
    return blocked_score_rows<M, J>(cur, ref, a, grid_h, grid_w, lr_w, lr_b, lane, bs);
      NSC_ROWS_CASE(1)
      NSC_ROWS_CASE(2)
      NSC_ROWS_CASE(3)
      NSC_ROWS_CASE(4)
      NSC_ROWS_CASE(5)
      NSC_ROWS_CASE(6)
#undef NSC_ROWS_CASE
      default:
        break;
    }
  }
  double z = lr_b;
  for (int by = 0; by < grid_h; ++by) {
    const int y0 = (int)((int64_t)by * a.dd_h / grid_h);
    const int y1 = (int)((int64_t)(by + 1) * a.dd_h / grid_h);
    for (int bx = 0; bx < grid_w; ++bx) {
      const int x0 = (int)((int64_t)bx * a.dd_w / grid_w);
      const int x1 = (int)((int64_t)(bx + 1) * a.dd_w / grid_w);
      const int rl = (x1 - x0) * 3;
      const int total = (y1 - y0) * rl;
      DiffSums<M> acc;
      for (int k = lane; k < total; k += 64) {
        const int r = k / rl, cc = k - r * rl;
        const int64_t off = ((int64_t)(y0 + r) * a.dd_w + x0) * 3 + cc;
        acc.add(cur[off], ref[off]);
      }
      acc.reduce();
      const double ncell = ((double)(y1 - y0) * (double)(x1 - x0)) * 3.0;
      const double m = acc.value(a, ncell);
      z = z + (double)lr_w[by * grid_w + bx] * m;
    }
  }
  return z;
}

// The global MSE score of frame i from the fused kernel's partial sums
// (exact integers, so their grouping does not matter), as frame_score
// computes it from the sums.
__device__ __forceinline__ double part_score(const DiffArgs& a, int64_t i, int lane) {
#pragma clang fp contract(off)
  const int units = a.part_bands * a.part_strips;
  const int64_t* p = a.part + i * units;
  int64_t e = 0;
  for (int u = lane; u < units; u += 64) e += p[u];
  DiffSums<NSC_METRIC_MSE> acc;
  acc.e = wave_sum_i64(e);
  return acc.value(a, (double)((int64_t)a.dd_h * a.dd_w * 3));
}

// The fixed-reference detector fused into the area kernel: a thread per
// frame adds the frame's per-unit partial sums (exact integers, so their order
// does not matter) and applies the metric as k_diff does.
template <int M>
__global__ void __launch_bounds__(256) k_diff_fixed_finish(DiffArgs a, const int64_t* __restrict__ part,
                                                           int32_t units) {
#pragma clang fp contract(off)
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  DiffSums<M> acc;
  const int64_t* p = part + i * units * 3;
  for (int u = 0; u < units; ++u) {
    acc.e += p[3 * u];
    acc.s += p[3 * u + 1];
    acc.r += p[3 * u + 2];
  }
  const double score = acc.value(a, (double)((int64_t)a.dd_h * a.dd_w * 3));
  a.fire[i] = score > a.delta_diff ? 1 : 0;
  if (a.score) a.score[i] = score;
}

template <int M, bool BLK>
__global__ void __launch_bounds__(256) k_diff(DiffArgs a) {
  __shared__ BlockRowSums bsums[4];
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= a.n) return;
  const int64_t t = a.t0 + i;
  const int64_t cells = (int64_t)a.dd_h * a.dd_w * 3;
  const bool forced = a.ref_mode == NSC_REF_PREV && t < a.delta;
  double score = INFINITY;
  const bool from_part = M == NSC_METRIC_MSE && !BLK && a.part != nullptr && !forced &&
                         (i / a.delta) % a.chain_r != 0;
  if (from_part) {
    score = part_score(a, i, lane);
  } else if (!forced) {
    const int32_t* cur = a.sums + i * cells;
    const int32_t* ref;
    if (a.ref_mode == NSC_REF_FIXED)
      ref = a.ref_sums;
    else if (i >= a.delta)
      ref = a.sums + (i - a.delta) * cells;
    else
      ref = a.prev_sums + i * cells;  // frame t - delta = t0 - delta + i
    score = frame_score<M, BLK>(cur, ref, a, a.grid_h, a.grid_w, a.lr_w, a.lr_b, lane,
                          &bsums[threadIdx.x >> 6]);
  }
  if (lane == 0) {
    a.fire[i] = (forced || score > a.delta_diff) ? 1 : 0;
    if (a.score) a.score[i] = score;
  }
}

// A camera group's frames: camera c's n = per_cam frames [t0, t0 + n) are
// frames c * n .. c * n + n - 1 of the batch, each scored with its camera's
// reference, blocks, weights and threshold; the frames before t0 come from
// the camera's state slot.
template <int M, bool BLK>
__global__ void __launch_bounds__(256) k_diff_group(DiffArgs a) {
  __shared__ BlockRowSums bsums[4];
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= a.n) return;
  const int64_t cam = i / a.per_cam;
  const int64_t j = i - cam * a.per_cam;
  const CamDiff cd = a.cams[cam];
  const int64_t t = a.t0 + j;
  const int64_t cells = (int64_t)a.dd_h * a.dd_w * 3;
  const bool forced = cd.ref_mode == NSC_REF_PREV && t < cd.delta;
  double score = INFINITY;
  if (!forced) {
    const int32_t* cur = a.sums + i * cells;
    const int32_t* ref;
    if (cd.ref_mode == NSC_REF_FIXED)
      ref = cd.ref_sums;
    else if (j >= cd.delta)
      ref = a.sums + (i - cd.delta) * cells;
    else  // frame t0 - delta + j, kept in the camera's state
      ref = reinterpret_cast<const int32_t*>(a.state + cam * a.state_stride) + j * cells;
    score = frame_score<M, BLK>(cur, ref, a, cd.grid_h, cd.grid_w, cd.lr_w, cd.lr_b, lane,
                          &bsums[threadIdx.x >> 6]);
  }
  if (lane == 0) {
    a.fire[i] = (forced || score > cd.delta_diff) ? 1 : 0;
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
  // wave strips: whole periods of the horizontal pattern in 16/4-byte
  // chunks; 32-byte chunks (two 16-byte loads per lane) only where 16-byte
  // ones leave more than a fifth of a wave's lanes idle.  (1920x1080 ->
  // 100x100, 54 of 64 lanes busy in 16-byte chunks against 63 in 32-byte
  // ones: 16-byte chunks 3.3 % faster; 1280x720 -> 50x50, 48 against 60:
  // 32-byte chunks 3 % faster; area kernels alone, alternating in one
  // process.)
  p.wave = false;
  if (p.chunk_bytes != 1) {
    int best_cb = 0, best_used = 0;
    int64_t best_glanes = 0, best_gpix = 0;
    const int cands[2] = {p.chunk_bytes, p.chunk_bytes == 16 ? 32 : 0};
    for (int cb : cands) {
      if (cb == 0) continue;
      int k = 1;
      while ((3 * (int64_t)p.ax.p * k) % cb != 0) k *= 2;
      const int64_t glanes = 3 * (int64_t)p.ax.p * k / cb;
      const int64_t gpix = (int64_t)p.ax.p * k;
      if (glanes > 64 || in_w % gpix != 0) continue;
      const int used = (int)(64 / glanes * glanes);
      if (best_cb == 0 || (5 * best_used < 4 * 64 && used > best_used)) {
        best_used = used;
        best_cb = cb;
        best_glanes = glanes;
        best_gpix = gpix;
      }
    }
    if (best_cb != 0) {
      WaveGeom& g = p.wg;
      g.chunk_bytes = best_cb;
      g.group_lanes = (int32_t)best_glanes;
      g.group_cols = (int32_t)(p.ax.q * (best_gpix / p.ax.p));
      g.groups_per_wave = (int32_t)(64 / best_glanes);
      g.groups_per_row = (int32_t)(in_w / best_gpix);
      g.waves_per_frame = (g.groups_per_row + g.groups_per_wave - 1) / g.groups_per_wave;
      // a workgroup reads whole source rows (all strips of its bands) at once, so that
      // the cache lines two strips share are fetched once, by one CU
      g.waves_per_block = g.waves_per_frame <= 4 ? g.waves_per_frame * (4 / g.waves_per_frame) : 4;
      // bands of two output rows with 16- or 32-byte lane chunks (more when
      // there are too few frames to fill the chip): with units this short,
      // the waves resident on an XCD at a time read fewer frames.  Measured
      // against bands of 10 rows (area sums alone, all heights timed in turn
      // in one process, on two machines): 640x480 -> 50x50 4.6 and 7.6 %
      // faster, 1280x720 -> 100x100 0 and 6 %, 1920x1080 -> 100x100 1.2 and
      // 1 %, 1280x720 -> 50x50 within 0.5 %; a single row was faster still at
      // 640x480 but 5 % slower at 1280x720 -> 100x100.  Rows of a few hundred
      // bytes (4-byte chunks) keep bands of about 10 rows: 100x100 -> 50x50,
      // 20,000 frames, 663 us against 847 with two rows.
      int64_t wb = best_cb >= 16 ? (out_h + 1) / 2 : (out_h + 9) / 10;
      const int64_t fill = (16384 + n * g.waves_per_frame - 1) / (n * g.waves_per_frame > 0 ? n * g.waves_per_frame : 1);
      if (fill > wb) wb = fill;
      if (wb > out_h) wb = out_h;
      g.bands = (int32_t)wb;
      g.band_rows = (int32_t)((out_h + wb - 1) / wb);
      const int64_t scols = (int64_t)g.groups_per_wave * g.group_cols;
      const int64_t cellb = p.packed ? 2 : 4;
      const int64_t per_wave = (64 * best_cb * cellb + (int64_t)g.band_rows * scols * 3 * 4 + 15) & ~(int64_t)15;
      g.lds_bytes = (size_t)(scols * 16 + g.waves_per_block * per_wave);
      p.wave = g.lds_bytes <= 64 * 1024;
    }
  }
  // split frames into bands of output rows when there are too few frames to fill the chip
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
  const size_t row_bytes = (size_t)p.ax.n_in * 3;
  dim3 grid((unsigned)blocks), block(p.threads);
  if (p.wave) {
    const WaveGeom& g = p.wg;
    const int64_t units = n * g.bands * g.waves_per_frame;
    const int64_t wblocks = (units + g.waves_per_block - 1) / g.waves_per_block;
    if (wblocks > 0x7FFFFFFF) return fail(NSC_E_SHAPE, "too many frames in one call");
#define NSC_WAVE_LAUNCH(CB, PK)                                                          \
  hipLaunchKernelGGL((k_area_sums_wave<CB, PK, CB == 32 ? NSC_ROWS_BATCH / 2 : NSC_ROWS_BATCH>), \
                     dim3((unsigned)wblocks), dim3(64 * g.waves_per_block),               \
                     g.lds_bytes, stream, frames, stride, p.ay, p.ax, g, g.bands, n, sums,   \
                     nullptr, nullptr)
    if (g.chunk_bytes == 32) {
      if (p.packed) NSC_WAVE_LAUNCH(32, true); else NSC_WAVE_LAUNCH(32, false);
    } else if (g.chunk_bytes == 16) {
      if (p.packed) NSC_WAVE_LAUNCH(16, true); else NSC_WAVE_LAUNCH(16, false);
    } else {
      if (p.packed) NSC_WAVE_LAUNCH(4, true); else NSC_WAVE_LAUNCH(4, false);
    }
#undef NSC_WAVE_LAUNCH
    NSC_CHECK_LAUNCH("k_area_sums_wave");
    return NSC_OK;
  }
  {
    const size_t cell = p.packed ? 2 : 4;
    const size_t lds = (2 * row_bytes * cell + 15) / 16 * 16 + (size_t)p.ax.n_out * 16;
#define NSC_ROWS_LAUNCH(CB, PK)                                                              \
  hipLaunchKernelGGL((k_area_sums_rows<CB, PK>), grid, block, lds, stream, frames, stride, p.ay, \
                     p.ax, p.lanes, p.bands, sums)
    if (p.chunk_bytes == 16) {
      if (p.packed) NSC_ROWS_LAUNCH(16, true); else NSC_ROWS_LAUNCH(16, false);
    } else if (p.chunk_bytes == 4) {
      if (p.packed) NSC_ROWS_LAUNCH(4, true); else NSC_ROWS_LAUNCH(4, false);
    } else {
      if (p.packed) NSC_ROWS_LAUNCH(1, true); else NSC_ROWS_LAUNCH(1, false);
    }
#undef NSC_ROWS_LAUNCH
  }
  NSC_CHECK_LAUNCH("k_area_sums");
  return NSC_OK;
}

int launch_diff(const DiffArgs& a, hipStream_t stream) {
  if (a.n <= 0) return NSC_OK;
  const int64_t blocks = (a.n + 3) / 4;
  if (blocks > 0x7FFFFFFF) return fail(NSC_E_SHAPE, "too many frames in one call");
#define NSC_DIFF_LAUNCH(M)                                                                    \
  if (a.cams && a.cams_blocked)                                                               \
    hipLaunchKernelGGL((k_diff_group<M, true>), dim3((unsigned)blocks), dim3(256), 0, stream, a); \
  else if (a.cams)                                                                            \
    hipLaunchKernelGGL((k_diff_group<M, false>), dim3((unsigned)blocks), dim3(256), 0, stream, a); \
  else if (a.grid_h * a.grid_w > 1)                                                           \
    hipLaunchKernelGGL((k_diff<M, true>), dim3((unsigned)blocks), dim3(256), 0, stream, a);   \
  else                                                                                        \
    hipLaunchKernelGGL((k_diff<M, false>), dim3((unsigned)blocks), dim3(256), 0, stream, a)
  switch (a.metric) {
    case NSC_METRIC_MSE:
      NSC_DIFF_LAUNCH(NSC_METRIC_MSE);
      break;
    case NSC_METRIC_SAD:
      NSC_DIFF_LAUNCH(NSC_METRIC_SAD);
      break;
    case NSC_METRIC_NRMSE:
      NSC_DIFF_LAUNCH(NSC_METRIC_NRMSE);
      break;
    case NSC_METRIC_PSNR:
      NSC_DIFF_LAUNCH(NSC_METRIC_PSNR);
      break;
    default:
      return fail(NSC_E_INVAL, "metric %d is unknown", a.metric);
  }
#undef NSC_DIFF_LAUNCH
  NSC_CHECK_LAUNCH("k_diff");
  return NSC_OK;
}

bool area_prev_plan(const AreaPlan& p, const DiffArgs& a, int64_t n, PrevFusePlan* out) {
  // Where it applies: a global MSE score with 16- or 4-byte lane chunks from
  // delta = 2 on.  Measured against the two passes (whole cascade per call,
  // alternating builds in one process): with 32-byte chunks it needs 126
  // registers against 102 (four waves per SIMD instead of five) and was 3 %
  // slower (1920x1080, delta 30, blocked); against the frame just before
  // (delta = 1) 3.5 % slower on 720p blocked; a blocked score, which needs a
  // band per block row, 9.7 % slower at 1920x1080, delta 30; and since the
  // area kernel's bands are two rows high, 6-7 % slower than the two passes
  // on 640x480 too (a chain spreads the frames the resident waves read over
  // R times as many frames).  The caller takes it only when the
  // configuration asks for it.
  if (!p.wave || p.wg.chunk_bytes == 32 || a.ref_mode != NSC_REF_PREV ||
      a.metric != NSC_METRIC_MSE || a.cams != nullptr || a.delta < 2 ||
      n < 2 * (int64_t)a.delta || a.grid_h * a.grid_w != 1)
    return false;
  const AreaPlan& q = p;
  const WaveGeom& g = q.wg;
  const int64_t scols = (int64_t)g.groups_per_wave * g.group_cols;
  if (scols * 3 > 64 * kPrevSlots) return false;
  // chains of R frames, as long as the launch keeps about 8 rounds of the
  // chip's resident waves (18 per CU) busy, between 2 and 16 frames
  const int64_t units = n * g.bands * g.waves_per_frame;
  int64_t R = units / (8LL * kNumCU * 18);
  const int64_t q_max = (n + a.delta - 1) / a.delta;
  if (R > 16) R = 16;
  if (R > q_max) R = q_max;
  if (R < 2) R = 2;
  out->ap = q;
  out->chain_r = (int32_t)R;
  out->part_elems = n * g.bands * g.waves_per_frame;
  return true;
}

int launch_area_prev(const PrevFusePlan& fp, const uint8_t* frames, int64_t stride, int64_t n,
                     int32_t* sums, const DiffArgs& a, int64_t* part, hipStream_t stream) {
  if (n <= 0) return NSC_OK;
  const WaveGeom& g = fp.ap.wg;
  const int64_t q = (n + a.delta - 1) / a.delta;        // frames per residue (at most)
  const int64_t chains = (q + fp.chain_r - 1) / fp.chain_r * a.delta;
  const int64_t units = chains * g.bands * g.waves_per_frame;
  const int64_t wblocks = (units + g.waves_per_block - 1) / g.waves_per_block;
  if (wblocks > 0x7FFFFFFF) return fail(NSC_E_SHAPE, "too many frames in one call");
  if (g.chunk_bytes != 16 && g.chunk_bytes != 4)
    return fail(NSC_E_SHAPE, "the fused earlier-frame detector takes 16- or 4-byte lane chunks");
#define NSC_PREV_LAUNCH(CB, PK)                                                                  \
  hipLaunchKernelGGL((k_area_prev_wave<CB, PK, NSC_ROWS_BATCH>), dim3((unsigned)wblocks),        \
                     dim3(64 * g.waves_per_block), g.lds_bytes, stream, frames, stride, fp.ap.ay,   \
                     fp.ap.ax, g, n, a.delta, fp.chain_r, sums, part)
  if (g.chunk_bytes == 16) {
    if (fp.ap.packed) NSC_PREV_LAUNCH(16, true); else NSC_PREV_LAUNCH(16, false);
  } else {
    if (fp.ap.packed) NSC_PREV_LAUNCH(4, true); else NSC_PREV_LAUNCH(4, false);
  }
#undef NSC_PREV_LAUNCH
  NSC_CHECK_LAUNCH("k_area_prev_wave");
  return NSC_OK;
}

void area_prev_diff_args(const PrevFusePlan& fp, const int64_t* part, DiffArgs* a) {
  a->part = part;
  a->chain_r = fp.chain_r;
  a->part_bands = fp.ap.wg.bands;
  a->part_strips = fp.ap.wg.waves_per_frame;
}

bool area_detect_fused(const AreaPlan& p, const DiffArgs& a) {
  return p.wave && a.ref_mode == NSC_REF_FIXED && a.grid_h * a.grid_w == 1 && a.cams == nullptr &&
         a.metric >= NSC_METRIC_MSE && a.metric <= NSC_METRIC_PSNR;
}

int64_t area_detect_part_count(const AreaPlan& p, int64_t n) {
  return p.wave ? n * p.wg.bands * p.wg.waves_per_frame : 0;
}

int launch_area_detect_fixed(const AreaPlan& p, const uint8_t* frames, int64_t stride, int64_t n,
                             int32_t* sums, const DiffArgs& a, int64_t* part, hipStream_t stream) {
  if (n <= 0) return NSC_OK;
  if (!area_detect_fused(p, a)) return fail(NSC_E_SHAPE, "the fused fixed-reference detector does not apply");
  const WaveGeom& g = p.wg;
  const int64_t units = n * g.bands * g.waves_per_frame;
  const int64_t wblocks = (units + g.waves_per_block - 1) / g.waves_per_block;
  if (wblocks > 0x7FFFFFFF) return fail(NSC_E_SHAPE, "too many frames in one call");
#define NSC_FUSED_LAUNCH(CB, PK, M)                                                              \
  hipLaunchKernelGGL((k_area_sums_wave<CB, PK, CB == 32 ? NSC_ROWS_BATCH / 2 : NSC_ROWS_BATCH, M>), \
                     dim3((unsigned)wblocks), dim3(64 * g.waves_per_block), g.lds_bytes, stream,  \
                     frames, stride, p.ay, p.ax, g, g.bands, n, sums, a.ref_sums, part)
#define NSC_FUSED_CB(M)                                                                          \
  if (g.chunk_bytes == 32) {                                                                     \
    if (p.packed) NSC_FUSED_LAUNCH(32, true, M); else NSC_FUSED_LAUNCH(32, false, M);            \
  } else if (g.chunk_bytes == 16) {                                                              \
    if (p.packed) NSC_FUSED_LAUNCH(16, true, M); else NSC_FUSED_LAUNCH(16, false, M);            \
  } else {                                                                                       \
    if (p.packed) NSC_FUSED_LAUNCH(4, true, M); else NSC_FUSED_LAUNCH(4, false, M);              \
  }                                                                                              \
  NSC_CHECK_LAUNCH("k_area_sums_wave (fused detector)");                                         \
  hipLaunchKernelGGL((k_diff_fixed_finish<M>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0,  \
                     stream, a, (const int64_t*)part, (int32_t)(g.bands * g.waves_per_frame));   \
  NSC_CHECK_LAUNCH("k_diff_fixed_finish")
  switch (a.metric) {
    case NSC_METRIC_MSE:
      NSC_FUSED_CB(NSC_METRIC_MSE);
      break;
    case NSC_METRIC_SAD:
      NSC_FUSED_CB(NSC_METRIC_SAD);
      break;
    case NSC_METRIC_NRMSE:
      NSC_FUSED_CB(NSC_METRIC_NRMSE);
      break;
    default:
      NSC_FUSED_CB(NSC_METRIC_PSNR);
      break;
  }
#undef NSC_FUSED_CB
#undef NSC_FUSED_LAUNCH
  return NSC_OK;
}

}  // namespace nsc
