// Shared device code of the box-convolution library (gfx950).
//
// Geometry (Section 3.1, Eq. 2-3): for output pixel x (cell [x, x+1)) a box
// with centre offset cx and half-width rx covers [x + a, x + b) with
// a = 1/2 + cx - rx and b = 1/2 + cx + rx (the paper's x_l = a, x_h = b - 1);
// likewise c, d in y.  The exclusive table S[u][v] = sum_{i<u, j<v} I[i][j]
// is sampled at the four corners by bilinear interpolation (Eq. 3), indices
// clamped to [0,H] x [0,W] (zero padding).  Because the fractions of the
// corners do not change under integer shifts (Section 3.1, after Eq. 4), each
// box reduces to 4 column offsets {fa, fa+1, fb, fb+1} and 4 row offsets
// {fc, fc+1, fd, fd+1} with separable signed weights; the 16 tap weights of
// the paper are the products wy[r] * wx[k].
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bc {

// Output columns per thread item.  Odd, so that the 64 lanes of a wave,
// reading consecutive 3-column groups of one table row, hit distinct banks.
constexpr int kQ = 3;
// Output rows per thread item (the length of one sliding-window walk).
constexpr int kSeg = 16;

__device__ __forceinline__ int clampi(int v, int lo, int hi) {
  return v < lo ? lo : (v > hi ? hi : v);
}

// One box, ready to evaluate on a map: tap offsets and separable weights.
template <typename T>
struct Taps {
  int ox[4];  // column offsets  fa, fa+1, fb, fb+1
  int oy[4];  // row offsets     fc, fc+1, fd, fd+1
  T wx[4];    // -(1-alpha_a), -alpha_a, 1-alpha_b, alpha_b
  T wy[4];    // -(1-beta_c),  -beta_c,  1-beta_d,  beta_d
};

// Floor and fraction of one edge, in fp64 (the edge is exact in fp64 for fp32
// parameters).  The floor is clamped to [-lim, lim]: with lim = n + 1 for a
// map of extent n every clamped tap index is unchanged, and it keeps absurd or
// non-finite parameters from overflowing the integer conversion.
__device__ __forceinline__ void edge_split(double e, int lim, int& f, double& frac) {
  double fl = floor(e);
  frac = e - fl;
  if (!(fl >= -(double)lim)) fl = -(double)lim;
  if (fl > (double)lim) fl = (double)lim;
  f = (int)fl;
}

// Builds the taps of box (cx, cy, rx, ry); `mirror` negates the centre offset,
// which gives the box whose correlation is the transpose of this one's.
__device__ __forceinline__ Taps<float> make_taps_f32(const float* p, bool mirror, int limx, int limy) {
  const double cx = mirror ? -(double)p[0] : (double)p[0];
  const double cy = mirror ? -(double)p[1] : (double)p[1];
  const double rx = (double)p[2], ry = (double)p[3];
  Taps<float> t;
  int fa, fb, fc, fd;
  double aa, ab, ac, ad;
  edge_split(0.5 + cx - rx, limx, fa, aa);
  edge_split(0.5 + cx + rx, limx, fb, ab);
  edge_split(0.5 + cy - ry, limy, fc, ac);
  edge_split(0.5 + cy + ry, limy, fd, ad);
  t.ox[0] = fa; t.ox[1] = fa + 1; t.ox[2] = fb; t.ox[3] = fb + 1;
  t.oy[0] = fc; t.oy[1] = fc + 1; t.oy[2] = fd; t.oy[3] = fd + 1;
  t.wx[0] = (float)(aa - 1.0); t.wx[1] = (float)(-aa);
  t.wx[2] = (float)(1.0 - ab); t.wx[3] = (float)ab;
  t.wy[0] = (float)(ac - 1.0); t.wy[1] = (float)(-ac);
  t.wy[2] = (float)(1.0 - ad); t.wy[3] = (float)ad;
  return t;
}

// Integer maps: corners are floored (the fractions are ignored), so the box is
// the plain sum of Eq. 1 and only the four corner taps have weight.
__device__ __forceinline__ Taps<int> make_taps_i32(const float* p, int limx, int limy) {
  Taps<float> f = make_taps_f32(p, false, limx, limy);
  Taps<int> t;
  for (int k = 0; k < 4; ++k) { t.ox[k] = f.ox[k]; t.oy[k] = f.oy[k]; }
  t.wx[0] = -1; t.wx[1] = 0; t.wx[2] = 1; t.wx[3] = 0;
  t.wy[0] = -1; t.wy[1] = 0; t.wy[2] = 1; t.wy[3] = 0;
  return t;
}

// fp32 -> bf16, round to nearest even; NaN stays NaN (quiet).  Branch-free
// (a select), so that it never splits a wave.
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rounded = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  const uint32_t quiet = (u >> 16) | 0x0040u;
  return (uint16_t)(((u & 0x7fffffffu) > 0x7f800000u) ? quiet : rounded);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// Table accessors.  Indices passed in are already clamped.
template <typename T>
struct LdsTable {
  const T* p;
  int pitch;
  __device__ __forceinline__ T operator()(int u, int v) const { return p[u * pitch + v]; }
};

template <typename T>
struct GlobalTable {
  const T* __restrict__ p;
  int pitch;
  __device__ __forceinline__ T operator()(int u, int v) const { return p[(size_t)u * pitch + v]; }
};

// The x-interpolated table row for kQ consecutive outputs: for q in [0,kQ)
//   U[q] = sum_k wx[k] * S(u, clamp(x0 + q + ox[k]))
// ca[k] = clamp(x0 + fa + k), cb[k] = clamp(x0 + fb + k), k in [0, kQ].
template <typename T, typename Src>
__device__ __forceinline__ void table_row(const Src& S, int u, const int* ca, const int* cb,
                                          const Taps<T>& tp, T* U) {
  T sa[kQ + 1], sb[kQ + 1];
#pragma unroll
  for (int k = 0; k <= kQ; ++k) { sa[k] = S(u, ca[k]); sb[k] = S(u, cb[k]); }
#pragma unroll
  for (int q = 0; q < kQ; ++q)
    U[q] = tp.wx[0] * sa[q] + tp.wx[1] * sa[q + 1] + tp.wx[2] * sb[q] + tp.wx[3] * sb[q + 1];
}

// Same row, also returning the column differences at the two x edges
// (the edge-column prefix integrals used by the box-parameter gradient).
template <typename Src>
__device__ __forceinline__ void table_row_grad(const Src& S, int u, const int* ca, const int* cb,
                                               const Taps<float>& tp, float* U, float* DA, float* DB) {
  float sa[kQ + 1], sb[kQ + 1];
#pragma unroll
  for (int k = 0; k <= kQ; ++k) { sa[k] = S(u, ca[k]); sb[k] = S(u, cb[k]); }
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    U[q] = tp.wx[0] * sa[q] + tp.wx[1] * sa[q + 1] + tp.wx[2] * sb[q] + tp.wx[3] * sb[q + 1];
    DA[q] = sa[q + 1] - sa[q];
    DB[q] = sb[q + 1] - sb[q];
  }
}

template <typename T>
__device__ __forceinline__ void column_indices(const Taps<T>& tp, int x0, int W, int* ca, int* cb) {
#pragma unroll
  for (int k = 0; k <= kQ; ++k) {
    ca[k] = clampi(x0 + tp.ox[0] + k, 0, W);
    cb[k] = clampi(x0 + tp.ox[2] + k, 0, W);
  }
}

// Box evaluation for one item: kQ columns starting at x0, rows [y0, y1).
// Each step reads two new table rows (one per y edge) and reuses the two
// from the step before.  `emit(y, o)` receives the kQ outputs of row y.
// With `offset`, the table holds the map minus mu and mu * (clipped box area)
// is added back; the clipped area is the same tap combination applied to the
// clamped coordinates (the table of a constant image is mu * u * v).
template <typename T, bool kOffset, typename Src, typename Emit>
__device__ __forceinline__ void box_item(const Src& S, const Taps<T>& tp, int H, int W,
                                         int x0, int y0, int y1, float mu, Emit emit) {
  int ca[kQ + 1], cb[kQ + 1];
  column_indices(tp, x0, W, ca, cb);
  T uc[kQ], ud[kQ];
  table_row(S, clampi(y0 + tp.oy[0], 0, H), ca, cb, tp, uc);
  table_row(S, clampi(y0 + tp.oy[2], 0, H), ca, cb, tp, ud);
  float ex[kQ];
  if (kOffset) {
#pragma unroll
    for (int q = 0; q < kQ; ++q)
      ex[q] = (float)tp.wx[0] * (float)ca[q] + (float)tp.wx[1] * (float)ca[q + 1] +
              (float)tp.wx[2] * (float)cb[q] + (float)tp.wx[3] * (float)cb[q + 1];
  }
  for (int y = y0; y < y1; ++y) {
    T uc1[kQ], ud1[kQ];
    table_row(S, clampi(y + tp.oy[1], 0, H), ca, cb, tp, uc1);
    table_row(S, clampi(y + tp.oy[3], 0, H), ca, cb, tp, ud1);
    T o[kQ];
#pragma unroll
    for (int q = 0; q < kQ; ++q)
      o[q] = tp.wy[0] * uc[q] + tp.wy[1] * uc1[q] + tp.wy[2] * ud[q] + tp.wy[3] * ud1[q];
    if (kOffset) {
      const float ey = (float)tp.wy[0] * (float)clampi(y + tp.oy[0], 0, H) +
                       (float)tp.wy[1] * (float)clampi(y + tp.oy[1], 0, H) +
                       (float)tp.wy[2] * (float)clampi(y + tp.oy[2], 0, H) +
                       (float)tp.wy[3] * (float)clampi(y + tp.oy[3], 0, H);
#pragma unroll
      for (int q = 0; q < kQ; ++q) o[q] = o[q] + (T)(mu * (ex[q] * ey));
    }
    emit(y, o);
#pragma unroll
    for (int q = 0; q < kQ; ++q) { uc[q] = uc1[q]; ud[q] = ud1[q]; }
  }
}

// Wave-level sum (wave64), result valid in every lane.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Wave-level inclusive prefix sum over the 64 lanes.
template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    T t = __shfl_up(v, off, 64);
    if (lane >= off) v += t;
  }
  return v;
}

}  // namespace bc
