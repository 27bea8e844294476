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
#include <type_traits>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bc {

// Output columns per thread item.  Odd, so that the 64 lanes of a wave,
// reading consecutive 3-column groups of one table row, hit distinct banks.
constexpr int kQ = 3;

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return min(max(v, lo), hi); }

// Columns of padding on each side of a table row kept in LDS: left pads hold
// 0 (= the table's column 0), right pads repeat column W.  A run of kQ + 1
// consecutive table columns starting anywhere then reads correctly clamped
// values once its start is clamped to [-kPad, W].
constexpr int kPad = 3;

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

// Taps of the adjoint (mirrored) box as the backward pass uses them.  Each
// edge e is split as e = f + alpha with alpha in (0, 1], i.e. f = ceil(e) - 1:
// the same table lookups as the floor split (interpolation is continuous),
// but at an edge on a pixel boundary the table difference between the edge's
// two taps is the column (row) just below the edge.  In the adjoint the
// original box's right derivative (Section 3.1, Eq. 4) is that one-sided
// derivative from below, so the backward reads it straight from the taps.
__device__ __forceinline__ void edge_split_upper(double e, int lim, int& f, double& frac) {
  double fl = ceil(e) - 1.0;
  if (!(fl >= -(double)lim)) fl = -(double)lim;
  if (fl > (double)lim) fl = (double)lim;
  frac = e - fl;
  f = (int)fl;
}

__device__ __forceinline__ Taps<float> make_taps_adjoint(const float* p, int limx, int limy) {
  const double cx = -(double)p[0], cy = -(double)p[1];
  const double rx = (double)p[2], ry = (double)p[3];
  Taps<float> t;
  int fa, fb, fc, fd;
  double aa, ab, ac, ad;
  edge_split_upper(0.5 + cx - rx, limx, fa, aa);
  edge_split_upper(0.5 + cx + rx, limx, fb, ab);
  edge_split_upper(0.5 + cy - ry, limy, fc, ac);
  edge_split_upper(0.5 + cy + ry, limy, fd, ad);
  t.ox[0] = fa; t.ox[1] = fa + 1; t.ox[2] = fb; t.ox[3] = fb + 1;
  t.oy[0] = fc; t.oy[1] = fc + 1; t.oy[2] = fd; t.oy[3] = fd + 1;
  t.wx[0] = (float)(aa - 1.0); t.wx[1] = (float)(-aa);
  t.wx[2] = (float)(1.0 - ab); t.wx[3] = (float)ab;
  t.wy[0] = (float)(ac - 1.0); t.wy[1] = (float)(-ac);
  t.wy[2] = (float)(1.0 - ad); t.wy[3] = (float)ad;
  return t;
}

// Taps of a box whose corners are rounded to integers (the inference form of
// the Conclusions: once the boxes have converged the sampling points are
// rounded, and each corner is one table sample).  Each edge e (fp64) is
// rounded to floor(e + 1/2), ties up.  The adjoint (mirrored) box of the
// rounded box has the integer edges 1 - b, 1 - a, 1 - d, 1 - c.  Weights are
// those of an integer edge, (-1, 0) and (1, 0): the general 16-tap walk reads
// the same sums from these records as the 4-tap walk.
__device__ __forceinline__ Taps<float> make_taps_rounded(const float* p, bool adjoint, int limx, int limy) {
  const double cx = (double)p[0], cy = (double)p[1], rx = (double)p[2], ry = (double)p[3];
  auto rnd = [](double e, int lim) {
    double r = floor(e + 0.5);
    if (!(r >= -(double)lim)) r = -(double)lim;
    if (r > (double)lim) r = (double)lim;
    return (int)r;
  };
  int a = rnd(0.5 + cx - rx, limx), b = rnd(0.5 + cx + rx, limx);
  int c = rnd(0.5 + cy - ry, limy), d = rnd(0.5 + cy + ry, limy);
  if (adjoint) {
    const int a2 = 1 - b, b2 = 1 - a, c2 = 1 - d, d2 = 1 - c;
    a = a2; b = b2; c = c2; d = d2;
  }
  Taps<float> t;
  t.ox[0] = a; t.ox[1] = a + 1; t.ox[2] = b; t.ox[3] = b + 1;
  t.oy[0] = c; t.oy[1] = c + 1; t.oy[2] = d; t.oy[3] = d + 1;
  t.wx[0] = -1.f; t.wx[1] = 0.f; t.wx[2] = 1.f; t.wx[3] = 0.f;
  t.wy[0] = -1.f; t.wy[1] = 0.f; t.wy[2] = 1.f; t.wy[3] = 0.f;
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

// v clamped to [lo, hi] in one instruction (hi wave-uniform).
__device__ __forceinline__ int med3_i32(int v, int hi) {
  int r;
  asm("v_med3_i32 %0, %1, 0, %2" : "=v"(r) : "v"(v), "s"(hi));
  return r;
}

// Table accessors.  A walk addresses a table row by an unclamped row
// coordinate in the table's own units (row_coord(v) for table row v; one row
// further is + row_step()), and the two runs of columns it reads by
// cols(ba, bb) with ba = x0 + fa, bb = x0 + fb unclamped.  runs<N>(coord, c,
// sa, sb) returns S(clamp(v, 0, H), clamp(ba + k, 0, W)) and the same at bb,
// k in [0, N); N = kQ + 1 for interpolated edges, kQ for integer ones.
//
// LDS table, padded: S(u, v) at p[u * pitch + kPad + v], v in [-kPad, W+kPad];
// coordinates are byte offsets, a row is clamped once (v_med3) and each run
// is kQ + 1 consecutive words from one address.
template <typename T>
struct LdsTable {
  const T* p;
  int pitch, W, H;
  struct Cols { const char* a; const char* b; };  // first word of each run in table row 0
  __device__ __forceinline__ Cols cols(int ba, int bb) const {
    const char* base = reinterpret_cast<const char*>(p + kPad);
    return {base + clampi(ba, -kPad, W) * (int)sizeof(T), base + clampi(bb, -kPad, W) * (int)sizeof(T)};
  }
  __device__ __forceinline__ int row_step() const { return pitch * (int)sizeof(T); }
  __device__ __forceinline__ int row_coord(int v) const { return v * row_step(); }
  // One column run at a time (the split-box corner walks): col(x) a clamped
  // column, row(coord) a clamped row, run4 the 4 words from there.
  using Col = const char*;
  using Row = int;
  __device__ __forceinline__ Col col(int x) const {
    return reinterpret_cast<const char*>(p + kPad) + clampi(x, -kPad, W) * (int)sizeof(T);
  }
  __device__ __forceinline__ Row row(int coord) const { return med3_i32(coord, H * row_step()); }
  __device__ __forceinline__ void run4(Row r, Col c, T* v) const {
    const T* s = reinterpret_cast<const T*>(c + r);
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = s[k];
  }
  template <int N = kQ + 1>
  __device__ __forceinline__ void runs(int coord, const Cols& c, T* sa, T* sb) const {
    const int row = med3_i32(coord, H * row_step());
    const T* ra = reinterpret_cast<const T*>(c.a + row);
    const T* rb = reinterpret_cast<const T*>(c.b + row);
#pragma unroll
    for (int k = 0; k < N; ++k) { sa[k] = ra[k]; sb[k] = rb[k]; }
  }
};

// Table in HBM, (H+1) x (W+1), unpadded: row coordinates are row indices and
// every index is clamped.
template <typename T, bool kVec = false>
struct GlobalTable {
  const T* __restrict__ p;
  int pitch, W, H;
  struct Cols { int a, b; };
  __device__ __forceinline__ Cols cols(int ba, int bb) const { return {ba, bb}; }
  __device__ __forceinline__ int row_step() const { return 1; }
  __device__ __forceinline__ int row_coord(int v) const { return v; }
  using Col = int;
  using Row = const T*;
  __device__ __forceinline__ Col col(int x) const { return x; }
  __device__ __forceinline__ Row row(int coord) const { return p + (size_t)clampi(coord, 0, H) * pitch; }
  __device__ __forceinline__ void run4(Row r, Col c, T* v) const { run<4>(r, c, v); }
  template <int N = kQ + 1>
  __device__ __forceinline__ void runs(int coord, const Cols& c, T* sa, T* sb) const {
    const T* r = p + (size_t)clampi(coord, 0, H) * pitch;
    run<N>(r, c.a, sa);
    run<N>(r, c.b, sb);
  }
  // N consecutive words of row r from column j, clamped to [0, W]; with
  // kVec, one 16-byte load (4-byte aligned) when the whole run of 4 is
  // inside the row (the backward gather keeps the scalar loads: the wider
  // path would cost it registers it does not have).
  template <int N>
  __device__ __forceinline__ void run(const T* r, int j, T* s) const {
    typedef T vec4u __attribute__((ext_vector_type(4))) __attribute__((aligned(sizeof(T))));
    if (kVec && N == 4 && j >= 0 && j + 3 <= W) {
      const vec4u q = *reinterpret_cast<const vec4u*>(r + j);
      s[0] = q.x; s[1] = q.y; s[2] = q.z;
      if constexpr (N == 4) s[3] = q.w;
    } else {
#pragma unroll
      for (int k = 0; k < N; ++k) s[k] = r[clampi(j + k, 0, W)];
    }
  }
};

// w0*a + w1*b + w2*c + w3*d in a fixed rounding sequence (one product, then
// three fused multiply-adds in term order), so that every kernel instance
// evaluating the same sum gets the same bits whatever the compiler would
// contract; exact for integers.
template <typename T>
__device__ __forceinline__ T wsum4(T w0, T a, T w1, T b, T w2, T c, T w3, T d) {
  if constexpr (std::is_same<T, float>::value) return fmaf(w3, d, fmaf(w2, c, fmaf(w1, b, w0 * a)));
  else return w0 * a + w1 * b + w2 * c + w3 * d;
}

// o + mu * e, the mean offset's contribution added back (fused for floats,
// for the same reason as wsum4).
template <typename T>
__device__ __forceinline__ T add_offset(T o, float mu, float e) {
  if constexpr (std::is_same<T, float>::value) return fmaf(mu, e, o);
  else return o + (T)(mu * e);
}

// The x-interpolated table row for kQ consecutive outputs x0 + q: for q in
// [0, kQ),  U[q] = sum_k wx[k] * S(v, clamp(x0 + q + ox[k])).
template <typename T, typename Src>
__device__ __forceinline__ void table_row(const Src& S, int coord, const typename Src::Cols& c, const Taps<T>& tp,
                                          T* U) {
  T sa[kQ + 1], sb[kQ + 1];
  S.runs(coord, c, sa, sb);
#pragma unroll
  for (int q = 0; q < kQ; ++q)
    U[q] = wsum4(tp.wx[0], sa[q], tp.wx[1], sa[q + 1], tp.wx[2], sb[q], tp.wx[3], sb[q + 1]);
}

// Same row for adjoint taps, also returning the column differences at the
// two x edges (the table differences across each edge column).  Adjoint x
// weights are (alpha - 1, -alpha) and (1 - beta, beta), so the interpolated
// row is (sb - sa) - alpha * DA + beta * DB.
template <typename Src>
__device__ __forceinline__ void table_row_grad(const Src& S, int coord, const typename Src::Cols& c,
                                               const Taps<float>& tp, float* U, float* DA, float* DB) {
  float sa[kQ + 1], sb[kQ + 1];
  S.runs(coord, c, sa, sb);
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    DA[q] = sa[q + 1] - sa[q];
    DB[q] = sb[q + 1] - sb[q];
    U[q] = fmaf(tp.wx[3], DB[q], fmaf(tp.wx[1], DA[q], sb[q] - sa[q]));
  }
}

// Taps of one box from its record in the table box_prep writes (16 words:
// floors of a, b, c, d; x weights; y weights).  Called with a wave-uniform
// record, so the record comes in through scalar loads.  The floors are
// clamped to [-(n+1), n+1] for a map of extent n, which leaves every clamped
// tap index unchanged and keeps row and column arithmetic in range.
__device__ __forceinline__ Taps<float> load_taps(const int* __restrict__ rec, int W, int H) {
  const float* f = reinterpret_cast<const float*>(rec);
  Taps<float> t;
  const int fa = clampi(rec[0], -(W + 1), W + 1), fb = clampi(rec[1], -(W + 1), W + 1);
  const int fc = clampi(rec[2], -(H + 1), H + 1), fd = clampi(rec[3], -(H + 1), H + 1);
  t.ox[0] = fa; t.ox[1] = fa + 1; t.ox[2] = fb; t.ox[3] = fb + 1;
  t.oy[0] = fc; t.oy[1] = fc + 1; t.oy[2] = fd; t.oy[3] = fd + 1;
#pragma unroll
  for (int k = 0; k < 4; ++k) { t.wx[k] = f[4 + k]; t.wy[k] = f[8 + k]; }
  return t;
}

// Integer maps: corners are floored (the fractions are ignored), so the box is
// the plain sum of Eq. 1 and only the four corner taps have weight.
__device__ __forceinline__ Taps<int> int_taps(const Taps<float>& f) {
  Taps<int> t;
#pragma unroll
  for (int k = 0; k < 4; ++k) { t.ox[k] = f.ox[k]; t.oy[k] = f.oy[k]; }
  t.wx[0] = -1; t.wx[1] = 0; t.wx[2] = 1; t.wx[3] = 0;
  t.wy[0] = -1; t.wy[1] = 0; t.wy[2] = 1; t.wy[3] = 0;
  return t;
}

// Sum over the 16 lanes of each DPP row, in every lane of the row: pair,
// quad, half-row and row steps through data-parallel lane moves (no LDS).
__device__ __forceinline__ float row16_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));  // row_half_mirror
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));  // row_mirror
  return v;
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

// Wave-level exclusive prefix sum: the inclusive sum of the lane before (0 in
// lane 0), so a lane's value never enters its own prefix (a NaN or infinity in
// it leaves the prefix exact).
template <typename T>
__device__ __forceinline__ T wave_excl_scan(T v, int lane) {
  const T incl = wave_incl_scan(v, lane);
  const T prev = __shfl_up(incl, 1, 64);
  return lane ? prev : (T)0;
}

}  // namespace bc
