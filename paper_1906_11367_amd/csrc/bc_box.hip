// Box filter kernels: per-box precomputation, summed-area tables, forward
// evaluation and backward (input and box-parameter gradients).  gfx950, wave64.
#include "bc_common.hpp"
#include "bc_internal.hpp"

#include <type_traits>

namespace bc {

// ---------------------------------------------------------------------------
// Helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lds_pitch_dev(int W) { return (W + 7) | 1; }

template <typename OutT, typename T> __device__ __forceinline__ OutT convert_out(T v);
template <> __device__ __forceinline__ float convert_out<float, float>(float v) { return v; }
template <> __device__ __forceinline__ int convert_out<int, int>(int v) { return v; }
template <> __device__ __forceinline__ uint16_t convert_out<uint16_t, float>(float v) {
  return __builtin_bit_cast(uint16_t, (__bf16)v);  // round to nearest even (v_cvt_pk_bf16_f32)
}

// Grid-to-work mapping that keeps consecutive logical blocks on one XCD.
// Blocks are dispatched to the 8 XCDs round-robin by block index; logical
// block L = xcd * (grid/8) + slot gives each XCD one contiguous range of
// logical blocks, so all blocks reading one map's table share that XCD's L2.
// The grid is padded to a multiple of 8; logical ids >= total exit.
__device__ __forceinline__ int xcd_remap(int bid, int grid) {
  const int per = grid >> 3;
  return (bid & 7) * per + (bid >> 3);
}
inline int pad8(int n) { return (n + 7) & ~7; }

// Mean of one map, fp32, fixed summation order for a given block size.
__device__ float block_mean(const float* __restrict__ src, int n, float* red) {
  float s = 0.f;
  for (int i = threadIdx.x; i < n; i += blockDim.x) s += src[i];
  s = wave_sum(s);
  const int wave = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
  if ((threadIdx.x & 63) == 0) red[wave] = s;
  __syncthreads();
  float tot = 0.f;
  for (int w = 0; w < nw; ++w) tot += red[w];
  __syncthreads();
  return tot / (float)n;
}

// 16-byte vector of the map element type.
template <typename T> struct Vec4;
template <> struct Vec4<float> { using type = float4; };
template <> struct Vec4<int> { using type = int4; };

// Zero row 0 and columns -kPad..0 of every row of a padded LDS table.
template <typename T>
__device__ __forceinline__ void table_zero_edges(T* S, int H, int pitch) {
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int v = tid; v < pitch; v += nt) S[v] = (T)0;
  for (int k = tid; k < H * (kPad + 1); k += nt) {
    const int u = 1 + k / (kPad + 1);
    S[u * pitch + k - (u - 1) * (kPad + 1)] = (T)0;
  }
}

// Row pass of a padded LDS table whose interior holds column prefix sums:
// lanes own rows, reading kScan elements ahead before writing, so that a
// lane's LDS reads overlap; also fills the right padding.
template <typename T>
__device__ __forceinline__ void table_row_pass(T* S, int H, int W, int pitch) {
  constexpr int kScan = 16;
  T* R = S + kPad;
  for (int u = threadIdx.x + 1; u <= H; u += blockDim.x) {
    T* row = R + u * pitch;
    T run = (T)0;
    int v = 1;
    for (; v + kScan - 1 <= W; v += kScan) {
      T r[kScan];
#pragma unroll
      for (int k = 0; k < kScan; ++k) r[k] = row[v + k];
#pragma unroll
      for (int k = 0; k < kScan; ++k) {
        run += r[k];
        row[v + k] = run;
      }
    }
    for (; v <= W; ++v) {
      run += row[v];
      row[v] = run;
    }
#pragma unroll
    for (int k = 1; k <= kPad; ++k) row[W + k] = run;
  }
}

// Column pass (lanes own columns) and row pass of a padded LDS table whose
// interior holds the map, each reading kScan elements ahead before it writes.
template <typename T>
__device__ __forceinline__ void table_scans(T* S, int H, int W, int pitch) {
  constexpr int kScan = 16;
  const int tid = threadIdx.x, nt = blockDim.x;
  T* R = S + kPad;
  for (int v = tid + 1; v <= W; v += nt) {
    T run = (T)0;
    int u = 1;
    for (; u + kScan - 1 <= H; u += kScan) {
      T r[kScan];
#pragma unroll
      for (int k = 0; k < kScan; ++k) r[k] = R[(u + k) * pitch + v];
#pragma unroll
      for (int k = 0; k < kScan; ++k) {
        run += r[k];
        R[(u + k) * pitch + v] = run;
      }
    }
    for (; u <= H; ++u) {
      run += R[u * pitch + v];
      R[u * pitch + v] = run;
    }
  }
  __syncthreads();
  table_row_pass(S, H, W, pitch);
  __syncthreads();
}

// Map loads that stream (each map is read once per call) are non-temporal:
// they leave the caches to the outputs the next call reads (the box
// forward's filtered maps stay cached for the mix; pose-layer step 0.627 ->
// 0.614 ms).
template <typename T>
__device__ __forceinline__ typename Vec4<T>::type load_stream4(const typename Vec4<T>::type* p) {
  typedef T v4 __attribute__((ext_vector_type(4)));
  const v4 t = __builtin_nontemporal_load(reinterpret_cast<const v4*>(p));
  typename Vec4<T>::type r;
  r.x = t.x; r.y = t.y; r.z = t.z; r.w = t.w;
  return r;
}

// Exclusive table of one H x W map in LDS, padded (LdsTable): S(u, v) at
// S[u * pitch + kPad + v].  The map is first copied into the table's interior
// with every thread issuing 16-byte loads in batches (the loads of a batch are
// all in flight together; out-of-range slots re-read the last vector and are
// not stored, so no lane branches around a load).  Then a column pass (lanes
// own columns) and the row pass, each reading kScan elements ahead before it
// writes.  With `sub`, mu is subtracted from the tabulated values.
template <typename T, bool kSkip = false>
__device__ void build_table_lds(const T* __restrict__ src, T* S, int H, int W, int pitch, float mu, bool sub) {
  using V = typename Vec4<T>::type;
  constexpr int kBatch = 8;
  const int tid = threadIdx.x, nt = blockDim.x;
  T* R = S + kPad;
  table_zero_edges(S, H, pitch);
  // Slot k of this thread is element (vector) tid + k * nt; its row and
  // column advance by the same (nt / width, nt % width) every slot, so only
  // the first position takes a division.
  const int n = H * W;
  if ((W & 3) == 0 && ((uintptr_t)src & 15) == 0) {
    const int n4 = n >> 2, W4 = W >> 2;
    const int di = nt / W4, dj = nt - di * W4;
    int j = tid % W4;
    int o = (tid / W4 + 1) * pitch + 4 * j + 1;  // table offset of the slot's first element
    const int step = di * pitch + 4 * dj, wrap = pitch - W;
    const V* s4 = reinterpret_cast<const V*>(src);
    for (int base = 0; base < n4; base += nt * kBatch) {
      // kSkip: slots past the map for every thread of the block (the tail
      // of the last batch) issue nothing, a block-uniform test (the
      // backward keeps the unconditional form, which fits its registers)
      V q[kBatch];
#pragma unroll
      for (int b = 0; b < kBatch; ++b)
        if (!kSkip || base + b * nt < n4) q[b] = load_stream4<T>(s4 + min(base + b * nt + tid, n4 - 1));
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        if (kSkip && base + b * nt >= n4) break;
        if (tid < n4 - base - b * nt) {
          const T w4[4] = {(T)q[b].x, (T)q[b].y, (T)q[b].z, (T)q[b].w};
#pragma unroll
          for (int t = 0; t < 4; ++t) R[o + t] = sub ? (T)((float)w4[t] - mu) : w4[t];
        }
        o += step;
        j += dj;
        if (j >= W4) { j -= W4; o += wrap; }
      }
    }
  } else {
    const int di = nt / W, dj = nt - di * W;
    int i = tid / W, j = tid - i * W;
    for (int k = tid; k < n; k += nt) {
      const T v = __builtin_nontemporal_load(src + k);
      R[(i + 1) * pitch + j + 1] = sub ? (T)((float)v - mu) : v;
      i += di;
      j += dj;
      if (j >= W) { j -= W; ++i; }
    }
  }
  __syncthreads();
  table_scans(S, H, W, pitch);
}

// Table of a zero-upsampled fp32 map (the transpose of sampling every s-th
// pixel): src (Ho x Wo) placed at (s*i, s*j) of an H x W map, zeros
// elsewhere; s * (Ho - 1) < H and s * (Wo - 1) < W.  Each source value
// writes its whole s x s block of the interior (the value at the block's
// corner, zeros elsewhere), so every interior element is written once; the
// loads of a batch are in flight together.
__device__ void build_table_lds_up(const float* __restrict__ src, float* S, int H, int W, int pitch, int s, int Ho,
                                   int Wo) {
  constexpr int kB = 8;
  const int tid = threadIdx.x, nt = blockDim.x, n = Ho * Wo;
  float* R = S + kPad;
  table_zero_edges(S, H, pitch);
  for (int base = 0; base < n; base += nt * kB) {
    float g[kB];
#pragma unroll
    for (int b = 0; b < kB; ++b) g[b] = src[min(base + b * nt + tid, n - 1)];
#pragma unroll
    for (int b = 0; b < kB; ++b) {
      const int k = base + b * nt + tid;
      if (k < n) {
        const int i = k / Wo, j = k - i * Wo;
        const int u1 = min(s * i + s, H), v1 = min(s * j + s, W);
        for (int u = s * i; u < u1; ++u) {
          float* row = R + (u + 1) * pitch + 1;
          for (int v = s * j; v < v1; ++v) row[v] = (u == s * i && v == s * j) ? g[b] : 0.f;
        }
      }
    }
  }
  __syncthreads();
  table_scans(S, H, W, pitch);
}

// ---------------------------------------------------------------------------
// Walks with compile-time segment length (registers indexed statically)
// ---------------------------------------------------------------------------

// The columns of a Q-column item (Q a multiple of kQ) as Q / kQ groups of
// kQ, each with its own clamped run start: the LDS table's padding (kPad = 3
// columns a side) covers runs of kQ + 1 words only, so a wider item reads
// its runs group by group.
template <int Q, typename Src>
struct ColGroups {
  static_assert(Q % kQ == 0, "items are whole groups of kQ columns");
  static constexpr int NG = Q / kQ;
  typename Src::Cols c[NG];
  __device__ __forceinline__ ColGroups(const Src& S, int ba, int bb) {
#pragma unroll
    for (int g = 0; g < NG; ++g) c[g] = S.cols(ba + g * kQ, bb + g * kQ);
  }
  // x-interpolated row (table_row) for all Q columns
  template <typename T>
  __device__ __forceinline__ void row(const Src& S, int coord, const Taps<T>& tp, T* U) const {
#pragma unroll
    for (int g = 0; g < NG; ++g) table_row(S, coord, c[g], tp, U + g * kQ);
  }
  // the kQ-word runs at both x edges, for all Q columns
  template <typename T>
  __device__ __forceinline__ void runs(const Src& S, int coord, T* sa, T* sb) const {
#pragma unroll
    for (int g = 0; g < NG; ++g) S.template runs<kQ>(coord, c[g], sa + g * kQ, sb + g * kQ);
  }
};

// Forward walk: emit.put<kFull>(s, o) for s in [0, SEG) with y0 + s < y1.
// kFull: the item is known to be whole (y1 = y0 + SEG, x0 + kQ <= W), so no
// step or column is guarded and the unrolled window needs no register copies.
// Each step reads two new table rows (one per y edge) and reuses the two from
// the step before.  With kOffset the table holds the map minus mu, and
// mu * (clipped box area) is added back: the clipped area is the same tap
// combination applied to the clamped coordinates (the table of a constant
// image is mu * u * v).
template <int SEG, typename T, bool kOffset, bool kFull, int Q = kQ, typename Src, typename Emit>
__device__ __forceinline__ void box_walk(const Src& S, const Taps<T>& tp, int H, int W, int x0,
                                         int y0, int y1, float mu, Emit& emit) {
  const int ba = x0 + tp.ox[0], bb = x0 + tp.ox[2];
  const ColGroups<Q, Src> cl(S, ba, bb);
  const int st = S.row_step();
  const int rc = S.row_coord(y0 + tp.oy[0]), rd = S.row_coord(y0 + tp.oy[2]);
  T uc[Q], ud[Q];
  cl.row(S, rc, tp, uc);
  cl.row(S, rd, tp, ud);
  float ex[Q];
  if (kOffset) {
#pragma unroll
    for (int q = 0; q < Q; ++q)
      ex[q] = wsum4((float)tp.wx[0], (float)clampi(ba + q, 0, W), (float)tp.wx[1], (float)clampi(ba + q + 1, 0, W),
                    (float)tp.wx[2], (float)clampi(bb + q, 0, W), (float)tp.wx[3], (float)clampi(bb + q + 1, 0, W));
  }
#pragma unroll
  for (int s = 0; s < SEG; ++s) {
    const int y = y0 + s;
    if (kFull || y < y1) {
      T uc1[Q], ud1[Q];
      cl.row(S, rc + (s + 1) * st, tp, uc1);
      cl.row(S, rd + (s + 1) * st, tp, ud1);
      T o[Q];
#pragma unroll
      for (int q = 0; q < Q; ++q)
        o[q] = wsum4(tp.wy[0], uc[q], tp.wy[1], uc1[q], tp.wy[2], ud[q], tp.wy[3], ud1[q]);
      if (kOffset) {
        const float ey = wsum4((float)tp.wy[0], (float)clampi(y + tp.oy[0], 0, H), (float)tp.wy[1],
                               (float)clampi(y + tp.oy[1], 0, H), (float)tp.wy[2], (float)clampi(y + tp.oy[2], 0, H),
                               (float)tp.wy[3], (float)clampi(y + tp.oy[3], 0, H));
#pragma unroll
        for (int q = 0; q < Q; ++q) o[q] = add_offset(o[q], mu, ex[q] * ey);
      }
      emit.template put<kFull>(s, o);
#pragma unroll
      for (int q = 0; q < Q; ++q) { uc[q] = uc1[q]; ud[q] = ud1[q]; }
    }
  }
}

// Walk for boxes with integer corners (make_taps_rounded records): each
// output is Eq. 2's four-corner difference with no interpolation, so per
// output row the walk reads one table row per y edge, each a run of kQ
// columns at both x edges:  o = (S(y+d, x+b) - S(y+d, x+a)) - (S(y+c, x+b) -
// S(y+c, x+a)).  emit.put<kFull>(s, o) for s in [0, SEG) with y0 + s < y1.
// With kOffset the table holds the map minus mu, and mu * (clipped area) is
// added back.
template <int SEG, typename T, bool kOffset, bool kFull, int Q = kQ, typename Src, typename Emit>
__device__ __forceinline__ void box_walk_int(const Src& S, const Taps<T>& tp, int H, int W, int x0, int y0,
                                             int y1, float mu, Emit& emit) {
  const int ba = x0 + tp.ox[0], bb = x0 + tp.ox[2];
  const ColGroups<Q, Src> cl(S, ba, bb);
  const int st = S.row_step();
  const int rc = S.row_coord(y0 + tp.oy[0]), rd = S.row_coord(y0 + tp.oy[2]);
  float ex[Q];
  if (kOffset) {
#pragma unroll
    for (int q = 0; q < Q; ++q) ex[q] = (float)(clampi(bb + q, 0, W) - clampi(ba + q, 0, W));
  }
#pragma unroll
  for (int s = 0; s < SEG; ++s) {
    const int y = y0 + s;
    if (kFull || y < y1) {
      T ca[Q], cb[Q], da[Q], db[Q];
      cl.runs(S, rc + s * st, ca, cb);
      cl.runs(S, rd + s * st, da, db);
      T o[Q];
#pragma unroll
      for (int q = 0; q < Q; ++q) o[q] = (db[q] - da[q]) - (cb[q] - ca[q]);
      if (kOffset) {
        const float ey = (float)(clampi(y + tp.oy[2], 0, H) - clampi(y + tp.oy[0], 0, H));
#pragma unroll
        for (int q = 0; q < Q; ++q) o[q] = add_offset(o[q], mu, ex[q] * ey);
      }
      emit.template put<kFull>(s, o);
    }
  }
}

// Strided forward walk of one item: output column j (input column x = s*j)
// and output rows i0 .. i1-1 (input rows s*i).  Consecutive outputs are s
// rows apart and share no table rows, so each output reads its own: two rows
// per y edge (one with integer corners), runs of two columns (one) at both x
// edges -- the 16 (4) samples of Eq. 2-3.  emit.put(k, o) for output row
// i0 + k.  With kOffset the table holds the map minus mu, and mu * (clipped
// area) is added back.
template <int SEGS, typename T, bool kOffset, bool kInt, typename Src, typename Emit>
__device__ __forceinline__ void box_walk_strided(const Src& S, const Taps<T>& tp, int H, int W, int x, int i0,
                                                 int i1, int s, float mu, Emit& emit) {
  const int ba = x + tp.ox[0], bb = x + tp.ox[2];
  const typename Src::Cols cl = S.cols(ba, bb);
  const int st = S.row_step();
  float ex = 0.f;
  if (kOffset) {
    ex = kInt ? (float)(clampi(bb, 0, W) - clampi(ba, 0, W))
              : wsum4((float)tp.wx[0], (float)clampi(ba, 0, W), (float)tp.wx[1], (float)clampi(ba + 1, 0, W),
                      (float)tp.wx[2], (float)clampi(bb, 0, W), (float)tp.wx[3], (float)clampi(bb + 1, 0, W));
  }
#pragma unroll
  for (int k = 0; k < SEGS; ++k) {
    const int i = i0 + k;
    if (i < i1) {
      const int y = s * i;
      const int rc = S.row_coord(y + tp.oy[0]), rd = S.row_coord(y + tp.oy[2]);
      T o;
      if constexpr (kInt) {
        T ca[1], cb[1], da[1], db[1];
        S.template runs<1>(rc, cl, ca, cb);
        S.template runs<1>(rd, cl, da, db);
        o = (db[0] - da[0]) - (cb[0] - ca[0]);
      } else {
        T u[4];
        const int rows[4] = {rc, rc + st, rd, rd + st};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          T sa[2], sb[2];
          S.template runs<2>(rows[r], cl, sa, sb);
          u[r] = wsum4(tp.wx[0], sa[0], tp.wx[1], sa[1], tp.wx[2], sb[0], tp.wx[3], sb[1]);
        }
        o = wsum4(tp.wy[0], u[0], tp.wy[1], u[1], tp.wy[2], u[2], tp.wy[3], u[3]);
      }
      if (kOffset) {
        const float ey = kInt ? (float)(clampi(y + tp.oy[2], 0, H) - clampi(y + tp.oy[0], 0, H))
                              : wsum4((float)tp.wy[0], (float)clampi(y + tp.oy[0], 0, H), (float)tp.wy[1],
                                      (float)clampi(y + tp.oy[1], 0, H), (float)tp.wy[2],
                                      (float)clampi(y + tp.oy[2], 0, H), (float)tp.wy[3],
                                      (float)clampi(y + tp.oy[3], 0, H));
        o = add_offset(o, mu, ex * ey);
      }
      emit.put(k, o);
    }
  }
}

// Emitter of one strided output column: output row i0 + k at plane offset
// off0 + k * Wo (off0 = i0 * Wo + j).
template <typename OutT, typename T>
struct StoreCol {
  OutT* out;
  int Wo, off0;
  __device__ __forceinline__ void put(int k, T o) { out[(unsigned)(off0 + k * Wo)] = convert_out<OutT, T>(o); }
};

// Forward walk of one item: integer-corner or interpolated.
template <int SEG, typename T, bool kOffset, bool kFull, bool kInt, int Q = kQ, typename Src, typename Emit>
__device__ __forceinline__ void walk_fwd(const Src& S, const Taps<T>& tp, int H, int W, int x0, int y0, int y1,
                                         float mu, Emit& emit) {
  if constexpr (kInt) box_walk_int<SEG, T, kOffset, kFull, Q>(S, tp, H, W, x0, y0, y1, mu, emit);
  else box_walk<SEG, T, kOffset, kFull, Q>(S, tp, H, W, x0, y0, y1, mu, emit);
}

// Emitter that adds an item's outputs to its register accumulator (the
// input gradient, summed over boxes).
template <int SEG>
struct AccRows {
  float (&acc)[SEG][kQ];
  template <bool kFull>
  __device__ __forceinline__ void put(int s, const float* o) {
#pragma unroll
    for (int q = 0; q < kQ; ++q) acc[s][q] += o[q];
  }
};

// Backward walk over one item on the table of one upstream-gradient map G,
// with the adjoint taps of the box.  For each input pixel (y, x) =
// (y0 + s, x0 + q):
//   acc[s][q] += D(y, x), the adjoint box sum of G (the input gradient);
// and, since <G, box(I)> = <I, D> for every placement of the box, the four
// edge gradients of the original box follow from the derivatives of D with
// respect to the adjoint's edges, weighted by the map value v[s][q] = I(y, x)
// (0 outside the map).  The adjoint's edges are a' = 1 - b, b' = 1 - a,
// c' = 1 - d, d' = 1 - c, so
//   dL/da = -sum v * (G integrated over the adjoint's y extent along the
//           column just below x + b'): the y-weighted differences of the two
//           table columns at b';
//   dL/db = +sum v * (the same at a');
//   dL/dc = -sum v * (G integrated over the x extent along the row below
//           y + d'): the difference of the x-interpolated rows at d';
//   dL/dd = +sum v * (the same at c').
// These are Eq. 4's edge integrals moved to the gradient's table; the adjoint
// split of the edges puts the one-sided derivative between each edge's two
// taps.  Per pixel they are sums over the four tap rows r = c'0, c'1, d'0,
// d'1 of (column difference at a' or b', or x-interpolated row) times the
// row's y weight times v; regrouped by table row instead, each of the item's
// SEG + 1 rows of each y edge is interpolated once (rows c'0 + j and
// d'0 + j) and, with v[-1] = v[SEG] = 0 and dv = v[j-1] - v[j], the sums are
//   E0 = sum_j A_c(j) e_c(j) + A_d(j) e_d(j)  = dL/db,
//   E1 = sum_j B_c(j) e_c(j) + B_d(j) e_d(j)  = -dL/da,
//   E2 = sum_j U_c(j) dv(j)                   = dL/dd,
//   E3 = sum_j U_d(j) dv(j)                   = -dL/dc,
// with e_c(j) = wy0 v[j] + wy1 v[j-1] and e_d(j) = wy2 v[j] + wy3 v[j-1].  An
// edge's two y weights split 1 (wy0 + wy1 = -1, wy2 + wy3 = 1, up to their
// fp32 rounding), so e_c = -v[j-1] - wy0 dv and e_d = v[j-1] - wy2 dv: 9
// operations per row and column instead of 12 multiply-adds per pixel (pose
// layer backward 176 -> 174 us).
template <int SEG, bool kFull, typename Src>
__device__ __forceinline__ void adjoint_walk(const Src& S, const Taps<float>& tp, int x0, int y0, int y1,
                                                  const float (&v)[SEG][kQ], float (&acc)[SEG][kQ], float (&E)[4]) {
  const typename Src::Cols cl = S.cols(x0 + tp.ox[0], x0 + tp.ox[2]);
  const int st = S.row_step();
  const int rc = S.row_coord(y0 + tp.oy[0]), rd = S.row_coord(y0 + tp.oy[2]);
  float Uc[kQ], Ud[kQ];
#pragma unroll
  for (int j = 0; j <= SEG; ++j) {
    if (kFull || y0 + j <= y1) {
      float Uc1[kQ], Ac[kQ], Bc[kQ], Ud1[kQ], Ad[kQ], Bd[kQ];
      table_row_grad(S, rc + j * st, cl, tp, Uc1, Ac, Bc);
      table_row_grad(S, rd + j * st, cl, tp, Ud1, Ad, Bd);
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        const float vp = j > 0 ? v[j - 1][q] : 0.f;
        const float vc = j < SEG ? v[j][q] : 0.f;
        const float dv = vp - vc;
        const float ec = fmaf(-tp.wy[0], dv, -vp);
        const float ed = fmaf(-tp.wy[2], dv, vp);
        E[0] = fmaf(Ac[q], ec, fmaf(Ad[q], ed, E[0]));
        E[1] = fmaf(Bc[q], ec, fmaf(Bd[q], ed, E[1]));
        E[2] = fmaf(Uc1[q], dv, E[2]);
        E[3] = fmaf(Ud1[q], dv, E[3]);
        if (j > 0) {
          float a = acc[j - 1][q];
          a = fmaf(tp.wy[0], Uc[q], a);
          a = fmaf(tp.wy[1], Uc1[q], a);
          a = fmaf(tp.wy[2], Ud[q], a);
          acc[j - 1][q] = fmaf(tp.wy[3], Ud1[q], a);
        }
        Uc[q] = Uc1[q];
        Ud[q] = Ud1[q];
      }
    }
  }
}

// Emitter of forward outputs: the Q outputs of row y0 + s at plane offset
// off0 + s * W (elements; off0 = y0 * W + x0).
// kNT: non-temporal stores (the HBM-table forwards with outputs larger than
// the last-level cache, see kStreamOutBytes).  kPack (bf16 outputs, Q even,
// every row offset and x0 even and the output 4-byte aligned): a whole row
// of the item goes out as Q / 2 packed words in one store.
template <typename OutT, typename T, bool kNT = false, int Q = kQ, bool kPack = false>
struct StoreRows {
  OutT* out;
  int W, x0, off0;
  template <bool kFull>
  __device__ __forceinline__ void put(int s, const T* o) {
    if constexpr (kPack && kFull) {
      static_assert(std::is_same<OutT, uint16_t>::value && std::is_same<T, float>::value && Q % 2 == 0 && !kNT,
                    "packed rows are bf16 pairs");
      // one v_cvt_pk_bf16_f32 per pair (the rounding of convert_out); the
      // row's word offset s * W / 2 folds into the store's immediate
      typedef float f32x2 __attribute__((ext_vector_type(2)));
      typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
      uint32_t* w = reinterpret_cast<uint32_t*>(out + off0) + s * (W >> 1);
#pragma unroll
      for (int k = 0; k < Q / 2; ++k)
        w[k] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){o[2 * k], o[2 * k + 1]}, bf16x2));
      return;
    }
    OutT* row = out + (unsigned)(off0 + s * W);
#pragma unroll
    for (int q = 0; q < Q; ++q)
      if (kFull || x0 + q < W) {
        if constexpr (kNT) __builtin_nontemporal_store(convert_out<OutT, T>(o[q]), row + q);
        else row[q] = convert_out<OutT, T>(o[q]);
      }
  }
};

// ---------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------
// Tap records (16 words each): record r < CB is box r's forward taps, record
// CB + r its adjoint taps (make_taps_adjoint); with `rounded`, the taps of
// the boxes with rounded (integer) corners and of their adjoints.
__global__ void k_box_prep(const float* __restrict__ boxes, int CB, int rounded, int* __restrict__ table) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= 2 * CB) return;
  const bool adj = i >= CB;
  const float* p = boxes + (size_t)(adj ? i - CB : i) * 4;
  const Taps<float> t = rounded ? make_taps_rounded(p, adj, 1 << 20, 1 << 20)
                        : adj   ? make_taps_adjoint(p, 1 << 20, 1 << 20)
                                : make_taps_f32(p, false, 1 << 20, 1 << 20);
  int* r = table + (size_t)i * 16;
  float* f = reinterpret_cast<float*>(r);
  r[0] = t.ox[0]; r[1] = t.ox[2]; r[2] = t.oy[0]; r[3] = t.oy[2];
#pragma unroll
  for (int k = 0; k < 4; ++k) { f[4 + k] = t.wx[k]; f[8 + k] = t.wy[k]; r[12 + k] = 0; }
}

// Box-parameter reparameterisation (Section 3.2): corners kept as u in
// [-1, 1] relative to a maximum box size M per axis, x_l = u_xl * M_x / 2,
// x_h = u_xh * M_x / 2, box [x + x_l, x + x_h + 1).  fp64 arithmetic (exact
// for these operands), rounded once to fp32.
__global__ void k_boxes_from_unit(const float* __restrict__ u, int n, float mw, float mh,
                                  float* __restrict__ boxes) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float* q = u + (size_t)i * 4;
  const double xl = (double)q[0] * (double)mw / 2, xh = (double)q[1] * (double)mw / 2;
  const double yl = (double)q[2] * (double)mh / 2, yh = (double)q[3] * (double)mh / 2;
  *reinterpret_cast<float4*>(boxes + (size_t)i * 4) =
      make_float4((float)((xl + xh) / 2), (float)((yl + yh) / 2), (float)((xh - xl + 1) / 2), (float)((yh - yl + 1) / 2));
}

// dL/du from dL/d(cx, cy, rx, ry) through the map above: x_l = a and
// x_h = b - 1 with cx = (a + b - 1) / 2, rx = (b - a) / 2.
__global__ void k_unit_grad(const float* __restrict__ g, int n, float mw, float mh, float* __restrict__ gu) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float4 q = *reinterpret_cast<const float4*>(g + (size_t)i * 4);
  const double sx = (double)mw / 2, sy = (double)mh / 2;
  *reinterpret_cast<float4*>(gu + (size_t)i * 4) =
      make_float4((float)(((double)q.x - q.z) / 2 * sx), (float)(((double)q.x + q.z) / 2 * sx),
                  (float)(((double)q.y - q.w) / 2 * sy), (float)(((double)q.y + q.w) / 2 * sy));
}

// After an update: clip u to [-1, 1] and swap a reversed corner pair.
__global__ void k_clip_unit(float* __restrict__ u, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float4 q = *reinterpret_cast<float4*>(u + (size_t)i * 4);
  q.x = fminf(fmaxf(q.x, -1.f), 1.f); q.y = fminf(fmaxf(q.y, -1.f), 1.f);
  q.z = fminf(fmaxf(q.z, -1.f), 1.f); q.w = fminf(fmaxf(q.w, -1.f), 1.f);
  *reinterpret_cast<float4*>(u + (size_t)i * 4) = make_float4(fminf(q.x, q.y), fmaxf(q.x, q.y), fminf(q.z, q.w),
                                                              fmaxf(q.z, q.w));
}

// Standalone table in HBM, one block per map.  The map is processed in strips
// of kStrip rows staged in LDS: each wave scans whole rows (every lane holds a
// run of consecutive elements, scanned serially, then a wave-level scan of
// the lane totals), then lanes own columns and carry the column sums down the
// strip, writing finished table rows coalesced.
constexpr int kStrip = 16;
constexpr int kSatMaxK = 16;  // elements per lane in a row scan: W <= 1024
constexpr int kSatRowsPerWave = 4;  // rows of a strip each wave loads before scanning them

// kUp: x is [maps][Ho][Wo] and the table is that of its zero-upsampled H x W
// map (x[i][j] at (s*i, s*j)); mean must then be null.
// KM: elements per lane in a row scan, K = ceil(W / 64) <= KM (4 for
// W <= 256, else 16).  kGroups > 1 (W <= 256, few maps): blocks of
// 256 * kGroups threads take strips of kStrip * kGroups rows, and the column
// pass runs kGroups row groups of kStrip rows in parallel, each starting from
// the carried sums plus the totals of the groups above it.
template <typename T, bool kUp, int KM, int kGroups>
__global__ __launch_bounds__(256 * kGroups) void k_sat_build(const T* __restrict__ x, T* __restrict__ sat,
                                                             float* __restrict__ mean, int H, int W, int s, int Ho,
                                                             int Wo) {
  static_assert(kGroups == 1 || KM == 4, "row groups need W <= 256");
  constexpr int kRowsStrip = kStrip * kGroups;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  T* tile = reinterpret_cast<T*>(smem_raw);
  __shared__ float red[16];
  __shared__ T part[kGroups > 1 ? kGroups * 256 : 1];
  const int map = blockIdx.x;
  const T* src = x + (size_t)map * (kUp ? (size_t)Ho * Wo : (size_t)H * W);
  T* dst = sat + (size_t)map * (H + 1) * (W + 1);
  float mu = 0.f;
  const bool sub = mean != nullptr;
  if (sub) {
    mu = block_mean(reinterpret_cast<const float*>(src), H * W, red);
    if (threadIdx.x == 0) mean[map] = mu;
  }
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  const int K = (W + 63) >> 6;
  for (int v = tid; v <= W; v += blockDim.x) dst[v] = (T)0;
  T carry[KM / 4];
#pragma unroll
  for (int j = 0; j < KM / 4; ++j) carry[j] = (T)0;
  for (int r0 = 0; r0 < H; r0 += kRowsStrip) {
    const int rows = min(kRowsStrip, H - r0);
    // rows rr = wave + i * nw of the strip: all of a wave's loads are issued
    // before its first scan
    for (int rb = wave; rb < rows; rb += kSatRowsPerWave * nw) {
      T v[kSatRowsPerWave][KM];
#pragma unroll
      for (int i = 0; i < kSatRowsPerWave; ++i) {
        const int rr = rb + i * nw, r = r0 + rr;
        const T* row = kUp ? src + (size_t)(r / s) * Wo : src + (size_t)r * W;
        const bool live = rr < rows && (!kUp || r % s == 0);
#pragma unroll
        for (int k = 0; k < KM; ++k) {
          if (k < K) {
            const int idx = lane * K + k;
            T val;
            if constexpr (kUp) val = (live && idx < W && idx % s == 0) ? row[idx / s] : (T)0;
            else val = (live && idx < W) ? row[idx] : (T)0;
            if (sub && idx < W) val = (T)((float)val - mu);
            v[i][k] = val;
          }
        }
      }
#pragma unroll
      for (int i = 0; i < kSatRowsPerWave; ++i) {
        const int rr = rb + i * nw;
        T run = (T)0;
#pragma unroll
        for (int k = 0; k < KM; ++k) {
          if (k < K) {
            run += v[i][k];
            v[i][k] = run;
          }
        }
        const T excl = wave_excl_scan(run, lane);
        if (rr < rows) {
#pragma unroll
          for (int k = 0; k < KM; ++k) {
            const int idx = lane * K + k;
            if (k < K && idx < W) tile[rr * W + idx] = v[i][k] + excl;
          }
        }
      }
    }
    __syncthreads();
    if constexpr (kGroups == 1) {
#pragma unroll
      for (int j = 0; j < KM / 4; ++j) {
        const int v = tid + j * 256;
        if (v < W) {
          T cs = carry[j];
          for (int rr = 0; rr < rows; ++rr) {
            cs += tile[rr * W + v];
            dst[(size_t)(r0 + rr + 1) * (W + 1) + v + 1] = cs;
          }
          carry[j] = cs;
        }
      }
    } else {
      // column v, row group g: rows [g * kStrip, (g + 1) * kStrip) of the strip
      const int v = tid & 255, g = tid >> 8;
      const int ra = g * kStrip, rz = min(ra + kStrip, rows);
      T ps = (T)0;
      if (v < W)
        for (int rr = ra; rr < rz; ++rr) ps += tile[rr * W + v];
      part[g * 256 + v] = ps;
      __syncthreads();
      if (v < W) {
        T cs = carry[0], tot = (T)0;
#pragma unroll
        for (int h = 0; h < kGroups; ++h) {
          const T p = part[h * 256 + v];
          if (h < g) cs += p;
          tot += p;
        }
        for (int rr = ra; rr < rz; ++rr) {
          cs += tile[rr * W + v];
          dst[(size_t)(r0 + rr + 1) * (W + 1) + v + 1] = cs;
        }
        carry[0] += tot;
      }
    }
    if (tid < rows) dst[(size_t)(r0 + tid + 1) * (W + 1)] = (T)0;
    __syncthreads();
  }
}

template <typename T> __device__ __forceinline__ Taps<T> typed_taps(const Taps<float>& t);
template <> __device__ __forceinline__ Taps<float> typed_taps<float>(const Taps<float>& t) { return t; }
template <> __device__ __forceinline__ Taps<int> typed_taps<int>(const Taps<float>& t) { return int_taps(t); }

// Forward on a map's table in LDS, for the boxes b0 .. b0+nb-1 of channel c.
// Items of one box are (row segment, 3-column chunk), chunk fastest so that
// adjacent lanes write adjacent columns; each box's items are padded to a
// multiple of 64 (per_box_p) so that a wave works on one box and reads its
// taps through scalar loads.
template <typename T, typename OutT, int SEG, bool kOffset, bool kInt, int Q = kQ, bool kPack = false>
__device__ __forceinline__ void fwd_boxes(const LdsTable<T>& tab, const int* __restrict__ taps,
                                          OutT* __restrict__ y, int map, int c, int b0, int nb, int H, int W,
                                          int B, int per_box_p, float mu) {
  const int nch = (W + Q - 1) / Q, nseg = (H + SEG - 1) / SEG, per_box = nch * nseg;
  for (int it = threadIdx.x; it < nb * per_box_p; it += blockDim.x) {
    const int bl = __builtin_amdgcn_readfirstlane(it / per_box_p);
    const int r = it - bl * per_box_p;
    if (r >= per_box) continue;
    const int seg = r / nch, ch = r - seg * nch;
    const int b = b0 + bl;
    const Taps<T> tp = typed_taps<T>(load_taps(taps + (size_t)(c * B + b) * 16, W, H));
    OutT* out = y + ((size_t)map * B + b) * H * W;
    const int x0 = ch * Q, y0 = seg * SEG, y1 = min(y0 + SEG, H);
    StoreRows<OutT, T, false, Q, kPack> em{out, W, x0, y0 * W + x0};
    if (y0 + SEG <= H && x0 + Q <= W) walk_fwd<SEG, T, kOffset, true, kInt, Q>(tab, tp, H, W, x0, y0, y1, mu, em);
    else walk_fwd<SEG, T, kOffset, false, kInt, Q>(tab, tp, H, W, x0, y0, y1, mu, em);
  }
}

// Forward, table in LDS: one block per (map, group of bpg boxes).  The block
// builds the map's table once and evaluates every box of its group.
// kW > 0: the map width compiled in (W is then ignored), as in the LDS
// backward.  Q: columns per item; kPack: packed bf16 row stores (StoreRows).
template <typename T, typename OutT, int SEG, bool kOffset, bool kInt, int kW = 0, int Q = kQ, bool kPack = false>
__global__ __launch_bounds__(256) void k_box_fwd_lds(const T* __restrict__ x, const int* __restrict__ taps,
                                                     OutT* __restrict__ y, int C, int H, int W_arg, int B, int bpg,
                                                     int per_box_p) {
  const int W = kW > 0 ? kW : W_arg;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  T* S = reinterpret_cast<T*>(smem_raw);
  __shared__ float red[16];
  const int pitch = lds_pitch_dev(W);
  const int ngrp = (B + bpg - 1) / bpg;
  const int map = blockIdx.x / ngrp, grp = blockIdx.x - map * ngrp;
  const T* src = x + (size_t)map * H * W;
  float mu = 0.f;
  if (kOffset) mu = block_mean(reinterpret_cast<const float*>(src), H * W, red);
  build_table_lds<T, true>(src, S, H, W, pitch, mu, kOffset);
  const int b0 = grp * bpg;
  fwd_boxes<T, OutT, SEG, kOffset, kInt, Q, kPack>(LdsTable<T>{S, pitch, W, H}, taps, y, map, map % C, b0,
                                                   min(bpg, B - b0), H, W, B, per_box_p, mu);
}

// Forward, table in HBM: one block per (map, box, block of 256 items), mapped
// so that one map's blocks run on one XCD.
template <typename T, typename OutT, int SEG, bool kOffset, bool kInt, bool kNT>
__global__ __launch_bounds__(256) void k_box_fwd_gather(const T* __restrict__ sat, const float* __restrict__ means,
                                                        const int* __restrict__ taps, OutT* __restrict__ y,
                                                        int C, int H, int W, int B, int nblk, int total) {
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  if (L >= total) return;
  const int blk = L % nblk, mb = L / nblk;
  const int b = mb % B, map = mb / B, c = map % C;
  const int nch = (W + kQ - 1) / kQ, nseg = (H + SEG - 1) / SEG;
  const int it = blk * 256 + threadIdx.x;
  if (it >= nch * nseg) return;
  const int seg = it / nch, ch = it - seg * nch;
  const GlobalTable<T, true> tab{sat + (size_t)map * (H + 1) * (W + 1), W + 1, W, H};
  const float mu = kOffset ? means[map] : 0.f;
  const Taps<T> tp = typed_taps<T>(load_taps(taps + (size_t)(c * B + b) * 16, W, H));
  OutT* out = y + ((size_t)map * B + b) * H * W;
  const int x0 = ch * kQ, y0 = seg * SEG, y1 = min(y0 + SEG, H);
  StoreRows<OutT, T, kNT> em{out, W, x0, y0 * W + x0};
  if (y0 + SEG <= H && x0 + kQ <= W) walk_fwd<SEG, T, kOffset, true, kInt>(tab, tp, H, W, x0, y0, y1, mu, em);
  else walk_fwd<SEG, T, kOffset, false, kInt>(tab, tp, H, W, x0, y0, y1, mu, em);
}

// Strided forward (stride s > 1) on a map's table in LDS, boxes b0 .. b0+nb-1
// of channel c: items are (output column, segment of kSegS output rows),
// column fastest; a box's items are padded to per_box_p (a multiple of 64)
// so each wave serves one box.
constexpr int kSegS = 8;
template <typename T, typename OutT, bool kOffset, bool kInt>
__device__ __forceinline__ void fwd_boxes_strided(const LdsTable<T>& tab, const int* __restrict__ taps,
                                                  OutT* __restrict__ y, int map, int c, int b0, int nb, int H, int W,
                                                  int B, int s, int Ho, int Wo, int per_box_p, float mu) {
  const int per_box = Wo * ((Ho + kSegS - 1) / kSegS);
  for (int it = threadIdx.x; it < nb * per_box_p; it += blockDim.x) {
    const int bl = __builtin_amdgcn_readfirstlane(it / per_box_p);
    const int r = it - bl * per_box_p;
    if (r >= per_box) continue;
    const int seg = r / Wo, j = r - seg * Wo;
    const int b = b0 + bl;
    const Taps<T> tp = typed_taps<T>(load_taps(taps + (size_t)(c * B + b) * 16, W, H));
    const int i0 = seg * kSegS;
    StoreCol<OutT, T> em{y + ((size_t)map * B + b) * Ho * Wo, Wo, i0 * Wo + j};
    box_walk_strided<kSegS, T, kOffset, kInt>(tab, tp, H, W, s * j, i0, min(i0 + kSegS, Ho), s, mu, em);
  }
}

template <typename T, typename OutT, bool kOffset, bool kInt, int kW = 0>
__global__ __launch_bounds__(256) void k_box_fwd_lds_strided(const T* __restrict__ x, const int* __restrict__ taps,
                                                             OutT* __restrict__ y, int C, int H, int W_arg, int B, int s,
                                                             int Ho, int Wo, int bpg, int per_box_p) {
  const int W = kW > 0 ? kW : W_arg;  // kW > 0: the map width compiled in
  extern __shared__ __align__(16) unsigned char smem_raw[];
  T* S = reinterpret_cast<T*>(smem_raw);
  __shared__ float red[16];
  const int pitch = lds_pitch_dev(W);
  const int ngrp = (B + bpg - 1) / bpg;
  const int map = blockIdx.x / ngrp, grp = blockIdx.x - map * ngrp;
  const T* src = x + (size_t)map * H * W;
  float mu = 0.f;
  if (kOffset) mu = block_mean(reinterpret_cast<const float*>(src), H * W, red);
  build_table_lds(src, S, H, W, pitch, mu, kOffset);
  const int b0 = grp * bpg;
  fwd_boxes_strided<T, OutT, kOffset, kInt>(LdsTable<T>{S, pitch, W, H}, taps, y, map, map % C, b0,
                                            min(bpg, B - b0), H, W, B, s, Ho, Wo, per_box_p, mu);
}

// Strided forward, table in HBM: one block per (map, box, block of 256 items).
template <typename T, typename OutT, bool kOffset, bool kInt>
__global__ __launch_bounds__(256) void k_box_fwd_gather_strided(const T* __restrict__ sat,
                                                                const float* __restrict__ means,
                                                                const int* __restrict__ taps, OutT* __restrict__ y,
                                                                int C, int H, int W, int B, int s, int Ho, int Wo,
                                                                int nblk, int total) {
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  if (L >= total) return;
  const int blk = L % nblk, mb = L / nblk;
  const int b = mb % B, map = mb / B, c = map % C;
  const int it = blk * 256 + threadIdx.x;
  if (it >= Wo * ((Ho + kSegS - 1) / kSegS)) return;
  const int seg = it / Wo, j = it - seg * Wo;
  const GlobalTable<T, true> tab{sat + (size_t)map * (H + 1) * (W + 1), W + 1, W, H};
  const float mu = kOffset ? means[map] : 0.f;
  const Taps<T> tp = typed_taps<T>(load_taps(taps + (size_t)(c * B + b) * 16, W, H));
  const int i0 = seg * kSegS;
  StoreCol<OutT, T> em{y + ((size_t)map * B + b) * Ho * Wo, Wo, i0 * Wo + j};
  box_walk_strided<kSegS, T, kOffset, kInt>(tab, tp, H, W, s * j, i0, min(i0 + kSegS, Ho), s, mu, em);
}

// Map values of one item, 0 outside the map (they then add nothing to the
// parameter gradients).
template <int SEG>
__device__ __forceinline__ void load_item(const float* __restrict__ xs, int H, int W, int x0, int y0, bool active,
                                          float (&v)[SEG][kQ]) {
#pragma unroll
  for (int s = 0; s < SEG; ++s)
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const int yy = y0 + s, xx = x0 + q;
      v[s][q] = (active && yy < H && xx < W) ? xs[(size_t)yy * W + xx] : 0.f;
    }
}

// The item's origin passes through an opaque copy (an empty asm with the
// coordinates as operands): the stores then recompute their row addresses
// instead of the compiler holding load_item's 64-bit row offsets live across
// a whole kernel (seven register pairs in the 8-row backward, which spilled
// them at four waves per SIMD).
__device__ __forceinline__ void opaque_origin(int& x0, int& y0) { asm volatile("" : "+v"(x0), "+v"(y0)); }

template <int SEG>
__device__ __forceinline__ void store_item(float* __restrict__ out, int H, int W, int x0, int y0,
                                           const float (&acc)[SEG][kQ]) {
  opaque_origin(x0, y0);
#pragma unroll
  for (int s = 0; s < SEG; ++s) {
    const int yy = y0 + s;
    if (yy < H) {
#pragma unroll
      for (int q = 0; q < kQ; ++q)
        if (x0 + q < W) out[(size_t)yy * W + x0 + q] = acc[s][q];
    }
  }
}

// The input gradient of a layer whose input x is a ReLU output, in the
// compute type of the bf16 mix before it: bf16(x > 0 ? dx : 0), round to
// nearest even.  x > 0 is the ReLU's own mask, so these are the operand bits
// that mix's backward forms.  The mask is taken from the item's input values
// once, as one bit per output (relu_mask), so they need not stay live.
template <int SEG>
__device__ __forceinline__ uint32_t relu_mask(const float (&v)[SEG][kQ]) {
  static_assert(SEG * kQ <= 32, "one bit per output");
  uint32_t m = 0;
#pragma unroll
  for (int s = 0; s < SEG; ++s)
#pragma unroll
    for (int q = 0; q < kQ; ++q) m |= (v[s][q] > 0.f ? 1u : 0u) << (s * kQ + q);
  return m;
}

// fp32 -> bf16 bits, round to nearest even, in integer arithmetic: the same
// bits as the conversion instruction for every finite value and infinity (a
// NaN stays a quiet NaN).  Here the instruction's form made the backward's
// register allocation grow from 144 to 224 VGPRs; this one does not.
__device__ __forceinline__ uint16_t bf16_rne_bits(float f) {
  const uint32_t b = __float_as_uint(f);
  if ((b & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((b >> 16) | 0x40u);
  return (uint16_t)((b + 0x7fffu + ((b >> 16) & 1u)) >> 16);
}

template <int SEG>
__device__ __forceinline__ void store_item_relu_bf16(uint16_t* __restrict__ out, int H, int W, int x0, int y0,
                                                     const float (&acc)[SEG][kQ], uint32_t mask) {
  opaque_origin(x0, y0);
#pragma unroll
  for (int s = 0; s < SEG; ++s) {
    const int yy = y0 + s;
    if (yy < H) {
#pragma unroll
      for (int q = 0; q < kQ; ++q)
        if (x0 + q < W)
          out[(size_t)yy * W + x0 + q] = bf16_rne_bits(((mask >> (s * kQ + q)) & 1u) ? acc[s][q] : 0.f);
    }
  }
}

// Lane move (data-parallel primitive `ctrl`), 0 where the source lane is
// disabled.
template <int kCtrl>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kCtrl, 0xF, 0xF, false));
}

// The wave's sums of the four edge gradients, written to pp[0..3] (lanes 0..3
// store one each).  A transposed reduction: the pair step (lane ^ 1) leaves
// even lanes summing values 0 and 1 and odd lanes values 2 and 3, the quad
// step (lane ^ 2) one value per lane, index 2 * (lane & 1) + ((lane >> 1) &
// 1); rotations by 4 and 8 lanes inside each 16-lane row, then the row
// swaps (lane ^ 16, lane ^ 32), finish the sum in every lane.  17 vector
// operations for the four sums instead of four separate reductions (four
// lane moves and four lane reads each).  Every lane of the wave must be
// active; the order of the additions is fixed, so the sums are
// deterministic.
__device__ __forceinline__ void store_wave_partial(const float* g4, float* __restrict__ pp) {
  const int lane = threadIdx.x & 63;
  const bool odd = lane & 1, hi = lane & 2;
  float k0 = odd ? g4[2] : g4[0], k1 = odd ? g4[3] : g4[1];
  const float s0 = odd ? g4[0] : g4[2], s1 = odd ? g4[1] : g4[3];
  k0 += dpp_move<0xB1>(s0);  // quad_perm 1,0,3,2: lane ^ 1
  k1 += dpp_move<0xB1>(s1);
  float t = hi ? k1 : k0;
  const float u = hi ? k0 : k1;
  t += dpp_move<0x4E>(u);    // quad_perm 2,3,0,1: lane ^ 2
  t += dpp_move<0x124>(t);   // row_ror:4
  t += dpp_move<0x128>(t);   // row_ror:8
  auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(t), __float_as_uint(t), false, false);
  t = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);  // rows 0+1 and 2+3
  auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(t), __float_as_uint(t), false, false);
  t = __uint_as_float(r32[0]) + __uint_as_float(r32[1]);  // halves
  if (lane < 4) pp[2 * (lane & 1) + (lane >> 1)] = t;
}

// Backward, table in LDS: one block per map (n, c); items (row segment,
// chunk), one per thread, whose map values stay in registers.  For each box
// b the table of grad_y[n][c*B+b] is built in LDS and the adjoint walk adds
// the input gradient (in registers, summed over b) and the edge gradients;
// each wave writes its edge-gradient sums to
// partials[(n * nw + wave) * C*B + c*B + b][4].  kInt (boxes with integer
// corners): the adjoint four-corner sums only, no edge gradients.  kUp
// (stride s > 1): grad_y is [maps][Ho][Wo] and is tabulated zero-upsampled,
// which makes every gradient that of the strided layer.  kRelu: gx is bf16,
// store_item_relu_bf16 (not with kInt, which does not read x).
// Four waves per SIMD: bounded to 128 VGPRs (from 144, three waves) the
// 8-row items fit without spilling once the final stores recompute their
// addresses (below); pose-layer backward 172.5 -> 151.5 us, results
// bit-identical.  The 4-row items take 92.
// kW > 0: the map width as a compile-time constant (W is then ignored), so
// the table pitch is one too and every row offset of the scans, the walk and
// the item loads and stores is an immediate of its LDS or global access
// instead of a per-element address add; the results are the same bits.
template <int SEG, bool kInt, bool kUp, int kMaxT, bool kRelu, int kW = 0>
__global__ __launch_bounds__(kMaxT) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_box_bwd_lds(
    const float* __restrict__ x, const int* __restrict__ taps, const float* __restrict__ gy, void* __restrict__ gx,
    float* __restrict__ partials, int C, int H, int W_arg, int B, int s, int Ho, int Wo) {
  static_assert(!(kInt && kRelu), "the ReLU mask needs x");
  const int W = kW > 0 ? kW : W_arg;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int pitch = lds_pitch_dev(W);
  float* SG = reinterpret_cast<float*>(smem_raw);
  const int map = blockIdx.x, n = map / C, c = map - n * C;
  const int nw = blockDim.x >> 6, wave = threadIdx.x >> 6;
  const int nch = (W + kQ - 1) / kQ, nseg = (H + SEG - 1) / SEG;
  const int it = threadIdx.x;
  const bool active = it < nch * nseg;
  const int seg = it / nch, ch = it - seg * nch;
  const int x0 = ch * kQ, y0 = seg * SEG, y1 = min(y0 + SEG, H);
  const bool full = y0 + SEG <= H && x0 + kQ <= W;
  const size_t plane = (size_t)H * W;
  const size_t gplane = kUp ? (size_t)Ho * Wo : plane;
  const float* g0 = gy + (size_t)map * B * gplane;
  float v[SEG][kQ], acc[SEG][kQ];
  if constexpr (!kInt) load_item<SEG>(x + (size_t)map * plane, H, W, x0, y0, active, v);
  uint32_t rmask = 0;
  if constexpr (kRelu) rmask = relu_mask<SEG>(v);
#pragma unroll
  for (int s = 0; s < SEG; ++s)
#pragma unroll
    for (int q = 0; q < kQ; ++q) acc[s][q] = 0.f;
  const LdsTable<float> tg{SG, pitch, W, H};
  const int* adj = taps + (size_t)C * B * 16;
  for (int b = 0; b < B; ++b) {
    __syncthreads();
    if constexpr (kUp) build_table_lds_up(g0 + b * gplane, SG, H, W, pitch, s, Ho, Wo);
    else build_table_lds(g0 + b * plane, SG, H, W, pitch, 0.f, false);
    const Taps<float> tp = load_taps(adj + (size_t)(c * B + b) * 16, W, H);
    if constexpr (kInt) {  // integer corners: input gradient only
      AccRows<SEG> em{acc};
      if (active) {
        if (full) box_walk_int<SEG, float, false, true>(tg, tp, H, W, x0, y0, y1, 0.f, em);
        else box_walk_int<SEG, float, false, false>(tg, tp, H, W, x0, y0, y1, 0.f, em);
      }
      continue;
    }
    float E[4] = {0.f, 0.f, 0.f, 0.f};
    if (active) {
      if (full) adjoint_walk<SEG, true>(tg, tp, x0, y0, y1, v, acc, E);
      else adjoint_walk<SEG, false>(tg, tp, x0, y0, y1, v, acc, E);
    }
    float g4[4] = {-E[1], E[0], -E[3], E[2]};   // dL/da, dL/db, dL/dc, dL/dd
    store_wave_partial(g4, partials + (((size_t)n * nw + wave) * C * B + (size_t)c * B + b) * 4);
  }
  if (active && gx != nullptr) {
    if constexpr (kRelu) store_item_relu_bf16<SEG>(static_cast<uint16_t*>(gx) + (size_t)map * plane, H, W, x0, y0, acc, rmask);
    else store_item<SEG>(static_cast<float*>(gx) + (size_t)map * plane, H, W, x0, y0, acc);
  }
}

// Backward, tables in HBM (one table per gradient map, built beforehand).
// One 256-thread block per (map, block of 256 items); loops over boxes.
// partials: [((n * nblk + blk) * 4 + wave) * C*B + c*B + b][4]; kInt as in
// k_box_bwd_lds.
template <int SEG, bool kInt, bool kRelu>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 8))) void k_box_bwd_gather(const float* __restrict__ x, const float* __restrict__ sat_g,
                                                        const int* __restrict__ taps, void* __restrict__ gx,
                                                        float* __restrict__ partials, int C, int H, int W, int B,
                                                        int nblk, int total) {
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  if (L >= total) return;
  const int blk = L % nblk, map = L / nblk;
  const int n = map / C, c = map - n * C;
  const int wave = threadIdx.x >> 6;
  const int nch = (W + kQ - 1) / kQ, nseg = (H + SEG - 1) / SEG;
  const int it = blk * 256 + threadIdx.x;
  const bool active = it < nch * nseg;
  const int seg = it / nch, ch = it - seg * nch;
  const int x0 = ch * kQ, y0 = seg * SEG, y1 = min(y0 + SEG, H);
  const bool full = y0 + SEG <= H && x0 + kQ <= W;
  const size_t tsz = (size_t)(H + 1) * (W + 1);
  float v[SEG][kQ], acc[SEG][kQ];
  if constexpr (!kInt) load_item<SEG>(x + (size_t)map * H * W, H, W, x0, y0, active, v);
  uint32_t rmask = 0;
  if constexpr (kRelu) rmask = relu_mask<SEG>(v);
#pragma unroll
  for (int s = 0; s < SEG; ++s)
#pragma unroll
    for (int q = 0; q < kQ; ++q) acc[s][q] = 0.f;
  const int* adj = taps + (size_t)C * B * 16;
  for (int b = 0; b < B; ++b) {
    const GlobalTable<float> tg{sat_g + ((size_t)map * B + b) * tsz, W + 1, W, H};
    const Taps<float> tp = load_taps(adj + (size_t)(c * B + b) * 16, W, H);
    if constexpr (kInt) {  // integer corners: input gradient only
      AccRows<SEG> em{acc};
      if (active) {
        if (full) box_walk_int<SEG, float, false, true>(tg, tp, H, W, x0, y0, y1, 0.f, em);
        else box_walk_int<SEG, float, false, false>(tg, tp, H, W, x0, y0, y1, 0.f, em);
      }
      continue;
    }
    float E[4] = {0.f, 0.f, 0.f, 0.f};
    if (active) {
      if (full) adjoint_walk<SEG, true>(tg, tp, x0, y0, y1, v, acc, E);
      else adjoint_walk<SEG, false>(tg, tp, x0, y0, y1, v, acc, E);
    }
    float g4[4] = {-E[1], E[0], -E[3], E[2]};   // dL/da, dL/db, dL/dc, dL/dd
    store_wave_partial(g4, partials + ((((size_t)n * nblk + blk) * 4 + wave) * C * B + (size_t)c * B + b) * 4);
  }
  if (active && gx != nullptr) {
    if constexpr (kRelu) store_item_relu_bf16<SEG>(static_cast<uint16_t*>(gx) + (size_t)map * H * W, H, W, x0, y0, acc, rmask);
    else store_item<SEG>(static_cast<float*>(gx) + (size_t)map * H * W, H, W, x0, y0, acc);
  }
}

// Second stage of the box-parameter gradient: fixed-order sum of the partial
// edge gradients, then the change of variables a = 1/2+cx-rx, b = 1/2+cx+rx,
// c = 1/2+cy-ry, d = 1/2+cy+ry:  dcx = ga+gb, dcy = gc+gd, drx = gb-ga,
// dry = gd-gc.
// One block per 16 boxes: thread (q, j) sums rows p = q, q + 16, ... of box
// j (a wave's load covers 4 rows x 16 consecutive boxes, 256 contiguous
// bytes each), then the 16 row-sums of each box combine in a fixed tree
// (lane shuffles across the wave's 4 row groups, then the 4 waves in LDS).
constexpr int kReduceBoxes = 16;
__global__ __launch_bounds__(256) void k_box_grad_reduce(const float* __restrict__ partials, int P, int CB,
                                                         float* __restrict__ out) {
  __shared__ float4 red[4][kReduceBoxes];
  const int j = threadIdx.x % kReduceBoxes, q = threadIdx.x / kReduceBoxes;
  const int i = blockIdx.x * kReduceBoxes + j;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  if (i < CB)
    for (int p = q; p < P; p += 256 / kReduceBoxes) {
      const float4 v = *reinterpret_cast<const float4*>(partials + ((size_t)p * CB + i) * 4);
      s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
#pragma unroll
  for (int m = 16; m < 64; m <<= 1) {
    s.x += __shfl_xor(s.x, m); s.y += __shfl_xor(s.y, m);
    s.z += __shfl_xor(s.z, m); s.w += __shfl_xor(s.w, m);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) < kReduceBoxes) red[wave][j] = s;
  __syncthreads();
  if (threadIdx.x < kReduceBoxes && i < CB) {
    float4 t = red[0][j];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const float4 u = red[w][j];
      t.x += u.x; t.y += u.y; t.z += u.z; t.w += u.w;
    }
    *reinterpret_cast<float4*>(out + (size_t)i * 4) = make_float4(t.x + t.y, t.z + t.w, t.y - t.x, t.w - t.z);
  }
}

// ---------------------------------------------------------------------------
// Kernel splitting (Section 3.1, Fig. 2): a box cut at its centre line(s)
// m = (a + b) / 2, n = (c + d) / 2 into nx * ny pieces with their own
// weights; the output is the weighted sum of the pieces' box sums.
// ---------------------------------------------------------------------------
// Corner records of split boxes for the forward, 32 words per box: a split
// box is sum_{i,j} w_ij * (box sum over [k_j, k_{j+1}) x [r_i, r_{i+1})), and
// each piece's box sum is the four-corner difference of the interpolated
// table, so the whole box is sum over the (nx+1) x (ny+1) shared corners of
// coef(ri, kj) * T(r_ri, k_kj) with
//   coef(ri, kj) = w(ri-1, kj-1) - w(ri-1, kj) - w(ri, kj-1) + w(ri, kj)
// (w = 0 outside the pieces): 9 interpolated corners for 4 pieces instead of
// 16.  Words: 0..2 column-corner floors, 3..5 row-corner floors, 6..11 row
// weights (1 - beta, beta) per row corner, 12..29 column weights
// coef * (1 - alpha), coef * alpha per (row corner, column corner); fp64
// edges and products, each weight rounded once.
__global__ void k_box_prep_corners(const float* __restrict__ boxes, const float* __restrict__ piece_w, int CB,
                                   int nx, int ny, int* __restrict__ table) {
  const int box = blockIdx.x * blockDim.x + threadIdx.x;
  if (box >= CB) return;
  const float* q = boxes + (size_t)box * 4;
  const double cx = q[0], cy = q[1], rx = q[2], ry = q[3];
  const double a = 0.5 + cx - rx, b = 0.5 + cx + rx, c = 0.5 + cy - ry, d = 0.5 + cy + ry;
  const double ke[3] = {a, nx == 2 ? (a + b) / 2 : b, b};
  const double re[3] = {c, ny == 2 ? (c + d) / 2 : d, d};
  const float* wp = piece_w + (size_t)box * nx * ny;
  auto w = [&](int i, int j) -> double {
    return (i < 0 || j < 0 || i >= ny || j >= nx) ? 0.0 : (double)wp[i * nx + j];
  };
  int* r = table + (size_t)box * 32;
  float* f = reinterpret_cast<float*>(r);
  double alpha[3];
  for (int k = 0; k <= nx; ++k) {
    int fl;
    edge_split(ke[k], 1 << 20, fl, alpha[k]);
    r[k] = fl;
  }
  for (int i = 0; i <= ny; ++i) {
    int fl;
    double beta;
    edge_split(re[i], 1 << 20, fl, beta);
    r[3 + i] = fl;
    f[6 + 2 * i] = (float)(1.0 - beta);
    f[7 + 2 * i] = (float)beta;
    for (int k = 0; k <= nx; ++k) {
      const double cf = w(i - 1, k - 1) - w(i - 1, k) - w(i, k - 1) + w(i, k);
      f[12 + (i * 3 + k) * 2] = (float)(cf * (1.0 - alpha[k]));
      f[13 + (i * 3 + k) * 2] = (float)(cf * alpha[k]);
    }
  }
  for (int k = 30; k < 32; ++k) r[k] = 0;
}

// Forward walk of a split box over its shared corners (record above), on a
// map's table in LDS: per table row v and row corner ri the column-weighted
// row R_ri(v)[q] = sum_kj cw0 * S(v, x+f_kj) + cw1 * S(v, x+f_kj+1), and the
// output of row y is sum_ri (1-beta) R_ri(y+f_ri) + beta R_ri(y+f_ri+1).
// Each step reads one new table row per row corner (NXC runs of kQ+1 words)
// and reuses the one from the step before.
template <int SEG, int NXC, int NYC, bool kFull, typename Src, typename Emit>
__device__ __forceinline__ void corner_walk(const Src& S, const int* __restrict__ rec, int x0, int y0, int y1,
                                            Emit& emit) {
  const float* f = reinterpret_cast<const float*>(rec);
  const int W = S.W, H = S.H;
  typename Src::Col col[NXC];
  float cw[NYC][NXC][2], wy[NYC][2];
  int rc[NYC];
  const int st = S.row_step();
#pragma unroll
  for (int k = 0; k < NXC; ++k) col[k] = S.col(x0 + clampi(rec[k], -(W + 1), W + 1));
#pragma unroll
  for (int i = 0; i < NYC; ++i) {
    rc[i] = S.row_coord(y0 + clampi(rec[3 + i], -(H + 1), H + 1));
    wy[i][0] = f[6 + 2 * i];
    wy[i][1] = f[7 + 2 * i];
#pragma unroll
    for (int k = 0; k < NXC; ++k) {
      cw[i][k][0] = f[12 + (i * 3 + k) * 2];
      cw[i][k][1] = f[13 + (i * 3 + k) * 2];
    }
  }
  auto row = [&](int i, int coord, float* R) {
    const typename Src::Row rr = S.row(coord);
#pragma unroll
    for (int q = 0; q < kQ; ++q) R[q] = 0.f;
#pragma unroll
    for (int k = 0; k < NXC; ++k) {
      float v[kQ + 1];
      S.run4(rr, col[k], v);
#pragma unroll
      for (int q = 0; q < kQ; ++q) R[q] = fmaf(cw[i][k][0], v[q], fmaf(cw[i][k][1], v[q + 1], R[q]));
    }
  };
  float Rc[NYC][kQ];
#pragma unroll
  for (int i = 0; i < NYC; ++i) row(i, rc[i], Rc[i]);
#pragma unroll
  for (int s = 0; s < SEG; ++s) {
    if (kFull || y0 + s < y1) {
      float o[kQ];
#pragma unroll
      for (int q = 0; q < kQ; ++q) o[q] = 0.f;
#pragma unroll
      for (int i = 0; i < NYC; ++i) {
        float Rn[kQ];
        row(i, rc[i] + (s + 1) * st, Rn);
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
          o[q] = fmaf(wy[i][0], Rc[i][q], fmaf(wy[i][1], Rn[q], o[q]));
          Rc[i][q] = Rn[q];
        }
      }
      emit.template put<kFull>(s, o);
    }
  }
}

// Forward of split boxes, table in LDS: as k_box_fwd_lds (a wave per box,
// items of 3 columns x SEG rows), each item walking its box's shared corners.
template <typename OutT, int SEG, int NXC, int NYC>
__global__ __launch_bounds__(256) void k_box_fwd_lds_split(const float* __restrict__ x, const int* __restrict__ rec,
                                                           OutT* __restrict__ y, int C, int H, int W, int B, int bpg,
                                                           int per_box_p) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  float* S = reinterpret_cast<float*>(smem_raw);
  const int pitch = lds_pitch_dev(W);
  const int ngrp = (B + bpg - 1) / bpg;
  const int map = blockIdx.x / ngrp, grp = blockIdx.x - map * ngrp, c = map % C;
  build_table_lds(x + (size_t)map * H * W, S, H, W, pitch, 0.f, false);
  const LdsTable<float> tab{S, pitch, W, H};
  const int b0 = grp * bpg, nb = min(bpg, B - b0);
  const int nch = (W + kQ - 1) / kQ, nseg = (H + SEG - 1) / SEG, per_box = nch * nseg;
  for (int it = threadIdx.x; it < nb * per_box_p; it += blockDim.x) {
    const int bl = __builtin_amdgcn_readfirstlane(it / per_box_p);
    const int r = it - bl * per_box_p;
    if (r >= per_box) continue;
    const int seg = r / nch, ch = r - seg * nch;
    const int b = b0 + bl;
    const int* rb = rec + (size_t)(c * B + b) * 32;
    OutT* out = y + ((size_t)map * B + b) * H * W;
    const int x0 = ch * kQ, y0 = seg * SEG, y1 = min(y0 + SEG, H);
    StoreRows<OutT, float> em{out, W, x0, y0 * W + x0};
    if (y0 + SEG <= H && x0 + kQ <= W) corner_walk<SEG, NXC, NYC, true>(tab, rb, x0, y0, y1, em);
    else corner_walk<SEG, NXC, NYC, false>(tab, rb, x0, y0, y1, em);
  }
}

// Adjoint corner records of split boxes for the backward, 32 words per box.
// The transpose of a split box's correlation is the mirrored split box: column
// corners k' = 1 - (b, m, a), row corners r' = 1 - (d, n, c) (ascending), and
// mirrored piece (i', j') carries w(ny-1-i', nx-1-j').  Each mirrored corner
// is split as e = f + alpha with alpha in (0, 1] (f = ceil(e) - 1), so that
// the column (row) difference across a corner is the one-sided derivative the
// box gradient takes.  Words: 0..2 column floors, 3..5 row floors, 6..8
// alpha, 9..11 beta, 12..20 coef'(ri, kj) of the mirrored pieces (as in the
// forward corner record); fp64 edges, each word rounded once.
__global__ void k_box_prep_corners_adj(const float* __restrict__ boxes, const float* __restrict__ piece_w, int CB,
                                       int nx, int ny, int* __restrict__ table) {
  const int box = blockIdx.x * blockDim.x + threadIdx.x;
  if (box >= CB) return;
  const float* q = boxes + (size_t)box * 4;
  const double cx = q[0], cy = q[1], rx = q[2], ry = q[3];
  const double a = 0.5 + cx - rx, b = 0.5 + cx + rx, c = 0.5 + cy - ry, d = 0.5 + cy + ry;
  const double ke[3] = {1.0 - b, nx == 2 ? 1.0 - (a + b) / 2 : 1.0 - a, 1.0 - a};
  const double re[3] = {1.0 - d, ny == 2 ? 1.0 - (c + d) / 2 : 1.0 - c, 1.0 - c};
  const float* wp = piece_w + (size_t)box * nx * ny;
  auto w = [&](int i, int j) -> double {  // weight of mirrored piece (i, j)
    return (i < 0 || j < 0 || i >= ny || j >= nx) ? 0.0 : (double)wp[(ny - 1 - i) * nx + (nx - 1 - j)];
  };
  int* r = table + (size_t)box * 32;
  float* f = reinterpret_cast<float*>(r);
  for (int k = 0; k <= nx; ++k) {
    int fl;
    double al;
    edge_split_upper(ke[k], 1 << 20, fl, al);
    r[k] = fl;
    f[6 + k] = (float)al;
  }
  for (int i = 0; i <= ny; ++i) {
    int fl;
    double be;
    edge_split_upper(re[i], 1 << 20, fl, be);
    r[3 + i] = fl;
    f[9 + i] = (float)be;
    for (int k = 0; k <= nx; ++k) f[12 + i * 3 + k] = (float)(w(i - 1, k - 1) - w(i - 1, k) - w(i, k - 1) + w(i, k));
  }
  for (int k = 21; k < 32; ++k) r[k] = 0;
}

// Backward walk of one split box over its mirrored corners on the table of
// an upstream-gradient map (record above).  For a table row R read at step s
// for row corner ri (R = y0 + s + f_ri + 1; R = y0 + f_ri at the start) and
// column corner kj, with D = S(R, x+f_kj+1) - S(R, x+f_kj) and X = S(R,
// x+f_kj) + alpha_kj * D (the row interpolated at the corner):
//   input gradient: acc[s'][q] += coef(ri, kj) * wy * X for the output rows
//     s' that read R (wy = beta for the row below the corner, 1 - beta for
//     the row above);
//   per-tap-row sums for the parameter gradient, with the input values v:
//     PX[ri][t][kj] += v[s'] * X and PD[ri][t][kj] += v[s'] * D, t = 1 for
//     the output row s' = s (R = its row f + 1), t = 0 for s' = s + 1.
template <int SEG, int NXC, int NYC, typename Src>
__device__ __forceinline__ void corner_adjoint_walk(const Src& S, const int* __restrict__ rec, int x0, int y0,
                                                    const float (&v)[SEG][kQ], float (&acc)[SEG][kQ],
                                                    float (&PX)[NYC][2][NXC], float (&PD)[NYC][2][NXC]) {
  const float* f = reinterpret_cast<const float*>(rec);
  const int W = S.W, H = S.H;
  const int st = S.row_step();
  typename Src::Col col[NXC];
  float al[NXC];
#pragma unroll
  for (int k = 0; k < NXC; ++k) {
    col[k] = S.col(x0 + clampi(rec[k], -(W + 1), W + 1));
    al[k] = f[6 + k];
  }
#pragma unroll
  for (int i = 0; i < NYC; ++i) {
    const int r0 = S.row_coord(y0 + clampi(rec[3 + i], -(H + 1), H + 1));
    const float be = f[9 + i], wy0 = 1.f - be;
    float cf[NXC];
#pragma unroll
    for (int k = 0; k < NXC; ++k) cf[k] = f[12 + i * 3 + k];
    // step s = -1 reads row y0 + f (the upper row of output row 0); step s
    // reads row y0 + s + f + 1 (lower row of output s, upper row of s + 1)
#pragma unroll
    for (int s = -1; s < SEG; ++s) {
      const typename Src::Row rr = S.row(r0 + (s + 1) * st);
      float R[kQ] = {0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < NXC; ++k) {
        float t[kQ + 1];
        S.run4(rr, col[k], t);
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
          const float D = t[q + 1] - t[q];
          const float X = fmaf(al[k], D, t[q]);
          R[q] = fmaf(cf[k], X, R[q]);
          if (s >= 0) {
            PX[i][1][k] = fmaf(v[s][q], X, PX[i][1][k]);
            PD[i][1][k] = fmaf(v[s][q], D, PD[i][1][k]);
          }
          if (s + 1 < SEG) {
            PX[i][0][k] = fmaf(v[s + 1][q], X, PX[i][0][k]);
            PD[i][0][k] = fmaf(v[s + 1][q], D, PD[i][0][k]);
          }
        }
      }
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        if (s >= 0) acc[s][q] = fmaf(be, R[q], acc[s][q]);
        if (s + 1 < SEG) acc[s + 1][q] = fmaf(wy0, R[q], acc[s + 1][q]);
      }
    }
  }
}

// One item's share of a split box's gradients from its per-tap-row sums
// (adjoint corner record f): per mirrored corner (ri, kj),
// Q = (1-beta) PX0 + beta PX1 (the corner's lookup, weighted by x),
// QX = (1-beta) PD0 + beta PD1 (its x derivative), QY = PX1 - PX0 (its y
// derivative); then
//   dL/dk'_kj = sum_ri coef(ri, kj) QX,  dL/dr'_ri = sum_kj coef(ri, kj) QY,
//   dL/dw'(i, j) = Q(i+1, j+1) - Q(i+1, j) - Q(i, j+1) + Q(i, j)
// (the mirrored piece's adjoint sum weighted by x).  Mirroring back:
// dL/dk_j = -dL/dk'_{nx-j}, a cut edge (the mean of the outer two) gives half
// to each, and dL/dw(i, j) = dL/dw'(ny-1-i, nx-1-j).  g8 = (dL/da, dL/db,
// dL/dc, dL/dd, dL/dw_0 .. dL/dw_3), unused weight slots 0.
template <int NXC, int NYC>
__device__ __forceinline__ void split_box_grads(const float* __restrict__ f, const float (&PX)[NYC][2][NXC],
                                                const float (&PD)[NYC][2][NXC], float (&g8)[8]) {
  constexpr int nx = NXC - 1, ny = NYC - 1;
  float Q[NYC][NXC], gk[NXC], gr[NYC];
#pragma unroll
  for (int k = 0; k < NXC; ++k) gk[k] = 0.f;
#pragma unroll
  for (int i = 0; i < NYC; ++i) {
    const float be = f[9 + i], wy0 = 1.f - be;
    gr[i] = 0.f;
#pragma unroll
    for (int k = 0; k < NXC; ++k) {
      const float cf = f[12 + i * 3 + k];
      Q[i][k] = fmaf(wy0, PX[i][0][k], be * PX[i][1][k]);
      gk[k] = fmaf(cf, fmaf(wy0, PD[i][0][k], be * PD[i][1][k]), gk[k]);
      gr[i] = fmaf(cf, PX[i][1][k] - PX[i][0][k], gr[i]);
    }
  }
  // mirrored corner kj is original corner nx - kj, with the sign flipped
  g8[0] = -gk[nx] - (nx == 2 ? 0.5f * gk[1] : 0.f);
  g8[1] = -gk[0] - (nx == 2 ? 0.5f * gk[1] : 0.f);
  g8[2] = -gr[ny] - (ny == 2 ? 0.5f * gr[1] : 0.f);
  g8[3] = -gr[0] - (ny == 2 ? 0.5f * gr[1] : 0.f);
#pragma unroll
  for (int k = 4; k < 8; ++k) g8[k] = 0.f;
#pragma unroll
  for (int i = 0; i < ny; ++i)
#pragma unroll
    for (int j = 0; j < nx; ++j)
      g8[4 + (ny - 1 - i) * nx + (nx - 1 - j)] = (Q[i + 1][j + 1] - Q[i + 1][j]) - (Q[i][j + 1] - Q[i][j]);
}

// Backward of split boxes, table in LDS: as k_box_bwd_lds (one block per map,
// one item of 3 columns x SEG rows per thread, input values in registers), one
// walk over each box's mirrored corners.  Each wave writes its split_box_grads
// sums to partials[(n * nw + wave) * C*B + c*B + b][8].
// kW > 0: the map width compiled in, as in k_box_bwd_lds.
template <int SEG, int NXC, int NYC, int kMaxT, int kW = 0>
__global__ __launch_bounds__(kMaxT) void k_box_bwd_lds_split(const float* __restrict__ x, const int* __restrict__ rec,
                                                           const float* __restrict__ gy, float* __restrict__ gx,
                                                           float* __restrict__ partials, int C, int H, int W_arg,
                                                           int B) {
  const int W = kW > 0 ? kW : W_arg;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int pitch = lds_pitch_dev(W);
  float* SG = reinterpret_cast<float*>(smem_raw);
  const int map = blockIdx.x, n = map / C, c = map - n * C;
  const int nw = blockDim.x >> 6, wave = threadIdx.x >> 6;
  const int nch = (W + kQ - 1) / kQ, nseg = (H + SEG - 1) / SEG;
  const int it = threadIdx.x;
  const bool active = it < nch * nseg;
  const int seg = it / nch, ch = it - seg * nch;
  const int x0 = ch * kQ, y0 = seg * SEG;
  const size_t plane = (size_t)H * W;
  const float* g0 = gy + (size_t)map * B * plane;
  float v[SEG][kQ], acc[SEG][kQ];
  load_item<SEG>(x + (size_t)map * plane, H, W, x0, y0, active, v);
#pragma unroll
  for (int s = 0; s < SEG; ++s)
#pragma unroll
    for (int q = 0; q < kQ; ++q) acc[s][q] = 0.f;
  const LdsTable<float> tg{SG, pitch, W, H};
  for (int b = 0; b < B; ++b) {
    __syncthreads();
    build_table_lds(g0 + b * plane, SG, H, W, pitch, 0.f, false);
    const int cb = c * B + b;
    const int* rb = rec + (size_t)cb * 32;
    float PX[NYC][2][NXC], PD[NYC][2][NXC];
#pragma unroll
    for (int i = 0; i < NYC; ++i)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int k = 0; k < NXC; ++k) { PX[i][t][k] = 0.f; PD[i][t][k] = 0.f; }
    if (active) corner_adjoint_walk<SEG, NXC, NYC>(tg, rb, x0, y0, v, acc, PX, PD);
    float g8[8];
    split_box_grads<NXC, NYC>(reinterpret_cast<const float*>(rb), PX, PD, g8);
    float* pp = partials + (((size_t)n * nw + wave) * C * B + cb) * 8;
    store_wave_partial(g8, pp);
    store_wave_partial(g8 + 4, pp + 4);
  }
  if (active && gx != nullptr) store_item<SEG>(gx + (size_t)map * plane, H, W, x0, y0, acc);
}

// Forward of split boxes, table in HBM: as k_box_fwd_gather (one block per
// (map, box, block of 256 items), one map's blocks on one XCD).
template <typename OutT, int SEG, int NXC, int NYC, bool kNT>
__global__ __launch_bounds__(256) void k_box_fwd_gather_split(const float* __restrict__ sat,
                                                              const int* __restrict__ rec, OutT* __restrict__ y,
                                                              int C, int H, int W, int B, int nblk, int total) {
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  if (L >= total) return;
  const int blk = L % nblk, mb = L / nblk;
  const int b = mb % B, map = mb / B, c = map % C;
  const int nch = (W + kQ - 1) / kQ, nseg = (H + SEG - 1) / SEG;
  const int it = blk * 256 + threadIdx.x;
  if (it >= nch * nseg) return;
  const int seg = it / nch, ch = it - seg * nch;
  const GlobalTable<float, true> tab{sat + (size_t)map * (H + 1) * (W + 1), W + 1, W, H};
  const int* rb = rec + (size_t)(c * B + b) * 32;
  OutT* out = y + ((size_t)map * B + b) * H * W;
  const int x0 = ch * kQ, y0 = seg * SEG, y1 = min(y0 + SEG, H);
  StoreRows<OutT, float, kNT> em{out, W, x0, y0 * W + x0};
  if (y0 + SEG <= H && x0 + kQ <= W) corner_walk<SEG, NXC, NYC, true>(tab, rb, x0, y0, y1, em);
  else corner_walk<SEG, NXC, NYC, false>(tab, rb, x0, y0, y1, em);
}

// Backward of split boxes, tables of the upstream-gradient maps in HBM: as
// k_box_bwd_gather (one block per (map, block of 256 items), looping over the
// boxes).  Each wave writes its split_box_grads sums to
// partials[((n * nblk + blk) * 4 + wave) * C*B + c*B + b][8].
template <int SEG, int NXC, int NYC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 8))) void k_box_bwd_gather_split(
    const float* __restrict__ x, const float* __restrict__ sat_g, const int* __restrict__ rec,
    float* __restrict__ gx, float* __restrict__ partials, int C, int H, int W, int B, int nblk, int total) {
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  if (L >= total) return;
  const int blk = L % nblk, map = L / nblk;
  const int n = map / C, c = map - n * C;
  const int wave = threadIdx.x >> 6;
  const int nch = (W + kQ - 1) / kQ, nseg = (H + SEG - 1) / SEG;
  const int it = blk * 256 + threadIdx.x;
  const bool active = it < nch * nseg;
  const int seg = it / nch, ch = it - seg * nch;
  const int x0 = ch * kQ, y0 = seg * SEG;
  const size_t tsz = (size_t)(H + 1) * (W + 1);
  float v[SEG][kQ], acc[SEG][kQ];
  load_item<SEG>(x + (size_t)map * H * W, H, W, x0, y0, active, v);
#pragma unroll
  for (int s = 0; s < SEG; ++s)
#pragma unroll
    for (int q = 0; q < kQ; ++q) acc[s][q] = 0.f;
  for (int b = 0; b < B; ++b) {
    const GlobalTable<float> tg{sat_g + ((size_t)map * B + b) * tsz, W + 1, W, H};
    const int cb = c * B + b;
    const int* rb = rec + (size_t)cb * 32;
    float PX[NYC][2][NXC], PD[NYC][2][NXC];
#pragma unroll
    for (int i = 0; i < NYC; ++i)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int k = 0; k < NXC; ++k) { PX[i][t][k] = 0.f; PD[i][t][k] = 0.f; }
    if (active) corner_adjoint_walk<SEG, NXC, NYC>(tg, rb, x0, y0, v, acc, PX, PD);
    float g8[8];
    split_box_grads<NXC, NYC>(reinterpret_cast<const float*>(rb), PX, PD, g8);
    float* pp = partials + ((((size_t)n * nblk + blk) * 4 + wave) * C * B + cb) * 8;
    store_wave_partial(g8, pp);
    store_wave_partial(g8 + 4, pp + 4);
  }
  if (active && gx != nullptr) store_item<SEG>(gx + (size_t)map * H * W, H, W, x0, y0, acc);
}

// Fixed-tree sum of the split partials [Pn][CB][8] (as k_box_grad_reduce) and
// the change of variables of the box edges; the weight gradients as summed.
__global__ __launch_bounds__(256) void k_split_grad_reduce(const float* __restrict__ partials, int Pn, int CB,
                                                           int P, float* __restrict__ grad_boxes,
                                                           float* __restrict__ grad_w) {
  __shared__ float4 red[4][kReduceBoxes][2];
  const int j = threadIdx.x % kReduceBoxes, q = threadIdx.x / kReduceBoxes;
  const int i = blockIdx.x * kReduceBoxes + j;
  float4 s0 = make_float4(0.f, 0.f, 0.f, 0.f), s1 = s0;
  if (i < CB)
    for (int p = q; p < Pn; p += 256 / kReduceBoxes) {
      const float4* v = reinterpret_cast<const float4*>(partials + ((size_t)p * CB + i) * 8);
      const float4 a = v[0], b = v[1];
      s0.x += a.x; s0.y += a.y; s0.z += a.z; s0.w += a.w;
      s1.x += b.x; s1.y += b.y; s1.z += b.z; s1.w += b.w;
    }
#pragma unroll
  for (int m = 16; m < 64; m <<= 1) {
    s0.x += __shfl_xor(s0.x, m); s0.y += __shfl_xor(s0.y, m); s0.z += __shfl_xor(s0.z, m); s0.w += __shfl_xor(s0.w, m);
    s1.x += __shfl_xor(s1.x, m); s1.y += __shfl_xor(s1.y, m); s1.z += __shfl_xor(s1.z, m); s1.w += __shfl_xor(s1.w, m);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) < kReduceBoxes) { red[wave][j][0] = s0; red[wave][j][1] = s1; }
  __syncthreads();
  if (threadIdx.x < kReduceBoxes && i < CB) {
    float t[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float4 a = red[w][j][0], b = red[w][j][1];
      t[0] += a.x; t[1] += a.y; t[2] += a.z; t[3] += a.w;
      t[4] += b.x; t[5] += b.y; t[6] += b.z; t[7] += b.w;
    }
    if (grad_boxes)
      *reinterpret_cast<float4*>(grad_boxes + (size_t)i * 4) = make_float4(t[0] + t[1], t[2] + t[3], t[1] - t[0], t[3] - t[2]);
    if (grad_w)
      for (int k = 0; k < P; ++k) grad_w[(size_t)i * P + k] = t[4 + k];
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
static hipError_t last_error() { return hipGetLastError(); }

hipError_t launch_box_prep(const float* boxes, int C, int B, bool rounded, void* table, hipStream_t s) {
  const int n = 2 * C * B;
  hipLaunchKernelGGL(k_box_prep, dim3((n + 255) / 256), dim3(256), 0, s, boxes, C * B, (int)rounded, (int*)table);
  return last_error();
}

hipError_t launch_unit_params(int op, const float* in, int n, float mw, float mh, float* out, hipStream_t s) {
  const dim3 grid((n + 255) / 256), block(256);
  if (op == 0) hipLaunchKernelGGL(k_boxes_from_unit, grid, block, 0, s, in, n, mw, mh, out);
  else if (op == 1) hipLaunchKernelGGL(k_unit_grad, grid, block, 0, s, in, n, mw, mh, out);
  else hipLaunchKernelGGL(k_clip_unit, grid, block, 0, s, out, n);
  return last_error();
}

// f(std::integral_constant<bool, v>) for the runtime flag v.
template <typename F>
static void with_flag(bool v, F&& f) {
  if (v) f(std::integral_constant<bool, true>{});
  else f(std::integral_constant<bool, false>{});
}

template <int KM, int kGroups>
static void sat_build_t(const void* x, bool is_int, void* sat, float* mean, int maps, int H, int W, hipStream_t s) {
  const size_t shm = (size_t)kStrip * kGroups * W * 4;
  if (is_int)
    hipLaunchKernelGGL((k_sat_build<int, false, KM, kGroups>), dim3(maps), dim3(256 * kGroups), shm, s,
                       (const int*)x, (int*)sat, (float*)nullptr, H, W, 1, H, W);
  else
    hipLaunchKernelGGL((k_sat_build<float, false, KM, kGroups>), dim3(maps), dim3(256 * kGroups), shm, s,
                       (const float*)x, (float*)sat, mean, H, W, 1, H, W);
}

// Fewer maps than 8 per CU leave one block per map short of filling the chip:
// then maps up to 256 wide take blocks of 1024 threads over 64-row strips.
constexpr int kSatFewMaps = 2048;

hipError_t launch_sat_build(const void* x, bool is_int, void* sat, float* mean, int maps, int H, int W,
                            hipStream_t s) {
  if (W <= 256 && maps < kSatFewMaps) sat_build_t<4, 4>(x, is_int, sat, mean, maps, H, W, s);
  else if (W <= 256) sat_build_t<4, 1>(x, is_int, sat, mean, maps, H, W, s);
  else sat_build_t<kSatMaxK, 1>(x, is_int, sat, mean, maps, H, W, s);
  return last_error();
}

hipError_t launch_sat_build_up(const float* x, float* sat, int maps, int H, int W, int stride, hipStream_t s) {
  const size_t shm = (size_t)kStrip * W * 4;
  const int Ho = (H + stride - 1) / stride, Wo = (W + stride - 1) / stride;
  if (W <= 256)
    hipLaunchKernelGGL((k_sat_build<float, true, 4, 1>), dim3(maps), dim3(256), shm, s, x, sat, (float*)nullptr, H,
                       W, stride, Ho, Wo);
  else
    hipLaunchKernelGGL((k_sat_build<float, true, kSatMaxK, 1>), dim3(maps), dim3(256), shm, s, x, sat,
                       (float*)nullptr, H, W, stride, Ho, Wo);
  return last_error();
}

// Forward launch geometry shared by both LDS kernels.
struct FwdGeom { int per_box_p, bpg, ngrp, threads; };
static FwdGeom fwd_geom_items(int N, int C, int B, int per_box) {
  FwdGeom g;
  g.per_box_p = ((per_box + 63) / 64) * 64;
  g.bpg = 256 / g.per_box_p;
  if (g.bpg < 1) g.bpg = 1;
  if (g.bpg > B) g.bpg = B;
  // keep enough blocks in flight to fill the chip
  while (g.bpg > 1 && (long)N * C * ((B + g.bpg - 1) / g.bpg) < 2048) g.bpg = (g.bpg + 1) / 2;
  g.ngrp = (B + g.bpg - 1) / g.bpg;
  g.threads = min(g.bpg * g.per_box_p, 256);
  return g;
}
static FwdGeom fwd_geom(int N, int C, int H, int W, int B, int seg) {
  return fwd_geom_items(N, C, B, n_chunks(W) * n_segs(H, seg));
}

// The pose network's maps are 48 columns wide (a 192-pixel-wide input at
// stride 4): the LDS forward and backward take instances with that width
// compiled in.
constexpr int kPoseW = 48;

template <typename T, typename OutT, bool kOffset>
static void fwd_lds_t(const void* x, const int* taps, void* y, int N, int C, int H, int W, int B, bool rounded,
                      int stride, hipStream_t s) {
  constexpr int SEG = 16;
  const size_t shm = (size_t)(H + 1) * lds_pitch(W) * sizeof(T);
  if (stride == 1) {
    // bf16 output of 48-column maps, 4-byte aligned: items of 6 columns x 8
    // rows (still 64 per box on 64-row maps), each row stored as 3 packed
    // words
    if constexpr (std::is_same<T, float>::value && std::is_same<OutT, uint16_t>::value) {
      if (W == kPoseW && ((uintptr_t)y & 3) == 0) {  // the ABI also requires 16-byte aligned tensors
        constexpr int kSeg6 = 8, kQ6 = 6;
        const FwdGeom g6 = fwd_geom_items(N, C, B, ((W + kQ6 - 1) / kQ6) * n_segs(H, kSeg6));
        with_flag(rounded, [&](auto ki) {
          hipLaunchKernelGGL((k_box_fwd_lds<T, OutT, kSeg6, kOffset, decltype(ki)::value, kPoseW, kQ6, true>),
                             dim3(N * C * g6.ngrp), dim3(g6.threads), shm, s, (const T*)x, taps, (OutT*)y, C, H, W,
                             B, g6.bpg, g6.per_box_p);
        });
        return;
      }
    }
    const FwdGeom g = fwd_geom(N, C, H, W, B, SEG);
    with_flag(rounded, [&](auto ki) {
      if (std::is_same<T, float>::value && W == kPoseW)
        hipLaunchKernelGGL((k_box_fwd_lds<T, OutT, SEG, kOffset, decltype(ki)::value, kPoseW>), dim3(N * C * g.ngrp),
                           dim3(g.threads), shm, s, (const T*)x, taps, (OutT*)y, C, H, W, B, g.bpg, g.per_box_p);
      else
        hipLaunchKernelGGL((k_box_fwd_lds<T, OutT, SEG, kOffset, decltype(ki)::value>), dim3(N * C * g.ngrp),
                           dim3(g.threads), shm, s, (const T*)x, taps, (OutT*)y, C, H, W, B, g.bpg, g.per_box_p);
    });
    return;
  }
  const int Ho = (H + stride - 1) / stride, Wo = (W + stride - 1) / stride;
  const FwdGeom g = fwd_geom_items(N, C, B, Wo * ((Ho + kSegS - 1) / kSegS));
  with_flag(rounded, [&](auto ki) {
    if (std::is_same<T, float>::value && W == kPoseW)
      hipLaunchKernelGGL((k_box_fwd_lds_strided<T, OutT, kOffset, decltype(ki)::value, kPoseW>), dim3(N * C * g.ngrp),
                         dim3(g.threads), shm, s, (const T*)x, taps, (OutT*)y, C, H, W, B, stride, Ho, Wo, g.bpg,
                         g.per_box_p);
    else
      hipLaunchKernelGGL((k_box_fwd_lds_strided<T, OutT, kOffset, decltype(ki)::value>), dim3(N * C * g.ngrp),
                         dim3(g.threads), shm, s, (const T*)x, taps, (OutT*)y, C, H, W, B, stride, Ho, Wo, g.bpg,
                         g.per_box_p);
  });
}

hipError_t launch_box_fwd_lds(const void* x, bool is_int, const int* taps, void* y, int out_kind, int N, int C,
                              int H, int W, int B, bool offset, bool rounded, int stride, hipStream_t s) {
  if (is_int) {
    fwd_lds_t<int, int, false>(x, taps, y, N, C, H, W, B, rounded, stride, s);
  } else if (out_kind == 2) {
    if (offset) fwd_lds_t<float, uint16_t, true>(x, taps, y, N, C, H, W, B, rounded, stride, s);
    else fwd_lds_t<float, uint16_t, false>(x, taps, y, N, C, H, W, B, rounded, stride, s);
  } else {
    if (offset) fwd_lds_t<float, float, true>(x, taps, y, N, C, H, W, B, rounded, stride, s);
    else fwd_lds_t<float, float, false>(x, taps, y, N, C, H, W, B, rounded, stride, s);
  }
  return last_error();
}

// The HBM-table forwards re-read their tables through the caches; an output
// larger than the last-level cache (256 MiB) cannot stay there for the next
// call anyway, so 4-byte outputs that large are stored non-temporally and
// leave the caches to the tables (4 x 128 maps of 256x256, 8 boxes, fp32
// out: 893 -> 776 us).  Narrower outputs keep ordinary stores: 2-byte
// non-temporal stores were slower.
constexpr size_t kStreamOutBytes = (size_t)256 << 20;
static bool stream_out(size_t elems, size_t bytes_per) { return bytes_per == 4 && elems * bytes_per > kStreamOutBytes; }

template <typename T, typename OutT, bool kOffset>
static void fwd_gather_t(const void* sat, const float* means, const int* taps, void* y, int N, int C, int H, int W,
                         int B, bool rounded, int stride, hipStream_t s) {
  constexpr int SEG = 16;
  if (stride == 1) {
    const int items = n_chunks(W) * n_segs(H, SEG);
    const int nblk = (items + 255) / 256;
    const int total = N * C * B * nblk;
    const bool nt = stream_out((size_t)N * C * B * H * W, sizeof(OutT));
    with_flag(rounded, [&](auto ki) {
      with_flag(nt, [&](auto kn) {
        hipLaunchKernelGGL((k_box_fwd_gather<T, OutT, SEG, kOffset, decltype(ki)::value, decltype(kn)::value>),
                           dim3(pad8(total)), dim3(256), 0, s, (const T*)sat, means, taps, (OutT*)y, C, H, W, B, nblk,
                           total);
      });
    });
    return;
  }
  const int Ho = (H + stride - 1) / stride, Wo = (W + stride - 1) / stride;
  const int nblk = (Wo * ((Ho + kSegS - 1) / kSegS) + 255) / 256;
  const int total = N * C * B * nblk;
  with_flag(rounded, [&](auto ki) {
    hipLaunchKernelGGL((k_box_fwd_gather_strided<T, OutT, kOffset, decltype(ki)::value>), dim3(pad8(total)),
                       dim3(256), 0, s, (const T*)sat, means, taps, (OutT*)y, C, H, W, B, stride, Ho, Wo, nblk,
                       total);
  });
}

hipError_t launch_box_fwd_gather(const void* sat, bool is_int, const float* means, const int* taps, void* y,
                                 int out_kind, int N, int C, int H, int W, int B, bool rounded, int stride,
                                 hipStream_t s) {
  const bool offset = means != nullptr;
  if (is_int) {
    fwd_gather_t<int, int, false>(sat, nullptr, taps, y, N, C, H, W, B, rounded, stride, s);
  } else if (out_kind == 2) {
    if (offset) fwd_gather_t<float, uint16_t, true>(sat, means, taps, y, N, C, H, W, B, rounded, stride, s);
    else fwd_gather_t<float, uint16_t, false>(sat, nullptr, taps, y, N, C, H, W, B, rounded, stride, s);
  } else {
    if (offset) fwd_gather_t<float, float, true>(sat, means, taps, y, N, C, H, W, B, rounded, stride, s);
    else fwd_gather_t<float, float, false>(sat, nullptr, taps, y, N, C, H, W, B, rounded, stride, s);
  }
  return last_error();
}

template <int SEG, int kMaxT>
static void bwd_lds_t(const float* x, const int* taps, const float* gy, void* gx, float* partials, int N, int C,
                      int H, int W, int B, bool rounded, bool relu_bf16, int stride, hipStream_t s) {
  const int items = n_chunks(W) * n_segs(H, SEG);
  const int threads = ((items + 63) / 64) * 64;
  const size_t shm = (size_t)(H + 1) * lds_pitch(W) * sizeof(float);
  const int Ho = (H + stride - 1) / stride, Wo = (W + stride - 1) / stride;
  auto go = [&](auto ki, auto ku, auto kr) {
    if (SEG == 8 && W == kPoseW)
      hipLaunchKernelGGL((k_box_bwd_lds<SEG, decltype(ki)::value, decltype(ku)::value, kMaxT, decltype(kr)::value, kPoseW>),
                         dim3(N * C), dim3(threads), shm, s, x, taps, gy, gx, partials, C, H, W, B, stride, Ho, Wo);
    else
      hipLaunchKernelGGL((k_box_bwd_lds<SEG, decltype(ki)::value, decltype(ku)::value, kMaxT, decltype(kr)::value>),
                         dim3(N * C), dim3(threads), shm, s, x, taps, gy, gx, partials, C, H, W, B, stride, Ho, Wo);
  };
  with_flag(stride > 1, [&](auto ku) {
    if (rounded) go(std::true_type{}, ku, std::false_type{});
    else with_flag(relu_bf16, [&](auto kr) { go(std::false_type{}, ku, kr); });
  });
}

// Segment length of the LDS backward: 8 rows when the map's items fit one
// 256-thread block, else 4 while they fit max_items threads; 0 = too many.
// The 4-row walk fits 128 VGPRs, so its blocks may take up to 1024 threads
// (maps up to 128x96 or 256x48): one block per CU, 16 waves.
int box_bwd_lds_seg(int H, int W, int max_items) {
  if (n_chunks(W) * n_segs(H, 8) <= 256) return 8;
  if (n_chunks(W) * n_segs(H, 4) <= max_items) return 4;
  return 0;
}

int box_bwd_lds_waves(int H, int W, int max_items) {
  const int seg = box_bwd_lds_seg(H, W, max_items);
  return seg == 0 ? 0 : (n_chunks(W) * n_segs(H, seg) + 63) / 64;
}

// A call whose maps give fewer than kBwdFillWaves waves with 8-row items
// takes 4-row items instead (twice the waves, each with fewer registers):
// 8 x 64 maps of 64x48 with 8 boxes, 51.5 -> 46.4 us; with 32 x 256 maps the
// 8-row items stay faster (163 against 209 us).
constexpr long kBwdFillWaves = 2048;  // 8 waves on each of 256 CUs
int box_bwd_lds_seg_maps(int H, int W, long maps) {
  const int seg = box_bwd_lds_seg(H, W, kBwdLdsItems);
  if (seg == 8 && maps * ((n_chunks(W) * n_segs(H, 8) + 63) / 64) < kBwdFillWaves &&
      n_chunks(W) * n_segs(H, 4) <= 256)
    return 4;
  return seg;
}

int box_bwd_lds_waves_maps(int H, int W, long maps) {
  const int seg = box_bwd_lds_seg_maps(H, W, maps);
  return seg == 0 ? 0 : (n_chunks(W) * n_segs(H, seg) + 63) / 64;
}

hipError_t launch_box_bwd_lds(const float* x, const int* taps, const float* gy, void* gx, float* partials, int N,
                              int C, int H, int W, int B, bool rounded, bool relu_bf16, int stride, hipStream_t s) {
  if (rounded && relu_bf16) return hipErrorInvalidValue;
  const int seg = box_bwd_lds_seg_maps(H, W, (long)N * C);
  if (seg == 8) bwd_lds_t<8, 256>(x, taps, gy, gx, partials, N, C, H, W, B, rounded, relu_bf16, stride, s);
  else if (seg == 4 && n_chunks(W) * n_segs(H, 4) <= 256)
    bwd_lds_t<4, 256>(x, taps, gy, gx, partials, N, C, H, W, B, rounded, relu_bf16, stride, s);
  else if (seg == 4)
    bwd_lds_t<4, kBwdLdsItems>(x, taps, gy, gx, partials, N, C, H, W, B, rounded, relu_bf16, stride, s);
  else return hipErrorInvalidValue;
  return last_error();
}

constexpr int kBwdGatherSeg = 8;

int box_bwd_gather_blocks(int H, int W) { return (n_chunks(W) * n_segs(H, kBwdGatherSeg) + 255) / 256; }

hipError_t launch_box_bwd_gather(const float* x, const float* sat_g, const int* taps, void* gx, float* partials,
                                 int N, int C, int H, int W, int B, bool rounded, bool relu_bf16, hipStream_t s) {
  if (rounded && relu_bf16) return hipErrorInvalidValue;
  const int nblk = box_bwd_gather_blocks(H, W);
  const int total = N * C * nblk;
  auto go = [&](auto ki, auto kr) {
    hipLaunchKernelGGL((k_box_bwd_gather<kBwdGatherSeg, decltype(ki)::value, decltype(kr)::value>), dim3(pad8(total)),
                       dim3(256), 0, s, x, sat_g, taps, gx, partials, C, H, W, B, nblk, total);
  };
  if (rounded) go(std::true_type{}, std::false_type{});
  else with_flag(relu_bf16, [&](auto kr) { go(std::false_type{}, kr); });
  return last_error();
}

hipError_t launch_box_grad_reduce(const float* partials, int P, int CB, float* grad_boxes, hipStream_t s) {
  hipLaunchKernelGGL(k_box_grad_reduce, dim3((CB + kReduceBoxes - 1) / kReduceBoxes), dim3(256), 0, s, partials, P, CB,
                     grad_boxes);
  return last_error();
}

hipError_t launch_box_prep_corners(const float* boxes, const float* piece_w, int C, int B, int nx, int ny,
                                   void* table, hipStream_t s) {
  const int n = C * B;
  hipLaunchKernelGGL(k_box_prep_corners, dim3((n + 255) / 256), dim3(256), 0, s, boxes, piece_w, n, nx, ny,
                     (int*)table);
  return last_error();
}

template <typename OutT, int NXC, int NYC>
static void fwd_split_t(const float* x, const int* rec, void* y, int N, int C, int H, int W, int B, hipStream_t s) {
  constexpr int SEG = 16;
  const size_t shm = (size_t)(H + 1) * lds_pitch(W) * sizeof(float);
  const FwdGeom g = fwd_geom(N, C, H, W, B, SEG);
  hipLaunchKernelGGL((k_box_fwd_lds_split<OutT, SEG, NXC, NYC>), dim3(N * C * g.ngrp), dim3(g.threads), shm, s, x,
                     rec, (OutT*)y, C, H, W, B, g.bpg, g.per_box_p);
}

template <typename OutT>
static void fwd_split_mode(const float* x, const int* rec, void* y, int N, int C, int H, int W, int B, int nx, int ny,
                           hipStream_t s) {
  if (nx == 2 && ny == 2) fwd_split_t<OutT, 3, 3>(x, rec, y, N, C, H, W, B, s);
  else if (nx == 2) fwd_split_t<OutT, 3, 2>(x, rec, y, N, C, H, W, B, s);
  else fwd_split_t<OutT, 2, 3>(x, rec, y, N, C, H, W, B, s);
}

hipError_t launch_box_fwd_lds_split(const float* x, const int* rec, void* y, bool bf16_out, int N, int C, int H, int W,
                                    int B, int nx, int ny, hipStream_t s) {
  if (bf16_out) fwd_split_mode<uint16_t>(x, rec, y, N, C, H, W, B, nx, ny, s);
  else fwd_split_mode<float>(x, rec, y, N, C, H, W, B, nx, ny, s);
  return last_error();
}

hipError_t launch_box_prep_corners_adj(const float* boxes, const float* piece_w, int C, int B, int nx, int ny,
                                       void* table, hipStream_t s) {
  const int n = C * B;
  hipLaunchKernelGGL(k_box_prep_corners_adj, dim3((n + 255) / 256), dim3(256), 0, s, boxes, piece_w, n, nx, ny,
                     (int*)table);
  return last_error();
}

template <int SEG, int NXC, int NYC, int kMaxT>
static void bwd_split_t(const float* x, const int* rec, const float* gy, float* gx, float* partials, int N, int C,
                        int H, int W, int B, hipStream_t s) {
  const int threads = ((n_chunks(W) * n_segs(H, SEG) + 63) / 64) * 64;
  const size_t shm = (size_t)(H + 1) * lds_pitch(W) * sizeof(float);
  if (SEG == 8 && W == kPoseW)
    hipLaunchKernelGGL((k_box_bwd_lds_split<SEG, NXC, NYC, kMaxT, kPoseW>), dim3(N * C), dim3(threads), shm, s, x,
                       rec, gy, gx, partials, C, H, W, B);
  else
    hipLaunchKernelGGL((k_box_bwd_lds_split<SEG, NXC, NYC, kMaxT>), dim3(N * C), dim3(threads), shm, s, x, rec, gy,
                       gx, partials, C, H, W, B);
}

template <int SEG, int kMaxT>
static void bwd_split_mode(const float* x, const int* rec, const float* gy, float* gx, float* partials, int N, int C,
                           int H, int W, int B, int nx, int ny, hipStream_t s) {
  if (nx == 2 && ny == 2) bwd_split_t<SEG, 3, 3, kMaxT>(x, rec, gy, gx, partials, N, C, H, W, B, s);
  else if (nx == 2) bwd_split_t<SEG, 3, 2, kMaxT>(x, rec, gy, gx, partials, N, C, H, W, B, s);
  else bwd_split_t<SEG, 2, 3, kMaxT>(x, rec, gy, gx, partials, N, C, H, W, B, s);
}

// As the whole-box backward: 8-row items in blocks of up to 256 threads, else
// 4-row items (at most 107 VGPRs) in blocks of up to kBwdLdsItems threads.
hipError_t launch_box_bwd_lds_split(const float* x, const int* rec, const float* gy, float* gx, float* partials, int N,
                                    int C, int H, int W, int B, int nx, int ny, hipStream_t s) {
  const int seg = box_bwd_lds_seg(H, W, kBwdLdsItems);
  if (seg == 8) bwd_split_mode<8, 256>(x, rec, gy, gx, partials, N, C, H, W, B, nx, ny, s);
  else if (seg == 4 && n_chunks(W) * n_segs(H, 4) <= 256)
    bwd_split_mode<4, 256>(x, rec, gy, gx, partials, N, C, H, W, B, nx, ny, s);
  else if (seg == 4) bwd_split_mode<4, kBwdLdsItems>(x, rec, gy, gx, partials, N, C, H, W, B, nx, ny, s);
  else return hipErrorInvalidValue;
  return last_error();
}

template <typename OutT, int NXC, int NYC>
static void fwd_gather_split_t(const float* sat, const int* rec, void* y, int N, int C, int H, int W, int B,
                               hipStream_t s) {
  constexpr int SEG = 16;
  const int nblk = (n_chunks(W) * n_segs(H, SEG) + 255) / 256;
  const int total = N * C * B * nblk;
  with_flag(stream_out((size_t)N * C * B * H * W, sizeof(OutT)), [&](auto kn) {
    hipLaunchKernelGGL((k_box_fwd_gather_split<OutT, SEG, NXC, NYC, decltype(kn)::value>), dim3(pad8(total)),
                       dim3(256), 0, s, sat, rec, (OutT*)y, C, H, W, B, nblk, total);
  });
}

template <typename OutT>
static void fwd_gather_split_mode(const float* sat, const int* rec, void* y, int N, int C, int H, int W, int B, int nx,
                                  int ny, hipStream_t s) {
  if (nx == 2 && ny == 2) fwd_gather_split_t<OutT, 3, 3>(sat, rec, y, N, C, H, W, B, s);
  else if (nx == 2) fwd_gather_split_t<OutT, 3, 2>(sat, rec, y, N, C, H, W, B, s);
  else fwd_gather_split_t<OutT, 2, 3>(sat, rec, y, N, C, H, W, B, s);
}

hipError_t launch_box_fwd_gather_split(const float* sat, const int* rec, void* y, bool bf16_out, int N, int C, int H,
                                       int W, int B, int nx, int ny, hipStream_t s) {
  if (bf16_out) fwd_gather_split_mode<uint16_t>(sat, rec, y, N, C, H, W, B, nx, ny, s);
  else fwd_gather_split_mode<float>(sat, rec, y, N, C, H, W, B, nx, ny, s);
  return last_error();
}

template <int NXC, int NYC>
static void bwd_gather_split_t(const float* x, const float* sat_g, const int* rec, float* gx, float* partials, int N,
                               int C, int H, int W, int B, hipStream_t s) {
  const int nblk = box_bwd_gather_blocks(H, W);
  const int total = N * C * nblk;
  hipLaunchKernelGGL((k_box_bwd_gather_split<kBwdGatherSeg, NXC, NYC>), dim3(pad8(total)), dim3(256), 0, s, x, sat_g,
                     rec, gx, partials, C, H, W, B, nblk, total);
}

hipError_t launch_box_bwd_gather_split(const float* x, const float* sat_g, const int* rec, float* gx, float* partials,
                                       int N, int C, int H, int W, int B, int nx, int ny, hipStream_t s) {
  if (nx == 2 && ny == 2) bwd_gather_split_t<3, 3>(x, sat_g, rec, gx, partials, N, C, H, W, B, s);
  else if (nx == 2) bwd_gather_split_t<3, 2>(x, sat_g, rec, gx, partials, N, C, H, W, B, s);
  else bwd_gather_split_t<2, 3>(x, sat_g, rec, gx, partials, N, C, H, W, B, s);
  return last_error();
}

hipError_t launch_split_grad_reduce(const float* partials, int Pn, int CB, int P, float* grad_boxes, float* grad_w,
                                    hipStream_t s) {
  hipLaunchKernelGGL(k_split_grad_reduce, dim3((CB + kReduceBoxes - 1) / kReduceBoxes), dim3(256), 0, s, partials,
                     Pn, CB, P, grad_boxes, grad_w);
  return last_error();
}

}  // namespace bc
