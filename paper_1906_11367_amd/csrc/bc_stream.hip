// Streaming box kernels: the summed-area table is never stored.  A group of
// lanes walks one box down the map, output row by output row, keeping the two
// table rows each y edge needs as running column prefix sums (two cursors);
// each step forms one row from them and scans it once across the group.
//
// Why this is the same computation (Section 3.1, Eq. 2-3).  With the
// exclusive table S(u, v) = sum_{i<u, j<v} I(i, j), the column prefix
// P(u, j) = sum_{i<u} I(i, j) and the row prefix of a row vector R,
// (scan R)(v) = sum_{j<v} R(j), the table row is S(u, .) = scan P(u, .).  A
// box's bilinear corner samples at output row y are
//   sum_r wy[r] * sum_k wx[k] * S(u_r, x + ox[k]),   u_r = y + oy[r] (clamped),
// and since the row scan is linear, sum_r wy[r] S(u_r, .) = scan Y with
//   Y = sum_r wy[r] P(u_r, .).
// The rows u_r come in pairs (f, f + 1) at each y edge, P(f + 1) = P(f) +
// I(f), and the two weights of a pair sum to -1 (upper edge) and +1 (lower
// edge), so
//   Y = P(y + fd) - P(y + fc) - beta_c * I(y + fc) + beta_d * I(y + fd)
// (beta the edges' fractions).  Per output row each cursor adds one map row,
// Y takes three operations per column, one scan gives scan Y, and the x
// taps are read from it exactly as from a table row.  Clamping a table
// index to [0, H] x [0, W] is zero padding; here a cursor outside the map
// adds nothing, and the scanned row is padded with 0 on the left and its
// last value on the right.
//
// Backward (the adjoint box on the upstream gradient G, as the table
// kernels do):
//   input gradient  sum_b of the adjoint box sums of G_b;
//   edge gradients  dL/da = -sum v * DB, dL/db = sum v * DA, where DA, DB
//                   are the differences of scan Y across the adjoint's two x
//                   edges (the y-weighted column differences) and v the input;
//                   dL/dc = -sum_j G(y + fd, j) * T(j), dL/dd =
//                   sum_j G(y + fc, j) * T(j), with T(j) = sum_k wx[k] *
//                   V(j + 1 - ox[k]) and V(t) = sum_{x >= t} v(y, x), the
//                   suffix sums of the input row: the x-interpolated row of the
//                   table of the single row G(y + f) weighted by v, moved onto
//                   the input row (sum_x v(x) sum_k wx[k] sum_{j < x+ox[k]} G(j)
//                   = sum_j G(j) T(j)).
// Lane layout: a group of LG lanes holds one box's row, CPL consecutive
// columns per lane (LG * CPL >= W); LG = 16 puts four boxes in a wave (one
// per DPP row, scans by row shifts), LG = 64 one box per wave.
#include "bc_common.hpp"
#include "bc_internal.hpp"

#include <algorithm>
#include <type_traits>

namespace bc {
namespace {

template <typename T> __device__ __forceinline__ int bits_of(T v) { return __builtin_bit_cast(int, v); }
template <typename T> __device__ __forceinline__ T of_bits(int v) { return __builtin_bit_cast(T, v); }

// Inclusive prefix (kRev: suffix) sum over the lanes of each group of LG
// lanes, for every lane.  LG = 16: row shifts within each DPP row; LG = 64:
// then the row broadcasts carry each row's total into the rows after it.
template <int LG, bool kRev, typename T>
__device__ __forceinline__ T group_scan(T v) {
  static_assert(LG == 16 || LG == 64, "groups are DPP rows or whole waves");
  if constexpr (!kRev) {
    v += of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(v), 0x111, 0xF, 0xF, true));  // row_shr:1
    v += of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(v), 0x112, 0xF, 0xF, true));  // row_shr:2
    v += of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(v), 0x114, 0xF, 0xF, true));  // row_shr:4
    v += of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(v), 0x118, 0xF, 0xF, true));  // row_shr:8
    if constexpr (LG == 64) {
      v += of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(v), 0x142, 0xA, 0xF, false));  // row_bcast:15
      v += of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(v), 0x143, 0xC, 0xF, false));  // row_bcast:31
    }
  } else {
    v += of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(v), 0x101, 0xF, 0xF, true));  // row_shl:1
    v += of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(v), 0x102, 0xF, 0xF, true));  // row_shl:2
    v += of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(v), 0x104, 0xF, 0xF, true));  // row_shl:4
    v += of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(v), 0x108, 0xF, 0xF, true));  // row_shl:8
    if constexpr (LG == 64) {
      // rows after this one: lane 0 of the next row holds that row's total,
      // then the rows beyond it (a reversed scan of the four row totals)
      const int lane = threadIdx.x & 63, row = lane >> 4;
      const T t1 = __shfl(v, ((row + 1) & 3) << 4, 64);
      const T t2 = __shfl(v, ((row + 2) & 3) << 4, 64);
      const T t3 = __shfl(v, ((row + 3) & 3) << 4, 64);
      v += (row < 3 ? t1 : (T)0) + (row < 2 ? t2 : (T)0) + (row < 1 ? t3 : (T)0);
    }
  }
  return v;
}

// Exclusive form of group_scan: the inclusive scan moved one lane along the
// scan direction (lane 0 of the group, or its last lane when reversed, gets 0
// from bound_ctrl).  Taking the neighbour's inclusive value, rather than
// subtracting the lane's own value from its inclusive scan, keeps a lane's
// earlier columns exact when a later column holds a NaN or an infinity, and
// costs the same one instruction.
template <int LG, bool kRev, typename T>
__device__ __forceinline__ T group_excl(T v) {
  const T incl = group_scan<LG, kRev>(v);
  constexpr int ctrl = kRev ? (LG == 16 ? 0x101 : 0x130)    // row_shl:1 / wave_shl:1
                            : (LG == 16 ? 0x111 : 0x138);   // row_shr:1 / wave_shr:1
  return of_bits<T>(__builtin_amdgcn_update_dpp(0, bits_of(incl), ctrl, 0xF, 0xF, true));
}

// Sum over the lanes of a group, in every lane of the group.
template <int LG>
__device__ __forceinline__ float group_sum(float v) {
  v = row16_sum(v);
  if constexpr (LG == 64) {
    v += __shfl_xor(v, 16, 64);
    v += __shfl_xor(v, 32, 64);
  }
  return v;
}

}  // namespace

// Padding of a group's scanned row in LDS, on each side: a run of CPL + 1
// consecutive entries whose start is clamped to [-pad, W] then reads exactly
// the clamped entries.
template <int CPL> constexpr int stream_pad() { return CPL + 1; }
// With an even CPL, lanes address a row CPL words apart, which puts lanes 32
// / CPL apart on one LDS bank; one skip word every 32 words (index i at
// i + i / 32) spreads them over all banks.  Odd CPL needs none.
template <int CPL> constexpr bool stream_skew() { return CPL % 2 == 0; }
template <int LG, int CPL> constexpr int stream_row_words() {
  constexpr int n = 2 * stream_pad<CPL>() + LG * CPL + 1;
  return stream_skew<CPL>() ? n + n / 32 + 1 : n;
}
// LDS index of row entry v (v in [-pad, LG * CPL + pad]).
template <int CPL>
__device__ __forceinline__ int stream_at(int v) {
  const int i = v + stream_pad<CPL>();
  return stream_skew<CPL>() ? i + (i >> 5) : i;
}
// LDS index of element j of a group's input-gradient slot (j in [0, LG*CPL)).
template <int CPL>
__device__ __forceinline__ int slot_at(int j) { return stream_skew<CPL>() ? j + (j >> 5) : j; }
template <int LG, int CPL> constexpr int slot_words() { return stream_skew<CPL>() ? LG * CPL + LG * CPL / 32 : LG * CPL; }

// Rows of a step are loaded kPrefetch steps ahead (a ring of registers), so
// that a step's loads are in flight while the steps before it compute.
constexpr int kPrefetch = 2;

// The lane's CPL columns of a map row: byte offsets within a row (columns
// outside the map clamped onto its last column, so every load is in bounds)
// and which of them lie in the map.  A row is then CPL loads from one uniform
// base plus a per-lane 32-bit offset.
template <int CPL>
struct LaneCols {
  unsigned off[CPL];
  bool in[CPL];
  __device__ __forceinline__ LaneCols(int x0, int W) {
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      in[k] = x0 + k < W;
      off[k] = 4u * (unsigned)min(x0 + k, W - 1);
    }
  }
  // row `row` of the map at byte offset `mapoff` from base (rows outside
  // [0, H) and columns outside the map read as 0).  The load is always made
  // (from a valid address) and its bits masked, so no branch surrounds it.
  // kVec: every lane's CPL columns lie in the map (W == LG * CPL) and rows
  // are 16-byte aligned, so a row is one 16-byte load per lane (CPL = 4).
  template <bool kVec, typename T>
  __device__ __forceinline__ void load(const T* base, unsigned mapoff, int row, int H, int W, bool live,
                                       T* r) const {
    const bool ok = live && row >= 0 && row < H;
    const unsigned ro = ok ? mapoff + 4u * (unsigned)(row * W) : 0u;
    const char* b = reinterpret_cast<const char*>(base);
    if constexpr (kVec && CPL == 4) {
      typedef int i4 __attribute__((ext_vector_type(4)));
      const i4 t = *reinterpret_cast<const i4*>(b + (ro + off[0]));
      const int m = ok ? -1 : 0;
      r[0] = __builtin_bit_cast(T, t.x & m);
      r[1] = __builtin_bit_cast(T, t.y & m);
      r[2] = __builtin_bit_cast(T, t.z & m);
      r[3] = __builtin_bit_cast(T, t.w & m);
    } else {
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        const int t = *reinterpret_cast<const int*>(b + (ro + off[k]));
        const int m = (ok && in[k]) ? -1 : 0;
        r[k] = __builtin_bit_cast(T, t & m);
      }
    }
  }
};

// ---------------------------------------------------------------------------
// Backward.  One block of NG groups per map (n, c); group g walks box b = g.
// dx: each group leaves its adjoint sums in LDS slots; every R rows the
// block adds the NG slots of each element in a fixed order and writes dx
// (two slot sets alternate, so one barrier per R rows orders every write
// before its reads and every read before the slot's next write).  kInt:
// boxes with integer corners (input gradient only, x not read).  kRelu: dx
// written as bf16(x > 0 ? dx : 0).  partials: [n][C*B][4] edge gradients
// (one row per image).
// ---------------------------------------------------------------------------
template <int LG, int CPL, int NG, bool kInt, bool kRelu, bool kVec>
__global__ __launch_bounds__(LG * NG) void k_box_bwd_stream(const float* __restrict__ x, const int* __restrict__ taps,
                                                            const float* __restrict__ gy, void* __restrict__ gx,
                                                            float* __restrict__ partials, int C, int H, int W, int B,
                                                            int R) {
  static_assert(!(kInt && kRelu), "the ReLU mask needs x");
  constexpr int PAD = stream_pad<CPL>();
  constexpr int RW = stream_row_words<LG, CPL>();
  constexpr int PF = kPrefetch;
  constexpr int LC = LG * CPL;            // columns a group covers
  constexpr int SW = slot_words<LG, CPL>();
  extern __shared__ __align__(16) float smem[];
  float* SY = smem;                       // [NG][RW]: scan Y of each group's box
  float* SV = SY + NG * RW;               // [NG][RW]: suffix sums of the input row
  float* DX = SV + NG * RW;               // [2][R][NG][SW]: adjoint sums, added over groups
  const int map = blockIdx.x, n = map / C, c = map - n * C;
  const int g = threadIdx.x / LG, p = threadIdx.x % LG;
  const int b = g;
  const bool live = b < B;
  const int x0 = p * CPL;
  const size_t plane = (size_t)H * W;
  const float* xs = x + (size_t)map * plane;
  const float* gbase = gy + (size_t)map * B * plane;
  const unsigned gmap = live ? 4u * (unsigned)(b * plane) : 0u;
  const LaneCols<CPL> cols(x0, W);
  float* sy = SY + g * RW;                // sy[stream_at(v)] = scan Y (v), v in [-PAD, LC + PAD]
  float* sv = SV + g * RW;
  // adjoint record of the box (each group its own; vector loads)
  const Taps<float> tp = load_taps(taps + (size_t)C * B * 16 + (size_t)(c * B + (live ? b : 0)) * 16, W, H);
  const int fa = tp.ox[0], fb = tp.ox[2], fc = tp.oy[0], fd = tp.oy[2];
  const float aa = -tp.wx[1], ab = tp.wx[3], bc_ = -tp.wy[1], bd = tp.wy[3];
  // LDS indices of the lane's tap runs (scan Y at the adjoint's x edges, the
  // suffix sums at the mirrored taps) and of the entries it writes
  int ia[CPL + 1], ib[CPL + 1], ja[CPL + 1], jb[CPL + 1], iw[CPL], jw[CPL];
  {
    const int ra0 = clampi(x0 + fa, -PAD, W), rb0 = clampi(x0 + fb, -PAD, W);
    const int va0 = clampi(x0 - fa, -PAD, W), vb0 = clampi(x0 - fb, -PAD, W);
#pragma unroll
    for (int k = 0; k <= CPL; ++k) {
      ia[k] = stream_at<CPL>(ra0 + k);
      ib[k] = stream_at<CPL>(rb0 + k);
      ja[k] = stream_at<CPL>(va0 + k);
      jb[k] = stream_at<CPL>(vb0 + k);
    }
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      iw[k] = stream_at<CPL>(x0 + k + 1);
      jw[k] = stream_at<CPL>(x0 + k);
    }
  }
  // constant parts of the LDS rows: scan Y is 0 left of column 0, the input
  // row's suffix sums are 0 right of column W
  for (int t = p; t <= PAD; t += LG) {
    sy[stream_at<CPL>(-PAD + t)] = 0.f;
    sv[stream_at<CPL>(LC + t)] = 0.f;
  }
  // cursors: P(clamp(y + fc)) and P(clamp(y + fd)) at the lane's columns
  float pc[CPL], pd[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) { pc[k] = 0.f; pd[k] = 0.f; }
  {
    const int upto = live ? min(max(fd, 0), H) : 0;
    for (int u0 = 0; u0 < upto; u0 += PF) {
      float r[PF][CPL];
#pragma unroll
      for (int i = 0; i < PF; ++i) cols.template load<kVec>(gbase, gmap, u0 + i < upto ? u0 + i : -1, H, W, live, r[i]);
#pragma unroll
      for (int i = 0; i < PF; ++i) {
        const bool inc = u0 + i < fc;
#pragma unroll
        for (int k = 0; k < CPL; ++k) {
          pd[k] += r[i][k];
          if (inc) pc[k] += r[i][k];
        }
      }
    }
  }
  float ca = 0.f, cb = 0.f, gcs = 0.f, gds = 0.f;
  // rows of step y: the input row v, gc_ = G(y + fc), gd_ = G(y + fd); a
  // queue of PF steps, step y at the front
  float qv[PF][CPL], qc[PF][CPL], qd[PF][CPL];
  auto issue = [&](int y, float (&v)[CPL], float (&gc_)[CPL], float (&gd_)[CPL]) {
    const bool in = y < H;
    if constexpr (!kInt) cols.template load<kVec>(xs, 0u, in ? y : -1, H, W, true, v);
    cols.template load<kVec>(gbase, gmap, in ? y + fc : -1, H, W, live, gc_);
    cols.template load<kVec>(gbase, gmap, in ? y + fd : -1, H, W, live, gd_);
  };
  // one output row
  auto step = [&](int y, const float* v, const float* gc_, const float* gd_) {
    // Y and its scan (inclusive within the lane, then across the group)
    float s[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      float yv = pd[k] - pc[k];
      if constexpr (!kInt) yv = fmaf(bd, gd_[k], fmaf(-bc_, gc_[k], yv));
      s[k] = k ? s[k - 1] + yv : yv;
      pc[k] += gc_[k];
      pd[k] += gd_[k];
    }
    const float tot = s[CPL - 1];
    const float off = group_excl<LG, false>(tot);
#pragma unroll
    for (int k = 0; k < CPL; ++k) sy[iw[k]] = s[k] + off;
    if (p == LG - 1) {
#pragma unroll
      for (int t = 1; t <= PAD; ++t) sy[stream_at<CPL>(LC + t)] = s[CPL - 1] + off;
    }
    // suffix sums of the input row (the same in every group)
    if constexpr (!kInt) {
      float sfx[CPL];
#pragma unroll
      for (int k = CPL - 1; k >= 0; --k) sfx[k] = k < CPL - 1 ? sfx[k + 1] + v[k] : v[k];
      const float vt = sfx[0];
      const float voff = group_excl<LG, true>(vt);
#pragma unroll
      for (int k = 0; k < CPL; ++k) sv[jw[k]] = sfx[k] + voff;
      if (p == 0) {
#pragma unroll
        for (int t = 1; t <= PAD; ++t) sv[stream_at<CPL>(-t)] = sfx[0] + voff;
      }
    }
    __builtin_amdgcn_wave_barrier();
    // the adjoint box sums of the lane's outputs and the edge terms
    float sa[CPL + 1], sb[CPL + 1];
#pragma unroll
    for (int k = 0; k <= CPL; ++k) { sa[k] = sy[ia[k]]; sb[k] = sy[ib[k]]; }
    const int bi = y / R, ri = y - bi * R;
    float* dxs = DX + (((bi & 1) * R + ri) * NG + g) * SW;
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      float d;
      if constexpr (kInt) {
        d = sb[k] - sa[k];
      } else {
        const float da = sa[k + 1] - sa[k], db = sb[k + 1] - sb[k];
        d = fmaf(ab, db, fmaf(-aa, da, sb[k] - sa[k]));
        ca = fmaf(v[k], da, ca);
        cb = fmaf(v[k], db, cb);
      }
      dxs[slot_at<CPL>(x0 + k)] = live ? d : 0.f;
    }
    if constexpr (!kInt) {
      float A[CPL + 1], Bv[CPL + 1];
#pragma unroll
      for (int k = 0; k <= CPL; ++k) { A[k] = sv[ja[k]]; Bv[k] = sv[jb[k]]; }
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        const float t = fmaf(-ab, Bv[k + 1] - Bv[k], fmaf(aa, A[k + 1] - A[k], Bv[k + 1] - A[k + 1]));
        gcs = fmaf(gc_[k], t, gcs);
        gds = fmaf(gd_[k], t, gds);
      }
    }
    __builtin_amdgcn_wave_barrier();
    // every R rows (and after the last): the slots of the batch, added over
    // the groups in a fixed order
    if (ri == R - 1 || y == H - 1) {
      __syncthreads();
      const float* slots = DX + (bi & 1) * R * NG * SW;
      for (int r = 0; r <= ri; ++r) {
        const int yy = bi * R + r;
        for (int j = threadIdx.x; j < W; j += LG * NG) {
          float acc = 0.f;
#pragma unroll
          for (int h = 0; h < NG; ++h) acc += slots[(r * NG + h) * SW + slot_at<CPL>(j)];
          const size_t o = (size_t)map * plane + (size_t)yy * W + j;
          if constexpr (kRelu) {
            static_cast<uint16_t*>(gx)[o] = f32_to_bf16_rne(xs[(size_t)yy * W + j] > 0.f ? acc : 0.f);
          } else if (gx != nullptr) {
            static_cast<float*>(gx)[o] = acc;
          }
        }
      }
    }
  };
#pragma unroll
  for (int i = 0; i < PF; ++i) issue(i, qv[i], qc[i], qd[i]);
  for (int y = 0; y < H; ++y) {
    float v[CPL], gc_[CPL], gd_[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) { v[k] = qv[0][k]; gc_[k] = qc[0][k]; gd_[k] = qd[0][k]; }
#pragma unroll
    for (int i = 0; i + 1 < PF; ++i)
#pragma unroll
      for (int k = 0; k < CPL; ++k) { qv[i][k] = qv[i + 1][k]; qc[i][k] = qc[i + 1][k]; qd[i][k] = qd[i + 1][k]; }
    issue(y + PF, qv[PF - 1], qc[PF - 1], qd[PF - 1]);
    step(y, v, gc_, gd_);
  }
  if constexpr (!kInt) {
    // (dL/da, dL/db, dL/dc, dL/dd) of the box, one partial per image
    ca = group_sum<LG>(ca);
    cb = group_sum<LG>(cb);
    gcs = group_sum<LG>(gcs);
    gds = group_sum<LG>(gds);
    if (live && p == 0) {
      float* pp = partials + ((size_t)n * C * B + (size_t)c * B + b) * 4;
      pp[0] = -cb;
      pp[1] = ca;
      pp[2] = -gds;
      pp[3] = gcs;
    }
  }
}

// ---------------------------------------------------------------------------
// Forward.  One block of NG groups per map (n, c); group g walks box b = g
// over the map's rows and writes that box's output row by row (no table, no
// exchange between groups).  T = int: integer maps (the sum of Eq. 1 over the
// floored box, exact).  kInt: boxes with integer corners (four table
// samples, no interpolation).  kOffset: the map's mean mu is subtracted
// before the cursors add its rows and mu times the clipped box area is added
// back (the same combination applied to the clamped coordinates).  kNT:
// non-temporal output stores (outputs larger than the last-level cache).
// ---------------------------------------------------------------------------
template <typename T, typename OutT, int LG, int CPL, int NG, bool kOffset, bool kInt, bool kNT, bool kVec>
__global__ __launch_bounds__(LG * NG) void k_box_fwd_stream(const T* __restrict__ x, const int* __restrict__ taps,
                                                            OutT* __restrict__ y, int C, int H, int W, int B) {
  constexpr bool kPlain = kInt || std::is_same<T, int>::value;   // corner weights (-1, 0, 1, 0)
  constexpr int PAD = stream_pad<CPL>();
  constexpr int RW = stream_row_words<LG, CPL>();
  constexpr int PF = kPrefetch;
  constexpr int LC = LG * CPL;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  T* SY = reinterpret_cast<T*>(smem_raw);
  __shared__ float red[(LG * NG + 63) / 64];
  const int map = blockIdx.x, c = map % C;
  const int g = threadIdx.x / LG, p = threadIdx.x % LG;
  const int b = g;
  const bool live = b < B;
  const int x0 = p * CPL;
  const size_t plane = (size_t)H * W;
  const T* xs = x + (size_t)map * plane;
  const LaneCols<CPL> cols(x0, W);
  T* sy = SY + g * RW;                    // sy[stream_at(v)] = scan Y (v)
  float mu = 0.f;
  if constexpr (kOffset) {
    float sum = 0.f;
    for (size_t i = threadIdx.x; i < plane; i += LG * NG) sum += (float)xs[i];
    sum = wave_sum(sum);
    constexpr int nw = (LG * NG + 63) / 64;
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = sum;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < nw; ++w) tot += red[w];
    mu = tot / (float)plane;
  }
  const Taps<float> tp = load_taps(taps + (size_t)(c * B + (live ? b : 0)) * 16, W, H);
  const int fa = tp.ox[0], fb = tp.ox[2], fc = tp.oy[0], fd = tp.oy[2];
  const float aa = -tp.wx[1], ab = tp.wx[3], bc_ = -tp.wy[1], bd = tp.wy[3];
  int ia[CPL + 1], ib[CPL + 1], iw[CPL];
  {
    const int ra0 = clampi(x0 + fa, -PAD, W), rb0 = clampi(x0 + fb, -PAD, W);
#pragma unroll
    for (int k = 0; k <= CPL; ++k) {
      ia[k] = stream_at<CPL>(ra0 + k);
      ib[k] = stream_at<CPL>(rb0 + k);
    }
#pragma unroll
    for (int k = 0; k < CPL; ++k) iw[k] = stream_at<CPL>(x0 + k + 1);
  }
  for (int t = p; t <= PAD; t += LG) sy[stream_at<CPL>(-PAD + t)] = (T)0;
  T pc[CPL], pd[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) { pc[k] = (T)0; pd[k] = (T)0; }
  // map row `row` at the lane's columns, minus mu (kOffset), 0 outside
  auto load_row = [&](int row, T (&r)[CPL]) {
    cols.template load<kVec>(xs, 0u, row, H, W, live, r);
    if constexpr (kOffset) {
      const bool ok = live && row >= 0 && row < H;
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        const float v = (float)r[k] - mu;
        r[k] = __builtin_bit_cast(T, __builtin_bit_cast(int, (T)v) & ((ok && cols.in[k]) ? -1 : 0));
      }
    }
  };
  {
    const int upto = live ? min(max(fd, 0), H) : 0;
    for (int u0 = 0; u0 < upto; u0 += PF) {
      T r[PF][CPL];
#pragma unroll
      for (int i = 0; i < PF; ++i) load_row(u0 + i < upto ? u0 + i : -1, r[i]);
#pragma unroll
      for (int i = 0; i < PF; ++i) {
        const bool inc = u0 + i < fc;
#pragma unroll
        for (int k = 0; k < CPL; ++k) {
          pd[k] += r[i][k];
          if (inc) pc[k] += r[i][k];
        }
      }
    }
  }
  // clipped extent of the box along x at the lane's outputs (kOffset)
  float ex[CPL];
  if constexpr (kOffset) {
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      const int xa = x0 + k + fa, xb = x0 + k + fb;
      const float wa = (float)(clampi(xa + 1, 0, W) - clampi(xa, 0, W));
      const float wb = (float)(clampi(xb + 1, 0, W) - clampi(xb, 0, W));
      ex[k] = (float)(clampi(xb, 0, W) - clampi(xa, 0, W)) + (kPlain ? 0.f : ab * wb - aa * wa);
    }
  }
  OutT* out = y + ((size_t)map * B + (live ? b : 0)) * plane;
  auto step = [&](int yy, const T* gc_, const T* gd_) {
    T s[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      T yv = pd[k] - pc[k];
      if constexpr (!kPlain) yv = fmaf(bd, gd_[k], fmaf(-bc_, gc_[k], yv));
      s[k] = k ? s[k - 1] + yv : yv;
      pc[k] += gc_[k];
      pd[k] += gd_[k];
    }
    const T tot = s[CPL - 1];
    const T off = group_excl<LG, false>(tot);
#pragma unroll
    for (int k = 0; k < CPL; ++k) sy[iw[k]] = s[k] + off;
    if (p == LG - 1) {
#pragma unroll
      for (int t = 1; t <= PAD; ++t) sy[stream_at<CPL>(LC + t)] = s[CPL - 1] + off;
    }
    __builtin_amdgcn_wave_barrier();
    T sa[CPL + 1], sb[CPL + 1];
#pragma unroll
    for (int k = 0; k <= CPL; ++k) { sa[k] = sy[ia[k]]; sb[k] = sy[ib[k]]; }
    float ey = 0.f;
    if constexpr (kOffset) {
      const int yc = yy + fc, yd = yy + fd;
      const float wc = (float)(clampi(yc + 1, 0, H) - clampi(yc, 0, H));
      const float wd = (float)(clampi(yd + 1, 0, H) - clampi(yd, 0, H));
      ey = (float)(clampi(yd, 0, H) - clampi(yc, 0, H)) + (kPlain ? 0.f : bd * wd - bc_ * wc);
    }
    if (live) {
      OutT* row = out + (size_t)yy * W;
      OutT ov[CPL];
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        T o;
        if constexpr (kPlain) o = sb[k] - sa[k];
        else o = fmaf(ab, sb[k + 1] - sb[k], fmaf(-aa, sa[k + 1] - sa[k], sb[k] - sa[k]));
        if constexpr (kOffset) o = o + (T)(mu * (ex[k] * ey));
        if constexpr (std::is_same<OutT, uint16_t>::value) ov[k] = f32_to_bf16_rne((float)o);
        else ov[k] = (OutT)o;
      }
      if constexpr (kVec && CPL == 4 && sizeof(OutT) == 4) {
        typedef OutT v4 __attribute__((ext_vector_type(4)));
        const v4 q = {ov[0], ov[1], ov[2], ov[3]};
        v4* dst = reinterpret_cast<v4*>(row + x0);
        if constexpr (kNT) __builtin_nontemporal_store(q, dst);
        else *dst = q;
      } else if constexpr (kVec && CPL == 4) {   // 2-byte outputs: one 8-byte store
        const uint2 q = make_uint2((uint32_t)ov[0] | ((uint32_t)ov[1] << 16), (uint32_t)ov[2] | ((uint32_t)ov[3] << 16));
        *reinterpret_cast<uint2*>(row + x0) = q;
      } else {
#pragma unroll
        for (int k = 0; k < CPL; ++k)
          if (cols.in[k]) {
            if constexpr (kNT) __builtin_nontemporal_store(ov[k], row + x0 + k);
            else row[x0 + k] = ov[k];
          }
      }
    }
    __builtin_amdgcn_wave_barrier();
  };
  // main loop, the rows of step yy loaded PF steps ahead (a queue, step yy
  // at the front)
  T qc[PF][CPL], qd[PF][CPL];
#pragma unroll
  for (int i = 0; i < PF; ++i) {
    load_row(i < H ? i + fc : -1, qc[i]);
    load_row(i < H ? i + fd : -1, qd[i]);
  }
  for (int yy = 0; yy < H; ++yy) {
    T gc_[CPL], gd_[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) { gc_[k] = qc[0][k]; gd_[k] = qd[0][k]; }
#pragma unroll
    for (int i = 0; i + 1 < PF; ++i)
#pragma unroll
      for (int k = 0; k < CPL; ++k) { qc[i][k] = qc[i + 1][k]; qd[i][k] = qd[i + 1][k]; }
    const int yn = yy + PF;
    load_row(yn < H ? yn + fc : -1, qc[PF - 1]);
    load_row(yn < H ? yn + fd : -1, qd[PF - 1]);
    step(yy, gc_, gd_);
  }
}

// ---------------------------------------------------------------------------
// Launchers.  Geometry: LG = 16 for maps up to 64 wide (four boxes per wave),
// LG = 64 up to 256 wide (a box per wave); CPL = ceil(W / LG); NG = 4 or 8
// groups (boxes) per block, so B <= 8.  The backward adds the groups' input
// gradients every R rows (R from an LDS budget of 2 KiB per slot set, which
// keeps the pose-shaped maps at 32 waves per CU).
// ---------------------------------------------------------------------------
struct StreamGeom { int lg, cpl, ng, R; };

static bool stream_geom(int H, int W, int B, StreamGeom& g) {
  if (W <= 64) {
    g.lg = 16;
    g.cpl = W <= 16 ? 1 : W <= 32 ? 2 : W <= 48 ? 3 : 4;
  } else if (W <= 256) {
    g.lg = 64;
    g.cpl = W <= 128 ? 2 : W <= 192 ? 3 : 4;
  } else {
    return false;
  }
  if (B > 8) return false;
  g.ng = B <= 4 ? 4 : 8;
  // per-lane 32-bit byte offsets into a block's gradient maps
  if ((size_t)g.ng * H * W * 4 >= ((size_t)1 << 31)) return false;
  const size_t slot_set = (size_t)g.ng * (g.lg * g.cpl + g.lg * g.cpl / 32) * 4;
  g.R = (int)std::max<size_t>(1, std::min<size_t>(8, (2u << 10) / slot_set));
  return true;
}

bool box_stream_supported(int H, int W, int B) {
  StreamGeom g;
  return stream_geom(H, W, B, g);
}

// Vector row accesses: every lane's columns inside the map and 16-byte
// aligned rows (W == LG * CPL, CPL = 4, base pointers 16-byte aligned).
static bool stream_vec(int W, int lg, int cpl) { return cpl == 4 && W == lg * cpl; }

template <int LG, int CPL, int NG>
static void bwd_stream_t(const float* x, const int* taps, const float* gy, void* gx, float* partials, int N, int C,
                         int H, int W, int B, bool rounded, bool relu_bf16, int R, hipStream_t s) {
  constexpr int RW = stream_row_words<LG, CPL>();
  const size_t shm = ((size_t)2 * NG * RW + (size_t)2 * R * NG * slot_words<LG, CPL>()) * sizeof(float);
  const dim3 grid(N * C), block(LG * NG);
  auto go = [&](auto ki, auto kr, auto kv) {
    hipLaunchKernelGGL((k_box_bwd_stream<LG, CPL, NG, decltype(ki)::value, decltype(kr)::value, decltype(kv)::value>),
                       grid, block, shm, s, x, taps, gy, gx, partials, C, H, W, B, R);
  };
  auto with_vec = [&](auto ki, auto kr) {
    if (CPL == 4 && stream_vec(W, LG, CPL)) go(ki, kr, std::true_type{});
    else go(ki, kr, std::false_type{});
  };
  if (rounded) with_vec(std::true_type{}, std::false_type{});
  else if (relu_bf16) with_vec(std::false_type{}, std::true_type{});
  else with_vec(std::false_type{}, std::false_type{});
}

hipError_t launch_box_bwd_stream(const float* x, const int* taps, const float* gy, void* gx, float* partials, int N,
                                 int C, int H, int W, int B, bool rounded, bool relu_bf16, hipStream_t s) {
  StreamGeom g;
  if (!stream_geom(H, W, B, g) || (rounded && relu_bf16)) return hipErrorInvalidValue;
#define BC_BWD_STREAM(LG, CPL, NG)                                                                            \
  if (g.lg == LG && g.cpl == CPL && g.ng == NG) {                                                           \
    bwd_stream_t<LG, CPL, NG>(x, taps, gy, gx, partials, N, C, H, W, B, rounded, relu_bf16, g.R, s);       \
    return hipGetLastError();                                                                               \
  }
  BC_BWD_STREAM(16, 1, 4) BC_BWD_STREAM(16, 2, 4) BC_BWD_STREAM(16, 3, 4) BC_BWD_STREAM(16, 4, 4)
  BC_BWD_STREAM(16, 1, 8) BC_BWD_STREAM(16, 2, 8) BC_BWD_STREAM(16, 3, 8) BC_BWD_STREAM(16, 4, 8)
  BC_BWD_STREAM(64, 2, 4) BC_BWD_STREAM(64, 3, 4) BC_BWD_STREAM(64, 4, 4)
  BC_BWD_STREAM(64, 2, 8) BC_BWD_STREAM(64, 3, 8) BC_BWD_STREAM(64, 4, 8)
#undef BC_BWD_STREAM
  return hipErrorInvalidValue;
}

template <typename T, typename OutT, int LG, int CPL, int NG, bool kOffset>
static void fwd_stream_t(const void* x, const int* taps, void* y, int N, int C, int H, int W, int B, bool rounded,
                         bool nt, hipStream_t s) {
  const size_t shm = (size_t)NG * stream_row_words<LG, CPL>() * sizeof(T);
  const bool vec = stream_vec(W, LG, CPL);
  auto go = [&](auto ki, auto kn) {
    if (CPL == 4 && vec)
      hipLaunchKernelGGL((k_box_fwd_stream<T, OutT, LG, CPL, NG, kOffset, decltype(ki)::value, decltype(kn)::value,
                                           true>),
                         dim3(N * C), dim3(LG * NG), shm, s, (const T*)x, taps, (OutT*)y, C, H, W, B);
    else
      hipLaunchKernelGGL((k_box_fwd_stream<T, OutT, LG, CPL, NG, kOffset, decltype(ki)::value, decltype(kn)::value,
                                           false>),
                         dim3(N * C), dim3(LG * NG), shm, s, (const T*)x, taps, (OutT*)y, C, H, W, B);
  };
  auto with_nt = [&](auto ki) {
    if (nt) go(ki, std::true_type{});
    else go(ki, std::false_type{});
  };
  if (rounded) with_nt(std::true_type{});
  else with_nt(std::false_type{});
}

template <int LG, int CPL, int NG>
static void fwd_stream_dispatch(const void* x, bool is_int, const int* taps, void* y, int out_kind, int N, int C,
                                int H, int W, int B, bool offset, bool rounded, bool nt, hipStream_t s) {
  if (is_int) fwd_stream_t<int, int, LG, CPL, NG, false>(x, taps, y, N, C, H, W, B, rounded, false, s);
  else if (out_kind == 2) {
    if (offset) fwd_stream_t<float, uint16_t, LG, CPL, NG, true>(x, taps, y, N, C, H, W, B, rounded, false, s);
    else fwd_stream_t<float, uint16_t, LG, CPL, NG, false>(x, taps, y, N, C, H, W, B, rounded, false, s);
  } else {
    if (offset) fwd_stream_t<float, float, LG, CPL, NG, true>(x, taps, y, N, C, H, W, B, rounded, nt, s);
    else fwd_stream_t<float, float, LG, CPL, NG, false>(x, taps, y, N, C, H, W, B, rounded, nt, s);
  }
}

hipError_t launch_box_fwd_stream(const void* x, bool is_int, const int* taps, void* y, int out_kind, int N, int C,
                                 int H, int W, int B, bool offset, bool rounded, hipStream_t s) {
  StreamGeom g;
  if (!stream_geom(H, W, B, g)) return hipErrorInvalidValue;
  // fp32 outputs larger than the last-level cache are stored non-temporally
  const bool nt = out_kind == 1 && (size_t)N * C * B * H * W * 4 > ((size_t)256 << 20);
#define BC_FWD_STREAM(LG, CPL, NG)                                                                                \
  if (g.lg == LG && g.cpl == CPL && g.ng == NG) {                                                               \
    fwd_stream_dispatch<LG, CPL, NG>(x, is_int, taps, y, out_kind, N, C, H, W, B, offset, rounded, nt, s);     \
    return hipGetLastError();                                                                                   \
  }
  BC_FWD_STREAM(16, 1, 4) BC_FWD_STREAM(16, 2, 4) BC_FWD_STREAM(16, 3, 4) BC_FWD_STREAM(16, 4, 4)
  BC_FWD_STREAM(16, 1, 8) BC_FWD_STREAM(16, 2, 8) BC_FWD_STREAM(16, 3, 8) BC_FWD_STREAM(16, 4, 8)
  BC_FWD_STREAM(64, 2, 4) BC_FWD_STREAM(64, 3, 4) BC_FWD_STREAM(64, 4, 4)
  BC_FWD_STREAM(64, 2, 8) BC_FWD_STREAM(64, 3, 8) BC_FWD_STREAM(64, 4, 8)
#undef BC_FWD_STREAM
  return hipErrorInvalidValue;
}

}  // namespace bc
