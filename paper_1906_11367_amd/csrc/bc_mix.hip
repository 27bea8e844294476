// 1x1 mix over the C*B filtered maps (Section 1 and 3.2 of the paper: the
// depthwise box filters are followed by a 1x1 convolution), as MFMA GEMMs on
// gfx950.  Per image n with P = H*W pixels:
//   FWD        out[n] (M x P) = w (M x K)   * in[n] (K x P)
//   BWD_DATA   out[n] (K x P) = w^T (K x M) * grad[n] (M x P)
//   BWD_WEIGHT out   (M x K) = sum_n grad[n] (M x P) * in[n]^T (P x K)
// One kernel template covers the three: C(i, j) = sum_l A(i, l) * B(l, j)
// with A and B either contiguous along the reduction index l ("KC") or along
// their row/column index.  Tiles are staged through LDS in l-contiguous
// layout (transposed on the way in where needed) and fed to
// v_mfma_f32_32x32x16_bf16 (bf16 operands) or v_mfma_f32_32x32x2_f32.
#include "bc_common.hpp"
#include "bc_internal.hpp"

#include <algorithm>
#include <type_traits>

namespace bc {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBN = 128;
constexpr int kMixThreads = 256;  // 4 waves in a 2 x 2 arrangement of 64 x 64 sub-tiles

// Storage dtype codes follow bc_dtype: 0 = int32, 1 = fp32, 2 = bf16.
template <int DT> struct StoreBytes { static constexpr int v = DT == 2 ? 2 : 4; };

// Raw storage bits of one element.
template <int DT>
__device__ __forceinline__ uint32_t ld_bits(const char* base, size_t idx) {
  if constexpr (DT == 2) return reinterpret_cast<const uint16_t*>(base)[idx];
  else return reinterpret_cast<const uint32_t*>(base)[idx];
}

// N consecutive elements as raw bits (one 32-bit word per element; bf16 in
// the low half).  `vec` = in range and aligned for one wide load.
template <int DT, int N>
__device__ __forceinline__ void ld_run(const char* base, size_t idx, bool vec, int avail, uint32_t* w) {
  if (vec) {
    if constexpr (DT == 2) {
      static_assert(N == 4 || N == 8, "bf16 runs are 4 or 8 long");
      if constexpr (N == 8) {
        const uint4 q = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(base) + idx);
        const uint32_t p[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) { w[2 * k] = p[k] & 0xffffu; w[2 * k + 1] = p[k] >> 16; }
      } else {
        const uint2 q = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(base) + idx);
        w[0] = q.x & 0xffffu; w[1] = q.x >> 16; w[2] = q.y & 0xffffu; w[3] = q.y >> 16;
      }
    } else {
#pragma unroll
      for (int k = 0; k < N; k += 4) {
        const uint4 q = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint32_t*>(base) + idx + k);
        w[k] = q.x; w[k + 1] = q.y; w[k + 2] = q.z; w[k + 3] = q.w;
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < N; ++k) w[k] = k < avail ? ld_bits<DT>(base, idx + k) : 0u;
  }
}

// Buffer-resource loads: a wave-uniform descriptor of one operand (base and
// byte size, so that the hardware returns zeros past its end), a per-thread
// byte offset and a wave-uniform byte offset.
constexpr int kBufWord3 = 0x00020000;  // raw 32-bit data, no format conversion

__device__ __forceinline__ uint4 buf_ld16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  const auto q = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
  return make_uint4(q[0], q[1], q[2], q[3]);
}
__device__ __forceinline__ uint2 buf_ld8(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  const auto q = __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, 0);
  return make_uint2(q[0], q[1]);
}

// N consecutive elements through a buffer descriptor, as raw bits (one word
// per element; bf16 in the low half).
template <int DT, int N>
__device__ __forceinline__ void buf_run(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, uint32_t* w) {
  if constexpr (DT == 2) {
    if constexpr (N == 8) {
      const uint4 q = buf_ld16(r, voff, soff);
      const uint32_t p[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) { w[2 * k] = p[k] & 0xffffu; w[2 * k + 1] = p[k] >> 16; }
    } else {
      const uint2 q = buf_ld8(r, voff, soff);
      w[0] = q.x & 0xffffu; w[1] = q.x >> 16; w[2] = q.y & 0xffffu; w[3] = q.y >> 16;
    }
  } else {
#pragma unroll
    for (int k = 0; k < N; k += 4) {
      const uint4 q = buf_ld16(r, voff, soff + k * 4);
      w[k] = q.x; w[k + 1] = q.y; w[k + 2] = q.z; w[k + 3] = q.w;
    }
  }
}

// Storage bits -> fp32 value.
template <int DT>
__device__ __forceinline__ float bits_to_f32(uint32_t b) {
  if constexpr (DT == 0) return (float)(int)b;
  else if constexpr (DT == 1) return __uint_as_float(b);
  else return __uint_as_float(b << 16);
}

// Two fp32 values -> packed bf16 pair (lo in bits 0..15), round to nearest
// even; lowers to one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  const __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

template <int DT, bool MASK>
__device__ __forceinline__ float operand_f32(uint32_t b, uint32_t m) {
  float f = bits_to_f32<DT>(b);
  if constexpr (MASK) f = (__uint_as_float(m) > 0.f) ? f : 0.f;
  return f;
}

// Element offset of (row r, reduction index l) in a bf16 LDS tile.  The
// 16-byte chunks of a row are XOR-swizzled by (r / 16) % 4: the transposed
// stores (lanes 4 rows apart) and the MFMA operand reads (32 consecutive rows)
// then both hit distinct banks.
template <int PITCH>
__device__ __forceinline__ int bf16_tile_off(int r, int l) {
  constexpr int kChunks = (PITCH - 8) / 8;  // 16-byte chunks per row: 8 (64 deep) or 16 (128 deep)
  static_assert((kChunks & (kChunks - 1)) == 0, "a power of two");
  return r * PITCH + ((((l >> 3) ^ (r >> 4)) & (kChunks - 1)) << 3) + (l & 7);
}

// One GEMM operand X(r, l): rows r in [0, rows), reduction index l in
// [0, depth).  KC: element (r, l) at p[r * ld + l] (l contiguous); otherwise
// at p[l * ld + r] (r contiguous).  Optional fp32 mask with the same indexing:
// elements whose mask is not > 0 read as zero (ReLU derivative).
//
// A block stages rows [r0, r0 + 128) x l in [l0, l0 + BK) into an LDS tile
// T[128][PITCH] in the compute type with l contiguous (what the MFMA operand
// registers hold).  Loading (global -> registers, issued a whole K-step ahead)
// is split from storing (registers -> LDS), so the loads of the next tile are
// in flight while the current one feeds the MFMAs.
//   KC:     a unit is UL consecutive l of one row        (NU = 4 per thread)
//   not KC: a unit is UL consecutive l x 4 consecutive r (1 per thread); the
//           4 x UL block is transposed in registers so every LDS write is
//           16 contiguous bytes of one row.
// bf16 storage without a mask is kept packed and never converted.
template <bool BF16, int DT, bool KC, bool MASK, int kDeep = 0>
struct Stager {
  static constexpr int BK = kDeep > 0 ? kDeep : (BF16 ? 64 : 32);
  static constexpr int PITCH = BF16 ? BK + 8 : BK + 1;  // elements; bf16 rows are 16-byte aligned
  static constexpr int UL = BF16 ? 8 : 4;               // l per unit
  static constexpr int NU = KC ? (kBM * BK / UL) / kMixThreads : 1;
  static constexpr bool kRaw = BF16 && DT == 2 && !MASK;
  // words held per thread: packed bf16 pairs, or one word per element
  static constexpr int NW = kRaw ? (KC ? NU * UL / 2 : UL * 2) : (KC ? NU * UL : 4 * UL);
  using E = typename std::conditional<BF16, uint16_t, float>::type;

  // Byte offset of this thread's first load inside a tile (the same for every
  // K-step); its other loads sit a wave-uniform step further each: KC units
  // are kMixThreads / (BK / UL) rows apart, non-KC rows one l apart.
  static constexpr int SB = DT == 2 ? 2 : 4;

  const char* p;
  const float* mask;
  long ld;
  int rows, depth;
  bool vec_ok;
  uint32_t off0;
  __amdgpu_buffer_rsrc_t rs, mrs;
  uint32_t v[NW];
  uint32_t m[MASK ? NW : 1];

  // Offsets, and buffer descriptors covering this image's operand (and mask).
  __device__ __forceinline__ void init_offsets() {
    const int tid = threadIdx.x;
    if constexpr (KC) off0 = (uint32_t)(((long)(tid / (BK / UL)) * ld + (tid % (BK / UL)) * UL) * SB);
    else off0 = (uint32_t)(((long)((tid / (kBM / 4)) * UL) * ld + (tid % (kBM / 4)) * 4) * SB);
    const long extent = KC ? (long)(rows - 1) * ld + depth : (long)(depth - 1) * ld + rows;  // elements
    rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(p), (short)0, (int)(extent * SB), kBufWord3);
    if constexpr (MASK)
      mrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(mask), (short)0, (int)(extent * 4), kBufWord3);
  }
  __device__ __forceinline__ long unit_step() const {
    return KC ? (long)(kMixThreads / (BK / UL)) * ld * SB : ld * SB;
  }
  // Whether an image's operand fits the 32-bit byte offsets of the buffer path.
  __device__ __forceinline__ bool buf_ok() const {
    const long extent = KC ? (long)(rows - 1) * ld + depth : (long)(depth - 1) * ld + rows;
    return extent * 4 < (1L << 31);
  }

  // Whole tile in range and aligned: the block takes the unguarded path
  // (the condition is uniform, so no lane diverges and the wide loads stay in
  // flight until store() consumes them).  The unguarded path reads through
  // the buffer descriptor: the thread's one offset plus a wave-uniform offset
  // per K-step and unit, so no address is computed in the loop.
  __device__ __forceinline__ void load(int r0, int l0) {
    if (vec_ok && r0 + kBM <= rows && l0 + BK <= depth) load_full(r0, l0);
    else load_tile<false>(r0, l0);
  }

  __device__ __forceinline__ void load_full(int r0, int l0) {
    const uint32_t origin = (uint32_t)(KC ? (long)r0 * ld + l0 : (long)l0 * ld + r0);
    const uint32_t step = (uint32_t)unit_step();
    const uint32_t moff = off0 / SB * 4;
    if constexpr (KC) {
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        const uint32_t so = origin * SB + u * step;
        if constexpr (kRaw) {
          const uint4 q = buf_ld16(rs, off0, so);
          uint32_t* w = v + u * (UL / 2);
          w[0] = q.x; w[1] = q.y; w[2] = q.z; w[3] = q.w;
        } else {
          buf_run<DT, UL>(rs, off0, so, v + u * UL);
          if constexpr (MASK) buf_run<1, UL>(mrs, moff, origin * 4 + u * (step / SB * 4), m + u * UL);
        }
      }
    } else {
#pragma unroll
      for (int e = 0; e < UL; ++e) {
        const uint32_t so = origin * SB + e * step;
        if constexpr (kRaw) {
          const uint2 q = buf_ld8(rs, off0, so);
          v[e * 2] = q.x; v[e * 2 + 1] = q.y;
        } else {
          buf_run<DT, 4>(rs, off0, so, v + e * 4);
          if constexpr (MASK) buf_run<1, 4>(mrs, moff, origin * 4 + e * (step / SB * 4), m + e * 4);
        }
      }
    }
  }

  template <bool kFull>
  __device__ __forceinline__ void load_tile(int r0, int l0) {
    const int tid = threadIdx.x;
    if constexpr (KC) {
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        const int unit = tid + u * kMixThreads;
        const int r = r0 + unit / (BK / UL), l = l0 + (unit % (BK / UL)) * UL;
        if constexpr (kRaw) {
          uint32_t* w = v + u * (UL / 2);
          if (kFull) {
            const uint4 q = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(p) + (size_t)r * ld + l);
            w[0] = q.x; w[1] = q.y; w[2] = q.z; w[3] = q.w;
          } else {
            uint32_t e[UL];
            const bool in = r < rows;
            const int avail = in ? min(UL, max(0, depth - l)) : 0;
            ld_run<2, UL>(p, (size_t)(in ? r : 0) * ld + (avail > 0 ? l : 0), false, avail, e);
#pragma unroll
            for (int k = 0; k < UL / 2; ++k) w[k] = e[2 * k] | (e[2 * k + 1] << 16);
          }
        } else if constexpr (kFull) {
          const size_t idx = (size_t)r * ld + l;
          ld_run<DT, UL>(p, idx, true, UL, v + u * UL);
          if constexpr (MASK) ld_run<1, UL>(reinterpret_cast<const char*>(mask), idx, true, UL, m + u * UL);
        } else {
          const bool in = r < rows;
          const int avail = in ? min(UL, max(0, depth - l)) : 0;
          const size_t idx = (size_t)(in ? r : 0) * ld + (avail > 0 ? l : 0);
          ld_run<DT, UL>(p, idx, false, avail, v + u * UL);
          if constexpr (MASK) ld_run<1, UL>(reinterpret_cast<const char*>(mask), idx, false, avail, m + u * UL);
        }
      }
    } else {
      const int r = r0 + (tid % (kBM / 4)) * 4, lb = l0 + (tid / (kBM / 4)) * UL;
      const int ravail = max(0, min(4, rows - r));
#pragma unroll
      for (int e = 0; e < UL; ++e) {
        const int l = lb + e;
        if constexpr (kRaw) {
          uint32_t* w = v + e * 2;
          if (kFull) {
            const uint2 q = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(p) + (size_t)l * ld + r);
            w[0] = q.x; w[1] = q.y;
          } else {
            uint32_t t[4];
            const int avail = l < depth ? ravail : 0;
            ld_run<2, 4>(p, (size_t)(avail > 0 ? l : 0) * ld + (avail > 0 ? r : 0), false, avail, t);
            w[0] = t[0] | (t[1] << 16);
            w[1] = t[2] | (t[3] << 16);
          }
        } else if constexpr (kFull) {
          const size_t idx = (size_t)l * ld + r;
          ld_run<DT, 4>(p, idx, true, 4, v + e * 4);
          if constexpr (MASK) ld_run<1, 4>(reinterpret_cast<const char*>(mask), idx, true, 4, m + e * 4);
        } else {
          const int avail = l < depth ? ravail : 0;
          const size_t idx = (size_t)(avail > 0 ? l : 0) * ld + (avail > 0 ? r : 0);
          ld_run<DT, 4>(p, idx, false, avail, v + e * 4);
          if constexpr (MASK) ld_run<1, 4>(reinterpret_cast<const char*>(mask), idx, false, avail, m + e * 4);
        }
      }
    }
  }

  __device__ __forceinline__ uint32_t mk(int i) const { return MASK ? m[i] : 0u; }
  __device__ __forceinline__ float f(int i) const { return operand_f32<DT, MASK>(v[i], mk(i)); }

  __device__ __forceinline__ void store(E* T) const {
    const int tid = threadIdx.x;
    if constexpr (KC) {
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        const int unit = tid + u * kMixThreads;
        const int r = unit / (BK / UL), l = (unit % (BK / UL)) * UL;
        if constexpr (BF16) {
          uint4 q;
          if constexpr (kRaw) {
            q.x = v[u * 4 + 0]; q.y = v[u * 4 + 1]; q.z = v[u * 4 + 2]; q.w = v[u * 4 + 3];
          } else {
            const int b = u * UL;
            q.x = pack2_bf16(f(b + 0), f(b + 1)); q.y = pack2_bf16(f(b + 2), f(b + 3));
            q.z = pack2_bf16(f(b + 4), f(b + 5)); q.w = pack2_bf16(f(b + 6), f(b + 7));
          }
          *reinterpret_cast<uint4*>(T + bf16_tile_off<PITCH>(r, l)) = q;
        } else {
          E* dst = T + r * PITCH + l;
#pragma unroll
          for (int k = 0; k < UL; ++k) dst[k] = f(u * UL + k);
        }
      }
    } else {
      const int r = (tid % (kBM / 4)) * 4, lb = (tid / (kBM / 4)) * UL;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (BF16) {
          uint4 q;
          if constexpr (kRaw) {
            // element i of rows (l, l+1) -> one packed word: bytes of the
            // low (i even) or high (i odd) halves of the two source words
            const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;
            const int h = i >> 1;
            q.x = __builtin_amdgcn_perm(v[1 * 2 + h], v[0 * 2 + h], sel);
            q.y = __builtin_amdgcn_perm(v[3 * 2 + h], v[2 * 2 + h], sel);
            q.z = __builtin_amdgcn_perm(v[5 * 2 + h], v[4 * 2 + h], sel);
            q.w = __builtin_amdgcn_perm(v[7 * 2 + h], v[6 * 2 + h], sel);
          } else {
            q.x = pack2_bf16(f(0 * 4 + i), f(1 * 4 + i));
            q.y = pack2_bf16(f(2 * 4 + i), f(3 * 4 + i));
            q.z = pack2_bf16(f(4 * 4 + i), f(5 * 4 + i));
            q.w = pack2_bf16(f(6 * 4 + i), f(7 * 4 + i));
          }
          *reinterpret_cast<uint4*>(T + bf16_tile_off<PITCH>(r + i, lb)) = q;
        } else {
          E* dst = T + (r + i) * PITCH + lb;
#pragma unroll
          for (int e = 0; e < UL; ++e) dst[e] = f(e * 4 + i);
        }
      }
    }
  }
};

// Stores the 2 x 2 accumulator tiles of one wave.  OK: 0 = fp32, 1 = int32
// (exact integer values), 3 = fp32 accumulate, 4 = fp32 with ReLU.  `full`
// (block-uniform) skips the bounds checks.  NT: non-temporal stores (0, 1, 4).
template <int OK, bool NT>
__device__ __forceinline__ void epilogue(const f32x16_t (&acc)[2][2], char* cbase, int ib, int jb, int rows,
                                         int cols, long ldc, bool full) {
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = ib + x * 32 + 8 * (r >> 2) + (r & 3);
        const int j = jb + y * 32;
        if (full || (i < rows && j < cols)) {
          const float v = acc[x][y][r];
          const size_t o = (size_t)i * ldc + j;
          if constexpr (OK == 3) {
            reinterpret_cast<float*>(cbase)[o] += v;
          } else if constexpr (OK == 1) {
            if constexpr (NT) __builtin_nontemporal_store((int)v, reinterpret_cast<int*>(cbase) + o);
            else reinterpret_cast<int*>(cbase)[o] = (int)v;
          } else {
            const float u = OK == 4 ? fmaxf(v, 0.f) : v;
            if constexpr (NT) __builtin_nontemporal_store(u, reinterpret_cast<float*>(cbase) + o);
            else reinterpret_cast<float*>(cbase)[o] = u;
          }
        }
      }
}

// Occupancy target (waves per SIMD) of one GEMM variant.  The kernel is
// bound by global-load latency (one K-step of each operand in flight per
// block), so a third resident block per CU pays whenever the variant still
// fits in 168 registers without spilling -- the accumulators then move from
// AGPRs to VGPRs.  Variants that would spill (l-contiguous masked or fp32
// operands in bf16 compute, the bf16 weight-gradient GEMM) keep two.
template <bool BF16, int ADT, bool AKC, bool AMASK, int BDT, bool BKC, bool BMASK>
constexpr int mix_waves() {
  if (!BF16) return (AKC && AMASK) ? 2 : 3;
  if (AMASK || BMASK) return 2;
  if (AKC && !BKC) return (ADT == 2 && BDT == 2) ? 3 : 2;
  if (!AKC && !BKC) return (ADT == 1 && BDT == 1) ? 2 : 3;
  return 2;
}

// out-kind: 0 = store fp32 (relu optional), 1 = store int32 (exact integers),
// 2 = store fp32 partial (BWD_WEIGHT split), 3 = fp32 with accumulate; plus
// kOutNT for non-temporal stores of 0 and 1.
constexpr int kOutNT = 8;

template <bool BF16, int ADT, bool AKC, bool AMASK, int BDT, bool BKC, bool BMASK>
__global__ __launch_bounds__(kMixThreads)
__attribute__((amdgpu_waves_per_eu(mix_waves<BF16, ADT, AKC, AMASK, BDT, BKC, BMASK>(), 8))) void k_mix_gemm(
    const void* __restrict__ a, const void* __restrict__ b, const float* __restrict__ aux, void* __restrict__ out,
    int rows, int cols, int depth, long lda, long ldb, long ldc, long a_bs, long b_bs, long c_bs,
    int mt, int nt, int zt, int nsplit_p, int pchunk, int out_kind, int relu) {
  // bf16 storage on both operands, both contiguous along the reduction
  // (BWD_WEIGHT): 128-deep K-steps, each operand row read as 256-byte runs
  constexpr int kDeep = (BF16 && AKC && BKC && !AMASK && !BMASK && ADT == 2 && BDT == 2) ? 128 : 0;
  using SA = Stager<BF16, ADT, AKC, AMASK, kDeep>;
  using SB = Stager<BF16, BDT, BKC, BMASK, kDeep>;
  constexpr int BK = SA::BK, PITCH = SA::PITCH;
  using E = typename SA::E;
  __shared__ __align__(16) E As[kBM * PITCH];
  __shared__ __align__(16) E Bs[kBN * PITCH];

  // logical tile id: XCD-contiguous, row tiles fastest (blocks sharing one B
  // tile run together on one XCD)
  const int total = mt * nt * zt;
  const int per = gridDim.x >> 3;
  const int L = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  if (L >= total) return;
  const int tm = L % mt, tn = (L / mt) % nt, z = L / (mt * nt);

  // batch item and reduction range of this block
  int n = z, l_begin = 0, l_end = depth;
  if (nsplit_p > 0) {  // BWD_WEIGHT: z = n * nsplit_p + sp
    n = z / nsplit_p;
    const int sp = z - n * nsplit_p;
    l_begin = sp * pchunk;
    l_end = min(depth, l_begin + pchunk);
  }
  SA sa;
  sa.p = reinterpret_cast<const char*>(a) + (size_t)n * a_bs * StoreBytes<ADT>::v;
  sa.mask = AMASK ? aux + (size_t)n * a_bs : nullptr;
  sa.ld = lda; sa.rows = rows; sa.depth = depth;
  sa.vec_ok = (lda & 7) == 0 && ((uintptr_t)sa.p & 15) == 0 && (!AMASK || ((uintptr_t)sa.mask & 15) == 0);
  SB sb;
  sb.p = reinterpret_cast<const char*>(b) + (size_t)n * b_bs * StoreBytes<BDT>::v;
  sb.mask = BMASK ? aux + (size_t)n * b_bs : nullptr;
  sb.ld = ldb; sb.rows = cols; sb.depth = depth;
  sb.vec_ok = (ldb & 7) == 0 && ((uintptr_t)sb.p & 15) == 0 && (!BMASK || ((uintptr_t)sb.mask & 15) == 0);
  sa.init_offsets();
  sb.init_offsets();
  sa.vec_ok = sa.vec_ok && sa.buf_ok();
  sb.vec_ok = sb.vec_ok && sb.buf_ok();
  // loads stop at this block's reduction range (a split chunk need not be a
  // whole number of K-steps; the descriptors keep the operand's extent)
  sa.depth = l_end;
  sb.depth = l_end;

  const int i0 = tm * kBM, j0 = tn * kBN;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  f32x16_t acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.f;

  if (l_begin < l_end) {
    sa.load(i0, l_begin);
    sb.load(j0, l_begin);
    sa.store(As);
    sb.store(Bs);
    __syncthreads();
  }
  for (int l0 = l_begin; l0 < l_end; l0 += BK) {
    const bool more = l0 + BK < l_end;
    if (more) {  // next tile's loads in flight during this tile's MFMAs
      sa.load(i0, l0 + BK);
      sb.load(j0, l0 + BK);
    }
    if constexpr (BF16) {
#pragma unroll
      for (int kk = 0; kk < BK; kk += 16) {
        bf16x8_t af[2], bfr[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          af[t] = *reinterpret_cast<const bf16x8_t*>(As + bf16_tile_off<PITCH>(wm * 64 + t * 32 + (lane & 31), kk + 8 * (lane >> 5)));
          bfr[t] = *reinterpret_cast<const bf16x8_t*>(Bs + bf16_tile_off<PITCH>(wn * 64 + t * 32 + (lane & 31), kk + 8 * (lane >> 5)));
        }
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
          for (int y = 0; y < 2; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[x], bfr[y], acc[x][y], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < BK; kk += 2) {
        float af[2], bfr[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          af[t] = As[(wm * 64 + t * 32 + (lane & 31)) * PITCH + kk + (lane >> 5)];
          bfr[t] = Bs[(wn * 64 + t * 32 + (lane & 31)) * PITCH + kk + (lane >> 5)];
        }
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
          for (int y = 0; y < 2; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[x], bfr[y], acc[x][y], 0, 0, 0);
      }
    }
    __syncthreads();
    if (more) {
      sa.store(As);
      sb.store(Bs);
      __syncthreads();
    }
  }

  // Epilogue.  Accumulator element r of lane t in a 32 x 32 tile is
  // C[8 * (r / 4) + 4 * (t / 32) + r % 4][t % 32].
  char* cbase = reinterpret_cast<char*>(out) + (size_t)z * c_bs * 4;
  const bool full = i0 + kBM <= rows && j0 + kBN <= cols;
  const int ib = i0 + wm * 64 + 4 * (lane >> 5), jb = j0 + wn * 64 + (lane & 31);
  switch (out_kind) {
    case 1: epilogue<1, false>(acc, cbase, ib, jb, rows, cols, ldc, full); break;
    case 1 | kOutNT: epilogue<1, true>(acc, cbase, ib, jb, rows, cols, ldc, full); break;
    case 3: epilogue<3, false>(acc, cbase, ib, jb, rows, cols, ldc, full); break;
    case kOutNT:
      if (relu) epilogue<4, true>(acc, cbase, ib, jb, rows, cols, ldc, full);
      else epilogue<0, true>(acc, cbase, ib, jb, rows, cols, ldc, full);
      break;
    default:
      if (relu) epilogue<4, false>(acc, cbase, ib, jb, rows, cols, ldc, full);
      else epilogue<0, false>(acc, cbase, ib, jb, rows, cols, ldc, full);
  }
}

// ---------------------------------------------------------------------------
// BWD_DATA in bf16, one block per column strip
// ---------------------------------------------------------------------------
// out[n] (K x P) = w^T (K x M) * grad[n] (M x P).  The reduction (the mix's
// M output channels) is short and the output (K rows) is the widest tensor
// of the layer, so the 128 x 128 tiles above spend most of their time on
// exposed load latency: each tile has only M / 64 K-steps.  Here a block
// owns kStripP columns of one image instead: it converts grad[n][:, strip]
// to bf16 once, into LDS in B-operand order (rows p, reduction m contiguous),
// and each wave then produces 64 output rows at a time with no further
// barrier, reading its A operand (w transposed, written in MFMA operand
// order by k_wt_frags) from L2 a group of m-steps ahead, and storing each
// finished 64 x 64 tile while the next one's MFMAs run.  The MFMA sequence
// of every output element is the one k_mix_gemm issues (m ascending in
// steps of 16), so both kernels give the same bits.
constexpr int kStripP = 64;     // output columns per block
constexpr int kWtGroup = 4;     // m-steps of 16 loaded together (one group ahead)

// Fragment count of w^T: K rounded up to 64 rows (two 32-row A fragments per
// wave tile), M to kWtGroup m-steps of 16.
__host__ __device__ __forceinline__ int wt_ksteps(int K) { return ((K + 63) / 64) * 2; }
__host__ __device__ __forceinline__ int wt_msteps(int M) { return ((M + 16 * kWtGroup - 1) / (16 * kWtGroup)) * kWtGroup; }

// w [M][K] -> A fragments of w^T: fragment (kb, ms) is 64 lanes x 8 bf16,
// lane l holding w[16 ms + 8 (l / 32) + e][32 kb + l % 32], e = 0..7 (zero
// outside w), stored at frags[(kb * msteps + ms) * 64 + l].
template <int ADT>
__global__ void k_wt_frags(const void* __restrict__ w, int M, int K, int msteps, size_t total,
                           uint4* __restrict__ frags) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int lane = (int)(i & 63);
  const size_t f = i >> 6;
  const int ms = (int)(f % msteps), kb = (int)(f / msteps);
  const int k = kb * 32 + (lane & 31), m0 = ms * 16 + 8 * (lane >> 5);
  uint32_t h[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int m = m0 + e;
    const bool in = m < M && k < K;
    const size_t idx = in ? (size_t)m * K + k : 0;
    if constexpr (ADT == 2) h[e] = in ? (uint32_t)reinterpret_cast<const uint16_t*>(w)[idx] : 0u;
    else h[e] = in ? (pack2_bf16(reinterpret_cast<const float*>(w)[idx], 0.f) & 0xffffu) : 0u;
  }
  frags[i] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
}

template <int BDT, bool BMASK>
__global__ __launch_bounds__(kMixThreads) __attribute__((amdgpu_waves_per_eu(3, 8))) void k_mix_bwd_data_strip(const uint4* __restrict__ frags,
                                                                    const void* __restrict__ g,
                                                                    const float* __restrict__ aux,
                                                                    float* __restrict__ out, int M, int K, int P,
                                                                    int msteps, int nstrips) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  uint16_t* Bs = reinterpret_cast<uint16_t*>(smem_raw);
  const int pitch = msteps * 16 + 8;   // bf16 elements; rows 16-byte aligned, 4 banks apart
  const int strip = blockIdx.x % nstrips, n = blockIdx.x / nstrips;
  const int p0 = strip * kStripP;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const size_t plane = (size_t)M * P;

  // grad[n][m][p0 + j] -> Bs[j * pitch + m]: units of 8 m x 4 p, transposed
  // in registers so each LDS write is 16 contiguous bytes of one row.
  {
    const bool vec = (P & 3) == 0;
    const char* gb = reinterpret_cast<const char*>(g) + (size_t)n * plane * StoreBytes<BDT>::v;
    const float* mb = BMASK ? aux + (size_t)n * plane : nullptr;
    const int units = (msteps * 16 / 8) * (kStripP / 4);
    for (int u = tid; u < units; u += kMixThreads) {
      const int pg = u % (kStripP / 4), mg = u / (kStripP / 4);
      const int pp = p0 + pg * 4, m0 = mg * 8;
      uint32_t v[8][4];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int m = m0 + e;
        const int avail = m < M ? max(0, min(4, P - pp)) : 0;
        const size_t idx = avail > 0 ? (size_t)m * P + pp : 0;
        uint32_t raw[4], mk[4] = {0u, 0u, 0u, 0u};
        ld_run<BDT, 4>(gb, idx, vec && avail == 4, avail, raw);
        if constexpr (BMASK) ld_run<1, 4>(reinterpret_cast<const char*>(mb), idx, vec && avail == 4, avail, mk);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if constexpr (BDT == 2 && !BMASK) v[e][i] = raw[i] & 0xffffu;
          else v[e][i] = i < avail ? (pack2_bf16(operand_f32<BDT, BMASK>(raw[i], mk[i]), 0.f) & 0xffffu) : 0u;
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint4 q = make_uint4(v[0][i] | (v[1][i] << 16), v[2][i] | (v[3][i] << 16), v[4][i] | (v[5][i] << 16),
                                   v[6][i] | (v[7][i] << 16));
        *reinterpret_cast<uint4*>(Bs + (pg * 4 + i) * pitch + m0) = q;
      }
    }
  }
  __syncthreads();

  // wave tiles: rows [64 (wave + 4 t), + 64) for t = 0, 1, ...; all 64 columns
  const int ntile = (K + 63) / 64;
  const int mytiles = ntile > wave ? (ntile - wave + 3) / 4 : 0;
  const int ngroups = msteps / kWtGroup;
  const int total = mytiles * ngroups;
  // Fragment loads and output stores go through buffer descriptors: one
  // per-lane offset plus a wave-uniform offset each, so the 8 loads of a
  // group and the 64 stores of a tile keep no per-element addresses in
  // registers.
  const __amdgpu_buffer_rsrc_t fr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint4*>(frags), (short)0,
                                                                      (int)((size_t)wt_ksteps(K) * msteps * 1024), kBufWord3);
  const __amdgpu_buffer_rsrc_t orr = __builtin_amdgcn_make_buffer_rsrc(out + (size_t)n * K * P, (short)0,
                                                                       (int)((size_t)K * P * 4), kBufWord3);
  auto load_group = [&](int t, uint4 (&a)[kWtGroup][2]) {
    const int kb = 2 * (wave + 4 * (t / ngroups));
    const int ms0 = (t % ngroups) * kWtGroup;
#pragma unroll
    for (int s = 0; s < kWtGroup; ++s)
#pragma unroll
      for (int x = 0; x < 2; ++x) a[s][x] = buf_ld16(fr, (uint32_t)lane * 16, (uint32_t)(((kb + x) * msteps + ms0 + s) * 1024));
  };
  f32x16_t acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.f;
  const uint16_t* brow = Bs + (lane & 31) * pitch + 8 * (lane >> 5);
  float* obase = out + (size_t)n * K * P;
  // the MFMAs of group t (m-steps of one tile), then the tile's store when
  // it is the tile's last group
  auto step = [&](int t, const uint4 (&a)[kWtGroup][2]) {
    const int ms0 = (t % ngroups) * kWtGroup;
#pragma unroll
    for (int s = 0; s < kWtGroup; ++s) {
      bf16x8_t bf[2];
#pragma unroll
      for (int y = 0; y < 2; ++y)
        bf[y] = *reinterpret_cast<const bf16x8_t*>(brow + y * 32 * pitch + (ms0 + s) * 16);
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const bf16x8_t af = __builtin_bit_cast(bf16x8_t, a[s][x]);
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bf[y], acc[x][y], 0, 0, 0);
      }
    }
    if (t % ngroups != ngroups - 1) return;
    const int i0 = 64 * (wave + 4 * (t / ngroups));
    const int ib = i0 + 4 * (lane >> 5), jb = p0 + (lane & 31);
    if (i0 + 64 <= K && p0 + kStripP <= P) {
      const uint32_t vo = (uint32_t)(ib * P + jb) * 4;
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[x][y][r]), orr, (int)vo,
                                                  ((x * 32 + 8 * (r >> 2) + (r & 3)) * P + y * 32) * 4, 2);
    } else {
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int i = ib + x * 32 + 8 * (r >> 2) + (r & 3), j = jb + y * 32;
            if (i < K && j < P) __builtin_nontemporal_store(acc[x][y][r], obase + (size_t)i * P + j);
          }
    }
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int y = 0; y < 2; ++y)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.f;
  };
  // groups alternate between two register sets, each loaded one group ahead
  uint4 a0[kWtGroup][2], a1[kWtGroup][2];
  if (total > 0) load_group(0, a0);
  for (int t = 0; t < total; t += 2) {
    if (t + 1 < total) load_group(t + 1, a1);
    step(t, a0);
    if (t + 1 >= total) break;
    if (t + 2 < total) load_group(t + 2, a0);
    step(t + 1, a1);
  }
}

// LDS bytes of the strip kernel's B operand, or 0 where it does not apply.
static size_t strip_lds_bytes(int M) {
  const size_t b = (size_t)kStripP * (wt_msteps(M) * 16 + 8) * 2;
  return b <= (64u << 10) ? b : 0;
}

static size_t wt_frag_bytes(int M, int K) { return (size_t)wt_ksteps(K) * wt_msteps(M) * 64 * 16; }

// dst[i] = bf16(src[i]), round to nearest even, 8 elements per thread.
__global__ void k_cast_bf16(const float* __restrict__ src, uint16_t* __restrict__ dst, size_t n) {
  const size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * 8;
  if (i + 8 <= n) {
    const float4 a = *reinterpret_cast<const float4*>(src + i);
    const float4 b = *reinterpret_cast<const float4*>(src + i + 4);
    uint4 q;
    q.x = pack2_bf16(a.x, a.y); q.y = pack2_bf16(a.z, a.w);
    q.z = pack2_bf16(b.x, b.y); q.w = pack2_bf16(b.z, b.w);
    *reinterpret_cast<uint4*>(dst + i) = q;
  } else {
    for (size_t k = i; k < n; ++k) dst[k] = (uint16_t)(pack2_bf16(src[k], 0.f) & 0xffffu);
  }
}

hipError_t launch_cast_bf16(const float* src, void* dst, size_t n, hipStream_t s) {
  const size_t threads = (n + 7) / 8;
  hipLaunchKernelGGL(k_cast_bf16, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, src, (uint16_t*)dst, n);
  return hipGetLastError();
}

// ReLU backward of the mix in its compute type: dst[i] = bf16(aux[i] > 0 ?
// g[i] : 0), round to nearest even, 8 elements per thread.  These are the
// operand bits a masked bf16 GEMM (MASK) forms from g and aux on load, so
// the unmasked GEMMs on dst compute exactly the same sums.
__global__ void k_relu_cast_bf16(const float* __restrict__ g, const float* __restrict__ aux,
                                 uint16_t* __restrict__ dst, size_t n) {
  const size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * 8;
  if (i >= n) return;
  if (i + 8 <= n) {
    const float4 a0 = *reinterpret_cast<const float4*>(g + i);
    const float4 a1 = *reinterpret_cast<const float4*>(g + i + 4);
    const float4 m0 = *reinterpret_cast<const float4*>(aux + i);
    const float4 m1 = *reinterpret_cast<const float4*>(aux + i + 4);
    uint4 q;
    q.x = pack2_bf16(m0.x > 0.f ? a0.x : 0.f, m0.y > 0.f ? a0.y : 0.f);
    q.y = pack2_bf16(m0.z > 0.f ? a0.z : 0.f, m0.w > 0.f ? a0.w : 0.f);
    q.z = pack2_bf16(m1.x > 0.f ? a1.x : 0.f, m1.y > 0.f ? a1.y : 0.f);
    q.w = pack2_bf16(m1.z > 0.f ? a1.z : 0.f, m1.w > 0.f ? a1.w : 0.f);
    *reinterpret_cast<uint4*>(dst + i) = q;
  } else {
    for (size_t k = i; k < n; ++k) dst[k] = (uint16_t)(pack2_bf16(aux[k] > 0.f ? g[k] : 0.f, 0.f) & 0xffffu);
  }
}

hipError_t launch_relu_cast_bf16(const float* g, const float* aux, void* dst, size_t n, hipStream_t s) {
  const size_t threads = (n + 7) / 8;
  hipLaunchKernelGGL(k_relu_cast_bf16, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, g, aux,
                     (uint16_t*)dst, n);
  return hipGetLastError();
}

// Fixed-order sum of split-K partials: out = (accumulate ? out : 0) + sum_s part[s].
__global__ void k_mix_reduce(const float* __restrict__ part, int S, size_t n, float* __restrict__ out, int accumulate) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = accumulate ? out[i] : 0.f;
  for (int k = 0; k < S; ++k) s += part[(size_t)k * n + i];
  out[i] = s;
}

// The same sum, four consecutive outputs per thread (n a multiple of 4), the
// partials' loads unrolled so that several are in flight; each output's
// additions keep their order, so the bits are those of k_mix_reduce.
__global__ void k_mix_reduce4(const float4* __restrict__ part, int S, size_t n4, float4* __restrict__ out,
                              int accumulate) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  float4 s = accumulate ? out[i] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8
  for (int k = 0; k < S; ++k) {
    const float4 p = part[(size_t)k * n4 + i];
    s.x += p.x;
    s.y += p.y;
    s.z += p.z;
    s.w += p.w;
  }
  out[i] = s;
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
struct WeightSplit { int sp, chunk, S; };

static WeightSplit weight_split(int N, int M, int K, int P, bool bf16) {
  const int BK = bf16 ? 64 : 32;
  const long tiles = (long)((M + kBM - 1) / kBM) * ((K + kBN - 1) / kBN);
  const int max_sp = (P + BK - 1) / BK;
  int sp = (int)std::min<long>(512, (512 + tiles * N - 1) / (tiles * N));
  if (sp < 1) sp = 1;
  if (sp > max_sp) sp = max_sp;
  int chunk = (P + sp - 1) / sp;
  chunk = ((chunk + BK - 1) / BK) * BK;
  sp = (P + chunk - 1) / chunk;
  return {sp, chunk, N * sp};
}

size_t mix_workspace_bytes(int mode, int N, int M, int K, int P, int compute_dt) {
  if (mode == 1)
    return (compute_dt == 2 && strip_lds_bytes(M) > 0 && (size_t)K * P * 4 < ((size_t)1 << 31)) ? wt_frag_bytes(M, K) : 0;
  if (mode != 2) return 0;
  const WeightSplit ws = weight_split(N, M, K, P, compute_dt == 2);
  return ws.S > 1 ? (size_t)ws.S * M * K * sizeof(float) : 0;
}

template <bool BF16, int ADT, bool AKC, bool AMASK, int BDT, bool BKC, bool BMASK>
static void gemm_launch(const void* a, const void* b, const float* aux, void* out, int rows, int cols, int depth,
                        long lda, long ldb, long ldc, long a_bs, long b_bs, long c_bs, int zt, int nsplit_p,
                        int pchunk, int out_kind, int relu, hipStream_t s) {
  const int mt = (rows + kBM - 1) / kBM, nt = (cols + kBN - 1) / kBN;
  const int total = mt * nt * zt;
  const int grid = (total + 7) & ~7;
  hipLaunchKernelGGL((k_mix_gemm<BF16, ADT, AKC, AMASK, BDT, BKC, BMASK>), dim3(grid), dim3(kMixThreads), 0, s,
                     a, b, aux, out, rows, cols, depth, lda, ldb, ldc, a_bs, b_bs, c_bs, mt, nt, zt, nsplit_p,
                     pchunk, out_kind, relu);
}

// Stored operand dtypes instantiated per compute type: bf16 compute reads
// fp32 or bf16 storage; fp32 compute reads int32 or fp32 storage.
template <bool BF16, typename F>
static void with_dt(int dt, F&& f) {
  if constexpr (BF16) {
    if (dt == 2) f(std::integral_constant<int, 2>{});
    else f(std::integral_constant<int, 1>{});
  } else {
    if (dt == 0) f(std::integral_constant<int, 0>{});
    else f(std::integral_constant<int, 1>{});
  }
}

// Non-temporal stores of the final outputs, per mode: they are read once, by
// a later call, and are larger than the caches; keeping them out leaves the
// caches to the operands the other calls re-read.  Measured on the whole
// layer step (each alone on one GEMM gains less): pose layer 0.657 ->
// 0.638 ms, six stacked layers with ReLU 4.64 -> 4.47 ms.  Run back to back
// with warm caches the GEMMs gain far more (BWD_DATA 171 -> 119 us), and
// after a cache flush they lose (165 -> 186 us): the step is what counts.
constexpr bool kNtFwd = true;
constexpr bool kNtBwdData = true;

template <bool BF16>
static hipError_t launch_mix_t(int mode, const void* a, int a_dt, const void* b, int b_dt, void* out, int out_dt,
                               int N, int M, int K, int P, int relu, const float* aux, int accumulate, void* ws,
                               hipStream_t s) {
  const int out_kind_plain = out_dt == 0 ? 1 : 0;
  const int ok_fwd = out_kind_plain | (kNtFwd ? kOutNT : 0);
  const int ok_bwd_data = out_kind_plain | (kNtBwdData ? kOutNT : 0);
  if (mode == 0) {
    // C = out[n] (M x P): A = w (row-major M x K), B(l=k, j=p) = in[n][k][p]
    with_dt<BF16>(a_dt, [&](auto ad) {
      with_dt<BF16>(b_dt, [&](auto bd) {
        gemm_launch<BF16, decltype(ad)::value, true, false, decltype(bd)::value, false, false>(
            a, b, nullptr, out, M, P, K, K, P, P, 0, (long)K * P, (long)M * P, N, 0, 0, ok_fwd, relu, s);
      });
    });
    return hipGetLastError();
  }
  if (mode == 1 && BF16 && strip_lds_bytes(M) > 0 && out_dt == 1 && (size_t)K * P * 4 < ((size_t)1 << 31)) {
    // strip kernel: w^T in fragment order in the workspace, then one block
    // per (image, kStripP columns)
    const int ms = wt_msteps(M);
    const size_t nfr = (size_t)wt_ksteps(K) * ms * 64;
    with_dt<true>(a_dt, [&](auto ad) {
      hipLaunchKernelGGL(k_wt_frags<decltype(ad)::value>, dim3((unsigned)((nfr + 255) / 256)), dim3(256), 0, s, a, M,
                         K, ms, nfr, (uint4*)ws);
    });
    const int nstrips = (P + kStripP - 1) / kStripP;
    const size_t shm = strip_lds_bytes(M);
    with_dt<true>(b_dt, [&](auto bd) {
      if (relu)
        hipLaunchKernelGGL((k_mix_bwd_data_strip<decltype(bd)::value, true>), dim3(N * nstrips), dim3(kMixThreads),
                           shm, s, (const uint4*)ws, b, aux, (float*)out, M, K, P, ms, nstrips);
      else
        hipLaunchKernelGGL((k_mix_bwd_data_strip<decltype(bd)::value, false>), dim3(N * nstrips), dim3(kMixThreads),
                           shm, s, (const uint4*)ws, b, aux, (float*)out, M, K, P, ms, nstrips);
    });
    return hipGetLastError();
  }
  if (mode == 1) {
    // C = out[n] (K x P): A(i=k, l=m) = w[m][k] (k contiguous), B(l=m, j=p) = grad[n][m][p]
    with_dt<BF16>(a_dt, [&](auto ad) {
      with_dt<BF16>(b_dt, [&](auto bd) {
        if (relu)
          gemm_launch<BF16, decltype(ad)::value, false, false, decltype(bd)::value, false, true>(
              a, b, aux, out, K, P, M, K, P, P, 0, (long)M * P, (long)K * P, N, 0, 0, ok_bwd_data, 0, s);
        else
          gemm_launch<BF16, decltype(ad)::value, false, false, decltype(bd)::value, false, false>(
              a, b, nullptr, out, K, P, M, K, P, P, 0, (long)M * P, (long)K * P, N, 0, 0, ok_bwd_data, 0, s);
      });
    });
    return hipGetLastError();
  }
  // C = out (M x K): A(i=m, l=p) = grad[n][m][p], B(l=p, j=k) = in[n][k][p]; both p-contiguous.
  // The reduction over (n, p) is split over images and p-chunks into fp32
  // partials, summed in a fixed order by k_mix_reduce.
  const WeightSplit sp = weight_split(N, M, K, P, BF16);
  const bool direct = sp.S == 1;
  void* dst = direct ? out : ws;
  const int ok = direct ? (accumulate ? 3 : 0) : 2;
  with_dt<BF16>(a_dt, [&](auto ad) {
    with_dt<BF16>(b_dt, [&](auto bd) {
      if (relu)
        gemm_launch<BF16, decltype(ad)::value, true, true, decltype(bd)::value, true, false>(
            a, b, aux, dst, M, K, P, P, P, K, (long)M * P, (long)K * P, direct ? 0 : (long)M * K, sp.S, sp.sp,
            sp.chunk, ok, 0, s);
      else
        gemm_launch<BF16, decltype(ad)::value, true, false, decltype(bd)::value, true, false>(
            a, b, nullptr, dst, M, K, P, P, P, K, (long)M * P, (long)K * P, direct ? 0 : (long)M * K, sp.S, sp.sp,
            sp.chunk, ok, 0, s);
    });
  });
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || direct) return e;
  const size_t n = (size_t)M * K;
  if ((n & 3) == 0 && ((uintptr_t)out & 15) == 0) {
    const size_t n4 = n / 4;
    hipLaunchKernelGGL(k_mix_reduce4, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, (const float4*)ws, sp.S,
                       n4, (float4*)out, accumulate);
  } else {
    hipLaunchKernelGGL(k_mix_reduce, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, (const float*)ws, sp.S, n,
                       (float*)out, accumulate);
  }
  return hipGetLastError();
}

hipError_t launch_mix(int mode, const void* a, int a_dt, const void* b, int b_dt, void* out, int out_dt, int N,
                      int M, int K, int P, int compute_dt, int relu, const float* aux, int accumulate, void* ws,
                      size_t ws_bytes, hipStream_t s) {
  (void)ws_bytes;
  if (compute_dt == 2)
    return launch_mix_t<true>(mode, a, a_dt, b, b_dt, out, out_dt, N, M, K, P, relu, aux, accumulate, ws, s);
  return launch_mix_t<false>(mode, a, a_dt, b, b_dt, out, out_dt, N, M, K, P, relu, aux, accumulate, ws, s);
}

}  // namespace bc
