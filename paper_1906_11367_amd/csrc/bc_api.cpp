// C-ABI front end: argument validation, path selection, workspace layout and
// launches.  Every check runs on the host before anything is enqueued.
#include <stdint.h>
#include <string.h>

#include <algorithm>

#include "../../include/boxconv.h"
#include "bc_internal.hpp"

namespace {

constexpr size_t kAlign = 256;           // workspace sub-buffer alignment
// LDS per block for the table paths.  A workgroup may take all 160 KiB of a
// CU here, but a table above 80 KiB leaves room for one block per CU, and then
// the HBM gather is faster (box forward, 4 x 64 maps, B = 4: 128x128 LDS 65 us
// against gather 112 us; 160x160 152 against 128; 190x190 346 against 151).
constexpr size_t kLdsBudget = 80 * 1024;
constexpr int kMaxStride = 1024;
constexpr long kMaxDim = 1 << 16;

inline size_t align_up(size_t v) { return (v + kAlign - 1) & ~(kAlign - 1); }
inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool dims_ok(long N, long C, long H, long W, long B) {
  if (N <= 0 || C <= 0 || H <= 0 || W <= 0 || B <= 0) return false;
  if (N > kMaxDim || C > kMaxDim || H > kMaxDim || W > kMaxDim || B > kMaxDim) return false;
  // plane and grid indices stay within int range
  if ((long)H * W > (1L << 30)) return false;
  if (N * C * B > (1L << 30)) return false;
  return true;
}

size_t table_elems(int H, int W) { return (size_t)(H + 1) * (W + 1); }

bool fwd_lds_fits(int H, int W) {
  return (size_t)(H + 1) * bc::lds_pitch(W) * 4 <= kLdsBudget;
}
bool bwd_lds_fits(int H, int W) {
  return (size_t)(H + 1) * bc::lds_pitch(W) * 4 <= kLdsBudget && bc::box_bwd_lds_seg(H, W, bc::kBwdLdsItems) > 0;
}

// Which kernels evaluate a box call: the map's table built in LDS, tables in
// HBM (built by sat_build, then gathered), or the streaming kernels (no
// stored table).  BC_FLAG_FORCE_HBM always takes the HBM tables.
enum class BoxPath { Lds, Hbm, Stream };
#ifndef BC_STREAM_POLICY
#define BC_STREAM_POLICY 1
#endif
// 0: never stream; 1: stream where the table does not fit LDS; 2: stream
// wherever the streaming kernels apply.
constexpr int kStreamPolicy = BC_STREAM_POLICY;
BoxPath box_path(bool bwd, int H, int W, int B, unsigned flags, int stride) {
  if (flags & BC_FLAG_FORCE_HBM) return BoxPath::Hbm;
  const bool fits = bwd ? bwd_lds_fits(H, W) : fwd_lds_fits(H, W);
  const bool can_stream = stride == 1 && bc::box_stream_supported(H, W, B);
  if (can_stream && (kStreamPolicy == 2 || (kStreamPolicy == 1 && !fits))) return BoxPath::Stream;
  return fits ? BoxPath::Lds : BoxPath::Hbm;
}

// Workspace layouts.  Every box entry point first writes the tap records of
// all boxes (box_prep) at offset 0; the HBM paths add their tables after it.
struct FwdWs { size_t taps, sat, means, total; };
FwdWs fwd_ws(int N, int C, int H, int W, int B, BoxPath path) {
  const bool hbm = path == BoxPath::Hbm;
  FwdWs w{};
  w.taps = 0;
  w.sat = align_up(bc::tap_table_bytes(C, B));
  if (!hbm) {
    w.total = w.sat;
    return w;
  }
  w.means = w.sat + align_up((size_t)N * C * table_elems(H, W) * 4);
  w.total = w.means + align_up((size_t)N * C * 4);
  return w;
}

struct BwdWs { size_t taps, sat_g, partials, total; int P; };
BwdWs bwd_ws(int N, int C, int H, int W, int B, BoxPath path) {
  BwdWs w{};
  w.taps = 0;
  const size_t after_taps = align_up(bc::tap_table_bytes(C, B));
  if (path == BoxPath::Stream) {   // one partial row per image
    w.P = N;
    w.partials = after_taps;
    w.total = w.partials + align_up((size_t)w.P * C * B * 4 * 4);
    return w;
  }
  if (path == BoxPath::Lds) {
    w.P = N * bc::box_bwd_lds_waves_maps(H, W, (long)N * C);
    w.partials = after_taps;
    w.total = w.partials + align_up((size_t)w.P * C * B * 4 * 4);
    return w;
  }
  w.P = N * bc::box_bwd_gather_blocks(H, W) * 4;
  w.sat_g = after_taps;
  w.partials = w.sat_g + align_up((size_t)N * C * B * table_elems(H, W) * 4);
  w.total = w.partials + align_up((size_t)w.P * C * B * 4 * 4);
  return w;
}

bc_status hip_status(hipError_t e) { return e == hipSuccess ? BC_OK : BC_ERR_HIP; }

}  // namespace

extern "C" {

int bc_abi_version(void) { return 2; }

const char* bc_status_string(int status) {
  switch (status) {
    case BC_OK: return "ok";
    case BC_ERR_NULL: return "a required pointer is NULL";
    case BC_ERR_SHAPE: return "invalid or unsupported shape";
    case BC_ERR_DTYPE: return "unsupported dtype or dtype combination";
    case BC_ERR_ALIGN: return "a tensor pointer is not 16-byte aligned";
    case BC_ERR_WORKSPACE: return "workspace missing or too small";
    case BC_ERR_HIP: return "HIP runtime error at launch";
    case BC_ERR_UNSUPPORTED: return "unsupported request";
  }
  return "unknown status";
}

bc_status box_prep(const float* boxes, int C, int B, unsigned flags, void* table, hipStream_t stream) {
  if (!boxes || !table) return BC_ERR_NULL;
  if (C <= 0 || B <= 0 || (long)C * B > (1L << 28)) return BC_ERR_SHAPE;
  if (flags & ~BC_FLAG_INTEGER_CORNERS) return BC_ERR_UNSUPPORTED;
  if (!aligned16(boxes) || !aligned16(table)) return BC_ERR_ALIGN;
  return hip_status(bc::launch_box_prep(boxes, C, B, (flags & BC_FLAG_INTEGER_CORNERS) != 0, table, stream));
}

bc_status sat_build(const void* x, int dt, void* sat, float* mean, int N, int C, int H, int W,
                    hipStream_t stream) {
  if (!x || !sat) return BC_ERR_NULL;
  if (!dims_ok(N, C, H, W, 1) || W > 1024) return BC_ERR_SHAPE;
  if (dt != BC_I32 && dt != BC_F32) return BC_ERR_DTYPE;
  if (mean && dt != BC_F32) return BC_ERR_DTYPE;
  if (!aligned16(x) || !aligned16(sat) || (mean && !aligned16(mean))) return BC_ERR_ALIGN;
  return hip_status(bc::launch_sat_build(x, dt == BC_I32, sat, mean, N * C, H, W, stream));
}

size_t bc_box_workspace_bytes_strided(int op, int N, int C, int H, int W, int B, int stride, unsigned flags) {
  if (!dims_ok(N, C, H, W, B) || stride < 1 || stride > kMaxStride) return 0;
  if (op == 0) return fwd_ws(N, C, H, W, B, box_path(false, H, W, B, flags, stride)).total;
  if (op == 1) return bwd_ws(N, C, H, W, B, box_path(true, H, W, B, flags, stride)).total;
  return 0;
}

size_t bc_box_workspace_bytes(int op, int N, int C, int H, int W, int B, unsigned flags) {
  return bc_box_workspace_bytes_strided(op, N, C, H, W, B, 1, flags);
}

bc_status box_conv_fwd_strided(const void* x, int x_dt, const float* boxes, int N, int C, int H, int W, int B,
                               int stride, void* y, int y_dt, unsigned flags, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  if (!x || !boxes || !y) return BC_ERR_NULL;
  if (!dims_ok(N, C, H, W, B) || stride < 1 || stride > kMaxStride) return BC_ERR_SHAPE;
  if (flags & ~(BC_FLAG_MEAN_OFFSET | BC_FLAG_FORCE_HBM | BC_FLAG_INTEGER_CORNERS)) return BC_ERR_UNSUPPORTED;
  const bool is_int = x_dt == BC_I32;
  const bool rounded = (flags & BC_FLAG_INTEGER_CORNERS) != 0;
  if (x_dt != BC_I32 && x_dt != BC_F32) return BC_ERR_DTYPE;
  if (is_int ? (y_dt != BC_I32) : (y_dt != BC_F32 && y_dt != BC_BF16)) return BC_ERR_DTYPE;
  if (is_int && (flags & BC_FLAG_MEAN_OFFSET)) return BC_ERR_DTYPE;
  if (!aligned16(x) || !aligned16(boxes) || !aligned16(y)) return BC_ERR_ALIGN;
  const int out_kind = y_dt == BC_BF16 ? 2 : (is_int ? 0 : 1);
  const bool offset = (flags & BC_FLAG_MEAN_OFFSET) != 0;
  const BoxPath path = box_path(false, H, W, B, flags, stride);
  const bool hbm = path == BoxPath::Hbm;
  if (hbm && W > 1024) return BC_ERR_SHAPE;
  const FwdWs L = fwd_ws(N, C, H, W, B, path);
  if (!ws) return BC_ERR_WORKSPACE;
  if (ws_bytes < L.total) return BC_ERR_WORKSPACE;
  if (!aligned16(ws)) return BC_ERR_ALIGN;
  char* base = static_cast<char*>(ws);
  const int* taps = reinterpret_cast<const int*>(base + L.taps);
  hipError_t e = bc::launch_box_prep(boxes, C, B, rounded, base + L.taps, stream);
  if (e != hipSuccess) return BC_ERR_HIP;
  if (path == BoxPath::Stream)
    return hip_status(bc::launch_box_fwd_stream(x, is_int, taps, y, out_kind, N, C, H, W, B, offset, rounded, stream));
  if (!hbm)
    return hip_status(
        bc::launch_box_fwd_lds(x, is_int, taps, y, out_kind, N, C, H, W, B, offset, rounded, stride, stream));
  float* means = offset ? reinterpret_cast<float*>(base + L.means) : nullptr;
  e = bc::launch_sat_build(x, is_int, base + L.sat, means, N * C, H, W, stream);
  if (e != hipSuccess) return BC_ERR_HIP;
  return hip_status(bc::launch_box_fwd_gather(base + L.sat, is_int, means, taps, y, out_kind, N, C, H, W, B, rounded,
                                              stride, stream));
}

bc_status box_conv_fwd(const void* x, int x_dt, const float* boxes, int N, int C, int H, int W, int B,
                       void* y, int y_dt, unsigned flags, void* ws, size_t ws_bytes, hipStream_t stream) {
  return box_conv_fwd_strided(x, x_dt, boxes, N, C, H, W, B, 1, y, y_dt, flags, ws, ws_bytes, stream);
}

// Both backward entry points: grad_x fp32, or (relu_bf16) bf16(x > 0 ? dx : 0).
static bc_status box_bwd_impl(const float* x, const float* boxes, const float* grad_y, int N, int C, int H, int W,
                              int B, int stride, void* grad_x, bool relu_bf16, float* grad_boxes, unsigned flags,
                              void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!x || !boxes || !grad_y) return BC_ERR_NULL;
  if (!dims_ok(N, C, H, W, B) || stride < 1 || stride > kMaxStride) return BC_ERR_SHAPE;
  if (flags & ~(BC_FLAG_MEAN_OFFSET | BC_FLAG_FORCE_HBM | BC_FLAG_INTEGER_CORNERS)) return BC_ERR_UNSUPPORTED;
  const bool rounded = (flags & BC_FLAG_INTEGER_CORNERS) != 0;
  // rounding the corners is not differentiable: with rounded corners the
  // boxes are frozen and only the input gradient is defined
  if (rounded && grad_boxes) return BC_ERR_UNSUPPORTED;
  if (rounded && relu_bf16) return BC_ERR_UNSUPPORTED;
  if (!aligned16(x) || !aligned16(boxes) || !aligned16(grad_y) || (grad_x && !aligned16(grad_x)) ||
      (grad_boxes && !aligned16(grad_boxes)))
    return BC_ERR_ALIGN;
  if (!grad_x && !grad_boxes) return BC_OK;
  // BC_FLAG_MEAN_OFFSET is accepted and has no effect here: the backward
  // tabulates only the upstream gradient, never x.
  const BoxPath path = box_path(true, H, W, B, flags, stride);
  const bool hbm = path == BoxPath::Hbm;
  if (hbm && W > 1024) return BC_ERR_SHAPE;
  const BwdWs L = bwd_ws(N, C, H, W, B, path);
  if (!ws) return BC_ERR_WORKSPACE;
  if (ws_bytes < L.total) return BC_ERR_WORKSPACE;
  if (!aligned16(ws)) return BC_ERR_ALIGN;
  char* base = static_cast<char*>(ws);
  float* partials = reinterpret_cast<float*>(base + L.partials);
  const int* taps = reinterpret_cast<const int*>(base + L.taps);
  hipError_t e = bc::launch_box_prep(boxes, C, B, rounded, base + L.taps, stream);
  if (e != hipSuccess) return BC_ERR_HIP;
  if (path == BoxPath::Stream) {
    e = bc::launch_box_bwd_stream(x, taps, grad_y, grad_x, partials, N, C, H, W, B, rounded, relu_bf16, stream);
  } else if (!hbm) {
    e = bc::launch_box_bwd_lds(x, taps, grad_y, grad_x, partials, N, C, H, W, B, rounded, relu_bf16, stride, stream);
  } else {
    float* sat_g = reinterpret_cast<float*>(base + L.sat_g);
    e = stride == 1 ? bc::launch_sat_build(grad_y, false, sat_g, nullptr, N * C * B, H, W, stream)
                    : bc::launch_sat_build_up(grad_y, sat_g, N * C * B, H, W, stride, stream);
    if (e == hipSuccess)
      e = bc::launch_box_bwd_gather(x, sat_g, taps, grad_x, partials, N, C, H, W, B, rounded, relu_bf16, stream);
  }
  if (e != hipSuccess) return BC_ERR_HIP;
  if (grad_boxes) e = bc::launch_box_grad_reduce(partials, L.P, C * B, grad_boxes, stream);
  return hip_status(e);
}

bc_status box_conv_bwd_strided(const float* x, const float* boxes, const float* grad_y, int N, int C, int H, int W,
                               int B, int stride, float* grad_x, float* grad_boxes, unsigned flags, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  return box_bwd_impl(x, boxes, grad_y, N, C, H, W, B, stride, grad_x, false, grad_boxes, flags, ws, ws_bytes,
                      stream);
}

bc_status box_conv_bwd_relu_bf16(const float* x, const float* boxes, const float* grad_y, int N, int C, int H, int W,
                                 int B, int stride, void* grad_x_bf16, float* grad_boxes, unsigned flags, void* ws,
                                 size_t ws_bytes, hipStream_t stream) {
  return box_bwd_impl(x, boxes, grad_y, N, C, H, W, B, stride, grad_x_bf16, true, grad_boxes, flags, ws, ws_bytes,
                      stream);
}

bc_status box_conv_bwd(const float* x, const float* boxes, const float* grad_y, int N, int C, int H, int W, int B,
                       float* grad_x, float* grad_boxes, unsigned flags, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
  return box_conv_bwd_strided(x, boxes, grad_y, N, C, H, W, B, 1, grad_x, grad_boxes, flags, ws, ws_bytes, stream);
}

// Kernel splitting: pieces per box along x and y of a split mode, or 0 (the
// BC_SPLIT_FORCE_HBM bit is ignored here).
static int split_pieces(int mode, int& nx, int& ny) {
  switch (mode & ~BC_SPLIT_FORCE_HBM) {
    case BC_SPLIT_2X: nx = 2; ny = 1; return 2;
    case BC_SPLIT_2Y: nx = 1; ny = 2; return 2;
    case BC_SPLIT_4: nx = 2; ny = 2; return 4;
  }
  return 0;
}

// Split workspaces: the boxes' corner records (32 words per box; the
// backward's are those of the mirrored boxes) at offset 0; on the HBM path
// the tables next (one per input map in the forward, one per upstream-gradient
// map in the backward); then (backward) the per-wave partials of 8 words
// (4 edge and 4 piece-weight gradients).
static size_t split_corner_bytes(int C, int B) { return align_up((size_t)C * B * 32 * 4); }

struct SplitWs { size_t sat, partials, total; int rows; };
static SplitWs split_fwd_ws(int N, int C, int H, int W, int B, bool hbm) {
  SplitWs w{};
  w.sat = split_corner_bytes(C, B);
  w.total = w.sat + (hbm ? align_up((size_t)N * C * table_elems(H, W) * 4) : 0);
  return w;
}
static SplitWs split_bwd_ws(int N, int C, int H, int W, int B, bool hbm) {
  SplitWs w{};
  w.sat = split_corner_bytes(C, B);
  w.partials = w.sat + (hbm ? align_up((size_t)N * C * B * table_elems(H, W) * 4) : 0);
  w.rows = hbm ? N * bc::box_bwd_gather_blocks(H, W) * 4 : N * bc::box_bwd_lds_waves(H, W, bc::kBwdLdsItems);
  w.total = w.partials + align_up((size_t)w.rows * C * B * 8 * 4);
  return w;
}

static bool split_dims_ok(int N, int C, int H, int W, int B) {
  return dims_ok(N, C, H, W, B) && (long)C * B <= (1L << 24);
}

size_t bc_split_workspace_bytes(int op, int N, int C, int H, int W, int B, int mode) {
  int nx, ny;
  const int P = split_pieces(mode, nx, ny);
  if (P == 0 || !split_dims_ok(N, C, H, W, B)) return 0;
  const bool force = (mode & BC_SPLIT_FORCE_HBM) != 0;
  if (op == 0) {
    const bool hbm = force || !fwd_lds_fits(H, W);
    return hbm && W > 1024 ? 0 : split_fwd_ws(N, C, H, W, B, hbm).total;
  }
  if (op == 1) {
    const bool hbm = force || !bwd_lds_fits(H, W);
    return hbm && W > 1024 ? 0 : split_bwd_ws(N, C, H, W, B, hbm).total;
  }
  return 0;
}

bc_status box_conv_split_fwd(const float* x, const float* boxes, const float* piece_w, int N, int C, int H, int W,
                             int B, int mode, void* y, int y_dt, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  if (!x || !boxes || !piece_w || !y) return BC_ERR_NULL;
  if (!split_dims_ok(N, C, H, W, B)) return BC_ERR_SHAPE;
  int nx, ny;
  const int P = split_pieces(mode, nx, ny);
  if (P == 0) return BC_ERR_UNSUPPORTED;
  if (y_dt != BC_F32 && y_dt != BC_BF16) return BC_ERR_DTYPE;
  const bool hbm = (mode & BC_SPLIT_FORCE_HBM) || !fwd_lds_fits(H, W);
  if (hbm && W > 1024) return BC_ERR_SHAPE;
  if (!aligned16(x) || !aligned16(boxes) || !aligned16(piece_w) || !aligned16(y)) return BC_ERR_ALIGN;
  const SplitWs L = split_fwd_ws(N, C, H, W, B, hbm);
  if (!ws || ws_bytes < L.total) return BC_ERR_WORKSPACE;
  if (!aligned16(ws)) return BC_ERR_ALIGN;
  char* base = static_cast<char*>(ws);
  const int* rec = reinterpret_cast<const int*>(base);
  hipError_t e = bc::launch_box_prep_corners(boxes, piece_w, C, B, nx, ny, base, stream);
  if (e != hipSuccess) return BC_ERR_HIP;
  if (!hbm)
    return hip_status(bc::launch_box_fwd_lds_split(x, rec, y, y_dt == BC_BF16, N, C, H, W, B, nx, ny, stream));
  float* sat = reinterpret_cast<float*>(base + L.sat);
  e = bc::launch_sat_build(x, false, sat, nullptr, N * C, H, W, stream);
  if (e != hipSuccess) return BC_ERR_HIP;
  return hip_status(bc::launch_box_fwd_gather_split(sat, rec, y, y_dt == BC_BF16, N, C, H, W, B, nx, ny, stream));
}

bc_status box_conv_split_bwd(const float* x, const float* boxes, const float* piece_w, const float* grad_y, int N,
                             int C, int H, int W, int B, int mode, float* grad_x, float* grad_boxes, float* grad_w,
                             void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!x || !boxes || !piece_w || !grad_y) return BC_ERR_NULL;
  if (!split_dims_ok(N, C, H, W, B)) return BC_ERR_SHAPE;
  int nx, ny;
  const int P = split_pieces(mode, nx, ny);
  if (P == 0) return BC_ERR_UNSUPPORTED;
  const bool hbm = (mode & BC_SPLIT_FORCE_HBM) || !bwd_lds_fits(H, W);
  if (hbm && W > 1024) return BC_ERR_SHAPE;
  if (!aligned16(x) || !aligned16(boxes) || !aligned16(piece_w) || !aligned16(grad_y) ||
      (grad_x && !aligned16(grad_x)) || (grad_boxes && !aligned16(grad_boxes)) || (grad_w && !aligned16(grad_w)))
    return BC_ERR_ALIGN;
  if (!grad_x && !grad_boxes && !grad_w) return BC_OK;
  const SplitWs L = split_bwd_ws(N, C, H, W, B, hbm);
  if (!ws || ws_bytes < L.total) return BC_ERR_WORKSPACE;
  if (!aligned16(ws)) return BC_ERR_ALIGN;
  char* base = static_cast<char*>(ws);
  const int* rec = reinterpret_cast<const int*>(base);
  float* partials = reinterpret_cast<float*>(base + L.partials);
  hipError_t e = bc::launch_box_prep_corners_adj(boxes, piece_w, C, B, nx, ny, base, stream);
  if (e == hipSuccess && !hbm)
    e = bc::launch_box_bwd_lds_split(x, rec, grad_y, grad_x, partials, N, C, H, W, B, nx, ny, stream);
  if (e == hipSuccess && hbm) {
    float* sat_g = reinterpret_cast<float*>(base + L.sat);
    e = bc::launch_sat_build(grad_y, false, sat_g, nullptr, N * C * B, H, W, stream);
    if (e == hipSuccess)
      e = bc::launch_box_bwd_gather_split(x, sat_g, rec, grad_x, partials, N, C, H, W, B, nx, ny, stream);
  }
  if (e == hipSuccess && (grad_boxes || grad_w))
    e = bc::launch_split_grad_reduce(partials, L.rows, C * B, P, grad_boxes, grad_w, stream);
  return hip_status(e);
}

static bool unit_args_ok(int C, int B, float mw, float mh) {
  return C > 0 && B > 0 && (long)C * B <= (1L << 28) && mw > 0.f && mh > 0.f && mw <= 1e6f && mh <= 1e6f;
}

bc_status box_params_from_unit(const float* u, int C, int B, float max_w, float max_h, float* boxes,
                               hipStream_t stream) {
  if (!u || !boxes) return BC_ERR_NULL;
  if (!unit_args_ok(C, B, max_w, max_h)) return BC_ERR_SHAPE;
  if (!aligned16(u) || !aligned16(boxes)) return BC_ERR_ALIGN;
  return hip_status(bc::launch_unit_params(0, u, C * B, max_w, max_h, boxes, stream));
}

bc_status box_params_unit_grad(const float* grad_boxes, int C, int B, float max_w, float max_h, float* grad_u,
                               hipStream_t stream) {
  if (!grad_boxes || !grad_u) return BC_ERR_NULL;
  if (!unit_args_ok(C, B, max_w, max_h)) return BC_ERR_SHAPE;
  if (!aligned16(grad_boxes) || !aligned16(grad_u)) return BC_ERR_ALIGN;
  return hip_status(bc::launch_unit_params(1, grad_boxes, C * B, max_w, max_h, grad_u, stream));
}

bc_status box_params_clip(float* u, int C, int B, hipStream_t stream) {
  if (!u) return BC_ERR_NULL;
  if (!unit_args_ok(C, B, 1.f, 1.f)) return BC_ERR_SHAPE;
  if (!aligned16(u)) return BC_ERR_ALIGN;
  return hip_status(bc::launch_unit_params(2, nullptr, C * B, 1.f, 1.f, u, stream));
}

bc_status bc_cast_bf16(const float* src, void* dst, size_t n, hipStream_t stream) {
  if (!src || !dst) return BC_ERR_NULL;
  if (n == 0 || n > ((size_t)1 << 40)) return BC_ERR_SHAPE;
  if (!aligned16(src) || !aligned16(dst)) return BC_ERR_ALIGN;
  return hip_status(bc::launch_cast_bf16(src, dst, n, stream));
}

bc_status bc_relu_grad_bf16(const float* grad, const float* out, void* dst, size_t n, hipStream_t stream) {
  if (!grad || !out || !dst) return BC_ERR_NULL;
  if (n == 0 || n > ((size_t)1 << 40)) return BC_ERR_SHAPE;
  if (!aligned16(grad) || !aligned16(out) || !aligned16(dst)) return BC_ERR_ALIGN;
  return hip_status(bc::launch_relu_cast_bf16(grad, out, dst, n, stream));
}

// The sizes pointwise_mix accepts (the workspace query answers 0 for others).
static bool mix_dims_ok(int N, int M, int K, int P) {
  if (N <= 0 || M <= 0 || K <= 0 || P <= 0 || N > kMaxDim || M > kMaxDim || K > kMaxDim) return false;
  return (long)K * P <= (1L << 30) && (long)M * P <= (1L << 30) && (long)M * K <= (1L << 30);
}

size_t bc_mix_workspace_bytes(int mode, int N, int M, int K, int P, int compute_dt) {
  if (!mix_dims_ok(N, M, K, P)) return 0;
  return bc::mix_workspace_bytes((int)mode, N, M, K, P, (int)compute_dt);
}

bc_status pointwise_mix(int mode, const void* a, int a_dt, const void* b, int b_dt, void* out,
                        int out_dt, int N, int M, int K, int P, int compute_dt, int relu, const float* aux,
                        int accumulate, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!a || !b || !out) return BC_ERR_NULL;
  if (mode != BC_MIX_FWD && mode != BC_MIX_BWD_DATA && mode != BC_MIX_BWD_WEIGHT) return BC_ERR_UNSUPPORTED;
  if (!mix_dims_ok(N, M, K, P)) return BC_ERR_SHAPE;
  if (compute_dt != BC_F32 && compute_dt != BC_BF16) return BC_ERR_DTYPE;
  for (int d : {a_dt, b_dt}) {
    if (d != BC_I32 && d != BC_F32 && d != BC_BF16) return BC_ERR_DTYPE;
    if (d == BC_BF16 && compute_dt != BC_BF16) return BC_ERR_DTYPE;
    if (d == BC_I32 && compute_dt != BC_F32) return BC_ERR_DTYPE;
  }
  const bool ints = a_dt == BC_I32 && b_dt == BC_I32;
  if ((a_dt == BC_I32) != (b_dt == BC_I32)) return BC_ERR_DTYPE;
  if (out_dt == BC_I32 ? (!ints || mode == BC_MIX_BWD_WEIGHT) : out_dt != BC_F32) return BC_ERR_DTYPE;
  if (ints && (relu || mode != BC_MIX_FWD)) return BC_ERR_DTYPE;
  if (relu && mode != BC_MIX_FWD && !aux) return BC_ERR_NULL;
  if (accumulate && mode != BC_MIX_BWD_WEIGHT) return BC_ERR_UNSUPPORTED;
  if (!aligned16(a) || !aligned16(b) || !aligned16(out) || (aux && !aligned16(aux))) return BC_ERR_ALIGN;
  const size_t need = bc::mix_workspace_bytes((int)mode, N, M, K, P, (int)compute_dt);
  if (need > 0) {
    if (!ws) return BC_ERR_WORKSPACE;
    if (ws_bytes < need) return BC_ERR_WORKSPACE;
    if (!aligned16(ws)) return BC_ERR_ALIGN;
  }
  return hip_status(bc::launch_mix((int)mode, a, (int)a_dt, b, (int)b_dt, out, (int)out_dt, N, M, K, P,
                                   (int)compute_dt, relu, mode == BC_MIX_FWD ? nullptr : aux, accumulate, ws,
                                   ws_bytes, stream));
}

}  // extern "C"
