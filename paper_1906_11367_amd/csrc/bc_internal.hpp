// Host-side launcher declarations shared by the C-ABI front end (bc_api.cpp)
// and the kernel translation units.  Not part of the public interface.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bc {

// Row pitch (elements) of a table kept in LDS: W+1 columns plus 3 columns of
// padding on each side, rounded up to odd so that lanes walking down
// different rows of one column hit distinct banks.
inline int lds_pitch(int W) { return (W + 7) | 1; }

// Items of the sliding-window walk: kQ-column chunks x seg-row segments.
inline int n_chunks(int W) { return (W + 2) / 3; }
inline int n_segs(int H, int seg) { return (H + seg - 1) / seg; }

// Tap records of every box (2*C*B records of 16 words: forward, then adjoint);
// the box kernels read their taps from this table.  rounded: boxes with their
// corners rounded to integers (the kernels then take the 4-tap walks).
hipError_t launch_box_prep(const float* boxes, int C, int B, bool rounded, void* table, hipStream_t s);
inline size_t tap_table_bytes(int C, int B) { return (size_t)2 * C * B * 16 * 4; }

hipError_t launch_sat_build(const void* x, bool is_int, void* sat, float* mean,
                            int maps, int H, int W, hipStream_t s);
// Tables of zero-upsampled maps: x [maps][ceil(H/stride)][ceil(W/stride)]
// placed at every stride-th pixel of an H x W map (stride > 1).
hipError_t launch_sat_build_up(const float* x, float* sat, int maps, int H, int W, int stride, hipStream_t s);

// Forward, table in LDS.  out_kind: 0 = same type as x, 1 = fp32, 2 = bf16.
// stride > 1: y is [N][C*B][ceil(H/stride)][ceil(W/stride)].
hipError_t launch_box_fwd_lds(const void* x, bool is_int, const int* taps, void* y, int out_kind,
                              int N, int C, int H, int W, int B, bool offset, bool rounded, int stride,
                              hipStream_t s);
// Forward, table read from HBM (built beforehand by sat_build into `sat`).
hipError_t launch_box_fwd_gather(const void* sat, bool is_int, const float* means, const int* taps,
                                 void* y, int out_kind, int N, int C, int H, int W, int B, bool rounded,
                                 int stride, hipStream_t s);

// Backward (fp32).  partials: [P][C*B][4] edge gradients (a, b, c, d).
// LDS path: one block of box_bwd_lds_waves() waves per map, P = N * waves;
// box_bwd_lds_seg() == 0 means the map has too many items for one block
// (max_items: kBwdLdsItems; blocks of more than 256 threads run the 4-row
// walk, which fits the 128 VGPRs such a block allows).
// rounded: input gradient only (partials unused).  stride > 1: gy is
// [N][C*B][ceil(H/stride)][ceil(W/stride)] (tabulated zero-upsampled).
// relu_bf16: gx is bf16 [N][C][H][W], bf16(x > 0 ? dx : 0) (not with rounded).
hipError_t launch_box_bwd_lds(const float* x, const int* taps, const float* gy, void* gx,
                              float* partials, int N, int C, int H, int W, int B, bool rounded, bool relu_bf16,
                              int stride, hipStream_t s);
constexpr int kBwdLdsItems = 1024;
int box_bwd_lds_seg(int H, int W, int max_items);
int box_bwd_lds_waves(int H, int W, int max_items);
// The plain and strided LDS backward (launch_box_bwd_lds) over `maps` = N*C
// maps: its segment length and waves per map (P = N * waves).
int box_bwd_lds_seg_maps(int H, int W, long maps);
int box_bwd_lds_waves_maps(int H, int W, long maps);
// HBM path: tables of every gradient map in sat_g (built by sat_build, or
// sat_build_up for stride > 1);
// P = N * box_bwd_gather_blocks() * 4.
int box_bwd_gather_blocks(int H, int W);
hipError_t launch_box_bwd_gather(const float* x, const float* sat_g, const int* taps, void* gx,
                                 float* partials, int N, int C, int H, int W, int B, bool rounded, bool relu_bf16,
                                 hipStream_t s);
// Box-parameter reparameterisation over n = C*B boxes: op 0 = boxes from
// unit corners (in -> out), 1 = unit gradient from box gradient (in -> out),
// 2 = clip and order unit corners in place (out).
hipError_t launch_unit_params(int op, const float* in, int n, float mw, float mh, float* out, hipStream_t s);
hipError_t launch_box_grad_reduce(const float* partials, int P, int CB, float* grad_boxes,
                                  hipStream_t s);

// Kernel splitting (nx x ny pieces per box, fp32 maps).  Forward: corner
// records [C*B][32] (the pieces' shared corners with the piece weights folded
// into per-corner coefficients).  Backward: adjoint corner records [C*B][32]
// (the mirrored split box), partials [rows][C*B][8] (rows = N * waves per map
// on the LDS path, N * box_bwd_gather_blocks * 4 on the HBM path), and the
// reduce to grad_boxes [C*B][4] and the piece weights' gradient [C*B][nx*ny].
// The *_gather_split launchers read the tables sat_build wrote: one per input
// map (forward), one per upstream-gradient map (backward).
hipError_t launch_box_prep_corners(const float* boxes, const float* piece_w, int C, int B, int nx, int ny,
                                   void* table, hipStream_t s);
hipError_t launch_box_fwd_lds_split(const float* x, const int* rec, void* y, bool bf16_out, int N, int C, int H, int W,
                                    int B, int nx, int ny, hipStream_t s);
hipError_t launch_box_prep_corners_adj(const float* boxes, const float* piece_w, int C, int B, int nx, int ny,
                                       void* table, hipStream_t s);
hipError_t launch_box_bwd_lds_split(const float* x, const int* rec, const float* gy, float* gx, float* partials, int N,
                                    int C, int H, int W, int B, int nx, int ny, hipStream_t s);
hipError_t launch_box_fwd_gather_split(const float* sat, const int* rec, void* y, bool bf16_out, int N, int C, int H,
                                       int W, int B, int nx, int ny, hipStream_t s);
hipError_t launch_box_bwd_gather_split(const float* x, const float* sat_g, const int* rec, float* gx, float* partials,
                                       int N, int C, int H, int W, int B, int nx, int ny, hipStream_t s);
hipError_t launch_split_grad_reduce(const float* partials, int Pn, int CB, int P, float* grad_boxes, float* grad_w,
                                    hipStream_t s);

// Streaming box kernels (no stored table): maps up to 256 wide, B <= 16
// (W <= 64) or B <= 8 (W <= 256).  Backward partials: [N][C*B][4] (P = N).
bool box_stream_supported(int H, int W, int B);
hipError_t launch_box_bwd_stream(const float* x, const int* taps, const float* gy, void* gx, float* partials, int N,
                                 int C, int H, int W, int B, bool rounded, bool relu_bf16, hipStream_t s);
hipError_t launch_box_fwd_stream(const void* x, bool is_int, const int* taps, void* y, int out_kind, int N, int C,
                                 int H, int W, int B, bool offset, bool rounded, hipStream_t s);

// 1x1 mix GEMMs.
hipError_t launch_mix(int mode, const void* a, int a_dt, const void* b, int b_dt, void* out,
                      int out_dt, int N, int M, int K, int P, int compute_dt, int relu,
                      const float* aux, int accumulate, void* ws, size_t ws_bytes, hipStream_t s);
size_t mix_workspace_bytes(int mode, int N, int M, int K, int P, int compute_dt);
hipError_t launch_cast_bf16(const float* src, void* dst, size_t n, hipStream_t s);
hipError_t launch_relu_cast_bf16(const float* g, const float* aux, void* dst, size_t n, hipStream_t s);

}  // namespace bc
