/*
 * boxconv.h -- C ABI of the MI355X (gfx950) summed-area-table box-convolution
 * layer: Zhang, Halber, Rusinkiewicz, "Accelerating Large-Kernel Convolution
 * Using Summed-Area Tables".
 *
 * The layer (Section 3.1 and 3.2 of the paper):
 *   1. per input channel, an exclusive summed-area table of the H x W map;
 *   2. B boxes per channel applied depthwise: each output pixel reads the
 *      table at the box's four corners (Eq. 2), a corner at a sub-pixel
 *      position by bilinear interpolation of the table (Eq. 3), whatever the
 *      box size;
 *   3. a 1x1 convolution mixing the C*B filtered maps;
 *   and their gradients: to the input, to the box parameters (Eq. 4) and to
 *   the 1x1 weights.
 *
 * Conventions common to every entry point
 *   - Tensors are dense, row-major, NCHW.  Every pointer argument that names a
 *     tensor is a DEVICE pointer, 16-byte aligned; otherwise BC_ERR_ALIGN.
 *   - Box parameters are device fp32 [C][B][4] = (cx, cy, rx, ry) in pixels:
 *     (cx, cy) offsets the box centre from the output pixel's centre, rx, ry
 *     are its half-width and half-height (the paper's four variables: the x,y
 *     location and the size).  For output pixel (x, y), whose cell is
 *     [x, x+1) x [y, y+1), the box covers [x + a, x + b) x [y + c, y + d),
 *     a = 1/2 + cx - rx, b = 1/2 + cx + rx, c = 1/2 + cy - ry,
 *     d = 1/2 + cy + ry; the paper's integer corners are x_l = a, x_h = b - 1,
 *     y_l = c, y_h = d - 1.  cx = cy = 0, rx = ry = 1/2 is the identity.
 *     rx, ry >= 0 is the caller's precondition (not checked: the values live
 *     on the device).
 *   - Output channel of box b on input channel c is c*B + b.  Stride 1,
 *     output size = input size, pixels outside the map are zero.
 *   - The caller owns every buffer and keeps it alive until the stream has
 *     finished the call.  The library allocates nothing and keeps no pointer
 *     after returning.  Workspaces are caller-provided device memory of at
 *     least bc_*_workspace_bytes() bytes; their contents on entry are ignored.
 *   - Every call is asynchronous on `stream` (0 = the null stream).  Argument
 *     errors return before anything is launched.  A failed launch returns
 *     BC_ERR_HIP.  Faults during execution surface at the caller's sync.
 *   - Outputs are overwritten (pointwise_mix with accumulate = 1 excepted).
 *   - Non-finite values are not looked for; they spread as the integral image
 *     spreads them.  A NaN or infinity at pixel (i, j) of a map makes every
 *     table entry below and to the right of it non-finite.  Of that map's
 *     outputs, every one whose box covers (i, j) is non-finite, every one whose
 *     box ends above row i or left of column j is finite and exact, and the
 *     ones in between (below and right of the pixel without covering it) may be
 *     either; other maps are untouched.  With BC_FLAG_MEAN_OFFSET the map's
 *     mean is non-finite too and so is every output of that map.  The
 *     backward follows the same rule through the mirrored boxes; the edge
 *     gradients of a box are non-finite when its input map or its gradient
 *     map holds such a value.  Inputs outside the bf16 or fp32 range are not
 *     clamped.
 */
#ifndef BOXCONV_H
#define BOXCONV_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BC_OK = 0,
  BC_ERR_NULL = 1,        /* a required pointer is NULL */
  BC_ERR_SHAPE = 2,       /* a size is non-positive, too large, or inconsistent */
  BC_ERR_DTYPE = 3,       /* unsupported dtype or dtype combination */
  BC_ERR_ALIGN = 4,       /* a tensor pointer is not 16-byte aligned */
  BC_ERR_WORKSPACE = 5,   /* workspace missing or smaller than required */
  BC_ERR_HIP = 6,         /* the HIP runtime reported an error at launch */
  BC_ERR_UNSUPPORTED = 7  /* valid request the library does not implement */
} bc_status;

typedef enum { BC_I32 = 0, BC_F32 = 1, BC_BF16 = 2 } bc_dtype;

typedef enum {
  BC_MIX_FWD = 0,         /* out[n] = w * in[n]                          */
  BC_MIX_BWD_DATA = 1,    /* out[n] = w^T * grad[n]                      */
  BC_MIX_BWD_WEIGHT = 2   /* out    = sum_n grad[n] * in[n]^T            */
} bc_mix_mode;

/* Arguments that select a dtype or a mix mode are plain ints holding one of
   the enumerators above; any other value is rejected (BC_ERR_DTYPE,
   BC_ERR_UNSUPPORTED, or a zero workspace size), never undefined. */

/* Flags of box_conv_fwd / box_conv_bwd. */
#define BC_FLAG_MEAN_OFFSET 1u   /* fp32 only: build the table of (map - mean of
                                    the map) and add mean * (clipped box area)
                                    back analytically; limits cancellation in
                                    large tables. */
#define BC_FLAG_FORCE_HBM 2u     /* use the HBM-table path even when a map's table
                                    fits in LDS (both paths compute the same). */
#define BC_FLAG_INTEGER_CORNERS 4u  /* inference form of the Conclusions: each box
                                    edge (a, b, c, d, in fp64) is rounded to the
                                    nearest integer, ties up (floor(e + 1/2)),
                                    and each corner is one table sample: four
                                    samples per box instead of sixteen, no
                                    interpolation.  The boxes are then frozen
                                    (rounding is not differentiable):
                                    box_conv_bwd computes grad_x only. */

/* ------------------------------------------------------------------------
 * box_prep -- the per-box precomputation of Section 3.1 (after Eq. 4): since
 * integer shifts leave the corner fractions unchanged, each box is reduced
 * once to integer tap offsets and bilinear weights.
 *
 * boxes : device fp32 [C][B][4] (cx, cy, rx, ry).
 * flags : 0, or BC_FLAG_INTEGER_CORNERS: the records of the boxes with
 *         rounded corners (floors = the rounded edges, and for the adjoint
 *         1 - b, 1 - a, 1 - d, 1 - c of them; weights -1, 0, 1, 0).  Other
 *         flags: BC_ERR_UNSUPPORTED.
 * table : device, 2*C*B records of 16 32-bit words.  Record r < C*B is box r
 *         (r = c*B + b); record C*B + r is its adjoint: the mirrored box
 *         (centre offset negated), whose correlation is the transpose of box
 *         r's.  Words:
 *           0..3  int32  floors of the edges a, b, c, d, each clamped to
 *                        [-2^20, 2^20]; edges evaluated in fp64.  Forward
 *                        records use floor(e); adjoint records split each
 *                        edge as e = f + alpha with alpha in (0, 1], i.e.
 *                        f = ceil(e) - 1, which equals floor(e) except on
 *                        integer edges (see box_conv_bwd);
 *           4..7  fp32   x weights of columns f_a, f_a+1, f_b, f_b+1:
 *                        alpha_a - 1, -alpha_a, 1 - alpha_b, alpha_b
 *                        (alpha = e - f, in fp64, then rounded once to fp32);
 *           8..11 fp32   y weights, same for c, d;
 *          12..15        zero.
 *         The 16 tap weights of the paper are the products of an x and a y
 *         weight.  box_conv_fwd and box_conv_bwd run this first, into their
 *         workspace, and read their taps from it.
 * ---------------------------------------------------------------------- */
bc_status box_prep(const float* boxes, int C, int B, unsigned flags, void* table, hipStream_t stream);

/* ------------------------------------------------------------------------
 * sat_build -- the summed-area table (Section 3.1, before Eq. 2), exclusive
 * form: sat[m][u][v] = sum_{i<u, j<v} x[m][i][j] for u in [0,H], v in [0,W]
 * (row 0 and column 0 are zero; rows/columns 1.. are the paper's inclusive
 * table).  m ranges over the N*C maps.
 *
 * x      : device [N*C][H][W], dtype dt (BC_I32 or BC_F32).
 * sat    : device [N*C][H+1][W+1], same dtype as x.  int32 arithmetic wraps
 *          if |x| * H * W >= 2^31 (the caller's precondition).
 * mean   : NULL, or (BC_F32 only) device fp32 [N*C]: the call then writes
 *          each map's mean there and tabulates (x - mean) instead of x.
 * Limits : 1 <= W <= 1024.
 * ---------------------------------------------------------------------- */
bc_status sat_build(const void* x, int dt, void* sat, float* mean,
                    int N, int C, int H, int W, hipStream_t stream);

/* ------------------------------------------------------------------------
 * box_conv_fwd -- depthwise box filter by four bilinear table lookups per box
 * (Section 3.1, Eq. 2-3; Section 3.2):
 *   y[n][c*B+b][v][u] = integral of the zero-padded map x[n][c] over the box
 *   [u+a, u+b) x [v+c, v+d) of box (c, b).
 *
 * x      : device [N][C][H][W], x_dt = BC_I32 or BC_F32.
 * y      : device [N][C*B][H][W]; y_dt = BC_I32 iff x_dt = BC_I32, else
 *          BC_F32 or BC_BF16 (the fp32 result rounded to nearest even).
 * BC_I32 : corners are floored (fractions ignored) and the sum is exact int32
 *          arithmetic -- callers pass integer corners (half-integer cx - rx).
 * flags  : BC_FLAG_MEAN_OFFSET (BC_F32), BC_FLAG_FORCE_HBM,
 *          BC_FLAG_INTEGER_CORNERS (the box with rounded corners: the
 *          four-sample sum of Eq. 2, exact int32 for BC_I32 maps).
 * ws     : >= bc_box_workspace_bytes(0, ...) bytes: the tap records of
 *          box_prep (2*C*B*64 bytes), plus the maps' tables on the HBM path.
 * Paths  : a map whose table fits in LDS ((H + 1) * ((W + 7) | 1) * 4 <=
 *          80 KiB) has it built there, once per map and block; a larger map
 *          up to 256 wide with B <= 8 is evaluated by the streaming kernels,
 *          which keep each box's two table rows per y edge as running column
 *          sums and scan one row per output row (no stored table, no extra
 *          workspace); otherwise (or with BC_FLAG_FORCE_HBM) the tables are
 *          built in HBM by sat_build and gathered (W <= 1024).
 * ---------------------------------------------------------------------- */
bc_status box_conv_fwd(const void* x, int x_dt, const float* boxes,
                       int N, int C, int H, int W, int B,
                       void* y, int y_dt, unsigned flags,
                       void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * box_conv_bwd -- gradients of L = <grad_y, y> (fp32):
 *   grad_x[n][c] = sum_b (box (c,b))^T grad_y[n][c*B+b]: the transposed box
 *     sum, evaluated as the adjoint box (centre offset negated) read from the
 *     summed-area table of each upstream-gradient map.
 *   grad_boxes[c][b] = d L / d(cx, cy, rx, ry): each edge's derivative is the
 *     integral of x along that edge (Eq. 4 differenced between the box's two
 *     corners on that edge); at an edge lying exactly on a pixel boundary the
 *     right derivative is taken.  Evaluated through L = <x, adjoint box sums
 *     of grad_y>: the edge derivatives of the adjoint sums are differences of
 *     the taps already read for grad_x, weighted by x.  Only the gradient maps
 *     are tabulated, so BC_FLAG_MEAN_OFFSET has no effect here.
 *   With BC_FLAG_INTEGER_CORNERS: grad_x of the boxes with rounded corners
 *     (the adjoint four-sample sums); grad_boxes must be NULL
 *     (BC_ERR_UNSUPPORTED otherwise) and x is not read.
 *
 * x          : device fp32 [N][C][H][W]     (the forward input)
 * grad_y     : device fp32 [N][C*B][H][W]
 * grad_x     : device fp32 [N][C][H][W] or NULL (skip)
 * grad_boxes : device fp32 [C][B][4] or NULL (skip); summed over n with a
 *              fixed-order (deterministic) reduction.
 * ws         : >= bc_box_workspace_bytes(1, ...) bytes: the tap records,
 *              the per-wave partial edge gradients, and with the HBM path
 *              the tables of all N*C*B gradient maps.  The table is built in
 *              LDS when it takes at most 80 KiB ((H + 1) * ((W + 7) | 1) * 4
 *              bytes) and the map has at most 1024 work items of 3 columns x
 *              4 rows; otherwise maps up to 256 wide with B <= 8 take the
 *              streaming kernels (no tables), and the rest (or any call with
 *              BC_FLAG_FORCE_HBM) the HBM tables, which need W <= 1024
 *              (BC_ERR_SHAPE otherwise).
 * ---------------------------------------------------------------------- */
bc_status box_conv_bwd(const float* x, const float* boxes, const float* grad_y,
                       int N, int C, int H, int W, int B,
                       float* grad_x, float* grad_boxes, unsigned flags,
                       void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * box_conv_bwd_relu_bf16 -- box_conv_bwd_strided for a layer whose input x
 * is the rectified output of a bf16 mix before it (stacked blocks of the
 * dense prediction network, Section 3.3): the input gradient is written as
 * that mix's backward operand,
 *   grad_x_bf16[i] = bf16(x[i] > 0 ? dL/dx[i] : 0), round to nearest even,
 * which is bc_relu_grad_bf16(dL/dx, x) bit for bit for every finite value
 * and infinity (x > 0 is the ReLU's mask; a NaN stays a NaN), without
 * writing the fp32 gradient or reading it back.
 * grad_x_bf16 : device bf16 codes [N][C][H][W] or NULL (skip).
 * Every other argument, flag and workspace size is as for
 * box_conv_bwd_strided; BC_FLAG_INTEGER_CORNERS is BC_ERR_UNSUPPORTED.
 * ---------------------------------------------------------------------- */
bc_status box_conv_bwd_relu_bf16(const float* x, const float* boxes, const float* grad_y,
                                 int N, int C, int H, int W, int B, int stride,
                                 void* grad_x_bf16, float* grad_boxes, unsigned flags,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * box_conv_fwd_strided / box_conv_bwd_strided -- the same layer with an
 * integer stride (Section 3.1 assumes an integer stride: shifting a box by
 * whole pixels leaves its interpolation weights unchanged).  Output pixel
 * (i, j) is the box placed at input pixel (stride*i, stride*j):
 *   y      : [N][C*B][Ho][Wo], Ho = ceil(H/stride), Wo = ceil(W/stride);
 *   grad_y : the same shape; the gradients are those of the strided layer
 *            (the backward tabulates grad_y placed at every stride-th pixel,
 *            zeros elsewhere: the transpose of the sampling).
 * stride : 1 .. 1024 (BC_ERR_SHAPE otherwise); stride 1 is box_conv_fwd /
 *          box_conv_bwd.  Every other argument and flag is as for those
 *          calls; the workspace is bc_box_workspace_bytes_strided(..., stride,
 *          flags), which takes the input size.
 * ---------------------------------------------------------------------- */
bc_status box_conv_fwd_strided(const void* x, int x_dt, const float* boxes,
                               int N, int C, int H, int W, int B, int stride,
                               void* y, int y_dt, unsigned flags,
                               void* ws, size_t ws_bytes, hipStream_t stream);
bc_status box_conv_bwd_strided(const float* x, const float* boxes, const float* grad_y,
                               int N, int C, int H, int W, int B, int stride,
                               float* grad_x, float* grad_boxes, unsigned flags,
                               void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Box-parameter reparameterisation (Section 3.2): the corners x_l, x_h, y_l,
 * y_h of each box are trained as u = (u_xl, u_xh, u_yl, u_yh) in [-1, 1],
 * relative to a maximum box size (max_w, max_h pixels):
 *   x_l = u_xl * max_w / 2, x_h = u_xh * max_w / 2 (likewise y), the box
 *   covering [x + x_l, x + x_h + 1) -- u = 0 is the 1x1 identity box.
 * u, boxes, grad_boxes, grad_u : device fp32 [C][B][4], 16-byte aligned.
 * All arithmetic in fp64, each result rounded once to fp32.
 *
 * box_params_from_unit : boxes (cx, cy, rx, ry) for box_conv_* from u.
 * box_params_unit_grad : grad_u = dL/du from grad_boxes = dL/d(cx, cy, rx, ry)
 *                        (the chain rule of box_params_from_unit).
 * box_params_clip      : after an update, in place: u clipped to [-1, 1] and
 *                        a reversed pair (u_xl > u_xh or u_yl > u_yh) swapped.
 * Errors: NULL pointers, C, B <= 0, max sizes not in (0, 1e6].
 * ---------------------------------------------------------------------- */
bc_status box_params_from_unit(const float* u, int C, int B, float max_w, float max_h,
                               float* boxes, hipStream_t stream);
bc_status box_params_unit_grad(const float* grad_boxes, int C, int B, float max_w, float max_h,
                               float* grad_u, hipStream_t stream);
bc_status box_params_clip(float* u, int C, int B, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Kernel splitting (Section 3.1, Fig. 2): each box is cut at its centre
 * line(s), m = (a + b) / 2 and/or n = (c + d) / 2, into P pieces with their
 * own learnable weights; the output is the weighted sum of the pieces' box
 * integrals (each piece is a box of its own: 16 taps, same interpolation):
 *   y[n][c*B+b] = sum_p piece_w[c][b][p] * (integral of x[n][c] over piece p).
 * mode : BC_SPLIT_2X (P = 2: left, right halves), BC_SPLIT_2Y (P = 2: top,
 *        bottom), BC_SPLIT_4 (P = 4: quadrants); piece p = i * nx + j covers
 *        columns [k_j, k_{j+1}) of k = (a, m, b) (or (a, b)) and rows
 *        [r_i, r_{i+1}) of r = (c, n, d) (or (c, d)); edges in fp64.
 *        OR-ed with BC_SPLIT_FORCE_HBM: take the HBM-table kernels even
 *        where the map's table fits in LDS (same results up to fp32
 *        rounding order).  Other values: BC_ERR_UNSUPPORTED.
 * x, boxes, grad_y, grad_x, grad_boxes : as box_conv_fwd / box_conv_bwd,
 *        fp32 maps, stride 1, no flags.
 * piece_w : device fp32 [C][B][P].
 * y      : device [N][C*B][H][W], BC_F32 or BC_BF16.
 * box_conv_split_bwd : gradients of L = <grad_y, y> (any of grad_x,
 *        grad_boxes, grad_w may be NULL; all NULL is a no-op).  grad_boxes:
 *        each piece's edge derivatives (Eq. 4) times its weight, summed onto
 *        the box's edges, a cut edge contributing half to each of the two
 *        edges it is the mean of; grad_w [C][B][P] = <grad_y, piece sum>.
 *        Sums over n are fixed-order (deterministic).
 * Paths : as box_conv_fwd / box_conv_bwd: the map's table in LDS when
 *        (H + 1) * ((W + 7) | 1) * 4 <= 80 KiB (and, for the backward, the
 *        map has at most 1024 work items of 3 columns x 4 rows: one block
 *        per map), else tables in HBM built into the workspace, which needs
 *        W <= 1024 (BC_ERR_SHAPE otherwise).
 *        C * B <= 2^24.
 * ws     : >= bc_split_workspace_bytes(op, ...) (op 0 = forward: one record
 *        of 128 bytes per box, its shared corners with the piece weights
 *        folded in, plus the HBM path's tables of the N*C input maps; op 1 =
 *        backward: the same records for the mirrored boxes, the HBM path's
 *        tables of the N*C*B upstream-gradient maps, and per-wave gradient
 *        partials).  The query takes the same mode (with its
 *        BC_SPLIT_FORCE_HBM bit) and returns 0 for an unsupported request.
 * ---------------------------------------------------------------------- */
#define BC_SPLIT_2X 1
#define BC_SPLIT_2Y 2
#define BC_SPLIT_4 3
#define BC_SPLIT_FORCE_HBM 0x100
bc_status box_conv_split_fwd(const float* x, const float* boxes, const float* piece_w,
                             int N, int C, int H, int W, int B, int mode,
                             void* y, int y_dt, void* ws, size_t ws_bytes, hipStream_t stream);
bc_status box_conv_split_bwd(const float* x, const float* boxes, const float* piece_w,
                             const float* grad_y, int N, int C, int H, int W, int B, int mode,
                             float* grad_x, float* grad_boxes, float* grad_w,
                             void* ws, size_t ws_bytes, hipStream_t stream);
size_t bc_split_workspace_bytes(int op, int N, int C, int H, int W, int B, int mode);

/* ------------------------------------------------------------------------
 * pointwise_mix -- the 1x1 convolution over the C*B filtered maps
 * (Section 1, Section 3.2), per image n with P = H*W pixels, on MFMA:
 *   BC_MIX_FWD        : a = w [M][K], b = in [N][K][P]   -> out [N][M][P]
 *   BC_MIX_BWD_DATA   : a = w [M][K], b = grad [N][M][P] -> out [N][K][P]
 *   BC_MIX_BWD_WEIGHT : a = grad [N][M][P], b = in [N][K][P] -> out [M][K]
 * compute_dt : BC_F32  (fp32 operands and accumulation; exact for integer
 *                       data while every partial sum stays below 2^24),
 *              BC_BF16 (operands rounded to bf16, nearest even, on load;
 *                       fp32 accumulation).
 * a_dt, b_dt : dtype of the stored operands: BC_F32, BC_BF16 (bf16 storage,
 *              compute_dt must be BC_BF16) or BC_I32 (compute_dt BC_F32,
 *              values converted exactly while |v| < 2^24).
 * out_dt     : BC_F32, or BC_I32 when both operands are BC_I32.
 * relu       : FWD: out = max(out, 0).  BWD_DATA / BWD_WEIGHT: the incoming
 *              gradient is multiplied by (aux > 0), aux = the forward output
 *              [N][M][P] fp32 (required then).
 * accumulate : BWD_WEIGHT only: 1 = out += result.
 * ws         : >= bc_mix_workspace_bytes(mode, ...) bytes (NULL when that is
 *              0): BWD_WEIGHT's split-K partials; in BC_BF16, BWD_DATA's copy
 *              of w^T in the MFMA operand order (2 * K * M bytes, rounded up
 *              to 64 rows and 64 columns) when M <= 448 and K * P * 4 < 2^31,
 *              the shapes its column-strip kernel takes.
 * ---------------------------------------------------------------------- */
bc_status pointwise_mix(int mode, const void* a, int a_dt,
                        const void* b, int b_dt, void* out, int out_dt,
                        int N, int M, int K, int P, int compute_dt,
                        int relu, const float* aux, int accumulate,
                        void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bc_cast_bf16 -- dst[i] = bf16(src[i]) for i < n, round to nearest even (NaN
 * stays NaN).  src: device fp32 [n]; dst: device bf16 codes [n].  Lets a
 * caller hold the 1x1 weights in the mix's compute type once per step instead
 * of every GEMM tile rounding them again (pointwise_mix accepts BC_BF16
 * storage for either operand).
 * ---------------------------------------------------------------------- */
bc_status bc_cast_bf16(const float* src, void* dst, size_t n, hipStream_t stream);

/* ------------------------------------------------------------------------
 * bc_relu_grad_bf16 -- the backward of a ReLU after the mix (a layer whose
 * mix output is rectified, as in the stacked blocks of the dense prediction
 * network, Section 3.3):
 *   dst[i] = bf16(out[i] > 0 ? grad[i] : 0), round to nearest even.
 * grad: device fp32 [n], dL/d(rectified output); out: device fp32 [n], the
 * rectified forward output; dst: device bf16 codes [n].  These are exactly
 * the operand values pointwise_mix(BC_BF16, relu = 1, aux = out) forms from
 * grad on load, so BWD_DATA and BWD_WEIGHT with relu = 0 on dst (BC_BF16
 * storage) return bitwise the same results, reading 2 bytes per element
 * instead of 8 in each GEMM.  Errors: BC_ERR_NULL, BC_ERR_SHAPE (n = 0),
 * BC_ERR_ALIGN (pointers not 16-byte aligned).
 * ---------------------------------------------------------------------- */
bc_status bc_relu_grad_bf16(const float* grad, const float* out, void* dst, size_t n, hipStream_t stream);

/* ------------------------------------------------------------------------
 * box_conv_bwd_noalloc -- for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): box_conv_bwd with its workspace taken from a fixed device array
 * the library owns, BC_NOALLOC_SCRATCH_BYTES bytes on each GPU it runs on,
 * held until the process ends.  The call allocates nothing.
 *
 * Arguments, flags, results and errors are those of box_conv_bwd, without
 * ws / ws_bytes.  A request whose workspace (bc_box_workspace_bytes(1, ...))
 * exceeds BC_NOALLOC_SCRATCH_BYTES returns BC_ERR_WORKSPACE before anything
 * runs: in practice the maps whose table fits in LDS (the pose-shaped layer:
 * about 1.2 MB at N = 32, C = 256, B = 4, 64 x 48); maps that need their
 * tables in HBM (256 x 256) do not fit.  bc_noalloc_scratch_bytes() returns
 * the array's size.
 *
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents (the call writes every word it reads, so nothing stale is used):
 * calls that overlap on one GPU -- on different streams, or from different
 * host threads -- race on it and must be serialised by the caller.  The
 * array's device address is looked up once per device, on the first call
 * made with that device current.
 * ---------------------------------------------------------------------- */
#define BC_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
bc_status box_conv_bwd_noalloc(const float* x, const float* boxes, const float* grad_y,
                               int N, int C, int H, int W, int B,
                               float* grad_x, float* grad_boxes, unsigned flags,
                               hipStream_t stream);
size_t bc_noalloc_scratch_bytes(void);

/* Workspace sizes in bytes.  op: 0 = box_conv_fwd, 1 = box_conv_bwd (and
 * box_conv_bwd_relu_bf16); the _strided form for the strided entry points
 * (stride 1 is the plain query).  0 for sizes the calls reject. */
size_t bc_box_workspace_bytes(int op, int N, int C, int H, int W, int B, unsigned flags);
size_t bc_box_workspace_bytes_strided(int op, int N, int C, int H, int W, int B, int stride,
                                      unsigned flags);
size_t bc_mix_workspace_bytes(int mode, int N, int M, int K, int P, int compute_dt);

/* Human-readable status; never NULL. */
const char* bc_status_string(int status);

/* ABI version of this library (incremented on incompatible changes). */
int bc_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* BOXCONV_H */
