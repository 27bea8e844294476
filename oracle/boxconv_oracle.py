"""Plain CPU oracle of the SAT box-convolution layer (fp64 / int64, NumPy).

TEST INFRASTRUCTURE ONLY: used by tests/, the smoke check and the benchmark's
CPU-baseline leg; never by the product path.

What the layer computes (Zhang, Halber, Rusinkiewicz, "Accelerating Large-Kernel
Convolution Using Summed-Area Tables"):

* Section 3.1, Eq. 1: a box filter sums the input over a rectangle placed
  relative to each output pixel (a cross-correlation, stride 1).
* Section 3.1, Eq. 2-3: the same sum is read from a summed-area table at the
  four box corners; corners at sub-pixel positions are sampled by bilinear
  interpolation of the table.  Bilinear interpolation of the exclusive table
  between integer nodes is exactly the integral of the piecewise-constant
  image, so the layer output is the *area integral* of the zero-padded image
  over a continuous rectangle.  That plain definition is what this oracle
  evaluates, by fractional-overlap weights; it never builds a table except in
  ``sat_exclusive``, whose definition is the table itself.
* Section 3.1, Eq. 4 and the text after it: derivatives with respect to the
  corner positions and to the table samples.  Here they are the analytic
  derivatives of the area integral (edge integrals), using the right
  derivative where an edge sits exactly on a pixel boundary (the paper's floor
  and ceiling coincide there, see the reading below).
* Section 3.2: B boxes per input channel applied depthwise, then a 1x1
  convolution mixing the C*B filtered maps.

Readings of points the paper leaves open (each is restated where it is used):

R1  The table is exclusive: S[u][v] = sum_{i<u, j<v} I[i][j], u in [0,H],
    v in [0,W].  Eq. 2 samples S at x+x_l and x+x_h+1, which is only right for
    this form; the text's "including" is the same data without the zero row
    and column.
R2  Eq. 1's second form swaps the roles of i and j; the first form (x offset
    over [x_l, x_h], y offset over [y_l, y_h]) is taken as meant.
R3  Box parameters are (cx, cy, rx, ry) in pixels: a centre offset from the
    output pixel's centre and a half-width / half-height.  For output pixel x
    (cell [x, x+1)) the box covers [x + a, x + b) with a = 1/2 + cx - rx and
    b = 1/2 + cx + rx (so the paper's x_l = a and x_h = b - 1); likewise
    c, d in y.  cx = cy = 0, rx = ry = 1/2 is the identity.
R4  Pixels outside the image are zero (table indices clamped to [0,H]x[0,W]).
R5  Edge positions and their floors are evaluated in fp64 from the fp32
    parameters.  At an integer edge the derivative is the right derivative.
R6  No area normalisation and no bias (Eq. 1 is a plain sum).
R7  Output channel of box b on input channel c is c*B + b.
R8  A bf16 1x1 mix rounds both operands to bf16 (round to nearest even) and
    accumulates exactly; the oracle accumulates in fp64.
R13 Integer stride s (Section 3.1 assumes an integer stride so that the
    interpolation weights stay fixed): output pixel (i, j) is the box placed
    at input pixel (s*i, s*j); the output is ceil(H/s) x ceil(W/s).  Stride 1
    is the plain layer.
R14 Box-parameter reparameterisation (Section 3.2): the corners x_l, x_h,
    y_l, y_h are kept as u in [-1, 1] relative to a maximum box size M (per
    axis): x_l = u_xl * M_x / 2 and x_h = u_xh * M_x / 2 (so u = 0 is the
    1x1 identity box), converted during the forward pass; after each update
    u is clipped to [-1, 1] and a reversed pair (x_l > x_h) is swapped.
R15 Kernel splitting (Section 3.1, Fig. 2): a split box is cut at its centre
    line(s) into 2 pieces side by side (mode 2x), 2 stacked (2y) or 4 (mode
    4); piece p has its own weight w[c, b, p] and the output is the weighted
    sum of the pieces' box sums.  The cut edges are m = (a + b) / 2 and
    n = (c + d) / 2, so a split box keeps the 4 parameters of the box plus
    the piece weights, and the pieces share the cut edges.
R12 Integer corners for inference (Conclusions: once the boxes have
    converged, round the sampling points to integers so that no interpolation
    is needed): each edge a, b, c, d is rounded to the nearest integer, a tie
    (an edge exactly halfway between two integers) rounding up:
    floor(e + 1/2).  The boxes are then fixed; only the input gradient is
    defined.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "box_edges", "rounded_edges", "mirrored_boxes", "overlap_matrix", "sat_exclusive",
    "map_mean", "box_forward", "box_backward_input", "box_backward_params",
    "box_param_grad_from_edges", "bf16_round", "mix_forward",
    "mix_backward_data", "mix_backward_weight", "relu", "layer_forward",
    "stack_forward", "stack_backward", "naive_box_forward_eq1", "strided_size", "zero_upsample",
    "boxes_from_unit", "unit_grad_from_box_grad", "clip_unit_params",
    "SPLIT_MODES", "split_edges", "box_forward_split", "box_backward_split_input",
    "box_backward_split_params",
    "naive_box_forward_overlap", "tolerance_ok", "rel_errors",
]


# ---------------------------------------------------------------------------
# Box geometry (Section 3.1, Eq. 2 corners; reading R3, R5)
# ---------------------------------------------------------------------------
def box_edges(boxes):
    """Edges (a, b, c, d) in fp64 of boxes given as fp32 (cx, cy, rx, ry).

    boxes: array [..., 4].  Returns four fp64 arrays of shape boxes.shape[:-1].
    For output pixel (x, y) the box covers [x+a, x+b) x [y+c, y+d); in the
    paper's integer notation x_l = a, x_h = b - 1, y_l = c, y_h = d - 1.
    """
    p = np.asarray(boxes, dtype=np.float32).astype(np.float64)
    cx, cy, rx, ry = p[..., 0], p[..., 1], p[..., 2], p[..., 3]
    return 0.5 + cx - rx, 0.5 + cx + rx, 0.5 + cy - ry, 0.5 + cy + ry


def rounded_edges(boxes):
    """Edges (a, b, c, d) of the boxes with their corners rounded to integers
    (reading R12): each fp64 edge e becomes floor(e + 1/2), so a tie rounds
    up.  Returns four fp64 arrays holding integers."""
    return tuple(np.floor(e + 0.5) for e in box_edges(boxes))


def mirrored_boxes(boxes):
    """The box whose correlation is the adjoint of the given box's correlation.

    With zero padding, the transpose of correlating with [a, b) is correlating
    with [1-b, 1-a): the centre offset changes sign, the size is kept.
    """
    m = np.array(boxes, dtype=np.float32, copy=True)
    m[..., 0] = -m[..., 0]
    m[..., 1] = -m[..., 1]
    return m


def overlap_matrix(n, lo, hi):
    """M[x, j] = length of [j, j+1) intersected with [x+lo, x+hi), x, j in [0, n).

    This is the 1-D weight with which input pixel j enters output pixel x when
    the box's extent along this axis is [x+lo, x+hi) and pixels outside
    [0, n) do not exist (zero padding, reading R4).
    """
    x = np.arange(n, dtype=np.float64)[:, None]
    j = np.arange(n, dtype=np.float64)[None, :]
    return np.maximum(0.0, np.minimum(j + 1.0, x + hi) - np.maximum(j, x + lo))


# ---------------------------------------------------------------------------
# Summed-area table (Section 3.1, the definition before Eq. 2; reading R1)
# ---------------------------------------------------------------------------
def sat_exclusive(x):
    """Exclusive SAT of every map: S[..., u, v] = sum_{i<u, j<v} x[..., i, j].

    x: [..., H, W] integer or float.  Returns [..., H+1, W+1] in int64 or fp64;
    row 0 and column 0 are zero.
    """
    x = np.asarray(x)
    dt = np.int64 if np.issubdtype(x.dtype, np.integer) else np.float64
    s = np.zeros(x.shape[:-2] + (x.shape[-2] + 1, x.shape[-1] + 1), dtype=dt)
    s[..., 1:, 1:] = np.cumsum(np.cumsum(x.astype(dt), axis=-2), axis=-1)
    return s


def map_mean(x):
    """Per-map mean (fp64) of a [..., H, W] array: the offset that can be
    subtracted before building a floating-point table to limit cancellation."""
    return np.asarray(x, dtype=np.float64).mean(axis=(-2, -1))


# ---------------------------------------------------------------------------
# Depthwise box filter, forward (Section 3.1 Eq. 1-3, Section 3.2)
# ---------------------------------------------------------------------------
def _is_int(x):
    return np.issubdtype(np.asarray(x).dtype, np.integer)


def strided_size(n, stride):
    """Output extent of a stride-s filter over n pixels (reading R13)."""
    return (n + stride - 1) // stride


def zero_upsample(g, H, W, stride):
    """[..., ceil(H/s), ceil(W/s)] -> [..., H, W]: g[..., i, j] at (s*i, s*j),
    zero elsewhere.  The transpose of sampling every s-th pixel."""
    g = np.asarray(g)
    if stride == 1:
        return g
    out = np.zeros(g.shape[:-2] + (H, W), dtype=g.dtype)
    out[..., ::stride, ::stride] = g
    return out


def box_forward(x, boxes, integer_corners=False, stride=1):
    """O[n, c*B+b] = integral of zero-padded x[n, c] over each box (fp64/int64).

    x: [N, C, H, W]; boxes: [C, B, 4] fp32 (cx, cy, rx, ry).
    Computed as O = Wy @ I @ Wx^T with the overlap matrices of each box.  For
    integer x the boxes must have integer corners (then every weight is 0 or
    1) and the result is exact int64.  integer_corners: the boxes with their
    corners rounded (reading R12) -- the plain sum of Eq. 1 over the rounded
    box, for any map type.  stride: the output at every stride-th pixel
    (reading R13), [N, C*B, ceil(H/s), ceil(W/s)].
    """
    x = np.asarray(x)
    N, C, H, W = x.shape
    B = boxes.shape[1]
    a, b, c, d = rounded_edges(boxes) if integer_corners else box_edges(boxes)
    integer = _is_int(x)
    dt = np.int64 if integer else np.float64
    xf = x.astype(dt)
    out = np.empty((N, C, B, H, W), dtype=dt)
    for ci in range(C):
        for bi in range(B):
            wx = overlap_matrix(W, a[ci, bi], b[ci, bi])
            wy = overlap_matrix(H, c[ci, bi], d[ci, bi])
            if integer:
                if not (np.all(wx == np.round(wx)) and np.all(wy == np.round(wy))):
                    raise ValueError("integer maps need integer box corners")
                wx = wx.astype(np.int64)
                wy = wy.astype(np.int64)
            out[:, ci, bi] = wy @ xf[:, ci] @ wx.T
    return out.reshape(N, C * B, H, W)[..., ::stride, ::stride]


def box_backward_input(grad_y, boxes, H, W, integer_corners=False, stride=1):
    """dI[n, c] = sum_b Wy^T @ dO[n, c*B+b] @ Wx  (transpose of box_forward).

    grad_y: [N, C*B, H, W]; returns fp64 [N, C, H, W].  The paper states only
    the local derivative of a table sample (its bilinear weight, the text after
    Eq. 4); this is the chain rule of the whole forward map.  integer_corners:
    the transpose of box_forward(..., integer_corners=True).  stride: grad_y
    is [N, C*B, ceil(H/s), ceil(W/s)]; the transpose of sampling every s-th
    pixel places it on the full grid (zero_upsample) first.
    """
    g = zero_upsample(np.asarray(grad_y, dtype=np.float64), H, W, stride)
    C, B = boxes.shape[0], boxes.shape[1]
    N = g.shape[0]
    g = g.reshape(N, C, B, H, W)
    a, b, c, d = rounded_edges(boxes) if integer_corners else box_edges(boxes)
    out = np.zeros((N, C, H, W), dtype=np.float64)
    for ci in range(C):
        for bi in range(B):
            wx = overlap_matrix(W, a[ci, bi], b[ci, bi])
            wy = overlap_matrix(H, c[ci, bi], d[ci, bi])
            out[:, ci] += wy.T @ g[:, ci, bi] @ wx
    return out


def _edge_selector(n, edge):
    """E[x, j] = 1 where j = floor(x + edge) lies in [0, n), else 0.

    Column floor(x+edge) is the pixel column that a right-moving edge at
    x+edge sweeps into (right derivative, reading R5); outside the image the
    swept column does not exist and contributes nothing (R4).
    """
    x = np.arange(n)
    j = np.floor(x.astype(np.float64) + edge).astype(np.int64)
    e = np.zeros((n, n), dtype=np.float64)
    ok = (j >= 0) & (j < n)
    e[x[ok], j[ok]] = 1.0
    return e


def box_param_grad_from_edges(x, grad_y, boxes):
    """Gradients of L = <grad_y, O> with respect to the edges a, b, c, d.

    Returns fp64 [C, B, 4] holding (dL/da, dL/db, dL/dc, dL/dd).
    dO/db at (y, x) is the integral of the image over the edge column
    floor(x+b) between y+c and y+d (Eq. 4 differenced between the two
    y-corners of the box); dO/da is minus the same at floor(x+a); dO/dc and
    dO/dd are the row analogues.
    """
    xf = np.asarray(x, dtype=np.float64)
    N, C, H, W = xf.shape
    B = boxes.shape[1]
    g = np.asarray(grad_y, dtype=np.float64).reshape(N, C, B, H, W)
    a, b, c, d = box_edges(boxes)
    out = np.zeros((C, B, 4), dtype=np.float64)
    for ci in range(C):
        for bi in range(B):
            out[ci, bi] = _edge_grads(xf[:, ci], g[:, ci, bi], a[ci, bi], b[ci, bi], c[ci, bi], d[ci, bi])
    return out


def _edge_grads(img, gb, a, b, c, d):
    """(dL/da, dL/db, dL/dc, dL/dd) of L = <gb, box sum of img over [a, b) x [c, d)>
    for one box; img, gb: [N, H, W]."""
    H, W = img.shape[-2:]
    wx = overlap_matrix(W, a, b)
    wy = overlap_matrix(H, c, d)
    return np.array([-np.sum(gb * (wy @ img @ _edge_selector(W, a).T)),
                     np.sum(gb * (wy @ img @ _edge_selector(W, b).T)),
                     -np.sum(gb * (_edge_selector(H, c) @ img @ wx.T)),
                     np.sum(gb * (_edge_selector(H, d) @ img @ wx.T))])


def box_backward_params(x, grad_y, boxes, stride=1):
    """Gradient of L = <grad_y, O> with respect to (cx, cy, rx, ry), fp64 [C, B, 4].

    a = 1/2+cx-rx, b = 1/2+cx+rx, c = 1/2+cy-ry, d = 1/2+cy+ry, so
    dcx = gA+gB, dcy = gC+gD, drx = gB-gA, dry = gD-gC.  stride: as in
    box_backward_input (the strided output is the full output sampled, so its
    gradient is the full one of the zero-upsampled grad_y).
    """
    H, W = np.asarray(x).shape[-2:]
    g = zero_upsample(np.asarray(grad_y, dtype=np.float64), H, W, stride)
    e = box_param_grad_from_edges(x, g, boxes)
    ga, gb, gc, gd = e[..., 0], e[..., 1], e[..., 2], e[..., 3]
    return np.stack([ga + gb, gc + gd, gb - ga, gd - gc], axis=-1)


# ---------------------------------------------------------------------------
# Kernel splitting (Section 3.1, Fig. 2; reading R15)
# ---------------------------------------------------------------------------
SPLIT_MODES = {"2x": (1, 2), "2y": (2, 1), "4": (2, 2)}   # (pieces along y, pieces along x)


def split_edges(boxes, mode):
    """Edges (a_p, b_p, c_p, d_p) fp64 [C, B, P, 4] of the pieces of split
    boxes: the box [a, b) x [c, d) cut at m = (a + b) / 2 (modes 2x, 4) and
    n = (c + d) / 2 (modes 2y, 4); piece p = i * nx + j covers rows
    [r_i, r_{i+1}) and columns [k_j, k_{j+1}) with k = (a, m, b) or (a, b)
    and r = (c, n, d) or (c, d)."""
    a, b, c, d = box_edges(boxes)
    ny, nx = SPLIT_MODES[mode]
    ks = [a, (a + b) / 2, b] if nx == 2 else [a, b]
    rs = [c, (c + d) / 2, d] if ny == 2 else [c, d]
    out = np.empty(a.shape + (ny * nx, 4), dtype=np.float64)
    for i in range(ny):
        for j in range(nx):
            out[..., i * nx + j, :] = np.stack([ks[j], ks[j + 1], rs[i], rs[i + 1]], axis=-1)
    return out


def box_forward_split(x, boxes, piece_w, mode):
    """O[n, c*B+b] = sum_p w[c, b, p] * integral of x[n, c] over piece p (fp64).
    piece_w: [C, B, P] with P = 2 (modes 2x, 2y) or 4."""
    xf = np.asarray(x, dtype=np.float64)
    N, C, H, W = xf.shape
    B = boxes.shape[1]
    e = split_edges(boxes, mode)
    w = np.asarray(piece_w, dtype=np.float64)
    out = np.zeros((N, C, B, H, W), dtype=np.float64)
    for ci in range(C):
        for bi in range(B):
            for p in range(e.shape[2]):
                a, b, c, d = e[ci, bi, p]
                out[:, ci, bi] += w[ci, bi, p] * (overlap_matrix(H, c, d) @ xf[:, ci] @ overlap_matrix(W, a, b).T)
    return out.reshape(N, C * B, H, W)


def box_backward_split_input(grad_y, boxes, piece_w, mode, H, W):
    """dI[n, c] = sum_b sum_p w[c, b, p] * Wy_p^T @ dO[n, c*B+b] @ Wx_p (the transpose)."""
    g = np.asarray(grad_y, dtype=np.float64)
    C, B = boxes.shape[0], boxes.shape[1]
    N = g.shape[0]
    g = g.reshape(N, C, B, H, W)
    e = split_edges(boxes, mode)
    w = np.asarray(piece_w, dtype=np.float64)
    out = np.zeros((N, C, H, W), dtype=np.float64)
    for ci in range(C):
        for bi in range(B):
            for p in range(e.shape[2]):
                a, b, c, d = e[ci, bi, p]
                out[:, ci] += w[ci, bi, p] * (overlap_matrix(H, c, d).T @ g[:, ci, bi] @ overlap_matrix(W, a, b))
    return out


def box_backward_split_params(x, grad_y, boxes, piece_w, mode):
    """Gradients of L = <grad_y, O> for split boxes: (d/d(cx, cy, rx, ry) fp64
    [C, B, 4], d/dw fp64 [C, B, P]).

    dL/dw_p is <grad_y, box sum of piece p>.  The edge derivatives of each
    piece (times its weight) are summed onto the edges of the box: the outer
    edges directly, and the cut edges m = (a + b) / 2, n = (c + d) / 2 half to
    each edge they are the mean of."""
    xf = np.asarray(x, dtype=np.float64)
    N, C, H, W = xf.shape
    B = boxes.shape[1]
    g = np.asarray(grad_y, dtype=np.float64).reshape(N, C, B, H, W)
    e = split_edges(boxes, mode)
    w = np.asarray(piece_w, dtype=np.float64)
    ny, nx = SPLIT_MODES[mode]
    gbox = np.zeros((C, B, 4), dtype=np.float64)
    gw = np.zeros((C, B, ny * nx), dtype=np.float64)
    for ci in range(C):
        for bi in range(B):
            img, gb = xf[:, ci], g[:, ci, bi]
            gk = np.zeros(nx + 1)          # dL/d(column edge k)
            gr = np.zeros(ny + 1)          # dL/d(row edge r)
            for i in range(ny):
                for j in range(nx):
                    p = i * nx + j
                    a, b, c, d = e[ci, bi, p]
                    gw[ci, bi, p] = np.sum(gb * (overlap_matrix(H, c, d) @ img @ overlap_matrix(W, a, b).T))
                    ge = w[ci, bi, p] * _edge_grads(img, gb, a, b, c, d)
                    gk[j] += ge[0]
                    gk[j + 1] += ge[1]
                    gr[i] += ge[2]
                    gr[i + 1] += ge[3]
            ga, gbb = gk[0], gk[-1]
            gc, gd = gr[0], gr[-1]
            if nx == 2:
                ga += gk[1] / 2
                gbb += gk[1] / 2
            if ny == 2:
                gc += gr[1] / 2
                gd += gr[1] / 2
            gbox[ci, bi] = [ga + gbb, gc + gd, gbb - ga, gd - gc]
    return gbox, gw


# ---------------------------------------------------------------------------
# Box-parameter reparameterisation (Section 3.2; reading R14)
# ---------------------------------------------------------------------------
def boxes_from_unit(u, max_w, max_h):
    """(cx, cy, rx, ry) fp32 [..., 4] of corners given as u = (u_xl, u_xh,
    u_yl, u_yh) in [-1, 1]: x_l = u_xl * max_w / 2, x_h = u_xh * max_w / 2,
    and the box covers [x + x_l, x + x_h + 1), i.e. cx = (x_l + x_h) / 2,
    rx = (x_h - x_l + 1) / 2 (likewise y).  fp64, rounded once to fp32."""
    u = np.asarray(u, dtype=np.float32).astype(np.float64)
    mw, mh = float(np.float32(max_w)), float(np.float32(max_h))
    xl, xh = u[..., 0] * mw / 2, u[..., 1] * mw / 2
    yl, yh = u[..., 2] * mh / 2, u[..., 3] * mh / 2
    return np.stack([(xl + xh) / 2, (yl + yh) / 2, (xh - xl + 1) / 2, (yh - yl + 1) / 2],
                    axis=-1).astype(np.float32)


def unit_grad_from_box_grad(grad_boxes, max_w, max_h):
    """Chain rule through boxes_from_unit: dL/du from dL/d(cx, cy, rx, ry).
    dL/du_xl = (dcx - drx) / 2 * max_w / 2, dL/du_xh = (dcx + drx) / 2 * max_w / 2
    (likewise y).  fp64, rounded once to fp32."""
    g = np.asarray(grad_boxes, dtype=np.float32).astype(np.float64)
    mw, mh = float(np.float32(max_w)), float(np.float32(max_h))
    dcx, dcy, drx, dry = g[..., 0], g[..., 1], g[..., 2], g[..., 3]
    return np.stack([(dcx - drx) / 2 * mw / 2, (dcx + drx) / 2 * mw / 2,
                     (dcy - dry) / 2 * mh / 2, (dcy + dry) / 2 * mh / 2], axis=-1).astype(np.float32)


def clip_unit_params(u):
    """After an update: each u clipped to [-1, 1], then a reversed pair
    (u_xl > u_xh, or u_yl > u_yh) swapped, so that x_l <= x_h and y_l <= y_h."""
    v = np.clip(np.asarray(u, dtype=np.float32), np.float32(-1), np.float32(1))
    out = v.copy()
    out[..., 0] = np.minimum(v[..., 0], v[..., 1])
    out[..., 1] = np.maximum(v[..., 0], v[..., 1])
    out[..., 2] = np.minimum(v[..., 2], v[..., 3])
    out[..., 3] = np.maximum(v[..., 2], v[..., 3])
    return out


# ---------------------------------------------------------------------------
# Naive per-pixel loops (tiny inputs only)
# ---------------------------------------------------------------------------
def naive_box_forward_eq1(x, boxes):
    """Eq. 1 written out: for integer corners, O(x, y) is the plain sum of the
    input over rows y+y_l..y+y_h and columns x+x_l..x+x_h, pixels outside the
    image counting as zero.  Pure Python loops; integer corners only."""
    x = np.asarray(x)
    N, C, H, W = x.shape
    B = boxes.shape[1]
    a, b, c, d = box_edges(boxes)
    out = np.zeros((N, C * B, H, W), dtype=np.int64 if _is_int(x) else np.float64)
    for n in range(N):
        for ci in range(C):
            for bi in range(B):
                xl, xh = a[ci, bi], b[ci, bi] - 1.0
                yl, yh = c[ci, bi], d[ci, bi] - 1.0
                if any(v != int(v) for v in (xl, xh, yl, yh)):
                    raise ValueError("Eq. 1 needs integer corners")
                xl, xh, yl, yh = int(xl), int(xh), int(yl), int(yh)
                for yy in range(H):
                    for xx in range(W):
                        s = 0
                        for i in range(yy + yl, yy + yh + 1):
                            for j in range(xx + xl, xx + xh + 1):
                                if 0 <= i < H and 0 <= j < W:
                                    s += x[n, ci, i, j]
                        out[n, ci * B + bi, yy, xx] = s
    return out


def naive_box_forward_overlap(x, boxes):
    """Per-pixel loop of the area integral with sub-pixel corners: every input
    pixel weighted by the area of its cell inside the box.  Tiny inputs only."""
    x = np.asarray(x, dtype=np.float64)
    N, C, H, W = x.shape
    B = boxes.shape[1]
    a, b, c, d = box_edges(boxes)
    out = np.zeros((N, C * B, H, W))
    for n in range(N):
        for ci in range(C):
            for bi in range(B):
                for yy in range(H):
                    for xx in range(W):
                        s = 0.0
                        for i in range(H):
                            oy = min(i + 1, yy + d[ci, bi]) - max(i, yy + c[ci, bi])
                            if oy <= 0:
                                continue
                            for j in range(W):
                                ox = min(j + 1, xx + b[ci, bi]) - max(j, xx + a[ci, bi])
                                if ox > 0:
                                    s += x[n, ci, i, j] * ox * oy
                        out[n, ci * B + bi, yy, xx] = s
    return out


# ---------------------------------------------------------------------------
# 1x1 mix (Section 1 and Section 3.2: depthwise box filters followed by a
# 1x1 convolution), reading R8 for bf16
# ---------------------------------------------------------------------------
def bf16_round(v):
    """Round fp32 values to bf16 (round to nearest, ties to even); returned as
    fp64 holding the bf16 value.  fp64 input is first rounded to fp32, the
    precision in which the layer's values exist before the mix reads them."""
    f = np.ascontiguousarray(np.asarray(v, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    r = r.astype(np.uint32)
    nan = np.isnan(f)
    out = r.view(np.float32).astype(np.float64)
    out[nan] = np.nan
    return out


def _operand(v, compute):
    if compute == "bf16":
        return bf16_round(v)
    if compute in ("f32", "i32"):
        a = np.asarray(v)
        return a.astype(np.int64) if _is_int(a) else a.astype(np.float64)
    raise ValueError(compute)


def relu(z):
    return np.maximum(z, 0)


def mix_forward(w, o, compute="f32", apply_relu=False):
    """Z[n] = w @ O[n] over the channel axis; w [M, K], O [N, K, H, W].

    compute: 'f32' (operands as given), 'bf16' (operands rounded to bf16) or
    'i32' (integer operands, exact int64).
    """
    wv = _operand(w, compute)
    ov = _operand(o, compute)
    N, K, H, W = ov.shape
    z = np.einsum("mk,nkp->nmp", wv, ov.reshape(N, K, H * W), optimize=True)
    z = z.reshape(N, wv.shape[0], H, W)
    return relu(z) if apply_relu else z


def mix_backward_data(w, grad_z, compute="f32", relu_out=None):
    """dO[n] = w^T @ dZ[n]; with relu_out given, dZ is first masked by
    relu_out > 0 (the derivative of max(z, 0), applied before rounding)."""
    g = np.asarray(grad_z, dtype=np.float64) if not _is_int(grad_z) else np.asarray(grad_z)
    if relu_out is not None:
        g = np.where(np.asarray(relu_out) > 0, g, 0.0)
    wv = _operand(w, compute)
    gv = _operand(g.astype(np.float32) if compute == "bf16" else g, compute)
    N, M, H, W = gv.shape
    d = np.einsum("mk,nmp->nkp", wv, gv.reshape(N, M, H * W), optimize=True)
    return d.reshape(N, wv.shape[1], H, W)


def mix_backward_weight(grad_z, o, compute="f32", relu_out=None):
    """dW = sum_n dZ[n] @ O[n]^T, [M, K]."""
    g = np.asarray(grad_z, dtype=np.float64)
    if relu_out is not None:
        g = np.where(np.asarray(relu_out) > 0, g, 0.0)
    gv = _operand(g.astype(np.float32) if compute == "bf16" else g, compute)
    ov = _operand(o, compute)
    N, M, H, W = gv.shape
    K = ov.shape[1]
    return np.einsum("nmp,nkp->mk", gv.reshape(N, M, H * W),
                     ov.reshape(N, K, H * W), optimize=True)


# ---------------------------------------------------------------------------
# Whole layer and a stack of layers: box filter -> 1x1 mix (-> ReLU)
# ---------------------------------------------------------------------------
def layer_forward(x, boxes, w, compute="f32", apply_relu=False):
    """One layer: returns (O, Z) with O the filtered maps and Z the mix output."""
    o = box_forward(x, boxes)
    z = mix_forward(w, o, compute=compute, apply_relu=apply_relu)
    return o, z


def stack_forward(x, layers, compute="f32", apply_relu=True):
    """layers: list of (boxes, w).  Returns the list of per-layer inputs, filtered
    maps and outputs, [(x_l, O_l, Z_l)]."""
    cache = []
    cur = np.asarray(x, dtype=np.float64)
    for boxes, w in layers:
        o, z = layer_forward(cur, boxes, w, compute=compute, apply_relu=apply_relu)
        cache.append((cur, o, z))
        cur = z
    return cache


def stack_backward(cache, layers, grad_out, compute="f32", apply_relu=True):
    """Backward through stack_forward's layers for L = <grad_out, Z_last>.

    Returns (dx, [(dboxes_l, dw_l)]) with dx the gradient to the stack's input.
    """
    g = np.asarray(grad_out, dtype=np.float64)
    grads = [None] * len(layers)
    for li in range(len(layers) - 1, -1, -1):
        boxes, w = layers[li]
        xin, o, z = cache[li]
        ro = z if apply_relu else None
        dw = mix_backward_weight(g, o, compute=compute, relu_out=ro)
        do = mix_backward_data(w, g, compute=compute, relu_out=ro)
        H, W = xin.shape[-2:]
        dboxes = box_backward_params(xin, do, boxes)
        g = box_backward_input(do, boxes, H, W)
        grads[li] = (dboxes, dw)
    return g, grads


# ---------------------------------------------------------------------------
# Comparison metric used by the parity tests
# ---------------------------------------------------------------------------
def rel_errors(got, ref):
    """(max_i |g-r| / (|r_i| + rms(r)), ||g-r|| / ||r||) in fp64."""
    g = np.asarray(got, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    if r.size == 0:
        return 0.0, 0.0
    rms = float(np.sqrt(np.mean(r * r)))
    den = np.abs(r) + rms
    den = np.where(den == 0, 1.0, den)
    pointwise = float(np.max(np.abs(g - r) / den))
    nr = float(np.linalg.norm(r))
    normwise = float(np.linalg.norm(g - r) / nr) if nr > 0 else float(np.linalg.norm(g - r))
    return pointwise, normwise


def tolerance_ok(got, ref, rtol):
    """|g - r| <= rtol * (|r| + rms(r)) elementwise (a per-tensor scale keeps the
    test meaningful where box sums are near zero)."""
    return rel_errors(got, ref)[0] <= rtol
