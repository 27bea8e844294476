"""Test-side reader of the box records the library's box_prep writes.

This is not part of the oracle: it encodes the record layout of the GPU path
(one 16-word record per box: floors of the four edges, then the x weights,
then the y weights) so that the tests can (1) check the integer decisions in
those records bit for bit and (2) evaluate the records the GPU wrote on exact
(fp64 / int64) summed-area tables and compare the result with the oracle's
plain definitions (box_forward, box_backward_input, box_backward_params).

The precomputation itself follows Section 3.1 (text after Eq. 4): integer
shifts leave the corner fractions unchanged, so a box reduces to the floors
of its edges and the bilinear weights of the two table columns (rows) around
each edge; the 16 tap weights are products of an x weight and a y weight.
"""
import numpy as np

import oracle as O


def _weights(e, fl):
    """Weights of the taps (fl, fl + 1) around each edge e = fl + f: the
    leading edge of an axis enters with a minus sign (Eq. 2).  Formed in fp64
    from the exact fraction and rounded once to fp32."""
    fr = e - fl
    w = np.stack([fr - 1.0, -fr, 1.0 - fr, fr], axis=-1)        # [..., edge, 4]
    wx = np.concatenate([w[..., 0, :2], w[..., 1, 2:]], axis=-1).astype(np.float32)
    wy = np.concatenate([w[..., 2, :2], w[..., 3, 2:]], axis=-1).astype(np.float32)
    return wx, wy


def box_records(boxes):
    """Expected forward records: (floors int64 [..., 4] of a, b, c, d; wx fp32
    [..., 4] for columns floor(a), floor(a)+1, floor(b), floor(b)+1; wy fp32
    [..., 4] likewise for rows)."""
    a, b, c, d = O.box_edges(boxes)
    e = np.stack([a, b, c, d], axis=-1)
    fl = np.floor(e)
    wx, wy = _weights(e, fl)
    return fl.astype(np.int64), wx, wy


def adjoint_records(boxes):
    """Expected records of the mirrored (adjoint) box as the backward uses
    them: each mirrored edge e is split as e = f + alpha with alpha in (0, 1]
    (f = ceil(e) - 1).  Interpolation is continuous, so the lookups equal the
    floor split's; at an integer edge the two taps straddle the column (row)
    just below the edge, where the right derivative of the original box's
    edge is read (moving an original edge up moves its mirror image down)."""
    a, b, c, d = O.box_edges(O.mirrored_boxes(boxes))
    e = np.stack([a, b, c, d], axis=-1)
    fl = np.ceil(e) - 1.0
    wx, wy = _weights(e, fl)
    return fl.astype(np.int64), wx, wy


def decode(table, C, B):
    """Splits box_prep's int32 table (2*C*B records of 16 words) into the
    forward and the adjoint records: two (floors, wx, wy) triples."""
    t = np.asarray(table).reshape(2, C, B, 16)
    out = []
    for half in range(2):
        r = t[half]
        assert np.all(r[..., 12:16] == 0), "reserved record words must be zero"
        out.append((r[..., 0:4].astype(np.int64), r[..., 4:8].view(np.float32).copy(),
                    r[..., 8:12].view(np.float32).copy()))
    return out


def _taps(fl):
    fa, fb, fc, fd = (int(v) for v in fl)
    return [fa, fa + 1, fb, fb + 1], [fc, fc + 1, fd, fd + 1]


def eval_forward(records, x):
    """Eq. 2-3 with the given records: O[n, c*B+b, y, x] = sum over the 16
    taps of wy[r] * wx[k] * S(clamp(y + oy[r]), clamp(x + ox[k])) on the exact
    exclusive table of each map (clamping is zero padding).  fp64."""
    fl, wx, wy = records
    x = np.asarray(x, dtype=np.float64)
    N, C, H, W = x.shape
    B = fl.shape[1]
    S = O.sat_exclusive(x)
    ys, xs = np.arange(H), np.arange(W)
    out = np.zeros((N, C, B, H, W))
    for c in range(C):
        for b in range(B):
            ox, oy = _taps(fl[c, b])
            for r in range(4):
                u = np.clip(ys + oy[r], 0, H)
                for k in range(4):
                    v = np.clip(xs + ox[k], 0, W)
                    out[:, c, b] += float(wy[c, b, r]) * float(wx[c, b, k]) * S[:, c][:, u][:, :, v]
    return out.reshape(N, C * B, H, W)


def eval_adjoint(records, x, g):
    """The backward read from adjoint records on the exact table of each
    upstream-gradient map g[n, c*B+b]:
      input gradient  dI[n, c] = sum_b adjoint box sum of g (Eq. 2-3 on g's
                                 table with the adjoint taps);
      edge gradients  through <g, box(x)> = <x, adjoint box sum of g>: each
                      edge derivative of the adjoint sum is the difference of
                      the two taps around the mirrored edge, weighted by x.
    Returns (dI fp64 [N, C, H, W], dtheta fp64 [C, B, 4] in (cx, cy, rx, ry))."""
    fl, wx, wy = records
    x = np.asarray(x, dtype=np.float64)
    N, C, H, W = x.shape
    B = fl.shape[1]
    g = np.asarray(g, dtype=np.float64).reshape(N, C, B, H, W)
    ys, xs = np.arange(H), np.arange(W)
    dI = np.zeros((N, C, H, W))
    dth = np.zeros((C, B, 4))
    for c in range(C):
        for b in range(B):
            S = O.sat_exclusive(g[:, c, b])                       # [N, H+1, W+1]
            ox, oy = _taps(fl[c, b])
            T = [[S[:, np.clip(ys + oy[r], 0, H)][:, :, np.clip(xs + ox[k], 0, W)] for k in range(4)]
                 for r in range(4)]
            wxb, wyb = wx[c, b].astype(np.float64), wy[c, b].astype(np.float64)
            U = [sum(wxb[k] * T[r][k] for k in range(4)) for r in range(4)]
            dI[:, c] += sum(wyb[r] * U[r] for r in range(4))
            colA = sum(wyb[r] * (T[r][1] - T[r][0]) for r in range(4))
            colB = sum(wyb[r] * (T[r][3] - T[r][2]) for r in range(4))
            v = x[:, c]
            ga = -np.sum(v * colB)            # a = 1 - b'
            gb = np.sum(v * colA)             # b = 1 - a'
            gc = -np.sum(v * (U[3] - U[2]))   # c = 1 - d'
            gd = np.sum(v * (U[1] - U[0]))    # d = 1 - c'
            dth[c, b] = [ga + gb, gc + gd, gb - ga, gd - gc]
    return dI, dth
