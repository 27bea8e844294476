"""Reference values with rigorous deviation bounds for layers whose 1x1 mix
rounds its operands to bf16.

Rounding a value to bf16 is a discrete decision.  The GPU takes it on its own
fp32 result, the oracle on the fp64 result; when the two straddle a rounding
boundary both codes are correct, and with few mix inputs one such flip moves
an output by far more than accumulation noise.  Likewise a ReLU mask decision
is ambiguous where the pre-activation is within its error bound of zero.

For one layer fed exact inputs these helpers compute, next to each oracle
value, an elementwise bound E on how far any correct implementation may
deviate because of such ambiguous decisions, propagated with the absolute
values of the (linear) operators.  Parity then requires
|gpu - ref| <= E + rtol*(|ref| + rms).  E is derived from the oracle's values
and the fp32 accuracy bound of the box filter; nothing in it comes from the
GPU.  Through several layers the worst-case propagation of such bounds is too
loose to be useful (it treats rounding noise as coherent); the stacked-layer
test uses a normwise bar there instead.
"""
import numpy as np

import oracle as O

# Bound on the box filter's fp32 error relative to |r| + rms(r).  The GPU's
# measured pointwise error is ~1.2e-7 (parity tests of the box filter), so this
# leaves a 30x margin.
E_F32 = 4e-6


def scale_err(r, rel):
    r = np.asarray(r, dtype=np.float64)
    rms = float(np.sqrt(np.mean(r * r))) if r.size else 0.0
    return rel * (np.abs(r) + rms)


def bf16_band(r, e):
    """Largest |bf16(v) - bf16(r)| over all v with |v - r| <= e (bf16
    rounding is monotone, so the extremes are at r - e and r + e)."""
    b = O.bf16_round(r)
    return np.maximum(np.abs(O.bf16_round(r + e) - b), np.abs(O.bf16_round(r - e) - b))


def _mm_abs_w(w_b, v):
    """|W| applied over the channel axis: [M, K] x [N, K, H, W] -> [N, M, H, W]."""
    return np.einsum("mk,nkhw->nmhw", np.abs(w_b), v, optimize=True)


def layer_forward(x, boxes, w, relu):
    """One layer on the exact oracle input.  The only discrete decisions are
    the bf16 codes of O: D bounds how far the GPU's code may be from the
    oracle's given the fp32 accuracy of the box filter, and E_z = |W| D bounds
    the resulting deviation of the mix output."""
    o = O.box_forward(x, boxes)
    D = bf16_band(o, scale_err(o, E_F32))
    zpre = O.mix_forward(w, o, compute="bf16")
    ez = _mm_abs_w(O.bf16_round(w), D)
    z = np.maximum(zpre, 0.0) if relu else zpre
    return {"x": x, "o": o, "D": D, "zpre": zpre, "ez": ez, "z": z}


def layer_backward(fw, boxes, w, g, relu=False, eg_in=None, mask_exact=False):
    """Backward of that layer for an upstream gradient g.  The reference
    values come from the oracle (mix_backward_weight / mix_backward_data on
    the masked gradient, box_backward_input / box_backward_params); this
    function adds only their deviation bounds.

    Ambiguous decisions: the bf16 codes of O (they enter dW only:
    sum_p |bf16(g)| * D); with ReLU, the mask where |zpre| is within its bound
    ez of zero (there the masked gradient may be g or 0); and the bf16 codes
    of the masked gradient itself where g carries an uncertainty eg_in (an
    incoming gradient the GPU computed in fp32 from ambiguous operands; None:
    g is exact, fp32 values whose codes agree on both sides).  mask_exact: the
    ReLU mask is taken from an exact input (the layer above's input, which is
    this layer's rectified output fed from the oracle), so it is unambiguous.
    The uncertainty of the masked gradient is propagated through the
    transposed mix and box operators with absolute values."""
    H, W = fw["o"].shape[-2:]
    eg = np.zeros_like(g) if eg_in is None else np.asarray(eg_in, dtype=np.float64)
    if relu:
        on = fw["zpre"] > 0
        gm = np.where(on, g, 0.0)
        if mask_exact:
            eg = np.where(on, eg, 0.0)
        else:
            amb = np.abs(fw["zpre"]) <= fw["ez"]
            # either choice of the mask is valid there
            eg = np.where(amb, np.abs(g) + eg, np.where(on, eg, 0.0))
    else:
        gm = g
    gb = O.bf16_round(gm)
    Dg = bf16_band(gm, eg)
    ob = O.bf16_round(fw["o"])
    wb = O.bf16_round(w)
    N, M = gb.shape[:2]
    K = ob.shape[1]
    dw = O.mix_backward_weight(gm, fw["o"], compute="bf16")
    do = O.mix_backward_data(w, gm, compute="bf16")
    g2, o2, D2, Dg2 = (a.reshape(a.shape[0], a.shape[1], -1) for a in (gb, ob, fw["D"], Dg))
    edw = (np.einsum("nmp,nkp->mk", np.abs(g2) + Dg2, D2, optimize=True)
           + np.einsum("nmp,nkp->mk", Dg2, np.abs(o2), optimize=True))
    edo = np.einsum("mk,nmp->nkp", np.abs(wb), Dg2, optimize=True).reshape(N, K, H, W)
    dx = O.box_backward_input(do, boxes, H, W)
    edx = O.box_backward_input(edo, boxes, H, W)          # box weights are >= 0
    dth = O.box_backward_params(fw["x"], do, boxes)
    e = np.abs(O.box_param_grad_from_edges(np.abs(fw["x"]), edo, boxes))
    ea, eb, ec, ed = (e[..., k] for k in range(4))
    edth = np.stack([ea + eb, ec + ed, ea + eb, ec + ed], axis=-1)
    return {"dw": dw, "edw": edw, "do": do, "edo": edo, "dx": dx, "edx": edx, "dth": dth, "edth": edth,
            "gm": gm, "eg": eg}


def bounded_error(got, ref, bound):
    """max over elements of max(0, |g - r| - bound) / (|r| + rms(r)), the
    plain pointwise error without the bound, and the largest relative bound."""
    g = np.asarray(got, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(r * r)))
    den = np.abs(r) + rms
    den = np.where(den == 0, 1.0, den)
    excess = np.maximum(0.0, np.abs(g - r) - bound) / den
    plain = np.abs(g - r) / den
    return float(excess.max()), float(plain.max()), float((bound / den).max())
