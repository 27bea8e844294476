"""Non-finite inputs (NaN, +Inf, -Inf) through the box filter, on every path.

The library does not look for non-finite values.  Every path reads a map
through its exclusive integral image (a stored table, or running column sums
that hold the same entries), and a NaN or infinity at pixel (i, j) makes
every table entry below and to the right of it non-finite.  So for a map
holding one such value:
  * every output whose box covers (i, j) with positive weight is non-finite;
  * every output whose box ends above row i or left of column j (its last
    sampled table row <= i, or its last sampled column <= j) is finite and
    exact;
  * outputs in between (boxes below and right of the pixel without covering
    it) may be either: the table differences do not cancel a non-finite entry;
  * every other map of the call is untouched.
With BC_FLAG_MEAN_OFFSET the map's mean is itself non-finite and every
output of that map is non-finite.  The backward follows from the same
reading of its adjoint (mirrored) boxes; the edge gradients of a box are
finite and exact when neither its input map nor its output-gradient map
holds a non-finite value.
The expected values of the finite outputs come from the oracle on the same
inputs with the planted values replaced by zero (those outputs do not read
them).
"""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from paper_1906_11367_amd import boxconv as bc

pytestmark = pytest.mark.gpu

RTOL_F32 = 1e-4
MARGIN = 1e-3   # keeps the "clean" test away from exact integer box edges


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _inputs(N, C, H, W, B, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    bx = np.empty((C, B, 4), dtype=np.float32)
    bx[..., :2] = rng.uniform(-H / 4, H / 4, size=(C, B, 2))
    bx[..., 2:] = rng.uniform(0.5, H / 6, size=(C, B, 2))
    g = rng.standard_normal((N, C * B, H, W)).astype(np.float32)
    return x, bx, g


def _plants(H, W, maps):
    """(n, map, i, j, value) for a NaN, a +Inf and a -Inf in three maps."""
    pix = [(H // 5, W // 7), (H - 3, W - 4), (H // 2, 1)]
    vals = [np.nan, np.inf, -np.inf]
    return [(n, m, i, j, v) for (n, m), (i, j), v in zip(maps, pix, vals)]


def _plant(a, plants):
    bad, clean = a.copy(), a.copy()
    for n, m, i, j, v in plants:
        bad[n, m, i, j] = v
        clean[n, m, i, j] = 0.0
    return bad, clean


def _regions(box, H, W, i, j):
    """(covers, clean) masks over the H x W outputs of one box and one bad
    pixel (i, j): the box covers it with positive weight / the box's sampled
    table rows all lie at or above row i, or its columns at or left of j."""
    a, b, c, d = (float(e) for e in O.box_edges(np.asarray(box, dtype=np.float32)))
    wy = O.overlap_matrix(H, c, d)[:, i]
    wx = O.overlap_matrix(W, a, b)[:, j]
    covers = (wy > MARGIN)[:, None] & (wx > MARGIN)[None, :]
    ys, xs = np.arange(H, dtype=np.float64), np.arange(W, dtype=np.float64)
    clean = (ys + d < i - MARGIN)[:, None] | (xs + b < j - MARGIN)[None, :]
    return covers, clean


def _check_map(got, want, covers, clean, what, seen):
    """seen: running counts of the outputs checked in each region."""
    assert not np.isfinite(got[covers]).any(), f"{what}: an output covering the bad pixel is finite"
    assert np.isfinite(got[clean]).all(), f"{what}: an output away from the bad pixel is not finite"
    if clean.any():
        pw, _ = O.rel_errors(got[clean], want[clean])
        assert pw <= RTOL_F32, f"{what}: clean outputs pointwise {pw}"
    seen[0] += int(covers.sum())
    seen[1] += int(clean.sum())


def _enough(seen, what):
    say(f"  {what}: {seen[0]} covering outputs non-finite, {seen[1]} clean outputs exact")
    assert seen[0] > 0 and seen[1] > 0, "the case should reach both regions"


def _check_rest(got, want, touched, what):
    keep = np.ones(got.shape[:2], dtype=bool)
    for t in touched:
        keep[t] = False
    assert np.isfinite(got[keep]).all(), f"{what}: a map without planted values is not finite"
    pw, _ = O.rel_errors(got[keep], want[keep])
    say(f"  {what}: untouched maps pointwise {pw:.3e}")
    assert pw <= RTOL_F32


SHAPES = [
    ((2, 3, 40, 36, 4), 0),                        # table in LDS
    ((2, 3, 40, 36, 4), bc.BC_FLAG_FORCE_HBM),     # table in HBM
    ((1, 3, 200, 256, 4), bc.BC_FLAG_FORCE_HBM),   # table in HBM, several columns per lane
    ((1, 3, 200, 256, 4), 0),                      # streaming kernels, whole-wave groups
    ((1, 3, 500, 47, 3), 0),                       # streaming kernels, 16-lane groups
]


@pytest.mark.parametrize("shape,flags", SHAPES)
def test_forward_nonfinite_inputs(shape, flags):
    N, C, H, W, B = shape
    say(f"forward non-finite {shape} flags={flags}")
    x, bx, _ = _inputs(*shape, seed=71)
    plants = _plants(H, W, [(0, 1), (N - 1, 2), (0, 0)])
    xb, xc = _plant(x, plants)
    y = torch.empty((N, C * B, H, W), dtype=torch.float32, device="cuda")
    bc.box_conv_fwd(dev(xb), dev(bx), y, flags)
    got = y.cpu().numpy()
    want = O.box_forward(xc, bx)
    touched, seen = [], [0, 0]
    for n, c, i, j, _ in plants:
        for b in range(B):
            covers, clean = _regions(bx[c, b], H, W, i, j)
            _check_map(got[n, c * B + b], want[n, c * B + b], covers, clean, f"y[{n},{c * B + b}]", seen)
            touched.append((n, c * B + b))
    _enough(seen, "y")
    _check_rest(got, want, touched, "y")


@pytest.mark.parametrize("shape,flags", SHAPES)
def test_backward_nonfinite_gradient(shape, flags):
    N, C, H, W, B = shape
    say(f"backward non-finite grad_y {shape} flags={flags}")
    x, bx, g = _inputs(*shape, seed=72)
    # one planted value in a gradient map of each channel
    plants = _plants(H, W, [(0, 1), (N - 1, B + 2 % B), (0, 2 * B + 3 % B)])
    gb_, gc = _plant(g, plants)
    gx = torch.empty((N, C, H, W), dtype=torch.float32, device="cuda")
    gbox = torch.empty((C, B, 4), dtype=torch.float32, device="cuda")
    bc.box_conv_bwd(dev(x), dev(bx), dev(gb_), gx, gbox, flags)
    got_x, got_b = gx.cpu().numpy(), gbox.cpu().numpy()
    want_x = O.box_backward_input(gc, bx, H, W)
    want_b = O.box_backward_params(x, gc, bx)
    mirrored = O.mirrored_boxes(bx)
    touched_x, bad_boxes, seen = [], set(), [0, 0]
    for n, k, i, j, _ in plants:
        c, b = divmod(k, B)
        covers, clean = _regions(mirrored[c, b], H, W, i, j)
        _check_map(got_x[n, c], want_x[n, c], covers, clean, f"dx[{n},{c}]", seen)
        touched_x.append((n, c))
        bad_boxes.add((c, b))
    _enough(seen, "dx")
    _check_rest(got_x, want_x, touched_x, "dx")
    for c in range(C):
        for b in range(B):
            if (c, b) in bad_boxes:
                assert not np.isfinite(got_b[c, b]).all(), f"dboxes[{c},{b}] should not be finite"
            else:
                assert np.isfinite(got_b[c, b]).all()
                pw, _ = O.rel_errors(got_b[c, b], want_b[c, b])
                assert pw <= RTOL_F32, f"dboxes[{c},{b}] pointwise {pw}"


@pytest.mark.parametrize("shape,flags", SHAPES)
def test_backward_nonfinite_input(shape, flags):
    """dx does not read x; a non-finite map poisons the edge gradients of its
    own channel's boxes only."""
    N, C, H, W, B = shape
    say(f"backward non-finite x {shape} flags={flags}")
    x, bx, g = _inputs(*shape, seed=73)
    plants = _plants(H, W, [(0, 1)])
    xb, xc = _plant(x, plants)
    gx = torch.empty((N, C, H, W), dtype=torch.float32, device="cuda")
    gbox = torch.empty((C, B, 4), dtype=torch.float32, device="cuda")
    bc.box_conv_bwd(dev(xb), dev(bx), dev(g), gx, gbox, flags)
    got_x, got_b = gx.cpu().numpy(), gbox.cpu().numpy()
    pw, _ = O.rel_errors(got_x, O.box_backward_input(g, bx, H, W))
    assert np.isfinite(got_x).all() and pw <= RTOL_F32
    want_b = O.box_backward_params(xc, g, bx)
    assert not np.isfinite(got_b[1]).all(axis=-1).any(), "every box of the channel sees the bad pixel"
    for c in (0, 2):
        assert np.isfinite(got_b[c]).all()
        pw, _ = O.rel_errors(got_b[c], want_b[c])
        assert pw <= RTOL_F32


@pytest.mark.parametrize("shape", [(2, 3, 40, 36, 4), (1, 3, 200, 256, 4)])
def test_mean_offset_spreads_nonfinite_over_the_map(shape):
    N, C, H, W, B = shape
    say(f"forward non-finite mean offset {shape}")
    x, bx, _ = _inputs(*shape, seed=74)
    plants = _plants(H, W, [(0, 1)])
    xb, xc = _plant(x, plants)
    y = torch.empty((N, C * B, H, W), dtype=torch.float32, device="cuda")
    bc.box_conv_fwd(dev(xb), dev(bx), y, bc.BC_FLAG_MEAN_OFFSET)
    got = y.cpu().numpy()
    assert not np.isfinite(got[0, B:2 * B]).any()
    _check_rest(got, O.box_forward(xc, bx), [(0, k) for k in range(B, 2 * B)], "y")
