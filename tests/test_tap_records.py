"""CPU pins of the test-side record reader (tests/tap_records.py).

The GPU test of the per-box precomputation compares the records the library
writes with tap_records.box_records / adjoint_records bit for bit and
evaluates them on exact tables.  These tests pin that reader to the oracle's
plain definitions: evaluated on the exact table, the expected records give
the forward box sums, the input gradient and the box-parameter gradient, also
for boxes whose edges lie on pixel boundaries (where the one-sided derivative
of the adjoint split matters).  A planted floor split of the adjoint edges is
caught.
"""
import numpy as np

import oracle as O
import tap_records as TR


def _real_boxes(rng, C, B, cmax, rmin, rmax):
    bx = np.empty((C, B, 4), dtype=np.float32)
    bx[..., :2] = rng.uniform(-cmax, cmax, size=(C, B, 2))
    bx[..., 2:] = rng.uniform(rmin, rmax, size=(C, B, 2))
    return bx


def _edge_boxes(rng):
    """Random boxes plus boxes with every edge on a pixel boundary, hanging
    over the border, or both."""
    bx = _real_boxes(rng, 2, 4, cmax=5.0, rmin=0.2, rmax=6.0)
    bx[0, 0] = [0.5, -1.0, 1.0, 1.5]
    bx[0, 1] = [-2.5, 2.0, 2.0, 0.5]
    bx[1, 0] = [3.0, 0.5, 1.5, 3.0]
    bx[1, 1] = [0.0, 0.0, 0.5, 0.5]      # identity
    return bx


def test_forward_records_on_exact_table_give_box_forward():
    rng = np.random.default_rng(20)
    x = rng.standard_normal((2, 2, 9, 8))
    bx = _edge_boxes(rng)
    got = TR.eval_forward(TR.box_records(bx), x)
    want = O.box_forward(x, bx)
    # the tap weights are fp32 (reading R5): ~1e-7 relative per weight
    assert np.max(np.abs(got - want)) <= 2e-6 * (1 + np.max(np.abs(want)))


def test_adjoint_records_match_mirror_off_integer_edges():
    """Away from integer edges the adjoint split is the floor split of the
    mirrored box; on an integer edge the floor is one lower and the weights
    put all of the edge on the upper tap."""
    rng = np.random.default_rng(21)
    bx = _real_boxes(rng, 3, 5, cmax=6.0, rmin=0.3, rmax=7.0)
    fa, wxa, wya = TR.adjoint_records(bx)
    fm, wxm, wym = TR.box_records(O.mirrored_boxes(bx))
    np.testing.assert_array_equal(fa, fm)
    np.testing.assert_array_equal(wxa, wxm)
    np.testing.assert_array_equal(wya, wym)
    bi = np.array([[[1.5, -2.0, 1.0, 2.5]]], dtype=np.float32)   # all four edges integer
    fa, wxa, wya = TR.adjoint_records(bi)
    fm, _, _ = TR.box_records(O.mirrored_boxes(bi))
    np.testing.assert_array_equal(fa, fm - 1)
    np.testing.assert_array_equal(wxa[0, 0], np.array([0, -1, 0, 1], np.float32))
    np.testing.assert_array_equal(wya[0, 0], np.array([0, -1, 0, 1], np.float32))


def _check_adjoint(adj_records):
    rng = np.random.default_rng(22)
    N, C, H, W = 2, 2, 7, 6
    bx = _edge_boxes(rng)
    x = rng.standard_normal((N, C, H, W))
    g = rng.standard_normal((N, C * bx.shape[1], H, W))
    dI, dth = TR.eval_adjoint(adj_records(bx), x, g)
    want_dI = O.box_backward_input(g, bx, H, W)
    want_dth = O.box_backward_params(x, g, bx)
    assert np.max(np.abs(dI - want_dI)) <= 2e-6 * (1 + np.max(np.abs(want_dI)))
    assert np.all(np.abs(dth - want_dth) <= 2e-6 * (1.0 + np.abs(want_dth))), (dth, want_dth)


def test_adjoint_records_on_exact_table_give_both_gradients():
    """Through <g, box(x)> = <x, adjoint box(g)>, the adjoint records on g's
    exact table give the input gradient and the box-parameter gradient,
    boxes with integer edges included."""
    _check_adjoint(TR.adjoint_records)


def test_floor_split_of_adjoint_edges_is_caught():
    """Planted mistake: splitting the mirrored edges at the floor gives the
    left derivative at integer edges, which the gradient pin rejects."""
    try:
        _check_adjoint(lambda b: TR.box_records(O.mirrored_boxes(b)))
    except AssertionError:
        return
    raise AssertionError("the floor split of the adjoint edges was not caught")


def test_decode_round_trip():
    rng = np.random.default_rng(23)
    C, B = 3, 2
    bx = _real_boxes(rng, C, B, 4.0, 0.5, 5.0)
    recs = [TR.box_records(bx), TR.adjoint_records(bx)]
    t = np.zeros((2, C, B, 16), dtype=np.int32)
    for h, (fl, wx, wy) in enumerate(recs):
        t[h, ..., 0:4] = fl
        t[h, ..., 4:8] = wx.view(np.int32)
        t[h, ..., 8:12] = wy.view(np.int32)
    for (fl, wx, wy), (fl2, wx2, wy2) in zip(recs, TR.decode(t.reshape(-1), C, B)):
        np.testing.assert_array_equal(fl, fl2)
        np.testing.assert_array_equal(wx, wx2)
        np.testing.assert_array_equal(wy, wy2)
