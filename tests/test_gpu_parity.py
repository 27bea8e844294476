"""GPU parity: the HIP library (through the C ABI) against the CPU oracle.

Inputs come from the seeded workload generators; the oracle computes in fp64
(int64 for integer data).  Bars: bit-exact for integer data and for the
per-box integer decisions; for fp32 results |g - r| <= rtol * (|r| + rms(r))
elementwise with rtol = 1e-4; for the bf16 mix output rtol = 1e-3 against an
oracle that rounds the same operands to bf16.
"""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from paper_1906_11367_amd import boxconv as bc
from paper_1906_11367_amd import workloads as wlmod
from paper_1906_11367_amd.layer import LayerPlan, Stack

import bf16_bounds as bb  # noqa: E402
import tap_records as TR  # noqa: E402

pytestmark = pytest.mark.gpu

RTOL_F32 = 1e-4
RTOL_BF16_MIX = 1e-3


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy()


def check(got, ref, rtol, what):
    pw, nw = O.rel_errors(got, ref)
    say(f"  {what}: pointwise {pw:.3e}  normwise {nw:.3e}  (rtol {rtol})")
    assert pw <= rtol, f"{what}: pointwise rel error {pw} > {rtol}"


def real_boxes(rng, C, B, cmax, rmin, rmax):
    bx = np.empty((C, B, 4), dtype=np.float32)
    bx[..., :2] = rng.uniform(-cmax, cmax, size=(C, B, 2))
    bx[..., 2:] = rng.uniform(rmin, rmax, size=(C, B, 2))
    return bx


# ---------------------------------------------------------------------------
# a1: per-box precomputation (integer decisions are bit-exact)
# ---------------------------------------------------------------------------
def test_box_prep_bit_exact():
    """The records box_prep writes: their integer decisions (edge floors,
    floor split forward, ceil - 1 split adjoint) and fp32 weights bit for bit
    against the record layout (tests/tap_records.py); then the GPU's own
    records, evaluated on exact tables, against the oracle's forward, input
    gradient and box-parameter gradient."""
    rng = np.random.default_rng(100)
    C, B = 7, 5
    bx = real_boxes(rng, C, B, 40.0, 0.0, 60.0)
    bx[0, 0] = [0.0, 0.0, 0.5, 0.5]          # identity: integer edges
    bx[1, 1] = [0.25, -0.25, 1.75, 0.75]      # edges on quarter pixels
    bx[2, 2] = [3.0, -2.5, 2.5, 4.0]          # integer corners
    bx[3, 3] = [0.5, -1.0, 1.0, 1.5]          # integer edges, one-sided derivatives
    table = torch.zeros(2 * C * B * 16, dtype=torch.int32, device="cuda")
    bc.box_prep(dev(bx), table)
    torch.cuda.synchronize()
    fwd, adj = TR.decode(table.cpu().numpy(), C, B)
    for got, want in [(fwd, TR.box_records(bx)), (adj, TR.adjoint_records(bx))]:
        for g, w in zip(got, want):
            np.testing.assert_array_equal(g, w)
    # the GPU's records on exact tables (maps large enough for every tap to
    # land inside or at the clamped border for the smaller boxes)
    H, W = 23, 19
    bs = bx.copy()
    bs[..., :2] = np.clip(bs[..., :2], -8, 8)
    bs[..., 2:] = np.clip(bs[..., 2:], 0.0, 9)
    bs[3, 3] = [0.5, -1.0, 1.0, 1.5]
    table.zero_()
    bc.box_prep(dev(bs), table)
    torch.cuda.synchronize()
    fwd, adj = TR.decode(table.cpu().numpy(), C, B)
    x = rng.standard_normal((1, C, H, W))
    g = rng.standard_normal((1, C * B, H, W))
    check(TR.eval_forward(fwd, x), O.box_forward(x, bs), 2e-6, "GPU forward records on exact tables")
    dI, dth = TR.eval_adjoint(adj, x, g)
    check(dI, O.box_backward_input(g, bs, H, W), 2e-6, "GPU adjoint records: input gradient")
    check(dth, O.box_backward_params(x, g, bs), 2e-6, "GPU adjoint records: box-parameter gradient")


# ---------------------------------------------------------------------------
# a2: summed-area table
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("shape", [(1, 3, 32, 32), (2, 2, 37, 29), (1, 2, 256, 256), (1, 1, 1, 1), (1, 1, 5, 1000)])
def test_sat_build_int_bit_exact(shape):
    say(f"sat int {shape}")
    rng = np.random.default_rng(101)
    x = rng.integers(-8, 9, size=shape).astype(np.int32)
    N, C, H, W = shape
    sat = torch.empty((N, C, H + 1, W + 1), dtype=torch.int32, device="cuda")
    bc.sat_build(dev(x), sat)
    np.testing.assert_array_equal(host(sat), O.sat_exclusive(x))


@pytest.mark.parametrize("shape", [(2, 3, 64, 48), (1, 2, 256, 256), (1, 1, 3, 70)])
def test_sat_build_f32(shape):
    say(f"sat f32 {shape}")
    rng = np.random.default_rng(102)
    x = (rng.standard_normal(shape) + 0.5).astype(np.float32)
    N, C, H, W = shape
    sat = torch.empty((N, C, H + 1, W + 1), dtype=torch.float32, device="cuda")
    bc.sat_build(dev(x), sat)
    ref = O.sat_exclusive(x)
    check(host(sat), ref, 1e-5, "sat")
    # with the per-map mean subtracted: table + mean * u * v reconstructs the plain table
    mean = torch.empty((N, C), dtype=torch.float32, device="cuda")
    bc.sat_build(dev(x), sat, mean)
    mu = host(mean).astype(np.float64)
    np.testing.assert_allclose(mu, O.map_mean(x), rtol=0, atol=1e-5)
    u = np.arange(H + 1)[:, None] * np.arange(W + 1)[None, :]
    recon = host(sat).astype(np.float64) + mu[..., None, None] * u
    check(recon, ref, 1e-5, "sat(x - mean) + mean*u*v")


# ---------------------------------------------------------------------------
# a3: forward box filter
# ---------------------------------------------------------------------------
def _fwd(x, bx, y_dtype=torch.float32, flags=0):
    N, C, H, W = x.shape
    B = bx.shape[1]
    y = torch.empty((N, C * B, H, W), dtype=y_dtype, device="cuda")
    bc.box_conv_fwd(dev(x), dev(bx), y, flags)
    return host(y)


@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM])
def test_fwd_tiny_integer_workload_bit_exact(flags):
    wl = wlmod.WORKLOADS[1]
    d = wlmod.make_inputs(wl)
    say(f"fwd {wl.key} flags={flags}")
    got = _fwd(d["x"], d["boxes"], torch.int32, flags)
    want = O.box_forward(d["x"], d["boxes"])
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("key,scale", [
    (2, dict(N=2, C=6)),
    (3, dict(N=2, C=8)),
    (2, dict(N=1, C=3, H=37, W=29, B=5)),   # ragged chunks and segments
    (3, dict(N=1, C=2, H=17, W=100, B=3)),
    (2, dict(N=1, C=3, H=60, W=40, B=3)),
    (2, dict(N=2, C=2, H=9, W=47, B=2)),
    (2, dict(N=1, C=2, H=120, W=48, B=1)),
    # maps whose table does not fit LDS, evaluated by the streaming kernels:
    # tall and narrow (four boxes per wave), ragged widths, full 16-byte rows
    (2, dict(N=1, C=2, H=500, W=47, B=3)),
    (4, dict(N=1, C=2, H=300, W=128, B=3)),
    (4, dict(N=1, C=1, H=200, W=200, B=5)),
    (4, dict(N=1, C=2, H=130, W=256, B=8)),
])
@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM, bc.BC_FLAG_MEAN_OFFSET])
def test_fwd_f32(key, scale, flags):
    wl = wlmod.WORKLOADS[key].scaled(**scale)
    d = wlmod.make_inputs(wl)
    say(f"fwd {wl.key} {scale} flags={flags}")
    got = _fwd(d["x"], d["boxes"], torch.float32, flags)
    check(got, O.box_forward(d["x"], d["boxes"]), RTOL_F32, "O")


@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_MEAN_OFFSET])
def test_fwd_large_maps_hbm_table(flags):
    wl = wlmod.WORKLOADS[4].scaled(N=1, C=2)
    d = wlmod.make_inputs(wl)
    say(f"fwd {wl.key} reduced flags={flags}")
    got = _fwd(d["x"], d["boxes"], torch.float32, flags)
    check(got, O.box_forward(d["x"], d["boxes"]), RTOL_F32, "O")


# the pose shape (table in LDS), and maps the streaming kernels take; each
# also with the tables in HBM
@pytest.mark.parametrize("key,scale", [(3, dict(N=1, C=4)), (4, dict(N=1, C=2, H=300, W=128, B=3)),
                                       (2, dict(N=1, C=2, H=500, W=47, B=3))])
@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM])
def test_fwd_bf16_output_is_rounded_fp32(key, scale, flags):
    wl = wlmod.WORKLOADS[key].scaled(**scale)
    d = wlmod.make_inputs(wl)
    say(f"fwd bf16 out {wl.key} {scale} flags={flags}")
    got = _fwd(d["x"], d["boxes"], torch.bfloat16, flags)
    ref = O.box_forward(d["x"], d["boxes"])
    # the kernel rounds its fp32 value; that value is within the fp32 error
    # bound of the oracle's, so its bf16 code is one of the codes reachable
    # from [r - e, r + e]
    e = bb.scale_err(ref, bb.E_F32)
    assert np.all(np.abs(got - O.bf16_round(ref)) <= bb.bf16_band(ref, e))
    assert np.mean(got == O.bf16_round(ref)) > 0.9


def test_fwd_identity_and_exact_integer_valued_floats():
    rng = np.random.default_rng(103)
    x = rng.integers(-50, 51, size=(2, 3, 19, 23)).astype(np.float32)
    bx = np.zeros((3, 2, 4), dtype=np.float32)
    bx[..., 2:] = 0.5                                   # identity box
    bx[:, 1] = [1.5, -2.5, 3.0, 2.0]                     # integer corners
    got = _fwd(x, bx)
    np.testing.assert_array_equal(got[:, 0::2], x)
    np.testing.assert_array_equal(got, O.box_forward(x, bx))


def test_fwd_degenerate_boxes():
    rng = np.random.default_rng(104)
    x = rng.standard_normal((1, 2, 9, 7)).astype(np.float32)
    bx = np.array([[[0, 0, 1000, 1000], [500, 0, 3, 3], [0, 0, 0, 0], [0.3, 0.2, 0.1, 0.05]],
                   [[-20, 30, 2, 2], [0, 0, 4.5, 0.5], [2.2, -1.1, 0.5, 6], [0, 0, 0.5, 0.5]]],
                  dtype=np.float32)
    got = _fwd(x, bx)
    ref = O.box_forward(x, bx)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-4 * (1 + np.abs(ref).max()))
    # a box covering everything gives the map total at every pixel
    np.testing.assert_allclose(got[0, 0], x[0, 0].sum(dtype=np.float64), rtol=1e-5)
    # boxes entirely outside the map and zero-size boxes give zero
    assert np.all(got[0, 1] == 0) and np.all(got[0, 2] == 0) and np.all(got[0, 4] == 0)


def test_fwd_single_pixel_maps():
    x = np.array([[[[2.5]]]], dtype=np.float32)
    bx = np.array([[[0, 0, 0.5, 0.5], [0.25, 0, 0.5, 0.5], [0, 0, 10, 10]]], dtype=np.float32)
    got = _fwd(x, bx)
    np.testing.assert_allclose(got.ravel(), [2.5, 1.875, 2.5], rtol=1e-6)


def test_fwd_deterministic():
    wl = wlmod.WORKLOADS[2].scaled(N=2, C=4)
    d = wlmod.make_inputs(wl)
    a = _fwd(d["x"], d["boxes"])
    b = _fwd(d["x"], d["boxes"])
    np.testing.assert_array_equal(a, b)


# ---------------------------------------------------------------------------
# Integer corners (the inference form): the rounded box, four samples per box
# ---------------------------------------------------------------------------
INT_CORNERS = bc.BC_FLAG_INTEGER_CORNERS


def rounding_boxes(rng, C, B):
    """Real-valued boxes, plus boxes whose edges are exact ties."""
    bx = real_boxes(rng, C, B, 20.0, 0.0, 30.0)
    bx[0, 0] = [0.0, 0.0, 1.0, 2.0]        # edges -0.5, 1.5, -1.5, 2.5
    bx[0, 1] = [-3.25, 2.0, 0.25, 0.75]    # edges -3.0, -2.5, 1.75, 3.25
    bx[1, 0] = [0.0, 0.0, 0.5, 0.5]        # identity
    bx[1, 1] = [0.1, 0.0, 0.2, 0.1]        # rounds to an empty box
    return bx


def test_box_prep_rounded_bit_exact():
    rng = np.random.default_rng(110)
    C, B = 5, 4
    bx = rounding_boxes(rng, C, B)
    table = torch.zeros(2 * C * B * 16, dtype=torch.int32, device="cuda")
    bc.box_prep(dev(bx), table, INT_CORNERS)
    torch.cuda.synchronize()
    t = table.cpu().numpy().reshape(2, C, B, 16)
    a, b, c, d = O.rounded_edges(bx)
    np.testing.assert_array_equal(t[0, ..., 0:4], np.stack([a, b, c, d], axis=-1))
    # the adjoint: the mirrored box [1-b, 1-a) x [1-d, 1-c) of the rounded box
    np.testing.assert_array_equal(t[1, ..., 0:4], np.stack([1 - b, 1 - a, 1 - d, 1 - c], axis=-1))
    w = np.broadcast_to(np.array([-1, 0, 1, 0], dtype=np.float32), (C, B, 4))
    for half in range(2):
        np.testing.assert_array_equal(t[half, ..., 4:8].view(np.float32), w)
        np.testing.assert_array_equal(t[half, ..., 8:12].view(np.float32), w)
        np.testing.assert_array_equal(t[half, ..., 12:16], 0)


@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM])
@pytest.mark.parametrize("shape", [(2, 3, 32, 32), (1, 2, 37, 29),
                                   (1, 2, 260, 200), (1, 2, 130, 256)])   # streamed int32 maps
def test_fwd_integer_corners_int_bit_exact(flags, shape):
    say(f"fwd integer corners int32 {shape} flags={flags}")
    rng = np.random.default_rng(111)
    x = rng.integers(-8, 9, size=shape).astype(np.int32)
    bx = rounding_boxes(rng, shape[1], 4)
    got = _fwd(x, bx, torch.int32, flags | INT_CORNERS)
    np.testing.assert_array_equal(got, O.box_forward(x, bx, integer_corners=True))


@pytest.mark.parametrize("key,scale", [
    (3, dict(N=2, C=8)),
    (2, dict(N=1, C=3, H=37, W=29, B=5)),   # ragged chunks and segments
    (3, dict(N=1, C=2, H=17, W=100, B=3)),
])
@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM, bc.BC_FLAG_MEAN_OFFSET])
def test_fwd_integer_corners_f32(key, scale, flags):
    wl = wlmod.WORKLOADS[key].scaled(**scale)
    d = wlmod.make_inputs(wl)
    say(f"fwd integer corners {wl.key} {scale} flags={flags}")
    got = _fwd(d["x"], d["boxes"], torch.float32, flags | INT_CORNERS)
    check(got, O.box_forward(d["x"], d["boxes"], integer_corners=True), RTOL_F32, "O")


@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_MEAN_OFFSET])
def test_fwd_integer_corners_large_maps(flags):
    wl = wlmod.WORKLOADS[4].scaled(N=1, C=2)
    d = wlmod.make_inputs(wl)
    say(f"fwd integer corners {wl.key} reduced flags={flags}")
    got = _fwd(d["x"], d["boxes"], torch.float32, flags | INT_CORNERS)
    check(got, O.box_forward(d["x"], d["boxes"], integer_corners=True), RTOL_F32, "O")


@pytest.mark.parametrize("H", [64, 37])
@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_MEAN_OFFSET, bc.BC_FLAG_INTEGER_CORNERS])
def test_fwd_bf16_rows_are_rounded_fp32_outputs(H, flags):
    """48-column maps with a bf16 output take 6-column items whose rows go out
    as packed words (a ragged last segment, when H is not a multiple of 8,
    takes per-element stores); the fp32 output takes 3-column items.  Every
    bf16 value is the round-to-nearest-even bf16 of the same call's fp32
    output, bit for bit."""
    wl = wlmod.WORKLOADS[3].scaled(N=2, C=4, H=H)
    d = wlmod.make_inputs(wl)
    N, C, B, W = wl.N, wl.C, wl.B, wl.W
    say(f"fwd bf16 rows 48 wide H={H} flags={flags}")
    xd, bd = dev(d["x"]), dev(d["boxes"])
    y32 = torch.empty((N, C * B, H, W), dtype=torch.float32, device="cuda")
    bc.box_conv_fwd(xd, bd, y32, flags)
    want = y32.to(torch.bfloat16)
    y16 = torch.empty_like(want)
    bc.box_conv_fwd(xd, bd, y16, flags)
    torch.cuda.synchronize()
    assert torch.equal(y16.view(torch.int16), want.view(torch.int16))


def test_fwd_integer_corners_bf16_output():
    wl = wlmod.WORKLOADS[3].scaled(N=1, C=4)
    d = wlmod.make_inputs(wl)
    got = _fwd(d["x"], d["boxes"], torch.bfloat16, INT_CORNERS)
    ref = O.box_forward(d["x"], d["boxes"], integer_corners=True)
    e = bb.scale_err(ref, bb.E_F32)
    assert np.all(np.abs(got - O.bf16_round(ref)) <= bb.bf16_band(ref, e))
    assert np.mean(got == O.bf16_round(ref)) > 0.9


@pytest.mark.parametrize("key,scale", [
    (3, dict(N=3, C=4)),
    (3, dict(N=4, C=256)),                      # enough maps for 8-row items
    (2, dict(N=1, C=3, H=37, W=29, B=5)),
    (3, dict(N=2, C=2, H=17, W=100, B=3)),
    (3, dict(N=1, C=2, H=96, W=97, B=3)),       # 792 items: one block of 832 threads
    (4, dict(N=1, C=1, B=3)),
])
@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM])
def test_bwd_integer_corners(key, scale, flags):
    wl = wlmod.WORKLOADS[key].scaled(**scale)
    d = wlmod.make_inputs(wl)
    rng = np.random.default_rng(112)
    g = rng.standard_normal((wl.N, wl.C * wl.B, wl.H, wl.W)).astype(np.float32)
    say(f"bwd integer corners {wl.key} {scale} flags={flags}")
    gx = torch.empty((wl.N, wl.C, wl.H, wl.W), dtype=torch.float32, device="cuda")
    bc.box_conv_bwd(dev(d["x"]), dev(d["boxes"]), dev(g), gx, None, flags | INT_CORNERS)
    check(host(gx), O.box_backward_input(g, d["boxes"], wl.H, wl.W, integer_corners=True), RTOL_F32, "dx")


def test_integer_corners_box_grad_rejected():
    x = torch.zeros((1, 1, 8, 8), device="cuda")
    bx = torch.zeros((1, 2, 4), device="cuda")
    g = torch.zeros((1, 2, 8, 8), device="cuda")
    gx = torch.empty_like(x)
    gb = torch.empty((1, 2, 4), device="cuda")
    with pytest.raises(bc.BoxConvError):
        bc.box_conv_bwd(x, bx, g, gx, gb, INT_CORNERS)


# ---------------------------------------------------------------------------
# Integer stride: the box at every s-th pixel
# ---------------------------------------------------------------------------
def _fwd_s(x, bx, stride, y_dtype=torch.float32, flags=0):
    N, C, H, W = x.shape
    B = bx.shape[1]
    y = torch.empty((N, C * B, O.strided_size(H, stride), O.strided_size(W, stride)), dtype=y_dtype, device="cuda")
    bc.box_conv_fwd(dev(x), dev(bx), y, flags, stride=stride)
    return host(y)


@pytest.mark.parametrize("stride", [2, 3])
@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM, INT_CORNERS, INT_CORNERS | bc.BC_FLAG_FORCE_HBM])
def test_fwd_strided_int_bit_exact(stride, flags):
    say(f"fwd strided int32 stride={stride} flags={flags}")
    wl = wlmod.WORKLOADS[1]
    d = wlmod.make_inputs(wl)
    bx = d["boxes"] if not flags & INT_CORNERS else rounding_boxes(np.random.default_rng(113), wl.C, wl.B)
    got = _fwd_s(d["x"], bx, stride, torch.int32, flags)
    want = O.box_forward(d["x"], bx, integer_corners=bool(flags & INT_CORNERS), stride=stride)
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("key,scale", [
    (3, dict(N=2, C=8)),
    (2, dict(N=1, C=3, H=37, W=29, B=5)),
    (3, dict(N=1, C=2, H=17, W=100, B=3)),
])
@pytest.mark.parametrize("stride", [2, 3])
@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM, bc.BC_FLAG_MEAN_OFFSET, INT_CORNERS])
def test_fwd_strided_f32(key, scale, stride, flags):
    wl = wlmod.WORKLOADS[key].scaled(**scale)
    d = wlmod.make_inputs(wl)
    say(f"fwd strided {wl.key} {scale} stride={stride} flags={flags}")
    got = _fwd_s(d["x"], d["boxes"], stride, torch.float32, flags)
    want = O.box_forward(d["x"], d["boxes"], integer_corners=bool(flags & INT_CORNERS), stride=stride)
    check(got, want, RTOL_F32, "O")


@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_MEAN_OFFSET])
def test_fwd_strided_large_maps(flags):
    wl = wlmod.WORKLOADS[4].scaled(N=1, C=2)
    d = wlmod.make_inputs(wl)
    say(f"fwd strided {wl.key} reduced stride=2 flags={flags}")
    got = _fwd_s(d["x"], d["boxes"], 2, torch.float32, flags)
    check(got, O.box_forward(d["x"], d["boxes"], stride=2), RTOL_F32, "O")


def test_strided_api_stride_one_is_plain():
    wl = wlmod.WORKLOADS[2].scaled(N=1, C=3)
    d = wlmod.make_inputs(wl)
    N, C, H, W, B = wl.N, wl.C, wl.H, wl.W, wl.B
    x, bx = dev(d["x"]), dev(d["boxes"])
    y1 = torch.empty((N, C * B, H, W), device="cuda")
    y2 = torch.empty_like(y1)
    bc.box_conv_fwd(x, bx, y1)
    lib = bc.load_library()
    ws = bc._workspace(bc.box_workspace_bytes(0, N, C, H, W, B, 0), x.device)
    st = lib.box_conv_fwd_strided(bc._ptr(x), bc.BC_F32, bc._ptr(bx), N, C, H, W, B, 1, bc._ptr(y2), bc.BC_F32, 0,
                                  bc._ptr(ws), ws.numel(), bc._stream())
    assert st == 0
    np.testing.assert_array_equal(host(y1), host(y2))


@pytest.mark.parametrize("key,scale", [
    (3, dict(N=2, C=4)),
    (2, dict(N=1, C=3, H=37, W=29, B=5)),
    (3, dict(N=2, C=2, H=17, W=100, B=3)),
    (3, dict(N=1, C=2, H=96, W=97, B=3)),       # 792 items of the full-size map: one wide block
    (4, dict(N=1, C=1, B=3)),
])
@pytest.mark.parametrize("stride", [2, 3])
@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM])
def test_bwd_strided(key, scale, stride, flags):
    wl = wlmod.WORKLOADS[key].scaled(**scale)
    d = wlmod.make_inputs(wl)
    Ho, Wo = O.strided_size(wl.H, stride), O.strided_size(wl.W, stride)
    g = np.random.default_rng(114).standard_normal((wl.N, wl.C * wl.B, Ho, Wo)).astype(np.float32)
    say(f"bwd strided {wl.key} {scale} stride={stride} flags={flags}")
    gx = torch.empty((wl.N, wl.C, wl.H, wl.W), dtype=torch.float32, device="cuda")
    gb = torch.empty((wl.C, wl.B, 4), dtype=torch.float32, device="cuda")
    bc.box_conv_bwd(dev(d["x"]), dev(d["boxes"]), dev(g), gx, gb, flags, stride=stride)
    check(host(gx), O.box_backward_input(g, d["boxes"], wl.H, wl.W, stride=stride), RTOL_F32, "dx")
    check(host(gb), O.box_backward_params(d["x"], g, d["boxes"], stride=stride), RTOL_F32, "dboxes")


@pytest.mark.parametrize("flags", [INT_CORNERS, INT_CORNERS | bc.BC_FLAG_FORCE_HBM])
def test_bwd_strided_integer_corners(flags):
    wl = wlmod.WORKLOADS[3].scaled(N=2, C=3, H=37, W=29)
    d = wlmod.make_inputs(wl)
    s = 2
    Ho, Wo = O.strided_size(wl.H, s), O.strided_size(wl.W, s)
    g = np.random.default_rng(115).standard_normal((wl.N, wl.C * wl.B, Ho, Wo)).astype(np.float32)
    say(f"bwd strided integer corners flags={flags}")
    gx = torch.empty((wl.N, wl.C, wl.H, wl.W), dtype=torch.float32, device="cuda")
    bc.box_conv_bwd(dev(d["x"]), dev(d["boxes"]), dev(g), gx, None, flags, stride=s)
    want = O.box_backward_input(g, d["boxes"], wl.H, wl.W, integer_corners=True, stride=s)
    check(host(gx), want, RTOL_F32, "dx")


def test_layer_strided_fp32():
    """The whole layer at stride 2 (fp32 mix): every output against the
    oracle's strided box filter composed with its mix."""
    wl = wlmod.WORKLOADS[2].scaled(N=2, C=8)
    d = wlmod.make_inputs(wl)
    s = 2
    Ho, Wo = O.strided_size(wl.H, s), O.strided_size(wl.W, s)
    g = np.random.default_rng(116).standard_normal((wl.N, wl.mix_out, Ho, Wo)).astype(np.float32)
    plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, torch.float32, "f32", False, 0, True, stride=s)
    xd, bd, wd = dev(d["x"]), dev(d["boxes"]), dev(d["w"])
    z = plan.forward(xd, bd, wd)
    dx, db, dw = plan.backward(xd, bd, wd, dev(g))
    torch.cuda.synchronize()
    o = O.box_forward(d["x"], d["boxes"], stride=s)
    check(host(z), O.mix_forward(d["w"], o, compute="f32"), RTOL_F32, "Z")
    do = O.mix_backward_data(d["w"], g, compute="f32")
    check(host(dw), O.mix_backward_weight(g, o, compute="f32"), RTOL_F32, "dW")
    check(host(dx), O.box_backward_input(do, d["boxes"], wl.H, wl.W, stride=s), RTOL_F32, "dx")
    check(host(db), O.box_backward_params(d["x"], do, d["boxes"], stride=s), RTOL_F32, "dboxes")


# ---------------------------------------------------------------------------
# Box-parameter reparameterisation: bit-exact (fp64 arithmetic, one rounding)
# ---------------------------------------------------------------------------
def test_unit_params_bit_exact():
    rng = np.random.default_rng(117)
    C, B, Mw, Mh = 9, 5, 64.0, 48.0
    u = rng.uniform(-1, 1, size=(C, B, 4)).astype(np.float32)
    u[0, 0] = 0
    boxes = torch.empty((C, B, 4), device="cuda")
    bc.box_params_from_unit(dev(u), Mw, Mh, boxes)
    np.testing.assert_array_equal(host(boxes), O.boxes_from_unit(u, Mw, Mh))
    g = rng.standard_normal((C, B, 4)).astype(np.float32)
    gu = torch.empty((C, B, 4), device="cuda")
    bc.box_params_unit_grad(dev(g), Mw, Mh, gu)
    np.testing.assert_array_equal(host(gu), O.unit_grad_from_box_grad(g, Mw, Mh))
    v = (rng.standard_normal((C, B, 4)) * 1.5).astype(np.float32)
    vd = dev(v)
    bc.box_params_clip(vd)
    np.testing.assert_array_equal(host(vd), O.clip_unit_params(v))


def test_layer_unit_params_gradient():
    """Layer trained through unit corners: box gradient in u equals the
    oracle's chain rule of its parameter gradient."""
    wl = wlmod.WORKLOADS[2].scaled(N=2, C=4)
    d = wlmod.make_inputs(wl)
    rng = np.random.default_rng(118)
    Mw, Mh = 32.0, 32.0
    u = O.clip_unit_params(rng.uniform(-0.5, 0.5, size=(wl.C, wl.B, 4)).astype(np.float32))
    g = rng.standard_normal((wl.N, wl.mix_out, wl.H, wl.W)).astype(np.float32)
    plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, torch.float32, "f32", False, 0, True,
                     unit_size=(Mw, Mh))
    xd, ud, wd = dev(d["x"]), dev(u), dev(d["w"])
    z = plan.forward(xd, ud, wd)
    dx, du, dw = plan.backward(xd, ud, wd, dev(g))
    torch.cuda.synchronize()
    bx = O.boxes_from_unit(u, Mw, Mh)
    o = O.box_forward(d["x"], bx)
    check(host(z), O.mix_forward(d["w"], o, compute="f32"), RTOL_F32, "Z")
    do = O.mix_backward_data(d["w"], g, compute="f32")
    want = O.unit_grad_from_box_grad(O.box_backward_params(d["x"], do, bx), Mw, Mh)
    check(host(du), want, RTOL_F32, "du")
    check(host(dx), O.box_backward_input(do, bx, wl.H, wl.W), RTOL_F32, "dx")


# ---------------------------------------------------------------------------
# a7 / a8: backward of the box filter
# ---------------------------------------------------------------------------
# ---------------------------------------------------------------------------
# f2: kernel splitting (pieces with their own weights)
# ---------------------------------------------------------------------------
SPLIT_CASES = [
    (2, dict(N=2, C=3)),
    (3, dict(N=3, C=2)),
    (2, dict(N=1, C=3, H=37, W=29, B=5)),
    (3, dict(N=2, C=2, H=17, W=100, B=3)),
    (3, dict(N=1, C=1, H=1, W=1, B=2)),
]


def _split(x, bx, w, mode, g=None, y_dtype=torch.float32, hbm=False):
    N, C, H, W = x.shape
    B = bx.shape[1]
    xd, bd, wd = dev(x), dev(bx), dev(w)
    y = torch.empty((N, C * B, H, W), dtype=y_dtype, device="cuda")
    bc.box_conv_split_fwd(xd, bd, wd, mode, y, force_hbm=hbm)
    if g is None:
        return host(y)
    gx = torch.empty((N, C, H, W), dtype=torch.float32, device="cuda")
    gb = torch.empty((C, B, 4), dtype=torch.float32, device="cuda")
    gw = torch.empty_like(wd)
    bc.box_conv_split_bwd(xd, bd, wd, mode, dev(g), gx, gb, gw, force_hbm=hbm)
    return host(y), host(gx), host(gb), host(gw)


@pytest.mark.parametrize("hbm", [False, True])
@pytest.mark.parametrize("mode", ["2x", "2y", "4"])
@pytest.mark.parametrize("key,scale", SPLIT_CASES)
def test_split_fwd_bwd(mode, key, scale, hbm):
    wl = wlmod.WORKLOADS[key].scaled(**scale)
    d = wlmod.make_inputs(wl)
    P = bc.SPLIT_PIECES[bc.SPLIT_MODES[mode]]
    w = wlmod.make_piece_weights(wl, P)
    g = np.random.default_rng(120).standard_normal((wl.N, wl.C * wl.B, wl.H, wl.W)).astype(np.float32)
    say(f"split {mode} {wl.key} {scale} hbm={hbm}")
    y, gx, gb, gw = _split(d["x"], d["boxes"], w, mode, g, hbm=hbm)
    check(y, O.box_forward_split(d["x"], d["boxes"], w, mode), RTOL_F32, "y")
    check(gx, O.box_backward_split_input(g, d["boxes"], w, mode, wl.H, wl.W), RTOL_F32, "dx")
    want_b, want_w = O.box_backward_split_params(d["x"], g, d["boxes"], w, mode)
    check(gb, want_b, RTOL_F32, "dboxes")
    check(gw, want_w, RTOL_F32, "dw")


@pytest.mark.parametrize("mode", ["2x", "2y", "4"])
def test_split_cut_on_pixel_boundaries(mode):
    """Boxes of even integer size: both the outer edges and the cut lie on
    pixel boundaries, where every edge derivative is one-sided."""
    rng = np.random.default_rng(121)
    N, C, B, H, W = 2, 2, 4, 23, 19
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    g = rng.standard_normal((N, C * B, H, W)).astype(np.float32)
    bx = np.empty((C, B, 4), dtype=np.float32)
    for ax in range(2):
        size = 2 * rng.integers(1, 6, size=(C, B))
        lo = rng.integers(-8, 8, size=(C, B))
        bx[..., ax] = lo + (size - 1) / 2.0
        bx[..., 2 + ax] = size / 2.0
    e = O.split_edges(bx, mode)
    assert np.all(e == np.floor(e))
    w = rng.uniform(-1, 1, size=(C, B, bc.SPLIT_PIECES[bc.SPLIT_MODES[mode]])).astype(np.float32)
    say(f"split {mode} integer cuts")
    y, gx, gb, gw = _split(x, bx, w, mode, g)
    check(y, O.box_forward_split(x, bx, w, mode), RTOL_F32, "y")
    check(gx, O.box_backward_split_input(g, bx, w, mode, H, W), RTOL_F32, "dx")
    want_b, want_w = O.box_backward_split_params(x, g, bx, w, mode)
    check(gb, want_b, RTOL_F32, "dboxes")
    check(gw, want_w, RTOL_F32, "dw")


def test_split_bf16_output_is_rounded_fp32():
    wl = wlmod.WORKLOADS[3].scaled(N=2, C=4)
    d = wlmod.make_inputs(wl)
    w = wlmod.make_piece_weights(wl, 4)
    say("split 4 bf16 output")
    got = _split(d["x"], d["boxes"], w, "4", y_dtype=torch.bfloat16)
    ref = O.box_forward_split(d["x"], d["boxes"], w, "4")
    # as for the unsplit forward: the fp32 value the kernel rounds is within
    # the fp32 error bound of the oracle's, so its bf16 code is reachable
    # from [r - e, r + e]
    e = bb.scale_err(ref, bb.E_F32)
    assert np.all(np.abs(got - O.bf16_round(ref)) <= bb.bf16_band(ref, e))
    assert np.mean(got == O.bf16_round(ref)) > 0.9


def test_split_unit_weights_equal_the_box_layer():
    """All piece weights 1: the pieces tile the box, so the split layer is the
    plain layer (same values up to rounding; the parameter gradients agree)."""
    wl = wlmod.WORKLOADS[2].scaled(N=2, C=3)
    d = wlmod.make_inputs(wl)
    g = np.random.default_rng(122).standard_normal((wl.N, wl.C * wl.B, wl.H, wl.W)).astype(np.float32)
    y0 = _fwd(d["x"], d["boxes"])
    gx0, gb0 = _bwd(d["x"], d["boxes"], g)
    for mode in ("2x", "2y", "4"):
        ones = np.ones((wl.C, wl.B, bc.SPLIT_PIECES[bc.SPLIT_MODES[mode]]), dtype=np.float32)
        say(f"split {mode} unit weights vs plain layer")
        y, gx, gb, _ = _split(d["x"], d["boxes"], ones, mode, g)
        check(y, y0, RTOL_F32, "y")
        check(gx, gx0, RTOL_F32, "dx")
        check(gb, gb0, RTOL_F32, "dboxes")


@pytest.mark.parametrize("relu", [False, True])
def test_layer_split_fp32(relu):
    """The whole layer with boxes split in four (fp32 mix): outputs and every
    gradient against the oracle's split box filter composed with its mix."""
    wl = wlmod.WORKLOADS[2].scaled(N=2, C=8)
    d = wlmod.make_inputs(wl)
    pw = wlmod.make_piece_weights(wl, 4)
    g = np.random.default_rng(126).standard_normal((wl.N, wl.mix_out, wl.H, wl.W)).astype(np.float32)
    plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, torch.float32, "f32", relu, 0, True, split="4")
    xd, wd = dev(d["x"]), dev(d["w"])
    params = (dev(d["boxes"]), dev(pw))
    say(f"layer split 4 relu={relu}")
    z = plan.forward(xd, params, wd)
    dx, (db, dpw), dw = plan.backward(xd, params, wd, dev(g))
    torch.cuda.synchronize()
    o = O.box_forward_split(d["x"], d["boxes"], pw, "4")
    zr = O.mix_forward(d["w"], o, compute="f32", apply_relu=relu)
    check(host(z), zr, RTOL_F32, "Z")
    # the ReLU mask is taken from the layer's fp32 output on both sides
    mask = host(z) if relu else None
    do = O.mix_backward_data(d["w"], g, compute="f32", relu_out=mask)
    check(host(dw), O.mix_backward_weight(g, o, compute="f32", relu_out=mask), RTOL_F32, "dW")
    check(host(dx), O.box_backward_split_input(do, d["boxes"], pw, "4", wl.H, wl.W), RTOL_F32, "dx")
    want_b, want_w = O.box_backward_split_params(d["x"], do, d["boxes"], pw, "4")
    check(host(db), want_b, RTOL_F32, "dboxes")
    check(host(dpw), want_w, RTOL_F32, "dpiece_w")


def test_layer_split_unit_params():
    """Split boxes trained as unit corners: the layer converts u to pixels,
    runs the split filter and returns dL/du and the piece weights' gradient."""
    wl = wlmod.WORKLOADS[2].scaled(N=2, C=4)
    d = wlmod.make_inputs(wl)
    u = wlmod.make_unit_corners(wl)
    pw = wlmod.make_piece_weights(wl, 2)
    g = np.random.default_rng(127).standard_normal((wl.N, wl.mix_out, wl.H, wl.W)).astype(np.float32)
    mw, mh = float(wl.W), float(wl.H)
    plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, torch.float32, "f32", False, 0, True,
                     split="2x", unit_size=(mw, mh))
    xd, wd = dev(d["x"]), dev(d["w"])
    params = (dev(u), dev(pw))
    say("layer split 2x with unit corners")
    z = plan.forward(xd, params, wd)
    dx, (du, dpw), dw = plan.backward(xd, params, wd, dev(g))
    torch.cuda.synchronize()
    bx = O.boxes_from_unit(u, mw, mh).astype(np.float32)
    o = O.box_forward_split(d["x"], bx, pw, "2x")
    check(host(z), O.mix_forward(d["w"], o, compute="f32"), RTOL_F32, "Z")
    do = O.mix_backward_data(d["w"], g, compute="f32")
    check(host(dx), O.box_backward_split_input(do, bx, pw, "2x", wl.H, wl.W), RTOL_F32, "dx")
    gbox, gw = O.box_backward_split_params(d["x"], do, bx, pw, "2x")
    check(host(du), O.unit_grad_from_box_grad(gbox, mw, mh), RTOL_F32, "du")
    check(host(dpw), gw, RTOL_F32, "dpiece_w")
    check(host(dw), O.mix_backward_weight(g, o, compute="f32"), RTOL_F32, "dW")


def test_split_deterministic():
    wl = wlmod.WORKLOADS[3].scaled(N=2, C=4)
    d = wlmod.make_inputs(wl)
    w = wlmod.make_piece_weights(wl, 4)
    g = np.random.default_rng(123).standard_normal((2, 16, 64, 48)).astype(np.float32)
    a = _split(d["x"], d["boxes"], w, "4", g)
    b = _split(d["x"], d["boxes"], w, "4", g)
    for u, v in zip(a, b):
        np.testing.assert_array_equal(u, v)


def test_split_full_size_sampled():
    """The pose-layer shape (32 x 256 maps of 64 x 48, 4 boxes each), split in
    four: outputs and gradients of sampled channels against the oracle."""
    wl = wlmod.WORKLOADS[3]
    d = wlmod.make_inputs(wl)
    w = wlmod.make_piece_weights(wl, 4)
    N, C, H, W, B = wl.N, wl.C, wl.H, wl.W, wl.B
    g = np.random.default_rng(124).standard_normal((N, C * B, H, W), dtype=np.float32)
    say(f"split 4 full size {wl.key}")
    y, gx, gb, gw = _split(d["x"], d["boxes"], w, "4", g)
    rng = np.random.default_rng(125)
    for c in rng.choice(C, size=3, replace=False):
        ns = rng.choice(N, size=2, replace=False)
        xs, bs, ws = d["x"][ns][:, [c]], d["boxes"][[c]], w[[c]]
        gs = g[ns][:, c * B:(c + 1) * B]
        check(y[ns][:, c * B:(c + 1) * B], O.box_forward_split(xs, bs, ws, "4"), RTOL_F32, f"y c={c}")
        check(gx[ns][:, [c]], O.box_backward_split_input(gs, bs, ws, "4", H, W), RTOL_F32, f"dx c={c}")
        want_b, want_w = O.box_backward_split_params(d["x"][:, [c]], g[:, c * B:(c + 1) * B], bs, ws, "4")
        check(gb[[c]], want_b, RTOL_F32, f"dboxes c={c}")
        check(gw[[c]], want_w, RTOL_F32, f"dw c={c}")


def _bwd(x, bx, g, flags=0):
    N, C, H, W = x.shape
    B = bx.shape[1]
    gx = torch.empty((N, C, H, W), dtype=torch.float32, device="cuda")
    gb = torch.empty((C, B, 4), dtype=torch.float32, device="cuda")
    bc.box_conv_bwd(dev(x), dev(bx), dev(g), gx, gb, flags)
    return host(gx), host(gb)


@pytest.mark.parametrize("key,scale", [
    (2, dict(N=2, C=4)),
    (3, dict(N=3, C=4)),
    (2, dict(N=1, C=3, H=37, W=29, B=5)),
    (3, dict(N=2, C=2, H=17, W=100, B=3)),
    (4, dict(N=1, C=1, B=3)),
    # ragged rows and columns, a last column inside an item, 256-row maps
    (2, dict(N=1, C=3, H=60, W=40, B=3)),
    (2, dict(N=2, C=2, H=9, W=47, B=2)),
    (2, dict(N=1, C=2, H=256, W=48, B=2)),
    # maps the streaming backward takes (no table in LDS or HBM)
    (2, dict(N=1, C=2, H=500, W=47, B=3)),
    (4, dict(N=1, C=2, H=300, W=128, B=3)),
    (4, dict(N=1, C=1, H=200, W=200, B=5)),
    (4, dict(N=1, C=2, H=130, W=256, B=8)),
])
@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM, bc.BC_FLAG_MEAN_OFFSET])
def test_bwd(key, scale, flags):
    wl = wlmod.WORKLOADS[key].scaled(**scale)
    d = wlmod.make_inputs(wl)
    rng = np.random.default_rng(105)
    g = rng.standard_normal((wl.N, wl.C * wl.B, wl.H, wl.W)).astype(np.float32)
    say(f"bwd {wl.key} {scale} flags={flags}")
    gx, gb = _bwd(d["x"], d["boxes"], g, flags)
    check(gx, O.box_backward_input(g, d["boxes"], wl.H, wl.W), RTOL_F32, "dx")
    check(gb, O.box_backward_params(d["x"], g, d["boxes"]), RTOL_F32, "dboxes")


@pytest.mark.parametrize("stride", [1, 2])
def test_bwd_eight_row_items(stride):
    """The LDS backward with 8-row items (two waves per 64x48 map), which it
    takes once a call has enough maps to fill the GPU with them (here 4 x 256
    maps, as in the pose layer): dx and the box gradient against the oracle,
    and the masked bf16 variant bit for bit against bc_relu_grad_bf16 of it.
    Smaller calls take 4-row items (the other backward tests)."""
    wl = wlmod.WORKLOADS[3].scaled(N=4, C=256)
    N, C, H, W, B = wl.N, wl.C, wl.H, wl.W, wl.B
    # 8-row items: 128 per map, two waves, so N * 2 partial rows per box
    taps = 2 * C * B * 16 * 4
    a256 = lambda v: (v + 255) // 256 * 256
    assert bc.box_workspace_bytes(1, N, C, H, W, B, 0, stride) == a256(taps) + a256(N * 2 * C * B * 16)
    d = wlmod.make_inputs(wl)
    x = np.maximum(d["x"], 0)          # a rectified map: the ReLU mask has zeros
    Ho, Wo = O.strided_size(H, stride), O.strided_size(W, stride)
    g = np.random.default_rng(116 + stride).standard_normal((N, C * B, Ho, Wo)).astype(np.float32)
    say(f"bwd 8-row items {N}x{C} stride={stride}")
    xd, bd, gd = dev(x), dev(d["boxes"]), dev(g)
    gx = torch.empty((N, C, H, W), dtype=torch.float32, device="cuda")
    gb = torch.empty((C, B, 4), dtype=torch.float32, device="cuda")
    bc.box_conv_bwd(xd, bd, gd, gx, gb, 0, stride=stride)
    check(host(gx), O.box_backward_input(g, d["boxes"], H, W, stride=stride), RTOL_F32, "dx")
    check(host(gb), O.box_backward_params(x, g, d["boxes"], stride=stride), RTOL_F32, "dboxes")
    want = torch.empty((N, C, H, W), dtype=torch.bfloat16, device="cuda")
    bc.relu_grad_bf16(gx, xd, want)
    got = torch.empty_like(want)
    gb2 = torch.empty_like(gb)
    bc.box_conv_bwd_relu_bf16(xd, bd, gd, got, gb2, 0, stride=stride)
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16), want.view(torch.int16))
    assert torch.equal(gb2, gb)


@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM])
def test_bwd_integer_edges(flags):
    """Boxes whose edges all sit on pixel boundaries: the parameter gradient
    is one-sided there (right derivative), which the backward takes through
    the adjoint split of the taps."""
    rng = np.random.default_rng(107)
    N, C, B, H, W = 2, 3, 4, 23, 19
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    g = rng.standard_normal((N, C * B, H, W)).astype(np.float32)
    bx = np.empty((C, B, 4), dtype=np.float32)
    for ax in range(2):
        size = rng.integers(1, 9, size=(C, B))
        lo = rng.integers(-10, 10, size=(C, B))
        bx[..., ax] = lo + (size - 1) / 2.0
        bx[..., 2 + ax] = size / 2.0
    a, b, c, d = O.box_edges(bx)
    assert np.all(a == np.floor(a)) and np.all(d == np.floor(d))
    say(f"bwd integer edges flags={flags}")
    gx, gb = _bwd(x, bx, g, flags)
    check(gx, O.box_backward_input(g, bx, H, W), RTOL_F32, "dx")
    check(gb, O.box_backward_params(x, g, bx), RTOL_F32, "dboxes")


# ---------------------------------------------------------------------------
# Edges of the path selection: widest maps, the LDS-table limit, the
# backward's 256-item LDS limit, and degenerate boxes in the backward
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("H,W", [(5, 1024), (3, 1021)])
@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM])
def test_widest_maps(H, W, flags):
    """W up to 1024 (the HBM row-scan limit): the tables fit LDS and the
    backward's 684 (342) items one block of up to 1024 threads; with
    BC_FLAG_FORCE_HBM both take the HBM tables."""
    rng = np.random.default_rng(130)
    x = rng.standard_normal((1, 2, H, W)).astype(np.float32)
    g = rng.standard_normal((1, 6, H, W)).astype(np.float32)
    bx = real_boxes(rng, 2, 3, 40.0, 0.5, 300.0)
    say(f"widest maps {H}x{W} flags={flags}")
    check(_fwd(x, bx, flags=flags), O.box_forward(x, bx), RTOL_F32, "O")
    gx, gb = _bwd(x, bx, g, flags)
    check(gx, O.box_backward_input(g, bx, H, W), RTOL_F32, "dx")
    check(gb, O.box_backward_params(x, g, bx), RTOL_F32, "dboxes")


@pytest.mark.parametrize("H,W", [(128, 128), (138, 138), (140, 140), (128, 48), (136, 48), (96, 96), (256, 48),
                                 (260, 48)])
def test_lds_limits(H, W):
    """Maps on both sides of the LDS limits: 138x138 is the largest square
    table the forward keeps in LDS (140x140 is not); the backward walks a map
    in one block of up to 256 threads to 128x48, of up to 1024 threads from
    136x48 (and 96x96) to 256x48, and takes the HBM tables from 260x48."""
    rng = np.random.default_rng(131)
    x = rng.standard_normal((2, 2, H, W)).astype(np.float32)
    g = rng.standard_normal((2, 4, H, W)).astype(np.float32)
    bx = real_boxes(rng, 2, 2, 30.0, 0.5, 40.0)
    say(f"lds limits {H}x{W}")
    check(_fwd(x, bx), O.box_forward(x, bx), RTOL_F32, "O")
    gx, gb = _bwd(x, bx, g)
    check(gx, O.box_backward_input(g, bx, H, W), RTOL_F32, "dx")
    check(gb, O.box_backward_params(x, g, bx), RTOL_F32, "dboxes")


@pytest.mark.parametrize("flags", [0, bc.BC_FLAG_FORCE_HBM])
def test_bwd_degenerate_boxes(flags):
    """Boxes covering everything, entirely outside the map, of zero size, or
    thin: the gradients against the oracle (zero where the box reads nothing)."""
    rng = np.random.default_rng(132)
    x = rng.standard_normal((2, 2, 9, 7)).astype(np.float32)
    g = rng.standard_normal((2, 8, 9, 7)).astype(np.float32)
    bx = np.array([[[0, 0, 1000, 1000], [500, 0, 3, 3], [0, 0, 0, 0], [0.3, 0.2, 0.1, 0.05]],
                   [[-20, 30, 2, 2], [0, 0, 4.5, 0.5], [2.2, -1.1, 0.5, 6], [0, 0, 0.5, 0.5]]],
                  dtype=np.float32)
    say(f"bwd degenerate boxes flags={flags}")
    gx, gb = _bwd(x, bx, g, flags)
    check(gx, O.box_backward_input(g, bx, 9, 7), RTOL_F32, "dx")
    want = O.box_backward_params(x, g, bx)
    check(gb, want, RTOL_F32, "dboxes")
    # a box entirely outside the map reads nothing: no gradient at all
    assert np.all(gb[0, 1] == 0) and np.all(gb[1, 0] == 0)


@pytest.mark.parametrize("hbm", [False, True])
@pytest.mark.parametrize("mode", ["2x", "2y", "4"])
def test_split_degenerate_boxes(mode, hbm):
    """Split boxes with zero-width pieces (rx = 0 or ry = 0), boxes outside
    the map and boxes covering everything."""
    rng = np.random.default_rng(133)
    x = rng.standard_normal((2, 2, 9, 7)).astype(np.float32)
    g = rng.standard_normal((2, 8, 9, 7)).astype(np.float32)
    bx = np.array([[[0, 0, 1000, 1000], [500, 0, 3, 3], [0, 0, 0, 0], [0.3, 0.2, 0.0, 2.5]],
                   [[-20, 30, 2, 2], [0, 0, 4.5, 0.0], [2.2, -1.1, 0.5, 6], [0, 0, 0.5, 0.5]]],
                  dtype=np.float32)
    w = rng.uniform(-1, 1, size=(2, 4, bc.SPLIT_PIECES[bc.SPLIT_MODES[mode]])).astype(np.float32)
    say(f"split {mode} degenerate boxes hbm={hbm}")
    y, gx, gb, gw = _split(x, bx, w, mode, g, hbm=hbm)
    check(y, O.box_forward_split(x, bx, w, mode), RTOL_F32, "y")
    check(gx, O.box_backward_split_input(g, bx, w, mode, 9, 7), RTOL_F32, "dx")
    want_b, want_w = O.box_backward_split_params(x, g, bx, w, mode)
    check(gb, want_b, RTOL_F32, "dboxes")
    check(gw, want_w, RTOL_F32, "dw")


@pytest.mark.parametrize("mode", ["2x", "4"])
@pytest.mark.parametrize("H,W", [(70, 100), (131, 133), (150, 151)])
def test_split_large_maps(H, W, mode):
    """Maps at and past the LDS limits, each taking its path by itself:
    70x100 walks its 612 backward items in one block of 640 threads; 131x133
    keeps its forward table in LDS (74 KiB) but has too many backward items
    for one block; 150x151 has neither in LDS (ragged in both directions)."""
    rng = np.random.default_rng(134)
    x = rng.standard_normal((1, 2, H, W)).astype(np.float32)
    g = rng.standard_normal((1, 6, H, W)).astype(np.float32)
    bx = real_boxes(rng, 2, 3, 35.0, 0.5, 45.0)
    w = rng.uniform(-1, 1, size=(2, 3, bc.SPLIT_PIECES[bc.SPLIT_MODES[mode]])).astype(np.float32)
    say(f"split {mode} large maps {H}x{W}")
    y, gx, gb, gw = _split(x, bx, w, mode, g)
    check(y, O.box_forward_split(x, bx, w, mode), RTOL_F32, "y")
    check(gx, O.box_backward_split_input(g, bx, w, mode, H, W), RTOL_F32, "dx")
    want_b, want_w = O.box_backward_split_params(x, g, bx, w, mode)
    check(gb, want_b, RTOL_F32, "dboxes")
    check(gw, want_w, RTOL_F32, "dw")


def test_bwd_deterministic():
    wl = wlmod.WORKLOADS[3].scaled(N=2, C=4)
    d = wlmod.make_inputs(wl)
    g = np.random.default_rng(106).standard_normal((2, 16, 64, 48)).astype(np.float32)
    a = _bwd(d["x"], d["boxes"], g)
    b = _bwd(d["x"], d["boxes"], g)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


# ---------------------------------------------------------------------------
# a4 / a5 / a6: 1x1 mix
# ---------------------------------------------------------------------------
# bf16 with bf16 storage takes the column-strip kernels where they apply
# (FWD: M <= 256, K % 128 == 0, P % 4 == 0; BWD_DATA: M <= 448): the pose
# shape at one image, rows ragged across waves, a ragged last strip, an odd
# number of reduction chunks, a single chunk
@pytest.mark.parametrize("dims", [(2, 64, 512, 3072), (1, 40, 72, 1000), (3, 8, 32, 1024), (2, 130, 260, 129),
                                  (1, 256, 1024, 3072), (2, 100, 256, 1000), (2, 200, 384, 132),
                                  (1, 16, 128, 64),
                                  # M * K odd: the split-K sum one output per thread
                                  (2, 7, 9, 200)])
@pytest.mark.parametrize("compute,storage", [("f32", torch.float32), ("bf16", torch.float32),
                                             ("bf16", torch.bfloat16)])
@pytest.mark.parametrize("relu", [0, 1])
def test_mix(dims, compute, storage, relu):
    N, M, K, P = dims
    say(f"mix {dims} {compute} {storage} relu={relu}")
    rng = np.random.default_rng(107)
    w = (rng.standard_normal((M, K)) / np.sqrt(K)).astype(np.float32)
    o = rng.standard_normal((N, K, P)).astype(np.float32)
    gz = rng.standard_normal((N, M, P)).astype(np.float32)
    cd = bc.BC_BF16 if compute == "bf16" else bc.BC_F32
    rtol = RTOL_F32 if compute == "f32" else 1e-3
    wd = dev(w).to(storage)
    od = dev(o).to(storage)
    z = torch.empty((N, M, P), dtype=torch.float32, device="cuda")
    bc.pointwise_mix(bc.BC_MIX_FWD, wd, od, z, N, M, K, P, cd, relu=relu)
    zr = O.mix_forward(w, o.reshape(N, K, P, 1), compute=compute, apply_relu=bool(relu)).reshape(N, M, P)
    check(host(z), zr, rtol, "Z")
    aux = z if relu else None
    auxr = zr if relu else None
    do = torch.empty((N, K, P), dtype=torch.float32, device="cuda")
    bc.pointwise_mix(bc.BC_MIX_BWD_DATA, wd, dev(gz), do, N, M, K, P, cd, relu=relu, aux=aux)
    dor = O.mix_backward_data(w, gz.reshape(N, M, P, 1), compute=compute,
                              relu_out=None if auxr is None else auxr.reshape(N, M, P, 1)).reshape(N, K, P)
    check(host(do), dor, rtol, "dO")
    dw = torch.empty((M, K), dtype=torch.float32, device="cuda")
    bc.pointwise_mix(bc.BC_MIX_BWD_WEIGHT, dev(gz), od, dw, N, M, K, P, cd, relu=relu, aux=aux)
    dwr = O.mix_backward_weight(gz.reshape(N, M, P, 1), o.reshape(N, K, P, 1), compute=compute,
                                relu_out=None if auxr is None else auxr.reshape(N, M, P, 1))
    check(host(dw), dwr, rtol, "dW")
    # accumulate adds onto the existing contents
    bc.pointwise_mix(bc.BC_MIX_BWD_WEIGHT, dev(gz), od, dw, N, M, K, P, cd, relu=relu, aux=aux, accumulate=1)
    check(host(dw), 2 * dwr, rtol, "dW accumulated")
    if storage == torch.bfloat16 and not relu:
        # dZ in bf16 storage too (both operands bf16: the 128-deep K-steps,
        # with split chunks that end inside a K-step for the small P); the
        # oracle rounds the same operands to bf16, so the reference is dwr
        dw2 = torch.empty_like(dw)
        bc.pointwise_mix(bc.BC_MIX_BWD_WEIGHT, dev(gz).to(storage), od, dw2, N, M, K, P, cd)
        check(host(dw2), dwr, rtol, "dW (bf16 dZ)")


def test_cast_bf16_bit_exact():
    rng = np.random.default_rng(110)
    v = np.concatenate([
        rng.standard_normal(100003).astype(np.float32) * np.float32(7.0),
        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 1.0078125, 65504.0, 3.3e38, -3.3e38,
                  np.inf, -np.inf, 1e-30, -1e-30], dtype=np.float32),
        (np.arange(256, dtype=np.uint32) << 16 | 0x3F808000).view(np.float32),   # exact ties
        (np.arange(256, dtype=np.uint32) << 16 | 0x3F807FFF).view(np.float32),
    ]).astype(np.float32)
    src = dev(v)
    dst = torch.empty(v.size, dtype=torch.bfloat16, device="cuda")
    bc.bc_cast_bf16(src, dst)
    np.testing.assert_array_equal(host(dst), O.bf16_round(v))


def test_relu_grad_bf16_bit_exact():
    """The ReLU backward in the mix's compute type, bf16(z > 0 ? g : 0),
    against the oracle's rounding of the same selection: exact ties, zeros of
    either sign and NaN in the mask (all mask out), n not a multiple of 8."""
    rng = np.random.default_rng(111)
    n = 100005
    g = (rng.standard_normal(n) * 7).astype(np.float32)
    z = rng.standard_normal(n).astype(np.float32)
    z[:64] = 0.0
    z[64:128] = -0.0
    z[128:136] = np.nan
    z[136:144] = np.inf
    g[200:456] = ((np.arange(256, dtype=np.uint32) << 16) | 0x3F808000).view(np.float32)
    z[200:456] = 1.0
    dst = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    bc.relu_grad_bf16(dev(g), dev(z), dst)
    with np.errstate(invalid="ignore"):
        want = O.bf16_round(np.where(z > 0, g, np.float32(0.0)))
    np.testing.assert_array_equal(host(dst), want)


@pytest.mark.parametrize("dims", [(2, 64, 192, 160), (1, 40, 72, 77)])
def test_relu_grad_prepass_matches_masked_gemms(dims):
    """BWD_DATA and BWD_WEIGHT on the pre-masked bf16 gradient return bitwise
    what the masked GEMMs return from the fp32 gradient and the forward
    output (the layer's ReLU path relies on it)."""
    N, M, K, P = dims
    rng = np.random.default_rng(112)
    gz = rng.standard_normal((N, M, P)).astype(np.float32)
    zf = rng.standard_normal((N, M, P)).astype(np.float32)
    w = (rng.standard_normal((M, K)) / np.sqrt(K)).astype(np.float32)
    o = rng.standard_normal((N, K, P)).astype(np.float32)
    cd = bc.BC_BF16
    wd, od, gd, zd = dev(w), dev(o), dev(gz), dev(zf)
    say(f"relu pre-pass vs masked GEMMs {dims}")
    gm = torch.empty((N, M, P), dtype=torch.bfloat16, device="cuda")
    bc.relu_grad_bf16(gd, zd, gm)
    do_a = torch.empty((N, K, P), dtype=torch.float32, device="cuda")
    do_b = torch.empty_like(do_a)
    bc.pointwise_mix(bc.BC_MIX_BWD_DATA, wd, gd, do_a, N, M, K, P, cd, relu=1, aux=zd)
    bc.pointwise_mix(bc.BC_MIX_BWD_DATA, wd, gm, do_b, N, M, K, P, cd)
    assert torch.equal(do_a, do_b)
    dw_a = torch.empty((M, K), dtype=torch.float32, device="cuda")
    dw_b = torch.empty_like(dw_a)
    bc.pointwise_mix(bc.BC_MIX_BWD_WEIGHT, gd, od, dw_a, N, M, K, P, cd, relu=1, aux=zd)
    bc.pointwise_mix(bc.BC_MIX_BWD_WEIGHT, gm, od, dw_b, N, M, K, P, cd)
    assert torch.equal(dw_a, dw_b)
    # and both against the oracle's masked backward
    zr = zf.reshape(N, M, P, 1)
    check(host(do_b), O.mix_backward_data(w, gz.reshape(N, M, P, 1), compute="bf16", relu_out=zr).reshape(N, K, P),
          RTOL_BF16_MIX, "dO")


@pytest.mark.parametrize("H,W,stride,flags", [(64, 48, 1, 0), (37, 29, 1, 0), (96, 97, 1, 0), (64, 48, 1, 2),
                                                (64, 48, 2, 0), (150, 151, 1, 0)])
def test_bwd_relu_bf16_matches_relu_grad(H, W, stride, flags):
    """box_conv_bwd_relu_bf16 writes bf16(x > 0 ? dx : 0) bit for bit as
    bc_relu_grad_bf16 forms it from box_conv_bwd's fp32 dx and x, and the same
    box gradient, on every backward path (LDS, wide LDS block, HBM tables,
    strided).  x is a rectified map (zeros where the ReLU cut)."""
    rng = np.random.default_rng(135)
    N, C, B = 2, 3, 4
    x = np.maximum(rng.standard_normal((N, C, H, W)), 0).astype(np.float32)
    Ho, Wo = O.strided_size(H, stride), O.strided_size(W, stride)
    g = rng.standard_normal((N, C * B, Ho, Wo)).astype(np.float32)
    bx = real_boxes(rng, C, B, 20.0, 0.5, 24.0)
    say(f"bwd relu bf16 {H}x{W} stride={stride} flags={flags}")
    xd, bd, gd = dev(x), dev(bx), dev(g)
    gx = torch.empty((N, C, H, W), dtype=torch.float32, device="cuda")
    gb = torch.empty((C, B, 4), dtype=torch.float32, device="cuda")
    bc.box_conv_bwd(xd, bd, gd, gx, gb, flags, stride=stride)
    want = torch.empty((N, C, H, W), dtype=torch.bfloat16, device="cuda")
    bc.relu_grad_bf16(gx, xd, want)
    got = torch.empty_like(want)
    gb2 = torch.empty_like(gb)
    bc.box_conv_bwd_relu_bf16(xd, bd, gd, got, gb2, flags, stride=stride)
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16), want.view(torch.int16))
    assert torch.equal(gb2, gb)


def test_mix_integer_exact():
    wl = wlmod.WORKLOADS[1]
    d = wlmod.make_inputs(wl)
    o = O.box_forward(d["x"], d["boxes"]).astype(np.int32)
    N, K, H, W = o.shape
    M = wl.mix_out
    z = torch.empty((N, M, H, W), dtype=torch.int32, device="cuda")
    bc.pointwise_mix(bc.BC_MIX_FWD, dev(d["w"]), dev(o), z, N, M, K, H * W, bc.BC_F32)
    np.testing.assert_array_equal(host(z), O.mix_forward(d["w"], o, compute="i32"))


# ---------------------------------------------------------------------------
# Whole layer / stack, reduced sizes of each workload
# ---------------------------------------------------------------------------
def check_bounded(got, ref, bound, rtol, what):
    excess, plain, bnd = bb.bounded_error(got, ref, bound)
    say(f"  {what}: beyond-bound {excess:.3e}  plain pointwise {plain:.3e}  max bound {bnd:.3e}  (rtol {rtol})")
    assert excess <= rtol, f"{what}: error beyond the ambiguity bound {excess} > {rtol}"


@pytest.mark.parametrize("key,scale", [(1, {}), (2, dict(N=2, C=8)), (4, dict(N=1, C=2, B=2)),
                                       (6, dict(N=1, C=4, B=2, mix_out=16))])
def test_layer_step_exact_decisions(key, scale):
    """Workloads without bf16 rounding or ReLU decisions: plain tolerances."""
    wl = wlmod.WORKLOADS[key].scaled(**scale)
    d = wlmod.make_inputs(wl)
    say(f"layer {wl.key} {scale}")
    x_dt = torch.int32 if wl.x_kind == "int8range" else torch.float32
    M = wl.mix_out
    flags = bc.BC_FLAG_MEAN_OFFSET if wl.mean_offset else 0
    plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, M, x_dt, wl.mix_dtype, wl.relu, flags, wl.backward)
    xd, bd = dev(d["x"]), dev(d["boxes"])
    wd = dev(d["w"]) if M is not None else None
    out = plan.forward(xd, bd, wd)
    o_ref = O.box_forward(d["x"], d["boxes"])
    if x_dt == torch.int32:
        np.testing.assert_array_equal(host(plan.o), o_ref)
        np.testing.assert_array_equal(host(out), O.mix_forward(d["w"], o_ref, compute="i32"))
        return
    if M is None:
        check(host(out), o_ref, RTOL_F32, "O")
        gz = d["grad"]
        dx, db, _ = plan.backward(xd, bd, None, dev(gz))
        check(host(dx), O.box_backward_input(gz, d["boxes"], wl.H, wl.W), RTOL_F32, "dx")
        check(host(db), O.box_backward_params(d["x"], gz, d["boxes"]), RTOL_F32, "dboxes")
        return
    check(host(out), O.mix_forward(d["w"], o_ref, compute="f32"), RTOL_F32, "Z")
    gz = d["grad"]
    dx, db, dw = plan.backward(xd, bd, wd, dev(gz))
    do_ref = O.mix_backward_data(d["w"], gz, compute="f32")
    check(host(plan.do), do_ref, RTOL_F32, "dO")
    check(host(dw), O.mix_backward_weight(gz, o_ref, compute="f32"), RTOL_F32, "dW")
    check(host(dx), O.box_backward_input(do_ref, d["boxes"], wl.H, wl.W), RTOL_F32, "dx")
    check(host(db), O.box_backward_params(d["x"], do_ref, d["boxes"]), RTOL_F32, "dboxes")


def test_layer_step_bf16_mix():
    """The pose-shaped layer (bf16 mix, K = 1024) at one image: each output
    within rtol of the oracle beyond the bound of its ambiguous bf16 codes."""
    wl = wlmod.WORKLOADS[3].scaled(N=1)
    d = wlmod.make_inputs(wl)
    say(f"layer {wl.key} N=1")
    plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, torch.float32, "bf16", False, 0, True)
    xd, bd, wd = dev(d["x"]), dev(d["boxes"]), dev(d["w"])
    z = plan.forward(xd, bd, wd)
    fw = bb.layer_forward(d["x"].astype(np.float64), d["boxes"], d["w"], relu=False)
    check_bounded(host(z), fw["z"], fw["ez"], RTOL_BF16_MIX, "Z")
    dx, db, dw = plan.backward(xd, bd, wd, dev(d["grad"]))
    bw = bb.layer_backward(fw, d["boxes"], d["w"], d["grad"].astype(np.float64))
    # without a ReLU, dO, dx and dboxes are fp32 results of the same bf16
    # operands on both sides: no ambiguous decision, the fp32 bar
    check_bounded(host(plan.do), bw["do"], bw["edo"], RTOL_F32, "dO")
    check_bounded(host(dw), bw["dw"], bw["edw"], RTOL_BF16_MIX, "dW")
    check_bounded(host(dx), bw["dx"], bw["edx"], RTOL_F32, "dx")
    check_bounded(host(db), bw["dth"], bw["edth"], RTOL_F32, "dboxes")


@pytest.mark.parametrize("relu", [False, True])
def test_layer_overlap_matches_in_order(relu):
    """A layer built with the weight gradient on a second stream gives the
    same bits as the in-order layer (the same kernels on the same operands;
    the caller's stream waits for the side stream before the backward
    returns), for the bf16 mix with the cast and with the masked gradient."""
    wl = wlmod.WORKLOADS[3].scaled(N=2, C=32)
    d = wlmod.make_inputs(wl)
    xd, bd, wd, gd = dev(d["x"]), dev(d["boxes"]), dev(d["w"]), dev(d["grad"])
    say(f"layer overlap relu={relu}")
    outs = []
    for overlap in (False, True):
        plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, torch.float32, "bf16", relu, 0, True,
                         overlap=overlap)
        z = plan.forward(xd, bd, wd)
        dx, db, dw = plan.backward(xd, bd, wd, gd)
        torch.cuda.synchronize()
        outs.append([t.clone() for t in (z, dx, db, dw)])
    for a_, b_, what in zip(outs[0], outs[1], ("Z", "dx", "dboxes", "dW")):
        assert torch.equal(a_, b_), what


def test_stack_layers_relu_bf16_each_on_oracle_input():
    """Each layer of the stacked workload (bf16 mix + ReLU), run on the
    oracle's input to that layer (the oracle's previous-layer output in fp32)
    with an exact upstream gradient: elementwise within rtol beyond the bound
    of its ambiguous bf16 codes and ReLU decisions."""
    wl = wlmod.WORKLOADS[5].scaled(N=1)          # all six layers of the stack
    d = wlmod.make_inputs(wl)
    x = d["x"].astype(np.float64)
    rng = np.random.default_rng(109)
    for li, (b, w) in enumerate(d["layers"]):
        say(f"stack layer {li} on oracle input")
        x32 = x.astype(np.float32)
        fw = bb.layer_forward(x32.astype(np.float64), b, w, relu=True)
        plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, torch.float32, "bf16", True, 0, True)
        xd, bd, wd = dev(x32), dev(b), dev(w)
        z = plan.forward(xd, bd, wd)
        check_bounded(host(z), fw["z"], fw["ez"], RTOL_BF16_MIX, f"Z[{li}]")
        g = rng.standard_normal(fw["z"].shape).astype(np.float32)
        dx, db, dw = plan.backward(xd, bd, wd, dev(g))
        bw = bb.layer_backward(fw, b, w, g.astype(np.float64), relu=True)
        check_bounded(host(dw), bw["dw"], bw["edw"], RTOL_BF16_MIX, f"dW[{li}]")
        check_bounded(host(plan.do), bw["do"], bw["edo"], RTOL_F32, f"dO[{li}]")
        check_bounded(host(dx), bw["dx"], bw["edx"], RTOL_F32, f"dx[{li}]")
        check_bounded(host(db), bw["dth"], bw["edth"], RTOL_F32, f"dboxes[{li}]")
        x = fw["z"]


def test_stack_two_layers_chained_elementwise():
    """Two stacked layers (bf16 mix + ReLU) through the chained backward the
    stack runs: the top layer's box backward writes the bottom layer's masked
    bf16 gradient operand (box_conv_bwd_relu_bf16) and the bottom layer's
    GEMMs read it as given (grad_premasked).  Each layer's forward runs on the
    oracle's input to that layer, so every gradient of both layers is checked
    element by element: dW, dO, dboxes and the input gradients, within the
    fp32 bar (1e-4; 1e-3 for dW, a bf16 mix result) beyond the bound of their
    ambiguous bf16 codes and ReLU decisions."""
    wl = wlmod.WORKLOADS[5].scaled(N=1, layers=2)
    d = wlmod.make_inputs(wl)
    (b0, w0), (b1, w1) = d["layers"]
    say("stack c5: 2 layers, chained backward, N=1")
    st = Stack(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, 2, "bf16", True)
    p0, p1 = st.plans
    assert p1.dx_relu_bf16 and p0.grad_premasked
    x0 = d["x"].astype(np.float32)
    fw0 = bb.layer_forward(x0.astype(np.float64), b0, w0, relu=True)
    x1 = fw0["z"].astype(np.float32)                 # the oracle's input to layer 1
    fw1 = bb.layer_forward(x1.astype(np.float64), b1, w1, relu=True)
    params = [(dev(b0), dev(w0)), (dev(b1), dev(w1))]
    inputs = [dev(x0), dev(x1)]
    z0 = p0.forward(inputs[0], *params[0])
    z1 = p1.forward(inputs[1], *params[1])
    check_bounded(host(z0), fw0["z"], fw0["ez"], RTOL_BF16_MIX, "Z[0]")
    check_bounded(host(z1), fw1["z"], fw1["ez"], RTOL_BF16_MIX, "Z[1]")
    G = np.random.default_rng(110).standard_normal(fw1["z"].shape).astype(np.float32)
    dx, grads = st.backward(inputs, params, dev(G))
    torch.cuda.synchronize()
    bw1 = bb.layer_backward(fw1, b1, w1, G.astype(np.float64), relu=True)
    check_bounded(host(grads[1][1]), bw1["dw"], bw1["edw"], RTOL_BF16_MIX, "dW[1]")
    check_bounded(host(p1.do), bw1["do"], bw1["edo"], RTOL_F32, "dO[1]")
    check_bounded(host(grads[1][0]), bw1["dth"], bw1["edth"], RTOL_F32, "dboxes[1]")
    # layer 1's input gradient, written masked and rounded: bf16(x1 > 0 ? dx1 : 0)
    eg0 = bw1["edx"] + bb.scale_err(bw1["dx"], bb.E_F32)
    on = x1 > 0
    g0 = np.where(on, bw1["dx"], 0.0)
    check_bounded(host(p1.dx), O.bf16_round(g0), bb.bf16_band(g0, np.where(on, eg0, 0.0)), RTOL_F32,
                  "dx[1] (masked bf16)")
    # layer 0 on that gradient: its mask comes from the exact x1, its bf16
    # codes carry the uncertainty of layer 1's fp32 input gradient
    bw0 = bb.layer_backward(fw0, b0, w0, bw1["dx"], relu=True, eg_in=eg0, mask_exact=True)
    check_bounded(host(grads[0][1]), bw0["dw"], bw0["edw"], RTOL_BF16_MIX, "dW[0]")
    check_bounded(host(p0.do), bw0["do"], bw0["edo"], RTOL_F32, "dO[0]")
    check_bounded(host(grads[0][0]), bw0["dth"], bw0["edth"], RTOL_F32, "dboxes[0]")
    check_bounded(host(dx), bw0["dx"], bw0["edx"], RTOL_F32, "dx[0]")


RTOL_STACK_NORMWISE_PER_LAYER = 5e-3


def test_stack_end_to_end_normwise():
    """Three stacked layers end to end on the GPU against the oracle's chain.
    Beyond the first bf16 rounding the GPU's inputs to later decisions (bf16
    codes, ReLU masks) differ from the oracle's by rounding, so elementwise
    agreement there is a statistical property; this checks every tensor's
    normwise relative error (sanity bar 1e-2; the elementwise parity of each
    layer is the test above)."""
    wl = wlmod.WORKLOADS[5].scaled(N=1, layers=3)
    d = wlmod.make_inputs(wl)
    say("stack c5: 3 layers end to end, N=1")
    st = Stack(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, 3, "bf16", True)
    params = [(dev(b), dev(w)) for b, w in d["layers"]]
    inputs, out = st.forward(dev(d["x"]), params)
    cache = O.stack_forward(d["x"], d["layers"], compute="bf16", apply_relu=True)
    G = np.random.default_rng(108).standard_normal(out.shape).astype(np.float32)
    dx, grads = st.backward(inputs, params, dev(G))
    dxr, gr = O.stack_backward(cache, d["layers"], G, compute="bf16", apply_relu=True)
    pairs = [("Z_last", out, cache[-1][2]), ("dx", dx, dxr)]
    for li in range(3):
        pairs += [(f"dboxes[{li}]", grads[li][0], gr[li][0]), (f"dW[{li}]", grads[li][1], gr[li][1])]
    for name, got, ref in pairs:
        pw, nw = O.rel_errors(host(got), ref)
        say(f"  {name}: normwise {nw:.3e}  pointwise {pw:.3e}")
        assert nw <= RTOL_STACK_NORMWISE_PER_LAYER * 3, f"{name}: normwise {nw}"
