"""Parity at the full workload sizes, in the launch configuration bench.py
times (LayerPlan / Stack over the whole batch), checked on outputs the oracle
can compute one image, one map or one box at a time.

* fp32 layer: the whole step, every output (the oracle finishes in seconds).
* pose layer (bf16 mix): images 0 and N-1 for O, Z, dO, dx; box-parameter and
  weight gradients for sampled boxes / mix inputs summed over every image.
* large maps (256x256, mean-offset table): sampled maps of O and dx, sampled
  boxes' parameter gradients over every image.
* 6-layer stack: image 0's output and input gradient (normwise).
* pose layer, inference (integer corners, forward only) and stride 2: the
  configurations bench.py --inference / --stride 2 time, sampled likewise.
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

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

RTOL_F32 = 1e-4
RTOL_BF16 = 1e-3


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
    assert pw <= rtol, f"{what}: {pw} > {rtol}"


def check_bounded(got, ref, bound, rtol, what):
    excess, plain, bnd = bb.bounded_error(got, ref, bound)
    say(f"  {what}: beyond-bound {excess:.3e}  plain {plain:.3e}  max bound {bnd:.3e}")
    assert excess <= rtol, f"{what}: {excess} > {rtol}"


def run_layer(wl, d):
    x_dt = torch.int32 if wl.x_kind == "int8range" else torch.float32
    flags = bc.BC_FLAG_MEAN_OFFSET if wl.mean_offset else 0
    plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, x_dt, wl.mix_dtype, wl.relu, flags, wl.backward)
    xd, bd = dev(d["x"]), dev(d["boxes"])
    wd = dev(d["w"]) if wl.mix_out is not None else None
    out = plan.forward(xd, bd, wd)
    grads = plan.backward(xd, bd, wd, dev(d["grad"])) if wl.backward else None
    torch.cuda.synchronize()
    return plan, out, grads


def test_fp32_layer_full_size_every_output():
    wl = wlmod.WORKLOADS[2]
    d = wlmod.make_inputs(wl)
    say(f"{wl.key} full size")
    plan, z, (dx, db, dw) = run_layer(wl, d)
    o = O.box_forward(d["x"], d["boxes"])
    check(host(plan.o), o, RTOL_F32, "O")
    check(host(z), O.mix_forward(d["w"], o, compute="f32"), RTOL_F32, "Z")
    do = O.mix_backward_data(d["w"], d["grad"], compute="f32")
    check(host(plan.do), do, RTOL_F32, "dO")
    check(host(dw), O.mix_backward_weight(d["grad"], o, compute="f32"), RTOL_F32, "dW")
    check(host(dx), O.box_backward_input(do, d["boxes"], wl.H, wl.W), RTOL_F32, "dx")
    check(host(db), O.box_backward_params(d["x"], do, d["boxes"]), RTOL_F32, "dboxes")


def test_pose_layer_full_size_sampled():
    wl = wlmod.WORKLOADS[3]
    d = wlmod.make_inputs(wl)
    say(f"{wl.key} full size")
    plan, z, (dx, db, dw) = run_layer(wl, d)
    B, K = wl.B, wl.C * wl.B
    for n in (0, wl.N - 1):
        fw = bb.layer_forward(d["x"][n:n + 1].astype(np.float64), d["boxes"], d["w"], relu=False)
        check_bounded(host(plan.o[n:n + 1]), O.bf16_round(fw["o"]), fw["D"], RTOL_BF16, f"O[{n}] (bf16)")
        check_bounded(host(z[n:n + 1]), fw["z"], fw["ez"], RTOL_BF16, f"Z[{n}]")
        bw = bb.layer_backward(fw, d["boxes"], d["w"], d["grad"][n:n + 1].astype(np.float64))
        # fp32 results of the same bf16 operands on both sides (no ReLU): the fp32 bar
        check(host(plan.do[n:n + 1]), bw["do"], RTOL_F32, f"dO[{n}]")
        check(host(dx[n:n + 1]), bw["dx"], RTOL_F32, f"dx[{n}]")
    # gradients summed over all images, for sampled boxes (c, b) = mix input k = c*B + b
    rng = np.random.default_rng(7)
    ks = sorted(rng.choice(K, size=12, replace=False).tolist())
    _sampled_mix_checks(wl, d, O.box_forward, host(dw), host(db), 1, ks)


# The large-map workload builds its forward tables from (map - mean); the
# plain fp32 table is the reported comparison.  Its values reach ~3e4
# (0.5-mean maps of 65536 pixels), so each four-corner difference loses about
# 1e-6 of relative precision (measured: outputs 1.8e-6 plain, 1.7e-7 with the
# offset).  The backward tabulates only the upstream gradient, so its results
# do not depend on the offset.  Bar 1e-4 for all.
@pytest.mark.parametrize("offset", [True, False])
def test_large_maps_full_size_sampled(offset):
    rtol_params = 1e-4
    wl = wlmod.WORKLOADS[4].scaled(mean_offset=offset)
    d = wlmod.make_inputs(wl)
    say(f"{wl.key} full size, mean offset {offset}")
    plan, o, (dx, db, _) = run_layer(wl, d)
    B = wl.B
    for (n, c) in [(0, 0), (wl.N - 1, wl.C - 1), (1, 77)]:
        o_ref = O.box_forward(d["x"][n:n + 1, c:c + 1], d["boxes"][c:c + 1])
        check(host(o[n:n + 1, c * B:(c + 1) * B]), o_ref, RTOL_F32, f"O[{n}, c={c}]")
        dx_ref = O.box_backward_input(d["grad"][n:n + 1, c * B:(c + 1) * B], d["boxes"][c:c + 1], wl.H, wl.W)
        check(host(dx[n:n + 1, c:c + 1]), dx_ref, RTOL_F32, f"dx[{n}, c={c}]")
    db_got = host(db)
    for (c, b) in [(0, 0), (5, 7), (wl.C - 1, 3)]:
        k = c * B + b
        ref = O.box_backward_params(d["x"][:, c:c + 1], d["grad"][:, k:k + 1], d["boxes"][c:c + 1, b:b + 1])[0, 0]
        pw = np.abs(db_got[c, b] - ref) / (np.abs(ref) + np.sqrt(np.mean(ref ** 2)))
        say(f"  dboxes[{c},{b}]: {pw.max():.3e}")
        assert pw.max() <= rtol_params


def test_stack6_full_size_image0():
    wl = wlmod.WORKLOADS[5]
    d = wlmod.make_inputs(wl)
    say(f"{wl.key} full size")
    st = Stack(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, wl.layers, "bf16", True)
    params = [(dev(b), dev(w)) for b, w in d["layers"]]
    inputs, out = st.forward(dev(d["x"]), params)
    dx, grads = st.backward(inputs, params, dev(d["grad"]))
    torch.cuda.synchronize()
    cache = O.stack_forward(d["x"][:1], d["layers"], compute="bf16", apply_relu=True)
    dxr, gr = O.stack_backward(cache, d["layers"], d["grad"][:1], compute="bf16", apply_relu=True)
    # end-to-end sanity bar, scaled with depth: ReLU decisions that the two
    # sides may legitimately take differently compound through the layers
    # (the elementwise parity of every layer is tested on oracle inputs)
    bar = 5e-3 * wl.layers
    pairs = [("Z_last[0]", out[:1], cache[-1][2]), ("dx[0]", dx[:1], dxr)]
    # every layer's weight and box gradients of image 0: the same stack at one
    # image (its gradients sum over that image only)
    say(f"{wl.key} full size, image 0 alone")
    st1 = Stack(1, wl.C, wl.H, wl.W, wl.B, wl.mix_out, wl.layers, "bf16", True)
    inputs1, _ = st1.forward(dev(d["x"][:1]), params)
    _, grads1 = st1.backward(inputs1, params, dev(d["grad"][:1]))
    torch.cuda.synchronize()
    for li in range(wl.layers):
        pairs += [(f"dboxes[{li}]", grads1[li][0], gr[li][0]), (f"dW[{li}]", grads1[li][1], gr[li][1])]
    for name, got, ref in pairs:
        pw, nw = O.rel_errors(host(got), ref)
        say(f"  {name}: normwise {nw:.3e}  pointwise {pw:.3e}  (bar {bar})")
        assert nw <= bar


def _sampled_mix_checks(wl, d, o_fn, dw_got, db_got, stride, ks):
    """dW columns and box-parameter gradients of sampled boxes k = c*B + b,
    summed over every image (bf16 mix operands, bounds as in bf16_bounds)."""
    B = wl.B
    g = np.ascontiguousarray(d["grad"][..., ::stride, ::stride])
    gb = O.bf16_round(g).reshape(wl.N, wl.mix_out, -1)
    for k in ks:
        c, b = divmod(k, B)
        bx = d["boxes"][c:c + 1, b:b + 1]
        o_k = o_fn(d["x"][:, c:c + 1], bx)                                    # [N, 1, Ho, Wo]
        D_k = bb.bf16_band(o_k, bb.scale_err(o_k, bb.E_F32))
        dw_ref = O.mix_backward_weight(g, o_k, compute="bf16")[:, 0]
        dw_bnd = np.einsum("nmp,np->m", np.abs(gb), D_k.reshape(wl.N, -1))   # the codes of o_k
        check_bounded(dw_got[:, k], dw_ref, dw_bnd, RTOL_BF16, f"dW[:, {k}]")
        if db_got is not None:
            # dO of this box is an fp32 result of the same bf16 operands on both
            # sides, so its box-parameter gradient takes the fp32 bar
            do_k = O.mix_backward_data(d["w"][:, k:k + 1], g, compute="bf16")
            db_ref = O.box_backward_params(d["x"][:, c:c + 1], do_k, bx, stride=stride)[0, 0]
            pw = np.abs(db_got[c, b] - db_ref) / (np.abs(db_ref) + np.sqrt(np.mean(db_ref ** 2)))
            say(f"  dboxes[{c},{b}]: {pw.max():.3e}")
            assert pw.max() <= RTOL_F32


def test_pose_layer_inference_full_size_sampled():
    """The inference forward bench.py --inference times: boxes with integer
    corners, bf16 filtered maps, bf16 mix; images 0 and N-1 of O and Z."""
    wl = wlmod.WORKLOADS[3]
    d = wlmod.make_inputs(wl)
    say(f"{wl.key} inference full size")
    plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, torch.float32, wl.mix_dtype, wl.relu,
                     bc.BC_FLAG_INTEGER_CORNERS, False)
    z = plan.forward(dev(d["x"]), dev(d["boxes"]), dev(d["w"]))
    torch.cuda.synchronize()
    wb = O.bf16_round(d["w"])
    for n in (0, wl.N - 1):
        o = O.box_forward(d["x"][n:n + 1], d["boxes"], integer_corners=True)
        D = bb.bf16_band(o, bb.scale_err(o, bb.E_F32))
        check_bounded(host(plan.o[n:n + 1]), O.bf16_round(o), D, RTOL_BF16, f"O[{n}] (bf16)")
        zr = O.mix_forward(d["w"], o, compute="bf16")
        ez = np.einsum("mk,nkhw->nmhw", np.abs(wb), D, optimize=True)
        check_bounded(host(z[n:n + 1]), zr, ez, RTOL_BF16, f"Z[{n}]")


def test_pose_layer_stride2_full_size_sampled():
    """The strided layer bench.py --stride 2 times: images 0 and N-1 of O, Z,
    dO and dx; dW columns and box-parameter gradients of sampled boxes."""
    wl = wlmod.WORKLOADS[3]
    d = wlmod.make_inputs(wl)
    s = 2
    say(f"{wl.key} stride {s} full size")
    plan = LayerPlan(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, torch.float32, wl.mix_dtype, wl.relu, 0, True,
                     stride=s)
    xd, bd, wd = dev(d["x"]), dev(d["boxes"]), dev(d["w"])
    g = np.ascontiguousarray(d["grad"][..., ::s, ::s])
    z = plan.forward(xd, bd, wd)
    dx, db, dw = plan.backward(xd, bd, wd, dev(g))
    torch.cuda.synchronize()
    wb = O.bf16_round(d["w"])
    for n in (0, wl.N - 1):
        o = O.box_forward(d["x"][n:n + 1], d["boxes"], stride=s)
        D = bb.bf16_band(o, bb.scale_err(o, bb.E_F32))
        check_bounded(host(plan.o[n:n + 1]), O.bf16_round(o), D, RTOL_BF16, f"O[{n}] (bf16)")
        zr = O.mix_forward(d["w"], o, compute="bf16")
        ez = np.einsum("mk,nkhw->nmhw", np.abs(wb), D, optimize=True)
        check_bounded(host(z[n:n + 1]), zr, ez, RTOL_BF16, f"Z[{n}]")
        do = O.mix_backward_data(d["w"], g[n:n + 1], compute="bf16")
        check(host(plan.do[n:n + 1]), do, RTOL_F32, f"dO[{n}]")
        check(host(dx[n:n + 1]), O.box_backward_input(do, d["boxes"], wl.H, wl.W, stride=s), RTOL_F32, f"dx[{n}]")
    ks = sorted(np.random.default_rng(8).choice(wl.C * wl.B, size=8, replace=False).tolist())
    _sampled_mix_checks(wl, d, lambda x, bx: O.box_forward(x, bx, stride=s), host(dw), host(db), s, ks)
