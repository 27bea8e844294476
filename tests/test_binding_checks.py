"""The Python binding rejects tensors whose shape or dtype the C ABI cannot
check (it receives only pointers), before any pointer is taken: a wrong-sized
or wrong-typed buffer would otherwise be read or written out of bounds on the
device.  CPU tensors are used, so every check must fire before the binding
asks for a device pointer."""
import pytest
import torch

from paper_1906_11367_amd import boxconv as bc

E = bc.BoxConvError
f32, bf16, i32 = torch.float32, torch.bfloat16, torch.int32


def t(*shape, dtype=f32):
    return torch.zeros(shape, dtype=dtype)


N, C, H, W, B = 2, 3, 8, 6, 4


def good_fwd():
    return dict(x=t(N, C, H, W), boxes=t(C, B, 4), y=t(N, C * B, H, W))


@pytest.mark.parametrize("bad", [
    dict(boxes=t(C + 1, B, 4)),            # boxes for the wrong channel count
    dict(boxes=t(C, B, 3)),                # not 4 parameters
    dict(boxes=t(C, B, 4, dtype=bf16)),    # not fp32
    dict(y=t(N, C * B, H, W + 1)),         # output of the wrong size
    dict(y=t(N, C * B, H, W, dtype=i32)),  # int output for fp32 maps
    dict(x=t(C, H, W)),                    # not 4-D
])
def test_box_conv_fwd_rejects(bad):
    a = good_fwd()
    a.update(bad)
    with pytest.raises(E):
        bc.box_conv_fwd(a["x"], a["boxes"], a["y"])


def test_box_conv_fwd_int_maps_need_int_output():
    with pytest.raises(E):
        bc.box_conv_fwd(t(N, C, H, W, dtype=i32), t(C, B, 4), t(N, C * B, H, W))


@pytest.mark.parametrize("bad", [
    dict(grad_x=t(N, C, H, W, dtype=bf16)),   # bf16 grad_x would take fp32 stores at twice its size
    dict(grad_x=t(N, C + 1, H, W)),
    dict(grad_boxes=t(C, B + 1, 4)),
    dict(grad_boxes=t(C, B, 4, dtype=bf16)),
    dict(grad_y=t(N, C * B, H, W - 1)),
    dict(grad_y=t(N, C * B, H, W, dtype=bf16)),
    dict(boxes=t(C, B, 4, dtype=torch.float64)),
    dict(x=t(N, C, H, W, dtype=i32)),          # the backward takes fp32 maps
])
def test_box_conv_bwd_rejects(bad):
    a = dict(x=t(N, C, H, W), boxes=t(C, B, 4), grad_y=t(N, C * B, H, W), grad_x=t(N, C, H, W),
             grad_boxes=t(C, B, 4))
    a.update(bad)
    with pytest.raises(E):
        bc.box_conv_bwd(a["x"], a["boxes"], a["grad_y"], a["grad_x"], a["grad_boxes"])


def test_box_conv_bwd_relu_bf16_rejects_fp32_grad_x():
    with pytest.raises(E):
        bc.box_conv_bwd_relu_bf16(t(N, C, H, W), t(C, B, 4), t(N, C * B, H, W), t(N, C, H, W), t(C, B, 4))


def test_strided_shapes_checked():
    s = 2
    with pytest.raises(E):   # the full-size grid instead of the strided one
        bc.box_conv_bwd(t(N, C, H, W), t(C, B, 4), t(N, C * B, H, W), t(N, C, H, W), None, stride=s)
    with pytest.raises(E):
        bc.box_conv_fwd(t(N, C, H, W), t(C, B, 4), t(N, C * B, H, W), stride=s)


@pytest.mark.parametrize("mode,shapes", [
    (bc.BC_MIX_FWD, dict(a=(5, 12), b=(N, 12, 7), out=(N, 5, 8))),        # out too large
    (bc.BC_MIX_FWD, dict(a=(5, 11), b=(N, 12, 7), out=(N, 5, 7))),        # w of the wrong size
    (bc.BC_MIX_BWD_DATA, dict(a=(5, 12), b=(N, 5, 7), out=(N, 12, 6))),
    (bc.BC_MIX_BWD_WEIGHT, dict(a=(N, 5, 7), b=(N, 12, 7), out=(5, 13))),
])
def test_pointwise_mix_rejects_sizes(mode, shapes):
    a, b, out = (t(*shapes[k]) for k in ("a", "b", "out"))
    with pytest.raises(E):
        bc.pointwise_mix(mode, a, b, out, N, 5, 12, 7, bc.BC_F32)


def test_pointwise_mix_rejects_dtypes_and_aux():
    M, K, P = 5, 12, 7
    with pytest.raises(E):   # bf16 output
        bc.pointwise_mix(bc.BC_MIX_FWD, t(M, K), t(N, K, P), t(N, M, P, dtype=bf16), N, M, K, P, bc.BC_BF16)
    with pytest.raises(E):   # aux of the wrong size
        bc.pointwise_mix(bc.BC_MIX_BWD_DATA, t(M, K), t(N, M, P), t(N, K, P), N, M, K, P, bc.BC_F32,
                         relu=1, aux=t(N, M, P + 1))
    with pytest.raises(E):
        bc.pointwise_mix(9, t(M, K), t(N, K, P), t(N, M, P), N, M, K, P, bc.BC_F32)


def test_other_entry_points_reject():
    with pytest.raises(E):
        bc.sat_build(t(N, C, H, W), t(N, C, H, W + 1))
    with pytest.raises(E):
        bc.sat_build(t(N, C, H, W), t(N, C, H + 1, W + 1, dtype=i32))
    with pytest.raises(E):
        bc.sat_build(t(N, C, H, W), t(N, C, H + 1, W + 1), mean=t(N, C + 1))
    with pytest.raises(E):
        bc.box_prep(t(C, B, 4), t(2 * C * B * 16 - 1, dtype=i32))
    with pytest.raises(E):
        bc.box_params_from_unit(t(C, B, 4), 8.0, 8.0, t(C, B + 1, 4))
    with pytest.raises(E):
        bc.box_params_unit_grad(t(C, B, 4), 8.0, 8.0, t(C, B, 4, dtype=bf16))
    with pytest.raises(E):
        bc.bc_cast_bf16(t(10), t(10))
    with pytest.raises(E):
        bc.box_conv_split_fwd(t(N, C, H, W), t(C, B, 4), t(C, B, 2), "4", t(N, C * B, H, W))
    with pytest.raises(E):
        bc.box_conv_split_bwd(t(N, C, H, W), t(C, B, 4), t(C, B, 4), "4", t(N, C * B, H, W),
                              t(N, C, H, W), t(C, B, 4), t(C, B, 2))
