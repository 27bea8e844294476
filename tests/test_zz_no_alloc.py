"""The box backward entry point that allocates nothing (box_conv_bwd_noalloc,
its workspace in the library's fixed device array) against box_conv_bwd with
a caller-allocated workspace, through the C ABI: two calls in a row, the
second with a smaller input (the array keeps the first call's contents), plus
the oracle on the second."""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from paper_1906_11367_amd import boxconv as bc

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _case(rng, N, C, H, W, B):
    x = np.abs(rng.standard_normal((N, C, H, W))).astype(np.float32)
    g = rng.standard_normal((N, C * B, H, W)).astype(np.float32)
    bx = np.empty((C, B, 4), dtype=np.float32)
    bx[..., :2] = rng.uniform(-16, 16, size=(C, B, 2))
    bx[..., 2:] = rng.uniform(0.5, 32, size=(C, B, 2))
    return x, g, bx


def test_noalloc_backward_matches_allocating_backward():
    rng = np.random.default_rng(300)
    assert bc.noalloc_scratch_bytes() == 16 << 20
    # maps whose table fits in LDS, then 200 x 256 maps (streaming kernels,
    # no table in the workspace), then a small ragged case
    for shape in [(8, 64, 64, 48, 4), (1, 8, 200, 256, 8), (2, 5, 37, 29, 3)]:
        N, C, H, W, B = shape
        say(f"noalloc backward {shape}")
        x, g, bx = _case(rng, *shape)
        assert bc.box_workspace_bytes(1, N, C, H, W, B) <= bc.noalloc_scratch_bytes()
        xd, gd, bd = dev(x), dev(g), dev(bx)
        gx_ref = torch.empty((N, C, H, W), dtype=torch.float32, device="cuda")
        gb_ref = torch.empty((C, B, 4), dtype=torch.float32, device="cuda")
        bc.box_conv_bwd(xd, bd, gd, gx_ref, gb_ref)
        gx = torch.full((N, C, H, W), float("nan"), dtype=torch.float32, device="cuda")
        gb = torch.full((C, B, 4), float("nan"), dtype=torch.float32, device="cuda")
        bc.box_conv_bwd_noalloc(xd, bd, gd, gx, gb)
        torch.cuda.synchronize()
        # the same kernels on the same inputs: bit for bit
        assert torch.equal(gx, gx_ref)
        assert torch.equal(gb, gb_ref)
    # the second, smaller call against the oracle as well (fp32 bar)
    for got, want in [(gx, O.box_backward_input(g, bx, H, W)), (gb, O.box_backward_params(x, g, bx))]:
        pw, _ = O.rel_errors(got.cpu().numpy(), want)
        say(f"  oracle: pointwise {pw:.3e}")
        assert pw <= 1e-4
    # input gradient only
    gx2 = torch.empty_like(gx)
    bc.box_conv_bwd_noalloc(xd, bd, gd, gx2, None)
    torch.cuda.synchronize()
    assert torch.equal(gx2, gx_ref)


def test_noalloc_backward_rejects_oversized_requests():
    # 256 x 256 maps with their gradient tables forced into HBM: far beyond the array
    N, C, H, W, B = 4, 128, 256, 256, 8
    assert bc.box_workspace_bytes(1, N, C, H, W, B, bc.BC_FLAG_FORCE_HBM) > bc.noalloc_scratch_bytes()
    x = torch.zeros((1, C, 8, 8), dtype=torch.float32, device="cuda")   # never read: rejected first
    st = bc.load_library().box_conv_bwd_noalloc(bc._ptr(x), bc._ptr(x), bc._ptr(x), N, C, H, W, B,
                                                bc._ptr(x), None, bc.BC_FLAG_FORCE_HBM, bc._stream())
    assert st == 5   # BC_ERR_WORKSPACE
