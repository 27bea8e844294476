"""The algorithmic bytes and FLOPs bench.py divides by the measured times
(the roofline numerators), checked against their closed forms at the
pose-shaped layer: N=32, C=256, 64x48 maps, B=4, mix 1024 -> 256 in bf16.
No GPU needed."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_1906_11367_amd import workloads as wlmod  # noqa: E402

MB = 1 << 20


def test_pose_layer_call_costs():
    wl = wlmod.WORKLOADS[3]
    px = 32 * 256 * 64 * 48              # input pixels
    pb = px * 4                          # output pixel*box
    nz = 32 * 256 * 64 * 48              # mix outputs
    c = bench.call_cost("box_conv_fwd", wl, 2)
    assert c == {"bound": "hbm", "bytes": 4 * px + 2 * pb}                # x read, bf16 O written
    assert c["bytes"] == 301_989_888                                      # 302.0 MB
    c = bench.call_cost("box_conv_bwd", wl, 2)
    assert c["bytes"] == 4 * px + 4 * pb + 4 * px == 603_979_776          # x, dO read; dx written
    c = bench.call_cost("mix_fwd", wl, 2)
    assert c["bound"] == "mfma" and c["flops"] == 2 * 32 * 256 * 1024 * 64 * 48
    assert c["bytes"] == 2 * pb + 4 * nz                                  # O read, Z written
    # the layer casts dZ to bf16 once for both backward GEMMs of a bf16 mix
    assert bench.call_cost("grad_cast", wl, 2)["bytes"] == 6 * nz          # fp32 read, bf16 written
    assert bench.call_cost("mix_bwd_data", wl, 2)["bytes"] == 2 * nz + 4 * pb
    assert bench.call_cost("mix_bwd_weight", wl, 2)["bytes"] == 2 * nz + 2 * pb


def test_stacked_relu_call_costs():
    wl = wlmod.WORKLOADS[5]
    px = 32 * 256 * 64 * 48
    pb = px * 4
    nz = 32 * 256 * 64 * 48
    assert bench.call_cost("relu_grad", wl, 2)["bytes"] == 10 * nz        # dZ, Z read; bf16 written
    assert bench.call_cost("mix_bwd_data", wl, 2)["bytes"] == 2 * nz + 4 * pb
    assert bench.call_cost("box_conv_bwd_relu_bf16", wl, 2)["bytes"] == 4 * px + 4 * pb + 2 * px


def test_strided_costs_count_the_output_grid():
    wl = wlmod.WORKLOADS[3]
    px = 32 * 256 * 64 * 48
    pb2 = 32 * 256 * 4 * 32 * 24           # outputs at stride 2
    assert bench.call_cost("box_conv_fwd", wl, 2, stride=2)["bytes"] == 4 * px + 2 * pb2
