"""Host-only checks of the C ABI: the library loads, exports every entry point
that include/boxconv.h declares, and rejects bad arguments before launching
anything (no kernel runs in these tests, so they need no GPU)."""
import ctypes
import os
import re

import pytest

from paper_1906_11367_amd import boxconv as bc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "boxconv.h")

pytestmark = pytest.mark.skipif(not os.path.exists(bc.LIB_PATH), reason="libboxconv.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([a-z_][a-z0-9_]*)\s*\(",
                       text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_four_entry_points():
    names = declared_functions()
    for n in ("sat_build", "box_conv_fwd", "box_conv_bwd", "pointwise_mix", "box_prep",
              "bc_box_workspace_bytes", "bc_box_workspace_bytes_strided", "bc_mix_workspace_bytes", "bc_status_string", "bc_abi_version",
              "box_conv_split_fwd", "box_conv_split_bwd", "bc_split_workspace_bytes"):
        assert n in names, n


def test_library_exports_every_declared_symbol():
    lib = bc.load_library()
    for n in declared_functions():
        assert hasattr(lib, n), f"missing export {n}"
        assert n in bc.SIGNATURES, f"binding lacks a signature for {n}"


def test_status_strings_and_version():
    lib = bc.load_library()
    assert lib.bc_abi_version() == 2
    for s in range(8):
        assert lib.bc_status_string(s)
    assert lib.bc_status_string(99) == b"unknown status"


FAKE = ctypes.c_void_p(0x100000)        # never dereferenced: every call below fails validation
FAKE_MISALIGNED = ctypes.c_void_p(0x100004)


def test_fwd_argument_errors():
    lib = bc.load_library()
    ok = (FAKE, bc.BC_F32, FAKE, 2, 3, 8, 8, 4, FAKE, bc.BC_F32, 0, None, 0, None)
    assert lib.box_conv_fwd(None, *ok[1:]) == 1
    a = list(ok); a[2] = None
    assert lib.box_conv_fwd(*a) == 1
    for idx in (3, 4, 5, 6, 7):
        a = list(ok); a[idx] = 0
        assert lib.box_conv_fwd(*a) == 2
    a = list(ok); a[1] = bc.BC_BF16
    assert lib.box_conv_fwd(*a) == 3
    a = list(ok); a[1] = bc.BC_I32          # int input needs int output
    assert lib.box_conv_fwd(*a) == 3
    a = list(ok); a[1] = bc.BC_I32; a[9] = bc.BC_I32; a[10] = bc.BC_FLAG_MEAN_OFFSET
    assert lib.box_conv_fwd(*a) == 3
    a = list(ok); a[0] = FAKE_MISALIGNED
    assert lib.box_conv_fwd(*a) == 4
    a = list(ok); a[10] = 1 << 7
    assert lib.box_conv_fwd(*a) == 7
    a = list(ok); a[10] = bc.BC_FLAG_INTEGER_CORNERS   # accepted: fails only for lack of a workspace
    assert lib.box_conv_fwd(*a) == 5
    # every forward needs a workspace (the boxes' tap records), larger when a
    # map's table does not fit LDS
    assert lib.box_conv_fwd(*ok) == 5
    a = list(ok); a[11] = FAKE; a[12] = 16
    assert lib.box_conv_fwd(*a) == 5
    a = list(ok); a[5] = 300; a[6] = 300
    a[11] = FAKE; a[12] = lib.bc_box_workspace_bytes(0, 2, 3, 8, 8, 4, 0)
    assert lib.box_conv_fwd(*a) == 5
    a = list(ok); a[10] = bc.BC_FLAG_FORCE_HBM
    assert lib.box_conv_fwd(*a) == 5


def test_bwd_argument_errors():
    lib = bc.load_library()
    ok = [FAKE, FAKE, FAKE, 2, 3, 8, 8, 4, FAKE, FAKE, 0, None, 0, None]
    assert lib.box_conv_bwd(*([None] + ok[1:])) == 1
    a = list(ok); a[7] = -1
    assert lib.box_conv_bwd(*a) == 2
    assert lib.box_conv_bwd(*ok) == 5      # workspace required (gradient partials)
    a = list(ok); a[11] = FAKE; a[12] = 1
    assert lib.box_conv_bwd(*a) == 5
    a = list(ok); a[8] = FAKE_MISALIGNED
    assert lib.box_conv_bwd(*a) == 4
    a = list(ok); a[8] = None; a[9] = None  # nothing requested: no-op
    assert lib.box_conv_bwd(*a) == 0
    # rounded corners are not differentiable: no box gradient with them
    a = list(ok); a[10] = bc.BC_FLAG_INTEGER_CORNERS
    assert lib.box_conv_bwd(*a) == 7
    a[9] = None                             # grad_x only: fails only for lack of a workspace
    assert lib.box_conv_bwd(*a) == 5


def test_strided_argument_errors():
    lib = bc.load_library()
    fwd = [FAKE, bc.BC_F32, FAKE, 2, 3, 8, 8, 4, 2, FAKE, bc.BC_F32, 0, None, 0, None]
    bwd = [FAKE, FAKE, FAKE, 2, 3, 8, 8, 4, 2, FAKE, FAKE, 0, None, 0, None]
    for args, fn in ((fwd, lib.box_conv_fwd_strided), (bwd, lib.box_conv_bwd_strided)):
        assert fn(*args) == 5                  # valid stride: fails only for lack of a workspace
        for bad in (0, -1, 1025):
            a = list(args); a[8] = bad
            assert fn(*a) == 2, bad
        a = list(args); a[0] = None
        assert fn(*a) == 1


def test_unit_params_argument_errors():
    lib = bc.load_library()
    assert lib.box_params_from_unit(None, 2, 4, 64.0, 48.0, FAKE, None) == 1
    assert lib.box_params_from_unit(FAKE, 0, 4, 64.0, 48.0, FAKE, None) == 2
    assert lib.box_params_from_unit(FAKE, 2, 4, 0.0, 48.0, FAKE, None) == 2
    assert lib.box_params_from_unit(FAKE, 2, 4, 64.0, 48.0, FAKE_MISALIGNED, None) == 4
    assert lib.box_params_unit_grad(FAKE, 2, 4, 64.0, -1.0, FAKE, None) == 2
    assert lib.box_params_unit_grad(FAKE, 2, 4, 64.0, 48.0, None, None) == 1
    assert lib.box_params_clip(None, 2, 4, None) == 1
    assert lib.box_params_clip(FAKE_MISALIGNED, 2, 4, None) == 4


def test_bwd_relu_bf16_argument_errors():
    lib = bc.load_library()
    ok = [FAKE, FAKE, FAKE, 2, 3, 8, 8, 4, 1, FAKE, FAKE, 0, None, 0, None]
    assert lib.box_conv_bwd_relu_bf16(*ok) == 5                        # valid: workspace missing
    a = list(ok); a[0] = None
    assert lib.box_conv_bwd_relu_bf16(*a) == 1
    a = list(ok); a[8] = 0
    assert lib.box_conv_bwd_relu_bf16(*a) == 2                         # stride
    a = list(ok); a[10] = None; a[11] = bc.BC_FLAG_INTEGER_CORNERS     # the mask needs x: not with rounded corners
    assert lib.box_conv_bwd_relu_bf16(*a) == 7
    a = list(ok); a[9] = FAKE_MISALIGNED
    assert lib.box_conv_bwd_relu_bf16(*a) == 4
    a = list(ok); a[9] = None; a[10] = None                            # nothing requested: no-op
    assert lib.box_conv_bwd_relu_bf16(*a) == 0


def test_relu_grad_argument_errors():
    lib = bc.load_library()
    assert lib.bc_relu_grad_bf16(None, FAKE, FAKE, 8, None) == 1
    assert lib.bc_relu_grad_bf16(FAKE, None, FAKE, 8, None) == 1
    assert lib.bc_relu_grad_bf16(FAKE, FAKE, None, 8, None) == 1
    assert lib.bc_relu_grad_bf16(FAKE, FAKE, FAKE, 0, None) == 2
    assert lib.bc_relu_grad_bf16(FAKE, FAKE_MISALIGNED, FAKE, 8, None) == 4


def test_split_argument_errors():
    lib = bc.load_library()
    fwd = [FAKE, FAKE, FAKE, 2, 3, 8, 8, 4, bc.BC_SPLIT_4, FAKE, bc.BC_F32, None, 0, None]
    assert lib.box_conv_split_fwd(*fwd) == 5                 # valid: fails only for lack of a workspace
    a = list(fwd); a[2] = None
    assert lib.box_conv_split_fwd(*a) == 1                   # piece weights are required
    for bad in (0, 4, -1, bc.BC_SPLIT_FORCE_HBM, bc.BC_SPLIT_4 | 0x200):
        a = list(fwd); a[8] = bad
        assert lib.box_conv_split_fwd(*a) == 7, bad
    a = list(fwd); a[8] = bc.BC_SPLIT_4 | bc.BC_SPLIT_FORCE_HBM
    assert lib.box_conv_split_fwd(*a) == 5
    a = list(fwd); a[10] = bc.BC_I32
    assert lib.box_conv_split_fwd(*a) == 3
    a = list(fwd); a[5] = 256; a[6] = 256                  # table does not fit LDS: HBM path
    assert lib.box_conv_split_fwd(*a) == 5
    a = list(fwd); a[5] = 4; a[6] = 1025                   # fits LDS: no width limit
    assert lib.box_conv_split_fwd(*a) == 5
    a[8] = bc.BC_SPLIT_4 | bc.BC_SPLIT_FORCE_HBM            # HBM path: W up to 1024
    assert lib.box_conv_split_fwd(*a) == 2
    a = list(fwd); a[2] = FAKE_MISALIGNED
    assert lib.box_conv_split_fwd(*a) == 4
    a = list(fwd); a[11] = FAKE; a[12] = lib.bc_split_workspace_bytes(0, 2, 3, 8, 8, 4, bc.BC_SPLIT_4) - 1
    assert lib.box_conv_split_fwd(*a) == 5
    bwd = [FAKE, FAKE, FAKE, FAKE, 2, 3, 8, 8, 4, bc.BC_SPLIT_2X, FAKE, FAKE, FAKE, None, 0, None]
    assert lib.box_conv_split_bwd(*bwd) == 5
    a = list(bwd); a[10] = None; a[11] = None; a[12] = None  # nothing requested: no-op
    assert lib.box_conv_split_bwd(*a) == 0
    a = list(bwd); a[12] = FAKE_MISALIGNED
    assert lib.box_conv_split_bwd(*a) == 4
    a = list(bwd); a[9] = 9
    assert lib.box_conv_split_bwd(*a) == 7
    a = list(bwd); a[6] = 256; a[7] = 256
    assert lib.box_conv_split_bwd(*a) == 5
    a = list(bwd); a[6] = 4; a[7] = 1025                   # 342 items: one LDS block, no width limit
    assert lib.box_conv_split_bwd(*a) == 5
    a[9] = bc.BC_SPLIT_2X | bc.BC_SPLIT_FORCE_HBM          # HBM path: W up to 1024
    assert lib.box_conv_split_bwd(*a) == 2
    # workspace: one 128-byte corner record per box, and for the backward the
    # 8-word partials of every wave of every image
    assert lib.bc_split_workspace_bytes(0, 32, 256, 64, 48, 4, bc.BC_SPLIT_4) == 256 * 4 * 128
    assert lib.bc_split_workspace_bytes(0, 32, 256, 64, 48, 4, bc.BC_SPLIT_2Y) == 256 * 4 * 128
    assert lib.bc_split_workspace_bytes(1, 32, 256, 64, 48, 4, bc.BC_SPLIT_4) >= \
        256 * 4 * 128 + 32 * 256 * 4 * 32
    assert lib.bc_split_workspace_bytes(0, 4, 8, 64, 48, 4, 0) == 0
    # HBM path (table too large, or forced): the tables come first after the
    # records; the backward's are those of the N*C*B upstream-gradient maps
    tab = 257 * 257 * 4
    assert lib.bc_split_workspace_bytes(0, 4, 8, 256, 256, 4, bc.BC_SPLIT_4) >= 8 * 4 * 128 + 4 * 8 * tab
    assert lib.bc_split_workspace_bytes(1, 4, 8, 256, 256, 4, bc.BC_SPLIT_4) >= 8 * 4 * 128 + 4 * 8 * 4 * tab
    forced = bc.BC_SPLIT_4 | bc.BC_SPLIT_FORCE_HBM
    assert lib.bc_split_workspace_bytes(0, 32, 256, 64, 48, 4, forced) >= 256 * 4 * 128 + 32 * 256 * 65 * 49 * 4
    assert lib.bc_split_workspace_bytes(0, 4, 8, 4, 1025, 4, forced) == 0
    assert lib.bc_split_workspace_bytes(1, 4, 8, 4, 1025, 4, forced) == 0
    assert lib.bc_split_workspace_bytes(1, 4, 8, 4, 1025, 4, bc.BC_SPLIT_4) > 0


def test_mix_argument_errors():
    lib = bc.load_library()
    ok = [bc.BC_MIX_FWD, FAKE, bc.BC_F32, FAKE, bc.BC_F32, FAKE, bc.BC_F32, 2, 64, 512, 3072, bc.BC_F32,
          0, None, 0, None, 0, None]
    a = list(ok); a[1] = None
    assert lib.pointwise_mix(*a) == 1
    a = list(ok); a[0] = 9
    assert lib.pointwise_mix(*a) == 7
    a = list(ok); a[8] = 0
    assert lib.pointwise_mix(*a) == 2
    a = list(ok); a[2] = bc.BC_BF16           # bf16 storage needs bf16 compute
    assert lib.pointwise_mix(*a) == 3
    a = list(ok); a[2] = bc.BC_I32            # mixed int / float operands
    assert lib.pointwise_mix(*a) == 3
    a = list(ok); a[0] = bc.BC_MIX_BWD_DATA; a[12] = 1   # relu without aux
    assert lib.pointwise_mix(*a) == 1
    a = list(ok); a[14] = 1                   # accumulate is BWD_WEIGHT only
    assert lib.pointwise_mix(*a) == 7
    a = list(ok); a[5] = FAKE_MISALIGNED
    assert lib.pointwise_mix(*a) == 4
    a = list(ok); a[0] = bc.BC_MIX_BWD_WEIGHT  # split-K partials need a workspace
    assert lib.pointwise_mix(*a) == 5


def test_sat_and_prep_argument_errors():
    lib = bc.load_library()
    assert lib.sat_build(FAKE, bc.BC_F32, FAKE, None, 1, 1, 8, 2000, None) == 2   # W > 1024
    assert lib.sat_build(FAKE, bc.BC_BF16, FAKE, None, 1, 1, 8, 8, None) == 3
    assert lib.sat_build(FAKE, bc.BC_I32, FAKE, FAKE, 1, 1, 8, 8, None) == 3      # mean needs fp32
    assert lib.sat_build(None, bc.BC_F32, FAKE, None, 1, 1, 8, 8, None) == 1
    assert lib.box_prep(FAKE, 0, 4, 0, FAKE, None) == 2
    assert lib.box_prep(FAKE_MISALIGNED, 2, 4, 0, FAKE, None) == 4
    assert lib.box_prep(FAKE, 2, 4, bc.BC_FLAG_MEAN_OFFSET, FAKE, None) == 7      # only INTEGER_CORNERS
    assert lib.box_prep(None, 2, 4, bc.BC_FLAG_INTEGER_CORNERS, FAKE, None) == 1


def test_workspace_queries():
    lib = bc.load_library()
    # 64x48 maps: tables fit LDS -> the forward needs the tap records only (2 per
    # box, 64 bytes each); the backward also needs its gradient partials
    taps = 2 * 256 * 4 * 64
    assert lib.bc_box_workspace_bytes(0, 32, 256, 64, 48, 4, 0) == taps
    assert lib.bc_box_workspace_bytes(1, 32, 256, 64, 48, 4, 0) >= taps + 32 * 256 * 4 * 16
    # the LDS backward's partials: one row per wave and image.  A call with
    # enough maps for 2048 waves of 8-row items takes them (two waves per
    # 64x48 map); fewer maps take 4-row items (four waves per map)
    a256 = lambda v: (v + 255) // 256 * 256
    for N, waves in ((32, 2), (4, 2), (3, 4), (1, 4)):
        assert lib.bc_box_workspace_bytes(1, N, 256, 64, 48, 4, 0) == a256(taps) + a256(N * waves * 256 * 4 * 16)
    # 256x256 maps take the streaming kernels: tap records plus one row of
    # edge-gradient partials per image, no tables
    assert lib.bc_box_workspace_bytes(0, 4, 128, 256, 256, 8, 0) == 2 * 128 * 8 * 64
    stream_bwd = lib.bc_box_workspace_bytes(1, 4, 128, 256, 256, 8, 0)
    assert 2 * 128 * 8 * 64 < stream_bwd < 1 << 20
    # the forced HBM path needs the tables in the workspace
    assert lib.bc_box_workspace_bytes(0, 4, 128, 256, 256, 8, bc.BC_FLAG_FORCE_HBM) >= 4 * 128 * 257 * 257 * 4
    assert lib.bc_box_workspace_bytes(0, 2, 3, 8, 8, 4, bc.BC_FLAG_FORCE_HBM) >= 2 * 3 * 81 * 4
    assert lib.bc_box_workspace_bytes(1, 4, 128, 256, 256, 8, bc.BC_FLAG_FORCE_HBM) >= 4 * 128 * 8 * 257 * 257 * 4
    # maps wider than the streaming kernels take (W > 256) need HBM tables
    assert lib.bc_box_workspace_bytes(0, 1, 4, 128, 300, 4, 0) >= 4 * 129 * 301 * 4
    # the strided query prices the path the strided call takes; stride 1 is the plain query
    for op in (0, 1):
        assert (lib.bc_box_workspace_bytes_strided(op, 4, 128, 256, 256, 8, 1, 0)
                == lib.bc_box_workspace_bytes(op, 4, 128, 256, 256, 8, 0))
    assert lib.bc_box_workspace_bytes_strided(0, 4, 128, 256, 256, 8, 0, 0) == 0
    assert lib.bc_mix_workspace_bytes(bc.BC_MIX_FWD, 32, 256, 1024, 3072, bc.BC_BF16) == 0
    assert lib.bc_mix_workspace_bytes(bc.BC_MIX_BWD_WEIGHT, 32, 256, 1024, 3072, bc.BC_BF16) > 0
    # bf16 BWD_DATA keeps w^T in MFMA operand order: K x M bf16, both sides
    # rounded up to 64; fp32 compute and wide M take the tiled GEMM (none)
    assert lib.bc_mix_workspace_bytes(bc.BC_MIX_BWD_DATA, 32, 256, 1024, 3072, bc.BC_BF16) == 1024 * 256 * 2
    assert lib.bc_mix_workspace_bytes(bc.BC_MIX_BWD_DATA, 2, 100, 70, 50, bc.BC_BF16) == 128 * 128 * 2
    assert lib.bc_mix_workspace_bytes(bc.BC_MIX_BWD_DATA, 32, 256, 1024, 3072, bc.BC_F32) == 0
    assert lib.bc_mix_workspace_bytes(bc.BC_MIX_BWD_DATA, 2, 512, 64, 64, bc.BC_BF16) == 0
    # a missing or short workspace is refused before any launch
    assert lib.pointwise_mix(bc.BC_MIX_BWD_DATA, FAKE, bc.BC_BF16, FAKE, bc.BC_F32, FAKE, bc.BC_F32, 32, 256,
                             1024, 3072, bc.BC_BF16, 0, None, 0, None, 0, None) == 5
    assert lib.pointwise_mix(bc.BC_MIX_BWD_DATA, FAKE, bc.BC_BF16, FAKE, bc.BC_F32, FAKE, bc.BC_F32, 32, 256,
                             1024, 3072, bc.BC_BF16, 0, None, 0, FAKE, 1024, None) == 5


def test_noalloc_backward_rejects_oversized_request_before_any_launch():
    """box_conv_bwd_noalloc compares the request's workspace with its fixed
    array first: 256 x 256 maps (tables in HBM) are rejected on the host."""
    lib = bc.load_library()
    assert lib.bc_noalloc_scratch_bytes() == 16 << 20
    F = bc.BC_FLAG_FORCE_HBM
    need = lib.bc_box_workspace_bytes(1, 4, 128, 256, 256, 8, F)
    assert need > lib.bc_noalloc_scratch_bytes()
    assert lib.box_conv_bwd_noalloc(FAKE, FAKE, FAKE, 4, 128, 256, 256, 8, FAKE, FAKE, F, None) == 5
    # invalid sizes are reported as such
    assert lib.box_conv_bwd_noalloc(FAKE, FAKE, FAKE, 0, 128, 64, 48, 4, FAKE, FAKE, 0, None) == 2
