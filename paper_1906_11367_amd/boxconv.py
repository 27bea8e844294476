"""Thin ctypes binding of libboxconv.so (C ABI: include/boxconv.h).

Argument marshalling only: tensors are passed as device pointers together with
torch's current HIP stream; every step of the layer runs in the library's
kernels.  The library is required: if it is not built, or a GPU is not
present, the calls raise -- there is no fallback implementation.

Entry points (same names as the C ABI): box_prep, sat_build, box_conv_fwd,
box_conv_bwd, box_conv_fwd_strided, box_conv_bwd_strided, pointwise_mix, the
box-parameter reparameterisation (box_params_from_unit, box_params_unit_grad,
box_params_clip), kernel splitting (box_conv_split_fwd, box_conv_split_bwd),
the bf16 helpers (bc_cast_bf16, bc_relu_grad_bf16), plus the workspace-size
queries.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libboxconv.so")

BC_I32, BC_F32, BC_BF16 = 0, 1, 2
BC_MIX_FWD, BC_MIX_BWD_DATA, BC_MIX_BWD_WEIGHT = 0, 1, 2
BC_FLAG_MEAN_OFFSET, BC_FLAG_FORCE_HBM, BC_FLAG_INTEGER_CORNERS = 1, 2, 4
BC_SPLIT_2X, BC_SPLIT_2Y, BC_SPLIT_4 = 1, 2, 3
BC_SPLIT_FORCE_HBM = 0x100
STATUS = {0: "BC_OK", 1: "BC_ERR_NULL", 2: "BC_ERR_SHAPE", 3: "BC_ERR_DTYPE", 4: "BC_ERR_ALIGN",
          5: "BC_ERR_WORKSPACE", 6: "BC_ERR_HIP", 7: "BC_ERR_UNSUPPORTED"}

# Exported symbols and their C signatures (kept in step with boxconv.h).
_vp, _i, _u, _sz, _f = ctypes.c_void_p, ctypes.c_int, ctypes.c_uint, ctypes.c_size_t, ctypes.c_float
SIGNATURES = {
    "box_prep": (_i, [_vp, _i, _i, _u, _vp, _vp]),
    "sat_build": (_i, [_vp, _i, _vp, _vp, _i, _i, _i, _i, _vp]),
    "box_conv_fwd": (_i, [_vp, _i, _vp, _i, _i, _i, _i, _i, _vp, _i, _u, _vp, _sz, _vp]),
    "box_conv_bwd": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp, _vp, _u, _vp, _sz, _vp]),
    "box_conv_fwd_strided": (_i, [_vp, _i, _vp, _i, _i, _i, _i, _i, _i, _vp, _i, _u, _vp, _sz, _vp]),
    "box_params_from_unit": (_i, [_vp, _i, _i, _f, _f, _vp, _vp]),
    "box_params_unit_grad": (_i, [_vp, _i, _i, _f, _f, _vp, _vp]),
    "box_params_clip": (_i, [_vp, _i, _i, _vp]),
    "box_conv_bwd_strided": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _vp, _u, _vp, _sz, _vp]),
    "pointwise_mix": (_i, [_i, _vp, _i, _vp, _i, _vp, _i, _i, _i, _i, _i, _i, _i, _vp, _i, _vp, _sz, _vp]),
    "box_conv_split_fwd": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _i, _vp, _sz, _vp]),
    "box_conv_split_bwd": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _sz, _vp]),
    "bc_split_workspace_bytes": (_sz, [_i, _i, _i, _i, _i, _i, _i]),
    "bc_box_workspace_bytes": (_sz, [_i, _i, _i, _i, _i, _i, _u]),
    "bc_box_workspace_bytes_strided": (_sz, [_i, _i, _i, _i, _i, _i, _i, _u]),
    "bc_mix_workspace_bytes": (_sz, [_i, _i, _i, _i, _i, _i]),
    "bc_cast_bf16": (_i, [_vp, _vp, _sz, _vp]),
    "bc_relu_grad_bf16": (_i, [_vp, _vp, _vp, _sz, _vp]),
    "box_conv_bwd_relu_bf16": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _vp, _u, _vp, _sz, _vp]),
    "box_conv_bwd_noalloc": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp, _vp, _u, _vp]),
    "bc_noalloc_scratch_bytes": (_sz, []),
    "bc_status_string": (ctypes.c_char_p, [_i]),
    "bc_abi_version": (_i, []),
}

_lib = None


class BoxConvError(RuntimeError):
    pass


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libboxconv.so (no GPU needed to load it)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise BoxConvError(f"{path} is not built: run `python -m paper_1906_11367_amd.build` "
                           "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, what: str):
    if status != 0:
        msg = load_library().bc_status_string(status).decode()
        raise BoxConvError(f"{what}: {STATUS.get(status, status)} ({msg})")


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise BoxConvError("tensors must be on the GPU")
    if not t.is_contiguous():
        raise BoxConvError("tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _need(t, shape, dtypes, what, name):
    """Shape and dtype checks the C ABI cannot make (it sees only pointers):
    a tensor of the wrong size or type would be read or written out of bounds
    on the device.  shape entries of None match any extent."""
    if t is None:
        return
    if not isinstance(t, torch.Tensor):
        raise BoxConvError(f"{what}: {name} must be a tensor")
    if isinstance(dtypes, torch.dtype):
        dtypes = (dtypes,)
    if t.dtype not in dtypes:
        raise BoxConvError(f"{what}: {name} has dtype {t.dtype}, expected one of {tuple(dtypes)}")
    if shape is not None:
        if t.dim() != len(shape) or any(e is not None and int(a) != int(e) for a, e in zip(t.shape, shape)):
            raise BoxConvError(f"{what}: {name} has shape {tuple(t.shape)}, expected "
                               f"{tuple('*' if e is None else e for e in shape)}")


def _need_numel(t, n, dtypes, what, name):
    if isinstance(dtypes, torch.dtype):
        dtypes = (dtypes,)
    if t.dtype not in dtypes:
        raise BoxConvError(f"{what}: {name} has dtype {t.dtype}, expected one of {tuple(dtypes)}")
    if t.numel() != n:
        raise BoxConvError(f"{what}: {name} has {t.numel()} elements, expected {n}")


_MAPS = (torch.int32, torch.float32)
_F32 = torch.float32


def _maps_and_boxes(x, boxes, what):
    if not isinstance(x, torch.Tensor) or x.dim() != 4:
        raise BoxConvError(f"{what}: x must be a 4-D [N, C, H, W] tensor")
    _need(x, None, _MAPS, what, "x")
    N, C, H, W = (int(v) for v in x.shape)
    _need(boxes, (C, None, 4), _F32, what, "boxes")
    return N, C, H, W, int(boxes.shape[1])


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.int32:
        return BC_I32
    if t.dtype == torch.float32:
        return BC_F32
    if t.dtype == torch.bfloat16:
        return BC_BF16
    raise BoxConvError(f"unsupported dtype {t.dtype}")


def _workspace(nbytes: int, device) -> torch.Tensor | None:
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def box_workspace_bytes(op: int, N, C, H, W, B, flags=0, stride: int = 1) -> int:
    return int(load_library().bc_box_workspace_bytes_strided(op, N, C, H, W, B, stride, flags))


def mix_workspace_bytes(mode: int, N, M, K, P, compute_dt) -> int:
    return int(load_library().bc_mix_workspace_bytes(mode, N, M, K, P, compute_dt))


def box_prep(boxes: torch.Tensor, table: torch.Tensor, flags: int = 0):
    """table: int32 tensor of 2*C*B*16 words (see boxconv.h)."""
    _need(boxes, (None, None, 4), _F32, "box_prep", "boxes")
    C, B = boxes.shape[0], boxes.shape[1]
    _need_numel(table, 2 * C * B * 16, torch.int32, "box_prep", "table")
    _check(load_library().box_prep(_ptr(boxes), C, B, flags, _ptr(table), _stream()), "box_prep")
    return table


def sat_build(x: torch.Tensor, sat: torch.Tensor, mean: torch.Tensor | None = None):
    """x [N, C, H, W] int32/fp32 -> sat [N, C, H+1, W+1] (exclusive table)."""
    if not isinstance(x, torch.Tensor) or x.dim() != 4:
        raise BoxConvError("sat_build: x must be a 4-D [N, C, H, W] tensor")
    _need(x, None, _MAPS, "sat_build", "x")
    N, C, H, W = x.shape
    _need(sat, (N, C, H + 1, W + 1), x.dtype, "sat_build", "sat")
    _need(mean, (N, C), _F32, "sat_build", "mean")
    _check(load_library().sat_build(_ptr(x), dtype_code(x), _ptr(sat), _ptr(mean), N, C, H, W, _stream()),
           "sat_build")
    return sat


def _strided_shape(N, C, H, W, B, stride):
    return (N, C * B, (H + stride - 1) // stride, (W + stride - 1) // stride)


def box_conv_fwd(x: torch.Tensor, boxes: torch.Tensor, y: torch.Tensor, flags: int = 0,
                 ws: torch.Tensor | None = None, stride: int = 1):
    """x [N, C, H, W], boxes [C, B, 4] fp32 -> y [N, C*B, ceil(H/stride), ceil(W/stride)]
    (int32, fp32 or bf16); stride > 1 calls box_conv_fwd_strided."""
    N, C, H, W, B = _maps_and_boxes(x, boxes, "box_conv_fwd")
    _need(y, _strided_shape(N, C, H, W, B, stride),
          torch.int32 if x.dtype == torch.int32 else (torch.float32, torch.bfloat16), "box_conv_fwd", "y")
    if ws is None:
        ws = _workspace(box_workspace_bytes(0, N, C, H, W, B, flags, stride), x.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    lib = load_library()
    if stride == 1:
        st = lib.box_conv_fwd(_ptr(x), dtype_code(x), _ptr(boxes), N, C, H, W, B, _ptr(y), dtype_code(y), flags,
                              _ptr(ws), nbytes, _stream())
    else:
        st = lib.box_conv_fwd_strided(_ptr(x), dtype_code(x), _ptr(boxes), N, C, H, W, B, stride, _ptr(y),
                                      dtype_code(y), flags, _ptr(ws), nbytes, _stream())
    _check(st, "box_conv_fwd")
    return y


def box_conv_fwd_strided(x, boxes, stride: int, y, flags: int = 0, ws=None):
    return box_conv_fwd(x, boxes, y, flags, ws, stride)


def box_conv_bwd(x: torch.Tensor, boxes: torch.Tensor, grad_y: torch.Tensor, grad_x: torch.Tensor | None,
                 grad_boxes: torch.Tensor | None, flags: int = 0, ws: torch.Tensor | None = None, stride: int = 1):
    """grad_y [N, C*B, ceil(H/stride), ceil(W/stride)]; stride > 1 calls box_conv_bwd_strided."""
    N, C, H, W, B = _maps_and_boxes(x, boxes, "box_conv_bwd")
    _need(x, None, _F32, "box_conv_bwd", "x")
    _need(grad_y, _strided_shape(N, C, H, W, B, stride), _F32, "box_conv_bwd", "grad_y")
    _need(grad_x, (N, C, H, W), _F32, "box_conv_bwd", "grad_x")
    _need(grad_boxes, (C, B, 4), _F32, "box_conv_bwd", "grad_boxes")
    if ws is None:
        ws = _workspace(box_workspace_bytes(1, N, C, H, W, B, flags, stride), x.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    lib = load_library()
    if stride == 1:
        st = lib.box_conv_bwd(_ptr(x), _ptr(boxes), _ptr(grad_y), N, C, H, W, B, _ptr(grad_x), _ptr(grad_boxes),
                              flags, _ptr(ws), nbytes, _stream())
    else:
        st = lib.box_conv_bwd_strided(_ptr(x), _ptr(boxes), _ptr(grad_y), N, C, H, W, B, stride, _ptr(grad_x),
                                      _ptr(grad_boxes), flags, _ptr(ws), nbytes, _stream())
    _check(st, "box_conv_bwd")
    return grad_x, grad_boxes


def box_conv_bwd_relu_bf16(x: torch.Tensor, boxes: torch.Tensor, grad_y: torch.Tensor,
                           grad_x_bf16: torch.Tensor | None, grad_boxes: torch.Tensor | None, flags: int = 0,
                           ws: torch.Tensor | None = None, stride: int = 1):
    """As box_conv_bwd, with the input gradient written as bf16(x > 0 ? dL/dx : 0)
    (x: the rectified output of a bf16 mix before this layer)."""
    what = "box_conv_bwd_relu_bf16"
    N, C, H, W, B = _maps_and_boxes(x, boxes, what)
    _need(x, None, _F32, what, "x")
    _need(grad_y, _strided_shape(N, C, H, W, B, stride), _F32, what, "grad_y")
    _need(grad_x_bf16, (N, C, H, W), torch.bfloat16, what, "grad_x")
    _need(grad_boxes, (C, B, 4), _F32, what, "grad_boxes")
    if ws is None:
        ws = _workspace(box_workspace_bytes(1, N, C, H, W, B, flags, stride), x.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load_library().box_conv_bwd_relu_bf16(_ptr(x), _ptr(boxes), _ptr(grad_y), N, C, H, W, B, stride,
                                                 _ptr(grad_x_bf16), _ptr(grad_boxes), flags, _ptr(ws), nbytes,
                                                 _stream()), "box_conv_bwd_relu_bf16")
    return grad_x_bf16, grad_boxes


def box_conv_bwd_noalloc(x: torch.Tensor, boxes: torch.Tensor, grad_y: torch.Tensor, grad_x: torch.Tensor | None,
                         grad_boxes: torch.Tensor | None, flags: int = 0):
    """box_conv_bwd with the library's own fixed scratch array as workspace:
    the call allocates nothing (bc_noalloc_scratch_bytes() is the limit)."""
    what = "box_conv_bwd_noalloc"
    N, C, H, W, B = _maps_and_boxes(x, boxes, what)
    _need(x, None, _F32, what, "x")
    _need(grad_y, (N, C * B, H, W), _F32, what, "grad_y")
    _need(grad_x, (N, C, H, W), _F32, what, "grad_x")
    _need(grad_boxes, (C, B, 4), _F32, what, "grad_boxes")
    _check(load_library().box_conv_bwd_noalloc(_ptr(x), _ptr(boxes), _ptr(grad_y), N, C, H, W, B, _ptr(grad_x),
                                               _ptr(grad_boxes), flags, _stream()), what)
    return grad_x, grad_boxes


def noalloc_scratch_bytes() -> int:
    return int(load_library().bc_noalloc_scratch_bytes())


def box_conv_bwd_strided(x, boxes, grad_y, stride: int, grad_x, grad_boxes, flags: int = 0, ws=None):
    return box_conv_bwd(x, boxes, grad_y, grad_x, grad_boxes, flags, ws, stride)


def box_params_from_unit(u: torch.Tensor, max_w: float, max_h: float, boxes: torch.Tensor):
    """u [C, B, 4] unit corners -> boxes [C, B, 4] (cx, cy, rx, ry) in pixels."""
    _need(u, (None, None, 4), _F32, "box_params_from_unit", "u")
    C, B = u.shape[0], u.shape[1]
    _need(boxes, (C, B, 4), _F32, "box_params_from_unit", "boxes")
    _check(load_library().box_params_from_unit(_ptr(u), C, B, max_w, max_h, _ptr(boxes), _stream()),
           "box_params_from_unit")
    return boxes


def box_params_unit_grad(grad_boxes: torch.Tensor, max_w: float, max_h: float, grad_u: torch.Tensor):
    _need(grad_boxes, (None, None, 4), _F32, "box_params_unit_grad", "grad_boxes")
    C, B = grad_boxes.shape[0], grad_boxes.shape[1]
    _need(grad_u, (C, B, 4), _F32, "box_params_unit_grad", "grad_u")
    _check(load_library().box_params_unit_grad(_ptr(grad_boxes), C, B, max_w, max_h, _ptr(grad_u), _stream()),
           "box_params_unit_grad")
    return grad_u


def box_params_clip(u: torch.Tensor):
    _need(u, (None, None, 4), _F32, "box_params_clip", "u")
    C, B = u.shape[0], u.shape[1]
    _check(load_library().box_params_clip(_ptr(u), C, B, _stream()), "box_params_clip")
    return u


SPLIT_MODES = {"2x": BC_SPLIT_2X, "2y": BC_SPLIT_2Y, "4": BC_SPLIT_4}
SPLIT_PIECES = {BC_SPLIT_2X: 2, BC_SPLIT_2Y: 2, BC_SPLIT_4: 4}


def _split_mode(mode) -> int:
    m = SPLIT_MODES.get(mode, mode)
    if m not in SPLIT_PIECES:
        raise BoxConvError(f"unknown split mode {mode!r}")
    return m


def split_workspace_bytes(op: int, N, C, H, W, B, mode, force_hbm: bool = False) -> int:
    code = _split_mode(mode) | (BC_SPLIT_FORCE_HBM if force_hbm else 0)
    return int(load_library().bc_split_workspace_bytes(op, N, C, H, W, B, code))


def box_conv_split_fwd(x: torch.Tensor, boxes: torch.Tensor, piece_w: torch.Tensor, mode, y: torch.Tensor,
                       ws: torch.Tensor | None = None, force_hbm: bool = False):
    """x [N, C, H, W] fp32, boxes [C, B, 4], piece_w [C, B, P] -> y [N, C*B, H, W] (fp32 or bf16).
    mode: "2x", "2y", "4" or a BC_SPLIT_* code; force_hbm: take the HBM-table
    kernels even where the map's table fits in LDS."""
    m = _split_mode(mode)
    code = m | (BC_SPLIT_FORCE_HBM if force_hbm else 0)
    what = "box_conv_split_fwd"
    N, C, H, W, B = _maps_and_boxes(x, boxes, what)
    _need(x, None, _F32, what, "x")
    _need(piece_w, (C, B, SPLIT_PIECES[m]), _F32, what, "piece_w")
    _need(y, (N, C * B, H, W), (torch.float32, torch.bfloat16), what, "y")
    if ws is None:
        ws = _workspace(split_workspace_bytes(0, N, C, H, W, B, m, force_hbm), x.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load_library().box_conv_split_fwd(_ptr(x), _ptr(boxes), _ptr(piece_w), N, C, H, W, B, code, _ptr(y),
                                             dtype_code(y), _ptr(ws), nbytes, _stream()), "box_conv_split_fwd")
    return y


def box_conv_split_bwd(x: torch.Tensor, boxes: torch.Tensor, piece_w: torch.Tensor, mode, grad_y: torch.Tensor,
                       grad_x: torch.Tensor | None, grad_boxes: torch.Tensor | None,
                       grad_w: torch.Tensor | None, ws: torch.Tensor | None = None, force_hbm: bool = False):
    m = _split_mode(mode)
    code = m | (BC_SPLIT_FORCE_HBM if force_hbm else 0)
    what = "box_conv_split_bwd"
    N, C, H, W, B = _maps_and_boxes(x, boxes, what)
    _need(x, None, _F32, what, "x")
    _need(piece_w, (C, B, SPLIT_PIECES[m]), _F32, what, "piece_w")
    _need(grad_y, (N, C * B, H, W), _F32, what, "grad_y")
    _need(grad_x, (N, C, H, W), _F32, what, "grad_x")
    _need(grad_boxes, (C, B, 4), _F32, what, "grad_boxes")
    _need(grad_w, (C, B, SPLIT_PIECES[m]), _F32, what, "grad_w")
    if ws is None:
        ws = _workspace(split_workspace_bytes(1, N, C, H, W, B, m, force_hbm), x.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load_library().box_conv_split_bwd(_ptr(x), _ptr(boxes), _ptr(piece_w), _ptr(grad_y), N, C, H, W, B, code,
                                             _ptr(grad_x), _ptr(grad_boxes), _ptr(grad_w), _ptr(ws), nbytes,
                                             _stream()), "box_conv_split_bwd")
    return grad_x, grad_boxes, grad_w


def bc_cast_bf16(src: torch.Tensor, dst: torch.Tensor):
    """dst (bf16, same numel) = src (fp32) rounded to nearest even."""
    _need_numel(src, src.numel(), _F32, "bc_cast_bf16", "src")
    _need_numel(dst, src.numel(), torch.bfloat16, "bc_cast_bf16", "dst")
    _check(load_library().bc_cast_bf16(_ptr(src), _ptr(dst), src.numel(), _stream()), "bc_cast_bf16")
    return dst


def relu_grad_bf16(grad: torch.Tensor, out: torch.Tensor, dst: torch.Tensor):
    """dst (bf16) = bf16(out > 0 ? grad : 0): the ReLU backward in the mix's compute type."""
    if not (grad.numel() == out.numel() == dst.numel()):
        raise BoxConvError("bc_relu_grad_bf16: size mismatch")
    if grad.dtype != torch.float32 or out.dtype != torch.float32 or dst.dtype != torch.bfloat16:
        raise BoxConvError("bc_relu_grad_bf16: grad and out fp32, dst bf16")
    _check(load_library().bc_relu_grad_bf16(_ptr(grad), _ptr(out), _ptr(dst), grad.numel(), _stream()),
           "bc_relu_grad_bf16")
    return dst


def pointwise_mix(mode: int, a: torch.Tensor, b: torch.Tensor, out: torch.Tensor, N: int, M: int, K: int,
                  P: int, compute_dt: int, relu: int = 0, aux: torch.Tensor | None = None,
                  accumulate: int = 0, ws: torch.Tensor | None = None):
    """The 1x1 mix (include/boxconv.h): FWD out[N,M,P] = a[M,K] * b[N,K,P];
    BWD_DATA out[N,K,P] = a[M,K]^T * b[N,M,P]; BWD_WEIGHT out[M,K] (+)=
    sum_n a[N,M,P] * b[N,K,P]^T.  aux: the FWD output Z [N,M,P] (ReLU mask)."""
    what = "pointwise_mix"
    sizes = {BC_MIX_FWD: (M * K, N * K * P, N * M * P), BC_MIX_BWD_DATA: (M * K, N * M * P, N * K * P),
             BC_MIX_BWD_WEIGHT: (N * M * P, N * K * P, M * K)}
    if mode not in sizes:
        raise BoxConvError(f"{what}: unknown mode {mode}")
    na, nb, no = sizes[mode]
    operand = (torch.int32, torch.float32, torch.bfloat16)
    _need_numel(a, na, operand, what, "a")
    _need_numel(b, nb, operand, what, "b")
    _need_numel(out, no, (torch.int32, torch.float32), what, "out")
    if aux is not None:
        _need_numel(aux, N * M * P, _F32, what, "aux")
    if ws is None:
        ws = _workspace(mix_workspace_bytes(mode, N, M, K, P, compute_dt), a.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load_library().pointwise_mix(mode, _ptr(a), dtype_code(a), _ptr(b), dtype_code(b), _ptr(out),
                                        dtype_code(out), N, M, K, P, compute_dt, relu, _ptr(aux), accumulate,
                                        _ptr(ws), nbytes, _stream()), "pointwise_mix")
    return out
