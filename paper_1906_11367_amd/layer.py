"""One box-convolution layer and a stack of them, composed from the C-ABI calls.

Forward:  O = box_conv_fwd(x)            (bf16 copy when the mix runs in bf16)
          Z = pointwise_mix(FWD, w, O)   (+ ReLU when configured)
Backward: dW = pointwise_mix(BWD_WEIGHT, dZ, O)
          dO = pointwise_mix(BWD_DATA, w, dZ)
          dx, dboxes = box_conv_bwd(x, dO)
With a bf16 mix, dZ is first rounded to bf16 once (bc_cast_bf16), or masked
and rounded with a ReLU (bc_relu_grad_bf16): both GEMMs then read those bf16
operands, the same operand bits they would form from the fp32 gradient
themselves, so the results are bitwise the same (pose layer 0.574 -> 0.556 ms
per step; six stacked layers 4.47 -> 3.71 ms).  In a stack the masked
operand of layer l comes straight from the box backward of layer l + 1
(box_conv_bwd_relu_bf16: its input is layer l's rectified output, so x > 0
is the mask), with no fp32 gradient written or read back.
With kernel splitting (`split` = "2x", "2y" or "4") the box filter is
box_conv_split_fwd / box_conv_split_bwd: the boxes argument is then the pair
(boxes, piece weights) and the backward returns the pair of their gradients.
The weight gradient depends on neither of the other two backward calls; a
plan built with `overlap` runs it on a second stream (default priority)
alongside them, and the caller's stream waits for it before the backward
returns.  By default every call runs in order on the caller's stream, which
was measured faster on every workload here.
All buffers and workspaces are allocated once per plan (torch is used for
device memory and streams only); every arithmetic step runs in libboxconv's
kernels.
"""
from __future__ import annotations

import dataclasses

import torch

from . import boxconv as bc


@dataclasses.dataclass
class LayerPlan:
    N: int
    C: int
    H: int
    W: int
    B: int
    M: int | None          # mix output channels; None = box filter only
    x_dtype: torch.dtype   # int32 or float32
    mix_dtype: str         # 'i32' | 'f32' | 'bf16'
    relu: bool = False
    flags: int = 0
    with_backward: bool = True
    device: str = "cuda"
    # weight gradient on a second stream during the backward (default off).
    # With the incoming gradient in bf16 (below) the two backward GEMMs run
    # faster in order than side by side (pose layer 0.556 against 0.587 ms),
    # and so do the stacked ReLU layers (3.465 against 3.515 ms) and the
    # compute-bound fp32 mix of the 256x256 layer (2.525 against 2.666 ms).
    overlap: bool = False
    stride: int = 1            # box filter stride: outputs ceil(H/stride) x ceil(W/stride)
    # (max_w, max_h): the boxes are given as unit corners u in [-1, 1] relative
    # to that maximum box size (converted in the forward; the backward returns
    # dL/du); None: the boxes are (cx, cy, rx, ry) in pixels
    unit_size: tuple | None = None
    split: str | None = None   # kernel splitting mode: None, "2x", "2y" or "4"
    # dx written as bf16(x > 0 ? dx : 0) for the ReLU + bf16 mix below this layer
    dx_relu_bf16: bool = False
    # grad_out arrives as that masked bf16 operand (from the layer above)
    grad_premasked: bool = False

    def __post_init__(self):
        dev = torch.device(self.device)
        N, C, H, W, B = self.N, self.C, self.H, self.W, self.B
        Ho, Wo = (H + self.stride - 1) // self.stride, (W + self.stride - 1) // self.stride
        self.Ho, self.Wo = Ho, Wo
        K = C * B
        P = Ho * Wo
        self.K, self.P = K, P
        integer = self.x_dtype == torch.int32
        if integer:
            o_dt = torch.int32
        elif self.M is not None and self.mix_dtype == "bf16":
            o_dt = torch.bfloat16
        else:
            o_dt = torch.float32
        self.o = torch.empty((N, K, Ho, Wo), dtype=o_dt, device=dev)
        self.compute = bc.BC_BF16 if self.mix_dtype == "bf16" else bc.BC_F32
        if self.dx_relu_bf16 and (integer or self.split is not None or self.flags & bc.BC_FLAG_INTEGER_CORNERS):
            raise ValueError("a bf16 masked input gradient needs fp32 maps, whole boxes and real corners")
        if self.grad_premasked and not (self.relu and self.M is not None and self.compute == bc.BC_BF16):
            raise ValueError("a pre-masked incoming gradient needs a ReLU after a bf16 mix")
        if self.split is not None:
            if integer or self.stride != 1 or self.flags:
                raise ValueError("kernel splitting takes fp32 maps, stride 1 and no box flags")
            self.pieces = bc.SPLIT_PIECES[bc.SPLIT_MODES[self.split]]
            self.ws_fwd = _ws(bc.split_workspace_bytes(0, N, C, H, W, B, self.split), dev)
        else:
            self.ws_fwd = _ws(bc.box_workspace_bytes(0, N, C, H, W, B, self.flags, self.stride), dev)
        if self.unit_size is not None:
            self.boxes_px = torch.empty((C, B, 4), dtype=torch.float32, device=dev)
        if self.M is not None:
            self.z = torch.empty((N, self.M, Ho, Wo), dtype=torch.int32 if integer else torch.float32, device=dev)
            # the mix's weights in its compute type, refreshed from w every forward
            self.w_c = (torch.empty((self.M, K), dtype=torch.bfloat16, device=dev)
                        if self.compute == bc.BC_BF16 else None)
        if self.with_backward:
            if self.split is not None:
                self.ws_bwd = _ws(bc.split_workspace_bytes(1, N, C, H, W, B, self.split), dev)
                self.dpiece = torch.empty((C, B, self.pieces), dtype=torch.float32, device=dev)
            else:
                self.ws_bwd = _ws(bc.box_workspace_bytes(1, N, C, H, W, B, self.flags, self.stride), dev)
            self.dx = torch.empty((N, C, H, W), dtype=torch.bfloat16 if self.dx_relu_bf16 else torch.float32,
                                  device=dev)
            self.dboxes = torch.empty((C, B, 4), dtype=torch.float32, device=dev)
            if self.unit_size is not None:
                self.du = torch.empty((C, B, 4), dtype=torch.float32, device=dev)
            if self.M is not None:
                self.do = torch.empty((N, K, Ho, Wo), dtype=torch.float32, device=dev)
                self.dw = torch.empty((self.M, K), dtype=torch.float32, device=dev)
                self.ws_mixw = _ws(bc.mix_workspace_bytes(bc.BC_MIX_BWD_WEIGHT, N, self.M, K, P,
                                                          self.compute), dev)
                self.ws_mixd = _ws(bc.mix_workspace_bytes(bc.BC_MIX_BWD_DATA, N, self.M, K, P,
                                                          self.compute), dev)
                # the incoming gradient in bf16, once, for both backward GEMMs of a
                # bf16 mix (masked by the ReLU if there is one): the GEMMs round it
                # to the same bits themselves, but read as bf16 it costs half the
                # bytes and arrives from cache (pose layer: BWD_DATA 145 -> 100 us,
                # BWD_WEIGHT 110 -> 97 us, for a 28 us cast; step 0.574 -> 0.556 ms)
                self.dz_bf16 = (torch.empty((N, self.M, Ho, Wo), dtype=torch.bfloat16, device=dev)
                                if self.compute == bc.BC_BF16 and not self.grad_premasked else None)
                self.side = torch.cuda.Stream(device=dev)   # default priority
                self.ev_in = torch.cuda.Event()
                self.ev_dw = torch.cuda.Event()

    def forward(self, x: torch.Tensor, boxes: torch.Tensor, w: torch.Tensor | None, tap=None):
        """tap(label), if given, is called after each library call (the benchmark
        records a stream event there)."""
        tap = tap or _no_tap
        piece_w = None
        if self.split is not None:
            boxes, piece_w = boxes
        if self.unit_size is not None:
            boxes = bc.box_params_from_unit(boxes, *self.unit_size, self.boxes_px)
        if piece_w is not None:
            bc.box_conv_split_fwd(x, boxes, piece_w, self.split, self.o, self.ws_fwd)
            tap("box_conv_split_fwd")
        else:
            bc.box_conv_fwd(x, boxes, self.o, self.flags, self.ws_fwd, stride=self.stride)
            tap("box_conv_fwd")
        if self.M is None:
            return self.o
        if self.w_c is not None:
            bc.bc_cast_bf16(w, self.w_c)
            w = self.w_c
        bc.pointwise_mix(bc.BC_MIX_FWD, w, self.o, self.z, self.N, self.M, self.K, self.P, self.compute,
                         relu=int(self.relu))
        tap("mix_fwd")
        return self.z

    def backward(self, x: torch.Tensor, boxes: torch.Tensor, w: torch.Tensor | None, grad_out: torch.Tensor,
                 tap=None):
        """grad_out: dL/dZ (or dL/dO without a mix).  Returns (dx, dboxes, dw).

        With a mix (and `overlap`), the weight gradient runs on the plan's
        second stream; given `tap`, every call runs in order on the current
        stream instead, so that the events the benchmark records there time
        each call alone."""
        overlap = tap is None and self.overlap
        tap = tap or _no_tap
        u = None
        piece_w = None
        if self.split is not None:
            boxes, piece_w = boxes
        if self.unit_size is not None:
            u, boxes = boxes, self.boxes_px      # the forward's conversion of u
        if self.M is None:
            do = grad_out
            dw = None
        else:
            aux = self.z if self.relu else None
            relu = int(self.relu)
            if self.grad_premasked:
                if grad_out.dtype != torch.bfloat16:
                    raise ValueError("grad_out must be the masked bf16 operand")
                aux, relu = None, 0
            elif self.dz_bf16 is not None and self.relu:
                grad_out = bc.relu_grad_bf16(grad_out, self.z, self.dz_bf16)
                tap("relu_grad")
                aux, relu = None, 0
            elif self.dz_bf16 is not None:
                grad_out = bc.bc_cast_bf16(grad_out, self.dz_bf16)
                tap("grad_cast")
            main = torch.cuda.current_stream()
            if overlap:
                self.ev_in.record(main)         # O, Z and dZ are ready on the caller's stream
                self.side.wait_event(self.ev_in)
                with torch.cuda.stream(self.side):
                    bc.pointwise_mix(bc.BC_MIX_BWD_WEIGHT, grad_out, self.o, self.dw, self.N, self.M, self.K,
                                     self.P, self.compute, relu=relu, aux=aux, ws=self.ws_mixw)
                self.ev_dw.record(self.side)
            else:
                bc.pointwise_mix(bc.BC_MIX_BWD_WEIGHT, grad_out, self.o, self.dw, self.N, self.M, self.K, self.P,
                                 self.compute, relu=relu, aux=aux, ws=self.ws_mixw)
                tap("mix_bwd_weight")
            if self.w_c is not None:
                w = self.w_c
            bc.pointwise_mix(bc.BC_MIX_BWD_DATA, w, grad_out, self.do, self.N, self.M, self.K, self.P,
                             self.compute, relu=relu, aux=aux, ws=self.ws_mixd)
            tap("mix_bwd_data")
            do = self.do
            dw = self.dw
        grad_boxes = None if self.flags & bc.BC_FLAG_INTEGER_CORNERS else self.dboxes
        if piece_w is not None:
            bc.box_conv_split_bwd(x, boxes, piece_w, self.split, do, self.dx, grad_boxes, self.dpiece, self.ws_bwd)
            tap("box_conv_split_bwd")
        elif self.dx_relu_bf16:
            bc.box_conv_bwd_relu_bf16(x, boxes, do, self.dx, grad_boxes, self.flags, self.ws_bwd, stride=self.stride)
            tap("box_conv_bwd_relu_bf16")
        else:
            bc.box_conv_bwd(x, boxes, do, self.dx, grad_boxes, self.flags, self.ws_bwd, stride=self.stride)
            tap("box_conv_bwd")
        if u is not None and grad_boxes is not None:
            grad_boxes = bc.box_params_unit_grad(grad_boxes, *self.unit_size, self.du)
            tap("box_params")
        if piece_w is not None:
            grad_boxes = (grad_boxes, self.dpiece)
        if self.M is not None and overlap:
            main.wait_event(self.ev_dw)         # dW (and the reuse of O, dZ) ordered after the side stream
        return self.dx, grad_boxes, dw


    def clip(self, u: torch.Tensor):
        """After an update of the unit corners: clip to [-1, 1], order each pair."""
        return bc.box_params_clip(u)


def _no_tap(label):
    return None


def _ws(nbytes: int, dev):
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=dev)


class Stack:
    """`layers` box-conv layers in sequence; layer l's mix output feeds layer l+1."""

    def __init__(self, N, C, H, W, B, M, layers, mix_dtype, relu, x_dtype=torch.float32, flags=0,
                 backward=True, device="cuda", stride=1, unit_size=None, split=None):
        if layers > 1 and (M != C or stride != 1):
            raise ValueError("stacked layers need M == C and stride 1")
        # a ReLU after a bf16 mix below: the layer above writes its input
        # gradient as that mix's masked bf16 operand
        chain = (layers > 1 and backward and relu and mix_dtype == "bf16" and M is not None and split is None
                 and x_dtype == torch.float32 and not flags & bc.BC_FLAG_INTEGER_CORNERS)
        self.plans = [LayerPlan(N, C, H, W, B, M, x_dtype, mix_dtype, relu, flags, backward, device,
                                stride=stride, unit_size=unit_size, split=split,
                                dx_relu_bf16=chain and l > 0, grad_premasked=chain and l < layers - 1)
                      for l in range(layers)]

    def forward(self, x, params, tap=None):
        """params: list of (boxes, w) device tensors.  Returns the inputs of every
        layer (for the backward) and the last output."""
        inputs = []
        cur = x
        for plan, (boxes, w) in zip(self.plans, params):
            inputs.append(cur)
            cur = plan.forward(cur, boxes, w, tap)
        return inputs, cur

    def backward(self, inputs, params, grad_out, tap=None):
        grads = [None] * len(self.plans)
        g = grad_out
        for li in range(len(self.plans) - 1, -1, -1):
            boxes, w = params[li]
            dx, dboxes, dw = self.plans[li].backward(inputs[li], boxes, w, g, tap)
            grads[li] = (dboxes, dw)
            g = dx
        return g, grads
