#!/usr/bin/env python3
"""Benchmark of the SAT box-convolution layer on one MI355X.

One step = one pass of the whole layer over one batch: box filter forward
(table + four-corner bilinear lookups), 1x1 mix forward (MFMA), mix backward
to the weights and to the filtered maps, and the box filter backward (input
and box-parameter gradients).  Inputs are seeded synthetic arrays shaped like
pose-estimation feature maps, already resident in HBM when timing starts.

Prints ONE JSON line.  `value` is filtered-map elements (pixel*box, summed over
layers) per second of the whole step, in Gpix*box/s, timed on steps run as the
layer runs them (every call in order on one stream; with --overlap the weight
gradient runs on a second stream).
`roofline` reports the dominant library call, timed with HIP events in a
second pass where every call runs in order on one stream (`serial_ms_per_step`
is that pass's step); `cpu_baseline` times the CPU oracle on a bounded sample
on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "box-conv fwd+bwd Gpix·box/s; SAT/box HBM GB/s and 1×1 MFMA util vs peak"
METRIC_INFERENCE = "box-conv inference fwd Gpix·box/s (integer corners); box HBM GB/s and 1×1 MFMA util vs peak"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
DEFAULT_WORKLOAD = 3


def parse():
    p = argparse.ArgumentParser(description=__doc__)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", type=int, default=DEFAULT_WORKLOAD, choices=[1, 2, 3, 4, 5, 6])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-budget-s", type=float, default=20.0,
                   help="rough CPU time the oracle sample may take")
    p.add_argument("--inference", action="store_true",
                   help="time the inference forward instead (boxes rounded to integer corners, "
                        "four table samples per box, then the 1x1 mix); no backward")
    p.add_argument("--stride", type=int, default=1,
                   help="box filter stride (outputs at every stride-th pixel; the 1x1 mix and the backward "
                        "run on the strided grid)")
    p.add_argument("--unit-params", action="store_true",
                   help="train the boxes as unit corners in [-1, 1] relative to a maximum box size equal to "
                        "the map size (drawn U[-0.5, 0.5]); the step then also converts them, takes their "
                        "gradient and clips them")
    p.add_argument("--split", choices=["2x", "2y", "4"], default=None,
                   help="kernel splitting: every box cut into 2 (along x or y) or 4 pieces with their own "
                        "weights (fp32 maps, stride 1; the table-offset flag is not used)")
    p.add_argument("--serial", action="store_true",
                   help="run every call in order on one stream in the timed pass (the layer's default; "
                        "overrides --overlap): the configuration the per-kernel profiles are taken in")
    p.add_argument("--overlap", action="store_true",
                   help="run each layer's weight gradient on a second stream beside its other backward "
                        "calls")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain elementwise kernel that reads 256 MiB and writes 256 MiB, 5 "
                        "times (reference for the FETCH_SIZE / WRITE_SIZE counters), and exit")
    return p.parse_args()


def source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1906_11367_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def call_cost(label, wl, o_bytes, stride=1):
    """Algorithmic bytes and FLOPs of one launch of a library call (one layer).

    box_conv_fwd : read x (4 B/pixel) + write O (o_bytes per output pixel*box)
    box_conv_bwd : read x + read dO (4 B/output pixel*box) + write dx (4 B/pixel;
                   2 B for box_conv_bwd_relu_bf16)
    mix_*        : 2*N*M*K*P FLOPs (one GEMM), reported against the MFMA
                   peak; also the operand bytes it must move (fwd: read O,
                   write Z; bwd_data: read dZ, write dO; bwd_weight: read dZ
                   and O), reported against the HBM peak; dZ is 2 bytes per
                   element for a bf16 mix (cast or masked once), else 4
    relu_grad    : read dZ and Z (fp32), write the masked dZ (bf16)
    grad_cast    : read dZ (fp32), write it in bf16
    """
    if label.startswith("box_params"):        # read and write [C][B][4] fp32
        return {"bound": "hbm", "bytes": 2 * wl.C * wl.B * 16}
    px = wl.N * wl.C * wl.H * wl.W
    Ho, Wo = (wl.H + stride - 1) // stride, (wl.W + stride - 1) // stride
    pb = wl.N * wl.C * wl.B * Ho * Wo          # output pixel*box
    if label in ("box_conv_fwd", "box_conv_split_fwd"):
        return {"bound": "hbm", "bytes": 4 * px + o_bytes * pb}
    if label in ("box_conv_bwd", "box_conv_split_bwd"):
        return {"bound": "hbm", "bytes": 4 * px + 4 * pb + 4 * px}
    if label == "box_conv_bwd_relu_bf16":                  # dx written in bf16
        return {"bound": "hbm", "bytes": 4 * px + 4 * pb + 2 * px}
    flops = 2 * wl.N * wl.mix_out * wl.C * wl.B * Ho * Wo
    nz = wl.N * wl.mix_out * Ho * Wo
    z = 4 * nz
    if label == "relu_grad":
        return {"bound": "hbm", "bytes": 10 * nz}
    if label == "grad_cast":
        return {"bound": "hbm", "bytes": 6 * nz}
    dz = 2 * nz if wl.mix_dtype == "bf16" else z
    mix_bytes = {"mix_fwd": o_bytes * pb + z, "mix_bwd_data": dz + 4 * pb, "mix_bwd_weight": dz + o_bytes * pb}
    return {"bound": "mfma", "flops": flops, "bytes": mix_bytes.get(label)}


def load_traffic(label, wl_key, src_hash):
    """HBM bytes per launch measured with rocprofv3 counters, if a committed
    summary for this call and workload exists and the sources have not
    changed since it was taken; else None."""
    path = os.path.join(ROOT, "profiles", f"{label}_{wl_key}_counters.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            d = json.load(f)
        if d.get("source_hash") != src_hash:
            return None
        return float(d["hbm_bytes_per_launch"])
    except Exception:
        return None


def cpu_baseline(wl, d, budget_s, inference=False, stride=1, split=None, piece_w=None):
    """Times the CPU oracle (fwd + bwd of the layer; with `inference`, the
    integer-corner forward only) on a sample of images.

    The sample keeps every channel and box of the workload and takes the
    first n images (n chosen from a one-image probe to fit the budget)."""
    import numpy as np
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = None

    def run(n):
        x = d["x"][:n]
        g = d["grad"][:n, ..., ::stride, ::stride] if d["grad"] is not None else None
        Ho, Wo = (wl.H + stride - 1) // stride, (wl.W + stride - 1) // stride
        if wl.layers > 1:
            layers = d["layers"][:1]   # one layer of the stack per sample image
            cache = O.stack_forward(x, layers, compute=wl.mix_dtype, apply_relu=wl.relu)
            O.stack_backward(cache, layers, g, compute=wl.mix_dtype, apply_relu=wl.relu)
            return n * wl.C * wl.B * wl.H * wl.W
        if inference:
            o = O.box_forward(x, d["boxes"], integer_corners=True, stride=stride)
            if wl.mix_out is not None:
                O.mix_forward(d["w"], o, compute=wl.mix_dtype, apply_relu=wl.relu)
            return n * wl.C * wl.B * Ho * Wo
        if split is not None:
            o = O.box_forward_split(x, d["boxes"], piece_w, split)
            if wl.mix_out is not None:
                O.mix_forward(d["w"], o, compute=wl.mix_dtype, apply_relu=wl.relu)
                if g is not None:
                    O.mix_backward_weight(g, o, compute=wl.mix_dtype)
                    g = O.mix_backward_data(d["w"], g, compute=wl.mix_dtype)
            if g is not None:
                O.box_backward_split_input(g, d["boxes"], piece_w, split, wl.H, wl.W)
                O.box_backward_split_params(x, g, d["boxes"], piece_w, split)
            return n * wl.C * wl.B * Ho * Wo
        o = O.box_forward(x, d["boxes"], stride=stride)
        if wl.mix_out is None:
            if g is not None:
                O.box_backward_input(g, d["boxes"], wl.H, wl.W, stride=stride)
                O.box_backward_params(x, g, d["boxes"], stride=stride)
            return n * wl.C * wl.B * Ho * Wo
        O.mix_forward(d["w"], o, compute=wl.mix_dtype, apply_relu=wl.relu)
        if g is not None:
            O.mix_backward_weight(g, o, compute=wl.mix_dtype)
            do = O.mix_backward_data(d["w"], g, compute=wl.mix_dtype)
            O.box_backward_input(do, d["boxes"], wl.H, wl.W, stride=stride)
            O.box_backward_params(x, do, d["boxes"], stride=stride)
        return n * wl.C * wl.B * Ho * Wo

    t0 = time.perf_counter()
    pb = run(1)
    t1 = time.perf_counter() - t0
    n = int(max(1, min(wl.N, budget_s / max(t1, 1e-3))))
    if n > 1:
        t0 = time.perf_counter()
        pb = run(n)
        t1 = time.perf_counter() - t0
    what = "integer-corner fwd" if inference else "fwd+bwd"
    if split is not None:
        what += f", boxes split {split}"
    return {"value": pb / t1 / 1e9, "unit": "Gpix·box/s", "cores": threads, "kind": "oracle",
            "affinity_cores": len(os.sched_getaffinity(0)),
            "sample": f"{n} of {wl.N} images, all {wl.C} channels x {wl.B} boxes, one layer, "
                      f"{what}, fp64 NumPy, {t1:.1f} s"}


def naive_eq1_baseline():
    """Times the oracle's naive per-pixel loop of Eq. 1 (pure Python, one
    core) on the whole tiny integer workload (one image, 8 channels x 4 boxes,
    32x32 int32 maps, integer corners; about a second).  The loop's result is
    checked against the oracle's forward before it is reported."""
    import numpy as np
    import oracle as O
    from paper_1906_11367_amd import workloads as wlmod
    wl = wlmod.WORKLOADS[1]
    d = wlmod.make_inputs(wl)
    x, bx = d["x"], d["boxes"]
    t0 = time.perf_counter()
    o = O.naive_box_forward_eq1(x, bx)
    t1 = time.perf_counter() - t0
    if not np.array_equal(o, O.box_forward(x, bx)):
        raise RuntimeError("naive Eq. 1 loop disagrees with the oracle's forward")
    pb = o.size
    return {"value": pb / t1 / 1e9, "unit": "Gpix·box/s", "cores": 1, "kind": "oracle naive Eq. 1 loop",
            "sample": f"{wl.key}: the whole workload, {wl.N} image, {wl.C} channels x {wl.B} boxes, "
                      f"{wl.H}x{wl.W}, forward only, int64 pure Python, {t1:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the layer's multi-GPU sharding is a design note only)", file=sys.stderr)
        return 2
    # the CPU oracle's BLAS uses every core this process may run on, unless
    # the environment already fixes the thread count
    ncpu = str(len(os.sched_getaffinity(0)))
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS"):
        os.environ.setdefault(var, ncpu)
    import numpy as np
    import torch

    if args.copy_calibration:
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            torch.mul(src, 2.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_per_launch": src.numel() * 4, "launches": 5}), flush=True)
        return 0

    from paper_1906_11367_amd import boxconv as bc
    from paper_1906_11367_amd import workloads as wlmod
    from paper_1906_11367_amd.layer import Stack

    bc.load_library()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    wl = wlmod.WORKLOADS[args.workload]
    print(f"[bench] workload {wl.key}: generating inputs", file=sys.stderr, flush=True)
    d = wlmod.make_inputs(wl)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    x = dev(d["x"])
    params = [(dev(b), dev(w) if w is not None else None) for b, w in d["layers"]]
    grad = dev(d["grad"]) if d["grad"] is not None else None
    x_dt = torch.int32 if wl.x_kind == "int8range" else torch.float32
    flags = bc.BC_FLAG_MEAN_OFFSET if wl.mean_offset else 0
    if args.split is not None:
        if args.inference or args.stride != 1 or wl.x_kind == "int8range" or wl.layers > 1:
            print("--split takes a one-layer fp32 workload with backward, stride 1", file=sys.stderr)
            return 2
        flags = 0
    backward = wl.backward and not args.inference
    if args.inference:
        flags |= bc.BC_FLAG_INTEGER_CORNERS
    s_ = args.stride
    unit = (float(wl.W), float(wl.H)) if args.unit_params else None
    st = Stack(wl.N, wl.C, wl.H, wl.W, wl.B, wl.mix_out, wl.layers, wl.mix_dtype, wl.relu, x_dt, flags,
               backward, stride=s_, unit_size=unit, split=args.split)
    if unit is not None:
        params = [(dev(wlmod.make_unit_corners(wl, li)), w) for li, (_, w) in enumerate(params)]
    piece_w = None
    if args.split is not None:
        piece_w = wlmod.make_piece_weights(wl, bc.SPLIT_PIECES[bc.SPLIT_MODES[args.split]])
        params = [((b, dev(piece_w)), w) for b, w in params]
    if grad is not None and s_ > 1:
        grad = grad[..., ::s_, ::s_].contiguous()
    for plan in st.plans:
        plan.overlap = args.overlap and not args.serial
    stream = torch.cuda.current_stream()
    timing = {"on": False, "events": [], "pool": []}

    def tap(label):
        if timing["on"]:
            e = timing["pool"].pop()
            e.record(stream)
            timing["events"].append((label, e))

    def step():
        # The plain pass runs the layer as a user would; the per-call pass
        # records an event after every call, in order on one stream.
        t = tap if timing["on"] else None
        if t:
            t("start")
        inputs, out = st.forward(x, params, t)
        if backward:
            st.backward(inputs, params, grad, t)
            if unit is not None:      # the per-update step on the unit corners
                for plan, (u, _) in zip(st.plans, params):
                    plan.clip(u[0] if args.split is not None else u)
                if t:
                    t("box_params_clip")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # Each timed pass starts behind ~100 ms of device-side spinning, queued
    # before its first event: the host enqueues the steps while the GPU is
    # busy, so no host launch gap lands inside a timed call or step.
    spin = torch.cuda._sleep
    probe = 1 << 20
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s0.record(stream)
    spin(probe)
    s1.record(stream)
    torch.cuda.synchronize()
    spin_cycles = int(probe * 100.0 / max(s0.elapsed_time(s1), 1e-3))

    # timed region: plain steps.  Untimed steps follow the spin before the
    # first event: after any pause in the step stream (the spin included) the
    # step time ramps down over ~40 steps (~25 ms; measured on the pose
    # layer: ~730 us at the 5th step, 588 us from the 45th on), and the
    # settle steps keep that ramp outside the timing, whatever --warmup and
    # --steps are.
    settle = 60
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    spin(spin_cycles)
    for _ in range(settle):
        step()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps

    # second timed pass with an event after every library call (events made
    # beforehand, so the pass itself only records them)
    # at most 8 calls per layer and step, plus the step's start and clip
    timing["pool"] = [torch.cuda.Event(enable_timing=True) for _ in range((8 * wl.layers + 2) * args.steps)]
    spin(spin_cycles)
    for _ in range(settle):
        step()
    timing["on"] = True
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    per = {}
    evs = timing["events"]
    for (l0, a), (l1, b) in zip(evs[:-1], evs[1:]):
        if l1 == "start":
            continue
        per.setdefault(l1, []).append(a.elapsed_time(b))
    # one step with every call in order on one stream (the per-call pass)
    serial_ms = sum(sum(ts) for ts in per.values()) / args.steps
    o_bytes = 2 if (wl.mix_out is not None and wl.mix_dtype == "bf16") else 4
    src_hash = source_hash()
    calls = {}
    for label, ts in per.items():
        avg_ms = sum(ts) / len(ts)
        c = call_cost(label, wl, o_bytes, args.stride)
        ent = {"avg_us": round(avg_ms * 1e3, 2), "launches": len(ts) // args.steps, "bound": c["bound"],
               "share": round(sum(ts) / args.steps / serial_ms, 3)}
        if c["bound"] == "hbm":
            ent["algo_bytes"] = c["bytes"]
            ent["achieved"] = c["bytes"] / (avg_ms * 1e-3) / 1e9
            ent["peak"] = HBM_PEAK_GBS
            ent["unit"] = "GB/s"
        else:
            ent["algo_flops"] = c["flops"]
            ent["achieved"] = c["flops"] / (avg_ms * 1e-3) / 1e12
            ent["peak"] = MFMA_PEAK_TFLOPS["bf16" if wl.mix_dtype == "bf16" else "f32"]
            ent["unit"] = "TFLOP/s"
            if c.get("bytes"):
                ent["algo_bytes"] = c["bytes"]
                ent["hbm_gbs"] = round(c["bytes"] / (avg_ms * 1e-3) / 1e9, 2)
                ent["hbm_frac"] = round(ent["hbm_gbs"] / HBM_PEAK_GBS, 4)
        ent["frac"] = ent["achieved"] / ent["peak"]
        ent["achieved"] = round(ent["achieved"], 2)
        ent["frac"] = round(ent["frac"], 4)
        calls[label] = ent
    dom = max(calls, key=lambda k: calls[k]["avg_us"] * calls[k]["launches"])
    dc = calls[dom]
    traffic = load_traffic(dom, wl.key + ("_inference" if args.inference else "")
                           + (f"_stride{args.stride}" if args.stride > 1 else "")
                           + (f"_split{args.split}" if args.split else ""), src_hash)
    roofline = {"bound": dc["bound"], "achieved": dc["achieved"], "peak": dc["peak"], "unit": dc["unit"],
                "frac": dc["frac"], "traffic": traffic, "kernel": dom, "avg_us": dc["avg_us"],
                "per_launch": ("algo_bytes=%d" % dc["algo_bytes"]) if dc["bound"] == "hbm"
                else ("algo_flops=%d" % dc["algo_flops"])}

    # HBM bandwidth a plain streaming kernel reaches on this GPU (the spec peak
    # beside it): an fp32 elementwise multiply, 256 MiB read and 256 MiB
    # written per launch, timed over 20 launches after 5
    src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        torch.mul(src, 2.0, out=dst)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(20):
        torch.mul(src, 2.0, out=dst)
    c1.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * src.numel() * 4 / (c0.elapsed_time(c1) / 20 * 1e-3) / 1e9
    del src, dst
    if roofline["bound"] == "hbm":
        roofline["frac_of_measured_copy"] = round(roofline["achieved"] / copy_gbs, 4)
    for ent in calls.values():
        gbs = ent["achieved"] if ent["bound"] == "hbm" else ent.get("hbm_gbs")
        if gbs is not None:
            ent["hbm_frac_of_measured_copy"] = round(gbs / copy_gbs, 4)

    pix_box = wl.N * wl.C * wl.B * st.plans[0].Ho * st.plans[0].Wo * wl.layers
    value = pix_box / (ms * 1e-3) / 1e9
    box_ms = sum(calls[k]["avg_us"] * calls[k]["launches"] for k in calls if k.startswith("box")) / 1e3
    line = {
        "metric": METRIC_INFERENCE if args.inference else METRIC, "value": round(value, 3), "unit": "Gpix·box/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "serial_ms_per_step": round(serial_ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32" if x_dt == torch.float32 else "i32",
        "data": "synthetic",
        "config": {"workload": wl.key, "N": wl.N, "C": wl.C, "H": wl.H, "W": wl.W, "B": wl.B,
                   "mix": None if wl.mix_out is None else f"{wl.C * wl.B}->{wl.mix_out} {wl.mix_dtype}",
                   "layers": wl.layers, "relu": wl.relu, "mean_offset": bool(flags & bc.BC_FLAG_MEAN_OFFSET),
                   "integer_corners": bool(args.inference), "backward": backward,
                   "overlap_weight_grad": backward and any(p.overlap for p in st.plans), "stride": args.stride,
                   "unit_params": bool(args.unit_params), "split": args.split,
                   "parallelism": "single GPU"},
        "box_only_gpixbox_s": round(pix_box / (box_ms * 1e-3) / 1e9, 3) if box_ms > 0 else None,
        "roofline": roofline,
        "hbm_measured_copy_gbs": round(copy_gbs, 1),
        "calls": calls,
        "source_hash": src_hash,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(wl, d, args.cpu_budget_s, args.inference, args.stride,
                                            args.split, piece_w)
        line["cpu_baseline_naive_eq1"] = naive_eq1_baseline()
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
