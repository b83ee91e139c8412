#!/usr/bin/env python3
"""Benchmark of the quantize-once MX convolution hot path on one MI355X.

Headline (`value`): one fwd+bwd training step of a YOLOv8n-shaped backbone
and neck (51 convolutions with SiLU, concatenations and 2x upsampling; see
paper_2609_28358_amd/workloads.py) at batch 64 on a 3x640x640 image, every
tensor in MXFP4 (E2M1 elements, E8M0 scales) and quantized exactly once:
weights from their bf16 masters, activations by the producing convolution's
epilogue, gradients once per layer from the sum its consumers hand back.
`value` = the step's GEMM flops (forward, input gradient, weight gradient;
real channels only) over the step's wall time; the step is captured once into
a HIP graph after warm-up and replayed `--steps` times between
synchronizations, inputs resident in HBM.

`roofline` belongs to the step's call that takes longest inside the step:
every call's in-step duration is measured with HIP events recorded on the
step's stream between consecutive calls of an eagerly enqueued step (behind
a GPU spin, so the events bracket kernels, not host launch latency);
`achieved` = the call's algorithmic bytes (or flops) / that duration.
`traffic` comes from the committed FETCH_SIZE / WRITE_SIZE counter summary of
the same step (profiles/), while the sources still hash to it.

Extra keys: `yolo_step` (every call's in-step time and roofline fraction,
time by kind, per-layer algorithmic bytes against the naive comparator);
`latent_replay_step` (the quantized-latent-replay back stack at batch 128,
MXFP4, measured the same way); `layer_sweep` (the three-layer sweep at batch
32 in MXFP8 and MXFP4 with steady-state per-op times, the measured naive
comparator, and the fused-epilogue, FP6, stochastic-rounding and NVFP4
legs, the NVFP GEMMs of every element-format combination); `cpu_baseline`
(the fp64 oracle on a bounded sample of the headline
workload, on the host).

    python bench.py [--steps K] [--warmup W] [--no-cpu-baseline] [--no-sweep] [--no-qlr]
    python bench.py --pmc-pass {yolo,qlr,sweep}        (under rocprofv3 --pmc)
    python bench.py --summarize-trace DIR LOG | --summarize-pmc FDIR WDIR FLOG WLOG
    python bench.py --summarize-sq LOG DIR [DIR ...]    (SQ counters of the MFMA-heavy calls)
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_GBS = 8000.0                                   # MI355X HBM3E
SPIN_CYCLES = 100000                               # GPU spin ahead of a timed eager launch
MFMA_TFLOPS = {0: 5000.0, 1: 10100.0}              # dense MXFP8 / MXFP4
FMT_NAME = {0: "mxfp8", 1: "mxfp4"}
# FP6 methods as (W, X, G_Y) element formats: MicroQonv+ (Sec. IV-D) keeps
# activations in E3M2 with FP4 weights and gradients; the "-6" methods
# (Sec. VI-B) use E2M3 throughout
FP6_METHODS = {"microqonv_plus": (1, 3, 1), "microqonv_6": (2, 2, 2)}
FP6_SLACK = 16                                     # read slack at the end of an FP6 code buffer
# NVFP methods besides NVFP4, as (W, X, G_Y) element formats: the "-8"
# methods, the "-6" methods (Sec. VI-B, E2M3) and MicroQonv+ (Sec. IV-D)
NV_METHODS = {"nvfp8": (0, 0, 0), "nvfp6_e2m3": (2, 2, 2), "microqonv_plus": (1, 3, 1)}


def layer_numbers(cv, fmt, mx):
    """Algorithmic flops and bytes of each op of one layer step."""
    from paper_2609_28358_amd import synth
    n, ci, co, kh, kw = cv["n"], cv["cin"], cv["cout"], cv["kh"], cv["kw"]
    ho, wo = synth.out_hw(cv)
    flops = 2.0 * n * co * ho * wo * ci * kh * kw

    def mxb(role, nn, c, h, w):
        return mx.codes_bytes(role, fmt, nn, c, h, w) + mx.scales_bytes(role, fmt, nn, c, h, w)

    X = mxb(mx.ACT, n, ci, cv["h"], cv["w"])
    W = mxb(mx.WEIGHT, co, ci, kh, kw)
    G = mxb(mx.ACT, n, co, ho, wo)
    import ctypes
    c = mx.conv_struct(cv)
    XC = (mx.lib().mxconv_im2col_codes_bytes(ctypes.byref(c), fmt) +
          mx.lib().mxconv_im2col_scales_bytes(ctypes.byref(c), fmt))
    return {
        "quant_x": (0.0, 4.0 * n * ci * cv["h"] * cv["w"] + X),
        "quant_w": (0.0, 4.0 * co * ci * kh * kw + W),
        "quant_xw": (0.0, 4.0 * n * ci * cv["h"] * cv["w"] + X + 4.0 * co * ci * kh * kw + W),
        # X and W quantized in one launch that also writes X's CBF im2col
        "quant_xw_im2col": (0.0, 4.0 * n * ci * cv["h"] * cv["w"] + X + 4.0 * co * ci * kh * kw + W + XC),
        "quant_gy": (0.0, 4.0 * n * co * ho * wo + G),
        "im2col": (0.0, X + XC),
        "fwd": (flops, W + X + 4.0 * n * co * ho * wo),
        "dgrad": (flops, W + G + 4.0 * n * ci * cv["h"] * cv["w"]),
        "wgrad": (flops, G + X + 4.0 * co * ci * kh * kw),
        # input gradient and weight-gradient GEMM in one launch, the split-K
        # reduction deferred to the step's batched reduction (credited with
        # the two products' flops and their distinct operands and results)
        "backward": (2.0 * flops, W + G + X + 4.0 * n * ci * cv["h"] * cv["w"] + 4.0 * co * ci * kh * kw),
    }


PMC_SUMMARY = os.path.join(ROOT, "profiles", "layer_sweep_b32_traffic_pmc.md")
PMC_YOLO = os.path.join(ROOT, "profiles", "yolo_b64_mxfp4_traffic_pmc.md")
COPY_BYTES = 256 << 20                             # calibration copy of the counter pass


def source_digest():
    """Digest of the HIP sources: counter figures taken from an older build
    no longer describe the kernels and are not reported."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_28358_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def counter_traffic(op_key, path=None):
    """HBM bytes per launch of `op_key` ("layer/format/op", or "workload/call")
    from a committed counter summary: FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch, summed over the op's kernels), each scaled by the factor the
    same counter gives for a copy of known size.  None if there is no
    summary, the op is missing, or the sources changed since the counters
    were taken."""
    path = path or PMC_SUMMARY
    if not os.path.exists(path):
        return None
    digest, fetch_f, write_f, rows = None, None, None, {}
    with open(path) as f:
        for line in f:
            t = line.strip()
            if t.startswith("source digest:"):
                digest = t.split(":", 1)[1].strip().strip("`")
            elif t.startswith("fetch factor:"):
                fetch_f = float(t.split(":", 1)[1])
            elif t.startswith("write factor:"):
                write_f = float(t.split(":", 1)[1])
            elif t.startswith("|") and "/" in t:
                c = [x.strip() for x in t.strip("|").split("|")]
                try:
                    rows[c[0]] = (float(c[2]), float(c[3]))
                except (ValueError, IndexError):
                    pass
    if digest != source_digest() or fetch_f is None or write_f is None or op_key not in rows:
        return None
    fk, wk = rows[op_key]
    return round((fk * fetch_f + wk * write_f) * 1024.0)


def naive_numbers(cv, fmt, mx):
    """Algorithmic bytes of one layer step of the naive comparator, and the
    elements it quantizes (X' twice, W twice, G_Y twice)."""
    from paper_2609_28358_amd import synth
    n, ci, co, kh, kw = cv["n"], cv["cin"], cv["cout"], cv["kh"], cv["kw"]
    ho, wo = synth.out_hw(cv)
    P, K = n * ho * wo, kh * kw * ci
    L = mx.lib()

    def line(lines, length):
        return L.mxconv_naive_codes_bytes(lines, length, fmt) + L.mxconv_naive_scales_bytes(lines, length)

    nx, ny, nw = n * ci * cv["h"] * cv["w"], P * co, co * K
    by = {
        "im2col_f32": 4.0 * nx + 4.0 * P * K,
        "quant_col_k": 4.0 * P * K + line(P, K), "quant_col_p": 4.0 * P * K + line(K, P),
        "quant_w_k": 4.0 * nw + line(co, K), "quant_w_co": 4.0 * nw + line(K, co),
        "quant_gy_co": 4.0 * ny + line(P, co), "quant_gy_p": 4.0 * ny + line(co, P),
        "fwd": line(P, K) + line(co, K) + 4.0 * ny,
        "dgrad": line(P, co) + line(K, co) + 4.0 * P * K + 4.0 * P * K + 4.0 * nx,   # GEMM + col2im
        "wgrad": line(co, P) + line(K, P) + 4.0 * nw,
    }
    return by, 2 * P * K + 2 * nw + 2 * ny


def cpu_baseline(min_s=10.0, max_steps=8):
    """The oracle on the benchmark's own workload: every layer of the sweep in
    both formats -- quantize X, W, G_Y, CBF im2col, fwd, dgrad, wgrad in fp64
    loops on the host -- i.e. one step on the CPU, repeated until at least
    min_s seconds of oracle work (at most max_steps steps)."""
    import oracle
    from paper_2609_28358_amd import synth
    inputs = []
    for li, (name, cv) in enumerate(synth.SWEEP_LAYERS):
        x, w, gy = synth.layer_inputs(cv, 1000 + li, kind="sweep")
        inputs.append((cv, x, w, gy))
    flops, dt, steps = 0.0, 0.0, 0
    while steps < max_steps and (steps == 0 or dt < min_s):
        for cv, x, w, gy in inputs:
            xn, wn, gn = x.numpy(), w.numpy(), gy.numpy()
            ho, wo = synth.out_hw(cv)
            for fmt in (0, 1):
                t0 = time.perf_counter()
                ox = oracle.quantize(xn, oracle.NCHW, oracle.ACT, fmt, *x.shape)
                ow = oracle.quantize(wn, oracle.NCHW, oracle.WEIGHT, fmt, *w.shape)
                og = oracle.quantize(gn, oracle.NCHW, oracle.ACT, fmt, *gy.shape)
                oracle.im2col_cbf(cv, fmt, *ox)
                oracle.fwd(cv, fmt, ow, ox)
                oracle.dgrad(cv, fmt, ow, og)
                oracle.wgrad(cv, fmt, og, ox)
                dt += time.perf_counter() - t0
                flops += 3 * 2.0 * cv["n"] * cv["cout"] * ho * wo * cv["cin"] * cv["kh"] * cv["kw"]
        steps += 1
    out = {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.get_threads(), "kind": "oracle",
           "sample": f"{steps} full step{'s' if steps > 1 else ''} of the benchmark workload (all three layers, MXFP8 and MXFP4, "
                     f"every op of the path) through the fp64 oracle: {dt:.1f} s"}
    # the same oracle on one thread, over one layer in one format (about 10 s)
    threads = oracle.get_threads()
    oracle.set_threads(1)
    try:
        cv, x, w, gy = inputs[0]
        ho, wo = synth.out_hw(cv)
        fmt = 1
        t0 = time.perf_counter()
        ox = oracle.quantize(x.numpy(), oracle.NCHW, oracle.ACT, fmt, *x.shape)
        ow = oracle.quantize(w.numpy(), oracle.NCHW, oracle.WEIGHT, fmt, *w.shape)
        og = oracle.quantize(gy.numpy(), oracle.NCHW, oracle.ACT, fmt, *gy.shape)
        oracle.im2col_cbf(cv, fmt, *ox)
        oracle.fwd(cv, fmt, ow, ox)
        oracle.dgrad(cv, fmt, ow, og)
        oracle.wgrad(cv, fmt, og, ox)
        t1 = time.perf_counter() - t0
    finally:
        oracle.set_threads(threads)
    fl1 = 3 * 2.0 * cv["n"] * cv["cout"] * ho * wo * cv["cin"] * cv["kh"] * cv["kw"]
    out["one_thread"] = {"value": fl1 / t1 / 1e12, "unit": "TFLOP/s", "cores": 1,
                         "sample": f"the 3x3 s1 64->64 56x56 layer in MXFP4, every op of the path: {t1:.1f} s"}
    return out


def naive_calls(jobs, mx, synth, dev):
    """The naive comparator's step for every (layer, format) job as separate
    calls (label "<layer>/<format>/naive_<op>", callable, 0 flops, the op's
    algorithmic bytes): fp32 im2col, the six 1-D quantizations (X' along K
    and along P, W along K and along Cout, G_Y along Cout and along P), the
    three GEMMs (dgrad with its col2im).  Line matrices persist in the
    returned dict so every call can be repeated on its own."""
    import torch
    calls, shared = {}, {}
    for j in jobs:
        cv, fmt = j["cv"], j["fmt"]
        ho, wo = synth.out_hw(cv)
        P, K, co = cv["n"] * ho * wo, cv["kh"] * cv["kw"] * cv["cin"], cv["cout"]
        key = j["name"].split("/")[0]
        if key not in shared:
            x = synth.cbf_to_nchw(j["x"].cpu(), cv["n"], cv["cin"], cv["h"], cv["w"], 32)
            gy = synth.cbf_to_nchw(j["gy"].cpu(), cv["n"], co, ho, wo, 32)
            shared[key] = dict(
                x=x.permute(0, 2, 3, 1).contiguous().to(dev),
                gy=gy.permute(0, 2, 3, 1).reshape(P, co).contiguous().to(dev),
                w=j["w"].permute(0, 2, 3, 1).reshape(co, K).contiguous(),
                col=torch.empty((P, K), dtype=torch.float32, device=dev),
                gcol=torch.empty((P, K), dtype=torch.float32, device=dev),
                y=torch.empty((P, co), dtype=torch.float32, device=dev),
                gx=torch.empty((cv["n"], cv["h"], cv["w"], cv["cin"]), dtype=torch.float32, device=dev),
                gw=torch.empty((co, K), dtype=torch.float32, device=dev))
        b = shared[key]
        q = {}
        nby, _ = naive_numbers(cv, fmt, mx)

        def qd(name, src, d, q=q, fmt=fmt):
            q[name] = mx.naive_quantize_1d(src, d, fmt, out=q.get(name))

        ops = [("im2col_f32", lambda b=b, cv=cv: mx.naive_im2col_f32(cv, b["x"], out=b["col"])),
               ("quant_col_k", lambda b=b, qd=qd: qd("c0", b["col"], 0)),
               ("quant_w_k", lambda b=b, qd=qd: qd("w0", b["w"], 0)),
               ("fwd", lambda b=b, cv=cv, q=q: mx.naive_fwd(cv, q["c0"], q["w0"], out=b["y"])),
               ("quant_gy_co", lambda b=b, qd=qd: qd("g0", b["gy"], 0)),
               ("quant_w_co", lambda b=b, qd=qd: qd("w1", b["w"], 1)),
               ("dgrad", lambda b=b, cv=cv, q=q: mx.naive_dgrad(cv, q["g0"], q["w1"], gcol=b["gcol"], out=b["gx"])),
               ("quant_gy_p", lambda b=b, qd=qd: qd("g1", b["gy"], 1)),
               ("quant_col_p", lambda b=b, qd=qd: qd("c1", b["col"], 1)),
               ("wgrad", lambda b=b, cv=cv, q=q: mx.naive_wgrad(cv, q["g1"], q["c1"], out=b["gw"]))]
        calls[j["name"]] = [(f"{j['name']}/naive_{op}", fn, 0.0, nby[op]) for op, fn in ops]
    return calls


def naive_leg(jobs, op_ms, mx, synth, dev, stream, reps=3):
    """Run the naive comparator once per (layer, format) on the same inputs
    (outside the timed region) and report its time, algorithmic bytes and
    quantized elements beside the method's; with a committed counter summary
    of the same sources, the measured HBM bytes of both too.  The method's
    bytes are its quantize x3 + fwd + dgrad + wgrad (the GEMMs take the
    im2col implicitly)."""
    import torch
    res = {}
    ncalls = naive_calls(jobs, mx, synth, dev)
    ours_ops = ("quant_xw", "quant_gy", "fwd", "dgrad", "wgrad")
    for j in jobs:
        cv, fmt = j["cv"], j["fmt"]
        ho, wo = synth.out_hw(cv)
        P, K, co = cv["n"] * ho * wo, cv["kh"] * cv["kw"] * cv["cin"], cv["cout"]
        calls = ncalls[j["name"]]
        for c in calls:
            c[1]()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SPIN_CYCLES)
        e0.record(stream)
        for _ in range(reps):
            for c in calls:
                c[1]()
        e1.record(stream)
        torch.cuda.synchronize()
        ms_naive = e0.elapsed_time(e1) / reps
        nby, nq = naive_numbers(cv, fmt, mx)
        oby = sum(j["nums"][op][1] for op in ours_ops)
        ms_ours = sum(op_ms[(j["name"], op)] for op in ours_ops)
        nx = cv["n"] * cv["cin"] * cv["h"] * cv["w"]
        oq = nx + co * K + P * co
        r = {"bytes_naive": round(sum(nby.values())), "bytes_ours": round(oby),
             "bytes_ratio": round(sum(nby.values()) / oby, 2),
             "ms_naive": round(ms_naive, 4), "ms_ours": round(ms_ours, 4),
             "speedup": round(ms_naive / ms_ours, 2),
             "quantized_naive": nq, "quantized_ours": oq}
        mo = [counter_traffic(f"sweep/{j['name']}/{op}") for op in ours_ops]
        mn = [counter_traffic(f"sweep/{c[0]}") for c in calls]
        if all(v is not None for v in mo + mn):
            r.update({"bytes_ours_measured": sum(mo), "bytes_naive_measured": sum(mn),
                      "bytes_ratio_measured": round(sum(mn) / sum(mo), 2)})
        res[j["name"]] = r
    return res


def sweep_leg(args):
    """The layer sweep at batch 32 (three layers, MXFP8 and MXFP4) as one
    step, with its per-op times, the naive comparator and the side legs."""
    import torch
    from paper_2609_28358_amd import mxconv as mx
    from paper_2609_28358_amd import synth
    dev = torch.device("cuda:0")

    layers = list(range(len(synth.SWEEP_LAYERS))) if args.layers == "all" else [int(v) for v in args.layers.split(",")]
    fmts = [int(v) for v in args.fmts.split(",")]
    jobs = []
    for li in layers:
        name, cv = synth.SWEEP_LAYERS[li]
        x, w, gy = synth.layer_inputs(cv, 1000 + li, kind="sweep")
        ho, wo = synth.out_hw(cv)
        xs, gs = tuple(x.shape), tuple(gy.shape)
        xd = synth.nchw_to_cbf(x, 32).to(dev)
        gd = synth.nchw_to_cbf(gy, 32).to(dev)
        wd = w.to(dev)
        for fmt in fmts:
            j = dict(name=f"{name}/{FMT_NAME[fmt]}", cv=cv, fmt=fmt, x=xd, w=wd, gy=gd, xs=xs, gs=gs,
                     qx=mx.MxTensor.empty(mx.ACT, fmt, xs, dev), qw=mx.MxTensor.empty(mx.WEIGHT, fmt, tuple(w.shape), dev),
                     qg=mx.MxTensor.empty(mx.ACT, fmt, gs, dev),
                     y=torch.empty((cv["n"] // 32, ho, wo, cv["cout"], 32), dtype=torch.float32, device=dev),
                     gx=torch.empty((cv["n"] // 32, cv["h"], cv["w"], cv["cin"], 32), dtype=torch.float32, device=dev),
                     gw=torch.empty(tuple(w.shape), dtype=torch.float32, device=dev),
                     ws=torch.empty(max(1, mx.wgrad_workspace_bytes(cv, fmt)), dtype=torch.uint8, device=dev),
                     nums=layer_numbers(cv, fmt, mx))
            jobs.append(j)

    stream = torch.cuda.current_stream()
    # a layer's forward operands X and W are quantized together, in one launch
    # that also writes X's explicit CBF im2col (the quantizer copies each block
    # to its im2col positions as it produces it)
    # a layer's input and weight gradients run as one launch (mxconv_backward),
    # and each weight gradient leaves its split-K partial sums for one batched
    # reduction of all layers at the end of the step (as at the end of a
    # backward pass)
    OPS = ("quant_xw_im2col", "quant_gy", "fwd", "backward")
    # timed beside the step, not part of it: the unfused forward-operand
    # quantize, the standalone im2col kernel and the whole weight gradient
    REF_OPS = ("quant_xw", "im2col", "dgrad", "wgrad")

    def run_op(j, op, src=None):
        cv, fmt = j["cv"], j["fmt"]
        if op == "quant_xw_im2col":
            mx.quantize_multi([(j["x"] if src is None else src, mx.ACT, fmt, mx.CBF, j["xs"], j["qx"],
                                (cv, j["col"][0], j["col"][1])),
                               (j["w"], mx.WEIGHT, fmt, mx.NCHW, tuple(j["w"].shape), j["qw"])])
        elif op == "quant_xw":
            mx.quantize_multi([(j["x"] if src is None else src, mx.ACT, fmt, mx.CBF, j["xs"], j["qx"]),
                               (j["w"], mx.WEIGHT, fmt, mx.NCHW, tuple(j["w"].shape), j["qw"])])
        elif op == "quant_x":
            mx.quantize(j["x"] if src is None else src, mx.ACT, fmt, layout=mx.CBF, shape=j["xs"], out=j["qx"])
        elif op == "quant_w":
            mx.quantize(j["w"], mx.WEIGHT, fmt, out=j["qw"])
        elif op == "quant_gy":
            mx.quantize(j["gy"] if src is None else src, mx.ACT, fmt, layout=mx.CBF, shape=j["gs"], out=j["qg"])
        elif op == "fwd":
            mx.fwd(cv, j["qw"], j["qx"], layout=mx.CBF, out=j["y"])
        elif op == "dgrad":
            mx.dgrad(cv, j["qw"], j["qg"], layout=mx.CBF, out=j["gx"])
        elif op == "backward":
            mx.backward(cv, j["qw"], j["qg"], j["qx"], layout=mx.CBF, gx_out=j["gx"], gw_out=j["gw"],
                        workspace=j["ws"], deferred=True)
        else:
            mx.wgrad(cv, j["qg"], j["qx"], out=j["gw"], workspace=j["ws"])

    # the explicit im2col output is written into a preallocated buffer too
    import ctypes
    for j in jobs:
        c = mx.conv_struct(j["cv"])
        j["col"] = (torch.empty(mx.lib().mxconv_im2col_codes_bytes(ctypes.byref(c), j["fmt"]), dtype=torch.uint8, device=dev),
                    torch.empty(mx.lib().mxconv_im2col_scales_bytes(ctypes.byref(c), j["fmt"]), dtype=torch.uint8, device=dev))

    def run_im2col(j):
        c = mx.conv_struct(j["cv"])
        rc = mx.lib().mxconv_im2col_cbf(ctypes.byref(c), j["fmt"], mx._ptr(j["qx"].codes), mx._ptr(j["qx"].scales),
                                        mx._ptr(j["col"][0]), mx._ptr(j["col"][1]), mx._stream(None))
        if rc:
            raise mx.MxconvError(mx.strerror(rc))

    # the step-level op: one launch finishing every layer's weight gradient
    red_bytes = sum(j["ws"].numel() + 4.0 * j["gw"].numel() for j in jobs
                    if mx.wgrad_workspace_bytes(j["cv"], j["fmt"]) > 0)
    step_job = {"name": "all_layers", "nums": {"wgrad_reduce_all": (0.0, red_bytes)}, "fmt": 0}
    seq = [(j, op) for j in jobs for op in OPS] + [(step_job, "wgrad_reduce_all")]

    def run(j, op):
        if op == "im2col":
            run_im2col(j)
        elif op == "wgrad_reduce_all":
            mx.wgrad_reduce_multi([(k["cv"], k["fmt"], k["ws"], k["gw"]) for k in jobs])
        else:
            run_op(j, op)

    def step():
        for j, op in seq:
            run(j, op)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    if args.pmc_pass:
        # every op of the step, the ops timed beside it and the naive
        # comparator's ops, one call each (see pmc_pass)
        calls = [(f"{j['name']}/{op}", (lambda j=j, op=op: run(j, op)), j["nums"][op][0], j["nums"][op][1])
                 for j, op in seq + [(j, op) for j in jobs for op in REF_OPS]]
        nc = naive_calls(jobs, mx, synth, dev)
        for j in jobs:
            calls += nc[j["name"]]
        for c in calls:
            c[1]()
        return pmc_pass(calls, "sweep")

    # Per-op GPU time: each op alone, behind a GPU spin so that the event pair
    # brackets the kernel(s) and not the host's launch latency.
    def op_time(j, op, reps=5):
        marks = []
        for _ in range(reps):
            torch.cuda._sleep(SPIN_CYCLES)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            run(j, op)
            e1.record(stream)
            marks.append((e0, e1))
        torch.cuda.synchronize()
        return sum(a.elapsed_time(b) for a, b in marks) / reps

    op_ms = {(j["name"], op): op_time(j, op) for j, op in seq + [(j, op) for j in jobs for op in REF_OPS]}

    # The step is launched as one HIP graph (captured once), so host-side
    # launch cost does not enter the step time.
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for _ in range(2):
        graph.replay()
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps

    # Steady-state kernel time of every op: a graph of back-to-back launches,
    # replayed.  Quantize sources rotate over copies totalling more than the
    # last-level cache, so that they come from HBM as they do in the step.
    def replay_ms(g, reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    import statistics
    LLC_BYTES = 256 << 20

    def rotated(base):
        # copies of a quantize source that together exceed the last-level cache
        ncopy = min(48, -(-(LLC_BYTES + (64 << 20)) // (base.numel() * base.element_size())))
        return [base] + [base.clone() for _ in range(ncopy - 1)]

    # measured device-copy bandwidth (read + write bytes / time) beside the
    # 8 TB/s datasheet peak: a graph of back-to-back 256 MiB copies
    csrc = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev)
    cdst = torch.empty_like(csrc)
    cdst.copy_(csrc)
    torch.cuda.synchronize()
    cg = torch.cuda.CUDAGraph()
    with torch.cuda.graph(cg):
        for _ in range(8):
            cdst.copy_(csrc)
    cg.replay()
    torch.cuda.synchronize()
    copy_ms = statistics.median(replay_ms(cg, 3) for _ in range(3)) / 8
    hbm_copy_gbps = 2 * COPY_BYTES / (copy_ms * 1e-3) / 1e9
    del cg, csrc, cdst

    steady = {}
    for j, op in seq + [(j, op) for j in jobs for op in REF_OPS]:
        srcs = [None]
        if op in ("quant_xw_im2col", "quant_xw", "quant_x", "quant_gy"):
            srcs = rotated(j["gy"] if op == "quant_gy" else j["x"])
        kl = max(12, len(srcs))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for k in range(kl):
                run_op(j, op, srcs[k % len(srcs)]) if op not in ("im2col", "wgrad_reduce_all") else run(j, op)
        g.replay()
        torch.cuda.synchronize()
        steady[(j["name"], op)] = statistics.median(replay_ms(g, 3) for _ in range(3)) / kl
        del g, srcs
    in_step = {(j["name"], op) for j, op in seq}
    dom = max(in_step, key=steady.get)
    dom_ms = steady[dom]

    naive = {} if args.no_naive else naive_leg(jobs, op_ms, mx, synth, dev, stream)

    # Fused quantizing epilogues (outside the step): the forward with its
    # output quantized in the epilogue (after SiLU, or none) against the
    # forward writing fp32 followed by a quantize of that output; the input
    # gradient likewise (SiLU' mask at a pre-activation z, or none).
    def steady_ms(fn, kl=12):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(kl):
                fn()
        g.replay()
        torch.cuda.synchronize()
        r = statistics.median(replay_ms(g, 3) for _ in range(3)) / kl
        del g
        return r

    fused = {}
    if not args.no_fused:
        for j in jobs:
            cv, fmt = j["cv"], j["fmt"]
            ho, wo = synth.out_hw(cv)
            ysh, xsh = (cv["n"], cv["cout"], ho, wo), (cv["n"], cv["cin"], cv["h"], cv["w"])
            yq = mx.MxTensor.empty(mx.ACT, fmt, ysh, dev)
            gq = mx.MxTensor.empty(mx.ACT, fmt, xsh, dev)
            z = j["x"]                                   # a CBF fp32 tensor of X's shape
            t = {
                "fwd_quant_silu": steady_ms(lambda: mx.fwd_quant(cv, j["qw"], j["qx"], fn=mx.FN_SILU, out=yq)),
                "fwd_quant": steady_ms(lambda: mx.fwd_quant(cv, j["qw"], j["qx"], out=yq)),
                "fwd_then_quantize": steady_ms(lambda: (run_op(j, "fwd"), mx.quantize(
                    j["y"], mx.ACT, fmt, layout=mx.CBF, shape=ysh, out=yq))),
                "dgrad_quant_silu": steady_ms(lambda: mx.dgrad_quant(cv, j["qw"], j["qg"], fn=mx.FN_SILU, z=z,
                                                                     out=gq)),
                "dgrad_quant": steady_ms(lambda: mx.dgrad_quant(cv, j["qw"], j["qg"], out=gq)),
                "dgrad_then_quantize": steady_ms(lambda: (run_op(j, "dgrad"), mx.quantize(
                    j["gx"], mx.ACT, fmt, layout=mx.CBF, shape=xsh, out=gq))),
            }
            W = mx.codes_bytes(mx.WEIGHT, fmt, *j["w"].shape) + mx.scales_bytes(mx.WEIGHT, fmt, *j["w"].shape)
            Xq = mx.codes_bytes(mx.ACT, fmt, *xsh) + mx.scales_bytes(mx.ACT, fmt, *xsh)
            Yq = mx.codes_bytes(mx.ACT, fmt, *ysh) + mx.scales_bytes(mx.ACT, fmt, *ysh)
            ny, nx = 4.0 * math.prod(ysh), 4.0 * math.prod(xsh)
            fl = j["nums"]["fwd"][0]
            fused[j["name"]] = {k + "_ms": round(v, 4) for k, v in t.items()}
            fused[j["name"]].update({
                "fwd_bytes_fused": round(W + Xq + Yq), "fwd_bytes_unfused": round(W + Xq + 2 * ny + Yq),
                "dgrad_bytes_fused": round(W + Yq + Xq), "dgrad_bytes_unfused": round(W + Yq + 2 * nx + Xq),
                "fwd_quant_tflops": round(fl / (t["fwd_quant"] * 1e-3) / 1e12, 1),
                "fwd_speedup": round(t["fwd_then_quantize"] / t["fwd_quant"], 2),
                "dgrad_speedup": round(t["dgrad_then_quantize"] / t["dgrad_quant"], 2)})

    # FP6 methods (outside the step): the same layers and ops with the FP6
    # operand formats, timed like `ops` (steady state, quantize sources
    # rotated through HBM), against the MXFP4 layer of the step.
    fp6 = {}
    if not args.no_fp6:
        def mxbytes(role, f, shape):
            b = mx.codes_bytes(role, f, *shape) + mx.scales_bytes(role, f, *shape)
            return b - (FP6_SLACK if f in (2, 3) else 0)

        seen = set()
        for j in jobs:
            cv = j["cv"]
            lname = j["name"].split("/")[0]
            if lname in seen:
                continue
            seen.add(lname)
            ho, wo = synth.out_hw(cv)
            wsh = tuple(j["w"].shape)
            xsrc, gsrc = rotated(j["x"]), rotated(j["gy"])
            fl = j["nums"]["fwd"][0]
            for meth, (fw, fx, fg) in FP6_METHODS.items():
                qx = mx.MxTensor.empty(mx.ACT, fx, j["xs"], dev)
                qw = mx.MxTensor.empty(mx.WEIGHT, fw, wsh, dev)
                qg = mx.MxTensor.empty(mx.ACT, fg, j["gs"], dev)
                wsb = torch.empty(max(1, mx.wgrad_workspace_bytes(cv, mx.pair(fg, fx))), dtype=torch.uint8, device=dev)
                it = {"x": 0, "g": 0}

                def qxwr():     # X and W in one call, as the MXFP4 layer's quant_xw
                    it["x"] += 1
                    mx.quantize_multi([(xsrc[it["x"] % len(xsrc)], mx.ACT, fx, mx.CBF, j["xs"], qx),
                                       (j["w"], mx.WEIGHT, fw, mx.NCHW, wsh, qw)])

                def qgr():
                    it["g"] += 1
                    mx.quantize(gsrc[it["g"] % len(gsrc)], mx.ACT, fg, layout=mx.CBF, shape=j["gs"], out=qg)

                qxwr(); qgr()
                kq = max(12, len(xsrc), len(gsrc))
                t = {"quant_xw": steady_ms(qxwr, kq),
                     "quant_gy": steady_ms(qgr, kq)}
                qxwr(); qgr()
                t["fwd"] = steady_ms(lambda: mx.fwd(cv, qw, qx, layout=mx.CBF, out=j["y"]))
                t["dgrad"] = steady_ms(lambda: mx.dgrad(cv, qw, qg, layout=mx.CBF, out=j["gx"]))
                t["wgrad"] = steady_ms(lambda: mx.wgrad(cv, qg, qx, out=j["gw"], workspace=wsb))
                X, W, G = mxbytes(mx.ACT, fx, j["xs"]), mxbytes(mx.WEIGHT, fw, wsh), mxbytes(mx.ACT, fg, j["gs"])
                # the MXFP4 layer measured the same way (every op timed beside or in the step)
                fp4 = sum(steady[(f"{lname}/mxfp4", op)] for op in ("quant_xw", "quant_gy", "fwd", "dgrad", "wgrad"))
                r = {k + "_ms": round(v, 4) for k, v in t.items()}
                r.update({"fwd_tflops": round(fl / (t["fwd"] * 1e-3) / 1e12, 1),
                          "dgrad_tflops": round(fl / (t["dgrad"] * 1e-3) / 1e12, 1),
                          "wgrad_tflops": round(fl / (t["wgrad"] * 1e-3) / 1e12, 1),
                          "quant_xw_gbps": round((4.0 * math.prod(j["xs"]) + X + 4.0 * math.prod(wsh) + W)
                                                 / (t["quant_xw"] * 1e-3) / 1e9, 1),
                          "x_bytes": X, "w_bytes": W, "gy_bytes": G,
                          "layer_ms": round(sum(t.values()), 4)})
                if fp4:
                    r["layer_ms_vs_mxfp4"] = round(sum(t.values()) / fp4, 3)
                fp6[f"{lname}/{meth}"] = r
            del xsrc, gsrc

    # Stochastic rounding (outside the step): the gradient quantize with
    # Eq. (6)'s stochastic option against the round-to-nearest one of the
    # step, same source rotation.
    sr = {}
    if not args.no_sr:
        for j in jobs:
            fmt = j["fmt"]
            gsrc = rotated(j["gy"])
            it = [0]

            def qsr():
                it[0] += 1
                mx.quantize_sr(gsrc[it[0] % len(gsrc)], mx.ACT, fmt, 7 + it[0], layout=mx.CBF, shape=j["gs"],
                               out=j["qg"])

            t_sr = steady_ms(qsr, max(12, len(gsrc)))
            t_rn = steady[(j["name"], "quant_gy")]
            by = j["nums"]["quant_gy"][1]
            sr[j["name"]] = {"quant_gy_sr_ms": round(t_sr, 4), "quant_gy_ms": round(t_rn, 4),
                             "sr_gbps": round(by / (t_sr * 1e-3) / 1e9, 1), "sr_over_rn": round(t_sr / t_rn, 3)}
            del gsrc
        # leave the step's G_Y codes as the round-to-nearest quantize made them
        for j in jobs:
            run_op(j, "quant_gy")
        torch.cuda.synchronize()

    # The paper-literal NVFP4 format (outside the step): per layer, the two-
    # launch quantize of X, W and G_Y and the three GEMMs on fp16 MFMAs,
    # timed like `ops`, against the MXFP4 layer of the step.
    nvfp = {}
    if not args.no_nvfp:
        seen = set()
        for j in jobs:
            cv = j["cv"]
            lname = j["name"].split("/")[0]
            if lname in seen:
                continue
            seen.add(lname)
            wsh = tuple(j["w"].shape)
            xsrc, gsrc = rotated(j["x"]), rotated(j["gy"])
            wsn = torch.empty(mx.lib().mxconv_nvfp_workspace_bytes(), dtype=torch.uint8, device=dev)
            it = {"x": 0, "g": 0}
            qx = mx.nvfp_quantize(j["x"], mx.ACT, 1, layout=mx.CBF, shape=j["xs"], workspace=wsn)
            qw = mx.nvfp_quantize(j["w"], mx.WEIGHT, 1, workspace=wsn)
            qg = mx.nvfp_quantize(j["gy"], mx.ACT, 1, layout=mx.CBF, shape=j["gs"], workspace=wsn)

            def nq(t, src_list, key, shape):
                it[key] += 1
                c = mx.lib().mxconv_nvfp_quantize(
                    mx._ptr(src_list[it[key] % len(src_list)]), mx.F32, mx.CBF, mx.ACT, 1, *shape,
                    mx._ptr(t.codes), mx._ptr(t.scales), mx._ptr(t.tscale), mx._ptr(wsn), wsn.numel(), mx._stream(None))
                if c:
                    raise mx.MxconvError(mx.strerror(c))

            kq = max(12, len(xsrc), len(gsrc))
            ws4 = torch.empty(max(1, mx.wgrad_workspace_bytes(cv, 1)), dtype=torch.uint8, device=dev)
            t = {"quant_x": steady_ms(lambda: nq(qx, xsrc, "x", j["xs"]), kq),
                 "quant_w": steady_ms(lambda: mx.nvfp_quantize(j["w"], mx.WEIGHT, 1, workspace=wsn)),
                 "quant_gy": steady_ms(lambda: nq(qg, gsrc, "g", j["gs"]), kq),
                 "fwd": steady_ms(lambda: mx.nvfp_fwd(cv, qw, qx, layout=mx.CBF, out=j["y"])),
                 "dgrad": steady_ms(lambda: mx.nvfp_dgrad(cv, qw, qg, layout=mx.CBF, out=j["gx"])),
                 "wgrad": steady_ms(lambda: mx.nvfp_wgrad(cv, qg, qx, out=j["gw"], workspace=ws4))}
            fl = j["nums"]["fwd"][0]
            fp4 = sum(steady[(f"{lname}/mxfp4", op)] for op in ("quant_xw", "quant_gy", "fwd", "dgrad", "wgrad"))
            r = {k + "_ms": round(v, 4) for k, v in t.items()}
            r.update({g + "_tflops": round(fl / (t[g] * 1e-3) / 1e12, 1) for g in ("fwd", "dgrad", "wgrad")})
            r["layer_ms"] = round(sum(t.values()), 4)
            r["layer_ms_vs_mxfp4"] = round(sum(t.values()) / fp4, 3)
            nvfp[f"{lname}/nvfp4"] = r
            # the GEMMs of the other NVFP methods: (W, X, G_Y) element formats
            for meth, (fw_, fx_, fg_) in NV_METHODS.items():
                mw = mx.nvfp_quantize(j["w"], mx.WEIGHT, fw_, workspace=wsn)
                mxq = mx.nvfp_quantize(j["x"], mx.ACT, fx_, layout=mx.CBF, shape=j["xs"], workspace=wsn)
                mg = mx.nvfp_quantize(j["gy"], mx.ACT, fg_, layout=mx.CBF, shape=j["gs"], workspace=wsn)
                wsm = torch.empty(max(1, mx.wgrad_workspace_bytes(cv, mx.pair(fg_, fx_))), dtype=torch.uint8,
                                  device=dev)
                tm = {"fwd": steady_ms(lambda: mx.nvfp_fwd(cv, mw, mxq, layout=mx.CBF, out=j["y"])),
                      "dgrad": steady_ms(lambda: mx.nvfp_dgrad(cv, mw, mg, layout=mx.CBF, out=j["gx"])),
                      "wgrad": steady_ms(lambda: mx.nvfp_wgrad(cv, mg, mxq, out=j["gw"], workspace=wsm))}
                rm = {k + "_ms": round(v, 4) for k, v in tm.items()}
                rm.update({g + "_tflops": round(fl / (tm[g] * 1e-3) / 1e12, 1) for g in tm})
                nvfp[f"{lname}/{meth}"] = rm
                del mw, mxq, mg, wsm
            del xsrc, gsrc

    gemm_flops = sum(j["nums"][op][0] for j in jobs for op in ("fwd", "dgrad", "wgrad"))
    value = gemm_flops / (ms_step * 1e-3) / 1e12

    def roof(job, op, ms):
        fl, by = job["nums"][op]
        fmt = job["fmt"]
        ai = fl / by if by else 0.0
        hbm_bound = fl == 0 or ai * HBM_GBS * 1e9 < MFMA_TFLOPS[fmt] * 1e12
        if hbm_bound:
            ach = by / (ms * 1e-3) / 1e9
            return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_GBS, "unit": "GB/s",
                    "frac": round(ach / HBM_GBS, 4)}
        ach = fl / (ms * 1e-3) / 1e12
        return {"bound": "mfma", "achieved": round(ach, 1), "peak": MFMA_TFLOPS[fmt], "unit": "TFLOP/s",
                "frac": round(ach / MFMA_TFLOPS[fmt], 4)}

    jmap = {j["name"]: j for j in jobs + [step_job]}
    rl = roof(jmap[dom[0]], dom[1], dom_ms)
    rl.update({"kernel": f"{dom[1]} {dom[0]}", "ms": round(dom_ms, 4),
               "ms_alone": round(op_ms[dom], 4),
               "traffic": counter_traffic(f"sweep/{dom[0]}/{dom[1]}")})
    ops = {}
    for (nm, op), ms in steady.items():
        fl, by = jmap[nm]["nums"][op]
        r = roof(jmap[nm], op, ms)
        ops[f"{nm}/{op}"] = {"ms": round(ms, 4), "ms_alone": round(op_ms[(nm, op)], 4),
                             "tflops": round(fl / (ms * 1e-3) / 1e12, 2) if fl else None,
                             "gbps": round(by / (ms * 1e-3) / 1e9, 1), "bound": r["bound"], "frac": r["frac"],
                             "in_step": (nm, op) in in_step}
        if fl:   # a GEMM: also its fraction of the MFMA peak, whatever bounds it
            ops[f"{nm}/{op}"]["mfma_frac"] = round(fl / (ms * 1e-3) / 1e12 / MFMA_TFLOPS[jmap[nm]["fmt"]], 4)

    out = {
        "value": round(value, 2), "unit": "TFLOP/s", "ms_per_step": round(ms_step, 4),
        "workload": "conv layer sweep, batch 32: 3x3 s1 64->64 56x56, 1x1 64->256 56x56, 3x3 s2 128->256 28x28; "
                    "each in MXFP8 and MXFP4; quantize X+W with X's CBF im2col (one launch) + quantize G_Y + fwd + "
                    "dgrad and wgrad in one launch per layer, the six weight gradients' split-K reductions in one "
                    "launch at the end",
        "layers": [n for n, _ in synth.SWEEP_LAYERS], "formats": ["mxfp8", "mxfp4"],
        "roofline": rl,
        "ops": ops,
        "ops_sum_ms": round(sum(steady[k] for k in in_step), 4),
        "hbm_copy_gbps": round(hbm_copy_gbps, 1),
    }
    if naive:
        out["vs_naive"] = naive
    if fused:
        out["fused_epilogues"] = fused
    if fp6:
        out["fp6_methods"] = fp6
    if sr:
        out["stochastic_rounding"] = sr
    if nvfp:
        out["nvfp4"] = nvfp
    return out


def roofline(fl, by, ms, fmt):
    """Roofline of one op from its algorithmic flops / bytes and time: HBM when
    its arithmetic intensity is below the ridge of its format's MFMA peak."""
    ai = fl / by if by else 0.0
    if fl == 0 or ai * HBM_GBS * 1e9 < MFMA_TFLOPS[fmt] * 1e12:
        ach = by / (ms * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_GBS, "unit": "GB/s", "frac": round(ach / HBM_GBS, 4)}
    ach = fl / (ms * 1e-3) / 1e12
    return {"bound": "mfma", "achieved": round(ach, 1), "peak": MFMA_TFLOPS[fmt], "unit": "TFLOP/s",
            "frac": round(ach / MFMA_TFLOPS[fmt], 4)}


def spin_rate():
    """GPU spin cycles per millisecond of torch.cuda._sleep (measured)."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    torch.cuda._sleep(2_000_000)
    e1.record()
    torch.cuda.synchronize()
    return 2_000_000 / max(e0.elapsed_time(e1), 1e-3)


def instep_times(calls, reps=3):
    """Duration of every call inside the step: the whole step enqueued
    eagerly behind a GPU spin long enough for the host to enqueue every
    call first, with a HIP event recorded on the step's stream between
    consecutive calls; mean over `reps` steps (ms per call)."""
    import torch
    stream = torch.cuda.current_stream()
    rate = spin_rate()
    # host enqueue time of one step, measured, with a wide margin
    t0 = time.perf_counter()
    for c in calls:
        c[1]()
    torch.cuda.synchronize()
    host_ms = (time.perf_counter() - t0) * 1e3
    cycles = int(rate * (3.0 * host_ms + 5.0))
    acc = [0.0] * len(calls)
    for _ in range(reps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]
        torch.cuda._sleep(cycles)
        ev[0].record(stream)
        for i, c in enumerate(calls):
            c[1]()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        for i in range(len(calls)):
            acc[i] += ev[i].elapsed_time(ev[i + 1]) / reps
    return acc


def step_leg(calls, flops, fmt, args, top=16):
    """Time one network step: warm-up, then the step captured once into a HIP
    graph and replayed args.steps times between synchronizations (value =
    the step's GEMM flops / wall time); every call's in-step duration; the
    roofline of the call that takes longest."""
    import torch
    for _ in range(args.warmup):
        for c in calls:
            c[1]()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for c in calls:
            c[1]()
    for _ in range(2):
        g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        g.replay()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    del g
    ins = instep_times(calls)
    rows = []
    for (lab, _, fl, by), ms in zip(calls, ins):
        r = roofline(fl, by, ms, fmt)
        row = {"call": lab, "ms": round(ms, 4), "bound": r["bound"], "frac": r["frac"],
               "gbps": round(by / (ms * 1e-3) / 1e9, 1) if ms > 0 else None}
        if fl:
            row["tflops"] = round(fl / (ms * 1e-3) / 1e12, 1)
            row["mfma_frac"] = round(fl / (ms * 1e-3) / 1e12 / MFMA_TFLOPS[fmt], 4)
        rows.append(row)
    dom = max(range(len(calls)), key=lambda i: ins[i])
    rl = roofline(calls[dom][2], calls[dom][3], ins[dom], fmt)
    rl.update({"kernel": calls[dom][0], "ms": round(ins[dom], 4), "algorithmic_flops": calls[dom][2],
               "algorithmic_bytes": calls[dom][3]})
    kinds = {}
    for row in rows:
        k = row["call"].split(" ")[0].rstrip("0123456789")
        kinds[k] = round(kinds.get(k, 0.0) + row["ms"], 4)
    return {"ms_per_step": round(ms_step, 4), "value": round(flops / (ms_step * 1e-3) / 1e12, 2),
            "gemm_gflop": round(flops / 1e9, 2), "calls": len(calls), "instep_sum_ms": round(sum(ins), 4),
            "ms_by_kind": kinds, "roofline": rl,
            "top_calls": sorted(rows, key=lambda r: -r["ms"])[:top], "all_calls": rows}


def net_bytes_vs_naive(net, n, fmt):
    """Per convolution of the network: algorithmic bytes of one layer step of
    the method (quantize X, W, G_Y once; the three GEMMs on MX operands,
    im2col implicit) against the naive comparator's (fp32 im2col, six 1-D
    quantizations, three GEMMs, col2im), by the same byte model as the layer
    sweep's measured comparison, and the elements each quantizes."""
    from paper_2609_28358_amd import mxconv as mx
    from paper_2609_28358_amd import workloads as wl
    per, ours_t, naive_t = {}, 0.0, 0.0
    for t in net.convs():
        cv = wl.conv_dict(t, n)
        nums = layer_numbers(cv, fmt, mx)
        ours = sum(nums[op][1] for op in ("quant_xw", "quant_gy", "fwd", "dgrad", "wgrad"))
        nby, nq = naive_numbers(cv, fmt, mx)
        nv = sum(nby.values())
        ho, wo = t["h"], t["w"]
        oq = n * cv["cin"] * cv["h"] * cv["w"] + cv["cout"] * cv["cin"] * cv["kh"] * cv["kw"] + n * cv["cout"] * ho * wo
        per[t["name"]] = {"k": t["k"], "s": t["s"], "bytes_ours": round(ours), "bytes_naive": round(nv),
                          "ratio": round(nv / ours, 2), "quantized_ours": oq, "quantized_naive": nq}
        ours_t += ours
        naive_t += nv
    return {"total_bytes_ours": round(ours_t), "total_bytes_naive": round(naive_t),
            "total_ratio": round(naive_t / ours_t, 2),
            "layers_at_least_3x": sum(1 for v in per.values() if v["ratio"] >= 3.0), "layers": per}


def cpu_baseline_net(net, n=32, fmt=1, min_s=10.0, max_s=30.0):
    """The oracle on a bounded sample of the network workload: the network's
    convolutions in order, each at one 32-sample group with its real shape
    -- quantize X, W and G_Y (seeded synthetic tensors), then fwd, dgrad and
    wgrad in fp64 -- until at least min_s seconds of oracle time."""
    import oracle
    from paper_2609_28358_amd import synth
    from paper_2609_28358_amd import workloads as wl
    flops, dt, done = 0.0, 0.0, []
    for li, t in enumerate(net.convs()):
        if dt >= min_s:
            break
        cv = wl.conv_dict(t, n)
        x, w, gy = synth.layer_inputs(cv, 7000 + li, kind="sweep")
        f = 2.0 * n * cv["cout"] * t["h"] * t["w"] * cv["cin"] * cv["kh"] * cv["kw"]
        if dt + 3 * f / 2.0e10 > max_s:     # would overrun the bound at about 0.02 TFLOP/s
            continue
        t0 = time.perf_counter()
        ox = oracle.quantize(x.numpy(), oracle.NCHW, oracle.ACT, fmt, *x.shape)
        ow = oracle.quantize(w.numpy(), oracle.NCHW, oracle.WEIGHT, fmt, *w.shape)
        og = oracle.quantize(gy.numpy(), oracle.NCHW, oracle.ACT, fmt, *gy.shape)
        oracle.fwd(cv, fmt, ow, ox)
        oracle.dgrad(cv, fmt, ow, og)
        oracle.wgrad(cv, fmt, og, ox)
        dt += time.perf_counter() - t0
        flops += 3 * f
        done.append(t["name"])
    return {"value": round(flops / dt / 1e12, 5), "unit": "TFLOP/s", "cores": oracle.get_threads(), "kind": "oracle",
            "sample": f"{len(done)} of the network's {len(net.convs())} convolutions in order ({done[0]} .. {done[-1]}), "
                      f"each at one 32-sample group of its real shape with seeded inputs: quantize X, W, G_Y, then "
                      f"fwd, dgrad and wgrad through the fp64 oracle; {dt:.1f} s, {flops / 1e9:.1f} GFLOP "
                      f"(the flops as the padded channels the oracle computes)"}


def pmc_pass(calls, label):
    """Counter pass: every call of the step once (eager), each preceded by a
    GPU spin kernel that delimits its dispatches in the counter output, then
    a 256 MiB device copy three times (the calibration)."""
    import torch
    torch.cuda.synchronize()
    for c in calls:
        torch.cuda._sleep(100)
        c[1]()
        torch.cuda.synchronize()
    torch.cuda._sleep(100)
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    return {"pmc_pass": label, "calls": [c[0] for c in calls], "algorithmic_bytes": [c[3] for c in calls],
            "algorithmic_flops": [c[2] for c in calls], "copy_bytes": COPY_BYTES, "source_digest": source_digest()}


def _bench_line(log):
    with open(log) as f:
        for line in f:
            if line.startswith("{"):
                try:
                    d = json.loads(line)
                except ValueError:
                    continue
                if "metric" in d or "pmc_pass" in d:
                    return d
    raise SystemExit(f"no bench JSON line in {log}")


def _csv_rows(d, suffix):
    import csv
    import glob
    paths = sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True))
    if not paths:
        raise SystemExit(f"no *{suffix} under {d}")
    with open(paths[0]) as f:
        return list(csv.DictReader(f))


def _short(name):
    return name.replace("mxc::(anonymous namespace)::", "").replace("void ", "").split("(")[0]


def summarize_trace(rdir, log):
    """Markdown summary of `rocprofv3 --kernel-trace --stats` over a default
    run of this script: the YOLO-shaped step's kernels in step order (median
    duration over every occurrence of the step in the run, beside the
    in-step times the bench line measured with HIP events), the roofline
    kernel's average, and every kernel of the run."""
    import statistics
    bench = _bench_line(log)
    calls = bench["yolo_step"]["all_calls"]
    rows = _csv_rows(rdir, "kernel_trace.csv")
    ks = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), _short(r["Kernel_Name"]),
                 int(r["Grid_Size_X"]) // max(1, int(r["Workgroup_Size_X"])), r) for r in rows)
    # the library's kernels only (not the runtime's copies and fills, nor torch's)
    ks = [k for k in ks if not k[4]["Kernel_Name"].startswith(("at::", "void at::", "__amd_rocclr"))]
    n = len(calls)
    # the step's kernel signature: the first n kernels of the run (its first warm-up step)
    sig = [(k[2], k[3]) for k in ks[:n]]
    wins, i = [], 0
    while i + n <= len(ks):
        if [(k[2], k[3]) for k in ks[i:i + n]] == sig:
            wins.append(ks[i:i + n])
            i += n
        else:
            i += 1
    L = ["# Kernel trace: YOLOv8n-shaped fwd+bwd step, batch 64, MXFP4\n"]
    L.append("Command (repository root on an MI355X machine, <out> an output directory; summary written by bench.py --summarize-trace):\n")
    L.append("    cd /tmp && export TMPDIR=/tmp && rocprofv3 --kernel-trace --stats --output-format csv "
             "-d <out>/ktrace -o run -- python3 <repo>/bench.py > <out>/ktrace.log\n")
    rl = bench["roofline"]
    L.append(f"Bench line of the same run: value {bench['value']} TFLOP/s, {bench['ms_per_step']} ms per step; "
             f"roofline call `{rl['kernel']}` {rl['ms'] * 1000:.1f} us in the step (bound {rl['bound']}, achieved "
             f"{rl['achieved']} {rl['unit']}, frac {rl['frac']}).\n")
    if not wins:
        L.append("The step's kernel sequence was not found as a repeating window; per-kernel stats only.\n")
    else:
        L.append(f"{len(wins)} occurrences of the step's {n}-kernel sequence in the trace (warm-up, graph replays, "
                 f"in-step timing runs); kernel i of the sequence is call i of the step.\n")
        L.append("| # | call | kernel | workgroups | median us (trace) | in-step us (bench, HIP events) |")
        L.append("|---|---|---|---|---|---|")
        dom = None
        for j in range(n):
            d = statistics.median([(w[j][1] - w[j][0]) / 1000 for w in wins])
            if calls[j]["call"] == rl["kernel"]:
                dom = (j, d)
            L.append(f"| {j} | {calls[j]['call']} | {sig[j][0]} | {sig[j][1]} | {d:.1f} | {calls[j]['ms'] * 1000:.1f} |")
        span = statistics.median([(w[-1][1] - w[0][0]) / 1000 for w in wins])
        L.append(f"\nMedian span of one step occurrence: {span:.1f} us (bench ms_per_step {bench['ms_per_step'] * 1000:.1f} us).\n")
        if dom:
            j, d = dom
            ds = [(w[j][1] - w[j][0]) / 1000 for w in wins]
            L.append(f"## Roofline call `{rl['kernel']}`\n")
            L.append(f"- kernel `{sig[j][0]}`, {sig[j][1]} workgroups: average {statistics.mean(ds):.1f} us over "
                     f"{len(ds)} launches in the trace (median {d:.1f} us); bench.py in-step {rl['ms'] * 1000:.1f} us\n")
    stats = {}
    for k in ks:
        stats.setdefault((k[2], k[3]), []).append((k[1] - k[0]) / 1000)
    tot = sum(sum(v) for v in stats.values())
    L.append("## Kernels of the run by total GPU time (top 30)\n")
    L.append("| kernel | workgroups | calls | avg us | min us | max us | % of GPU time |")
    L.append("|---|---|---|---|---|---|---|")
    for key, v in sorted(stats.items(), key=lambda kv: -sum(kv[1]))[:30]:
        L.append(f"| {key[0]} | {key[1]} | {len(v)} | {statistics.mean(v):.1f} | {min(v):.1f} | {max(v):.1f} | "
                 f"{100 * sum(v) / tot:.1f} |")
    return "\n".join(L) + "\n"


def summarize_pmc(fdir, wdir, flog, wlog):
    """Markdown summary of two `rocprofv3 --pmc` runs (FETCH_SIZE, then
    WRITE_SIZE) of `bench.py --pmc-pass <workload>`: every call's counters
    (KiB per dispatch, summed over its kernels; calls are delimited by the
    spin kernel the pass launches before each), scaled by what the same
    counter reads for the pass's 256 MiB copy, beside its algorithmic bytes."""
    fi, wi = _bench_line(flog), _bench_line(wlog)
    assert fi["calls"] == wi["calls"] and fi["source_digest"] == wi["source_digest"]

    def per_call(d, ctr):
        rows = [r for r in _csv_rows(d, "counter_collection.csv") if r["Counter_Name"] == ctr]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        segs, cur = [], None
        for r in rows:
            nm = _short(r["Kernel_Name"])
            if "spin_kernel" in r["Kernel_Name"]:
                cur = []
                segs.append(cur)
            elif cur is not None:
                cur.append((nm, float(r["Counter_Value"])))
        segs = segs[-(len(fi["calls"]) + 1):]       # the pass: one segment per call, then the copies
        if len(segs) != len(fi["calls"]) + 1:
            raise SystemExit(f"{ctr}: found {len(segs)} delimited segments, expected {len(fi['calls']) + 1}")
        copy = sorted(v for _, v in segs[-1])
        return segs[:-1], copy[len(copy) // 2]

    fs, fcopy = per_call(fdir, "FETCH_SIZE")
    ws, wcopy = per_call(wdir, "WRITE_SIZE")
    kib = fi["copy_bytes"] / 1024
    ff, wf = kib / fcopy, kib / wcopy
    label = fi["pmc_pass"]
    L = [f"# HBM traffic per call from FETCH_SIZE / WRITE_SIZE counters: {label} step\n"]
    L.append("Two counter passes over the same command, one counter each (repository root on an MI355X machine, "
             "<out> an output directory; "
             "summary by bench.py --summarize-pmc):\n")
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        L.append(f"    cd /tmp && export TMPDIR=/tmp && timeout -s KILL 180 rocprofv3 --pmc {c} --output-format csv "
                 f"-d <out>/pmc_{label}_{c} -o p -- python3 <repo>/bench.py --pmc-pass {label} --warmup 2 "
                 f"> <out>/pmc_{label}_{c}.log")
    L.append("\nThe pass runs every call of the step once (eager, in step order, each after a spin kernel that "
             "delimits it), then copies 256 MiB device to device three times; the counters of that copy "
             f"calibrate both: FETCH_SIZE {fcopy:.1f} KiB, WRITE_SIZE {wcopy:.1f} KiB for {kib:.0f} KiB moved.\n")
    L.append(f"fetch factor: {ff:.4f}\n\nwrite factor: {wf:.4f}\n")
    L.append(f"source digest: `{fi['source_digest']}`\n")
    L.append("| call | kernels | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM bytes (calibrated) | algorithmic bytes | ratio |")
    L.append("|---|---|---|---|---|---|---|")
    for c, a, f, w in zip(fi["calls"], fi["algorithmic_bytes"], fs, ws):
        fk, wk = sum(v for _, v in f), sum(v for _, v in w)
        hb = (fk * ff + wk * wf) * 1024
        names = "+".join(sorted({nm for nm, _ in f}))
        L.append(f"| {label}/{c} | {names} | {fk:.1f} | {wk:.1f} | {hb:.0f} | {a:.0f} | {hb / a if a else 0:.2f} |")
    return "\n".join(L) + "\n"


# Shader-sequencer counters of the MFMA-heavy calls, two passes of eight
SQ_PASSES = (("SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_VALU_MFMA_BUSY_CYCLES",
              "SQ_INSTS_MFMA", "SQ_ACTIVE_INST_ANY", "SQ_BUSY_CYCLES"),
             ("SQ_WAVES", "SQ_INSTS_LDS", "SQ_INSTS_VALU", "SQ_INSTS_SALU", "SQ_INSTS_VMEM", "SQ_WAIT_INST_LDS",
              "SQ_LDS_BANK_CONFLICT", "SQ_ACTIVE_INST_LDS"))


def summarize_sq(log, *dirs):
    """Markdown summary of `rocprofv3 --pmc` runs with the SQ_PASSES counter
    sets over `bench.py --pmc-pass <workload>`: for every call with matrix
    products, where its waves spend their time (wave-cycles waiting, matrix
    core busy cycles, instructions issued per wave)."""
    import statistics
    info = _bench_line(log)
    calls, flops = info["calls"], info["algorithmic_flops"]
    vals = [dict() for _ in calls]
    durs = [None] * len(calls)
    names = [set() for _ in calls]
    for d in dirs:
        disp = {}
        for r in _csv_rows(d, "counter_collection.csv"):
            disp.setdefault(int(r["Dispatch_Id"]), []).append(r)
        segs, cur = [], None
        for k in sorted(disp):
            if "spin_kernel" in disp[k][0]["Kernel_Name"]:
                cur = []
                segs.append(cur)
            elif cur is not None:
                cur.append(disp[k])
        segs = segs[-(len(calls) + 1):-1]
        if len(segs) != len(calls):
            raise SystemExit(f"{d}: found {len(segs)} delimited segments, expected {len(calls)}")
        for i, seg in enumerate(segs):
            got = {}
            for rs in seg:
                names[i].add(_short(rs[0]["Kernel_Name"]))
                for r in rs:
                    got[r["Counter_Name"]] = got.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
            for k, v in got.items():
                vals[i].setdefault(k, v)
            if durs[i] is None:
                durs[i] = sum((int(rs[0]["End_Timestamp"]) - int(rs[0]["Start_Timestamp"])) / 1000.0 for rs in seg)
    label = info["pmc_pass"]
    L = [f"# Shader-sequencer counters of the matrix-product calls: {label} step, MXFP4\n"]
    L.append("Two counter passes (repository root on an MI355X machine, <out> an output directory; "
             "summary by bench.py --summarize-sq):\n")
    for j, ps in enumerate(SQ_PASSES):
        L.append(f"    cd /tmp && export TMPDIR=/tmp && timeout -s KILL 180 rocprofv3 --pmc {' '.join(ps)} "
                 f"--output-format csv -d <out>/sq_{label}_{j} -o p -- python3 <repo>/bench.py "
                 f"--pmc-pass {label} --warmup 2 > <out>/sq_{label}_{j}.log")
    L.append(f"\nsource digest: `{info['source_digest']}`\n")
    L.append("Columns: kernel time under counter collection; fraction of the MXFP4 peak (10.1 PFLOP/s) the call's "
             "flops reach in that time; matrix-core busy cycles over the SIMD-cycles of the call (1024 SIMDs at "
             "2.4 GHz); a wave's lifetime (SQ_WAVE_CYCLES x 4 / SQ_WAVES); the share of it spent waiting for "
             "anything (SQ_WAIT_ANY / SQ_WAVE_CYCLES) and waiting to issue (SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES); "
             "instructions issued per wave; LDS bank-conflict cycles per LDS-active cycle.\n")
    L.append("| call | kernel | us | frac of peak | MFMA busy | wave cycles | waiting | issue wait | MFMA / VALU / "
             "SALU / LDS / VMEM per wave | LDS conflict |")
    L.append("|---|---|---|---|---|---|---|---|---|---|")
    for i, c in enumerate(calls):
        v = vals[i]
        if not flops[i] or not v.get("SQ_INSTS_MFMA"):
            continue
        us, w = durs[i], max(v.get("SQ_WAVES", 0.0), 1.0)
        wc = max(v.get("SQ_WAVE_CYCLES", 0.0), 1.0)
        per = " / ".join(f"{v.get(k, 0.0) / w:.0f}" for k in ("SQ_INSTS_MFMA", "SQ_INSTS_VALU", "SQ_INSTS_SALU",
                                                              "SQ_INSTS_LDS", "SQ_INSTS_VMEM"))
        L.append(f"| {c} | {'+'.join(sorted(names[i]))} | {us:.1f} | {flops[i] / (us * 1e-6) / 10.1e15:.3f} | "
                 f"{v.get('SQ_VALU_MFMA_BUSY_CYCLES', 0.0) / (1024 * us * 2400.0):.3f} | {4 * wc / w:.0f} | "
                 f"{v.get('SQ_WAIT_ANY', 0.0) / wc:.2f} | {v.get('SQ_WAIT_INST_ANY', 0.0) / wc:.2f} | {per} | "
                 f"{v.get('SQ_LDS_BANK_CONFLICT', 0.0) / max(v.get('SQ_ACTIVE_INST_LDS', 0.0), 1.0):.3f} |")
    return "\n".join(L) + "\n"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true", help="skip the layer-sweep leg")
    ap.add_argument("--no-qlr", action="store_true", help="skip the latent-replay leg")
    ap.add_argument("--no-naive", action="store_true", help="skip the naive comparator leg")
    ap.add_argument("--no-fused", action="store_true", help="skip the fused-epilogue leg")
    ap.add_argument("--no-fp6", action="store_true", help="skip the FP6-method leg")
    ap.add_argument("--no-sr", action="store_true", help="skip the stochastic-rounding leg")
    ap.add_argument("--no-nvfp", action="store_true", help="skip the NVFP4 leg")
    ap.add_argument("--pmc-pass", default=None, choices=["yolo", "qlr", "sweep"],
                    help="counter-collection pass over one workload's step (see pmc_pass)")
    ap.add_argument("--layers", default="all", help="layer sweep: comma list of layer indices (profiling aid)")
    ap.add_argument("--fmts", default="0,1", help="layer sweep: formats")
    ap.add_argument("--summarize-trace", nargs=2, metavar=("ROCPROF_DIR", "BENCH_LOG"),
                    help="write the kernel-trace summary of a rocprofv3 run of this script to stdout")
    ap.add_argument("--summarize-sq", nargs="+", metavar="LOG_THEN_DIRS",
                    help="SQ-counter summary: the --pmc-pass log, then the rocprofv3 output directories")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "FETCH_LOG", "WRITE_LOG"),
                    help="write the counter summary of two rocprofv3 --pmc runs of --pmc-pass to stdout")
    args = ap.parse_args()
    if args.summarize_trace:
        print(summarize_trace(*args.summarize_trace))
        return
    if args.summarize_pmc:
        print(summarize_pmc(*args.summarize_pmc))
        return
    if args.summarize_sq:
        print(summarize_sq(*args.summarize_sq))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: the path has no multi-GPU part",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_28358_amd import mxconv as mx
    from paper_2609_28358_amd import workloads as wl
    mx.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.pmc_pass == "sweep":
        print(json.dumps(sweep_leg(args)))
        return
    N4, F4 = 64, mx.E2M1
    if args.pmc_pass == "qlr":
        q = wl.QlrStep(dev, fmt=mx.E2M1)
        calls = q.calls()
        for _ in range(2):
            for c in calls:
                c[1]()
        print(json.dumps(pmc_pass(calls, "qlr")))
        return

    net = wl.yolo_net(640)
    st = wl.NetStep(net, N4, F4, dev)
    calls = st.calls()
    if args.pmc_pass == "yolo":
        for _ in range(2):
            for c in calls:
                c[1]()
        print(json.dumps(pmc_pass(calls, "yolo")))
        return
    yolo = step_leg(calls, st.flops(), F4, args)
    yolo["bytes_vs_naive"] = net_bytes_vs_naive(net, N4, F4)
    print(f"bench: yolo step {yolo['ms_per_step']} ms", file=sys.stderr, flush=True)
    del st, calls
    torch.cuda.empty_cache()

    qlr = None
    if not args.no_qlr:
        q = wl.QlrStep(dev, fmt=mx.E2M1)
        qlr = step_leg(q.calls(), q.flops(), mx.E2M1, args)
        print(f"bench: latent replay step {qlr['ms_per_step']} ms", file=sys.stderr, flush=True)
        qlr["workload"] = ("quantized latent replay, MXFP4: buffer of 8192 latents 128x16x16 kept as MX codes; batch "
                           "128 = 3 replayed 32-sample groups (copied codes) + 32 fresh 3x128x128 inputs through the "
                           "frozen front stack (3x3 s2 convs 3->32->64->128, SiLU); trainable back stack of four 3x3 "
                           "convs 128->256, 256->256 x3 at 16x16, SiLU, fwd + bwd")
        del q
        torch.cuda.empty_cache()

    sweep = None if args.no_sweep else sweep_leg(args)
    print("bench: layer sweep done", file=sys.stderr, flush=True)

    rl = dict(yolo["roofline"])
    rl["traffic"] = counter_traffic(f"yolo/{rl['kernel']}", PMC_YOLO)
    out = {
        "metric": "conv fwd+bwd TFLOPS (MXFP8/MXFP4) + quantize/im2col HBM GB/s, % of roofline",
        "value": yolo["value"], "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": yolo["ms_per_step"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "mxfp4 (exact block products, fp32 accumulation)", "data": "synthetic",
        "config": {"workload": "YOLOv8n-shaped backbone+neck, one fwd+bwd training step at batch 64, 3x640x640 "
                               "input, MXFP4 E2M1 activations/weights/gradients: 51 convolutions with SiLU "
                               "(stride-2 3x3 downsampling at widths 16-256, C2f-style 1x1/3x3 blocks, top-down "
                               "and bottom-up neck with 2x upsampling and concatenation), every tensor quantized "
                               "once; value = the step's GEMM flops (real channels) / step time",
                   "global_batch": N4, "image": [3, 640, 640], "format": "mxfp4", "convolutions": len(net.convs()),
                   "parallelism": "single GPU"},
        "roofline": rl,
        "yolo_step": yolo,
    }
    if qlr:
        out["latent_replay_step"] = qlr
    if sweep:
        out["layer_sweep"] = sweep
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_net(net)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
