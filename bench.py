#!/usr/bin/env python3
"""Benchmark of the quantize-once MX convolution hot path on one MI355X.

One step = one pass of the whole path over the layer sweep (batch 32, inputs
resident in HBM): for each layer
    3x3 s1 p1 64->64 at 56x56,  1x1 64->256 at 56x56,  3x3 s2 p1 128->256 at 28x28
and each format (MXFP8 E4M3, MXFP4 E2M1): quantize X, W and G_Y once
(activations arrive channel-batch-first in fp32, weights OIHW fp32), with the
explicit CBF im2col of X written by the same launch that quantizes X and W
(the forward operands), then the forward GEMM, and the input-gradient and
weight-gradient GEMMs as one launch per layer (both read the quantized G_Y),
the weight gradients' split-K partial sums of all layers finished by one
reduction launch at the end: 25 kernels.  Activations are SiLU(N(0,1)),
weights Kaiming-normal, gradients N(0, 1e-3), all seeded.

`value` is the conv fwd+bwd GEMM throughput of the whole step: the three
GEMMs' algorithmic flops (2 N Cout Ho Wo Cin Kh Kw each, real channels) over
the step's wall time, quantize and im2col included.  The timed step is
replayed from one HIP graph (captured once after warm-up), so it measures
GPU time, not Python launch cost.

Per op, two times are reported in `ops`: `ms`, the op's kernel time in
steady state -- a HIP graph of K back-to-back launches of the op, replayed on
the stream its kernels run on and bracketed by HIP events (median of
rounds); quantize launches rotate over enough copies of their fp32 source
that it is read from HBM, not from the 256 MB last-level cache -- and
`ms_alone`, one eager launch bracketed by HIP events behind a GPU spin
(launch and event overhead included).  The op of the step with the largest
`ms` gets the `roofline` object.  The unfused X+W quantize, the standalone
im2col kernel, the input gradient alone and the whole weight gradient (GEMM
and its own reduction) are timed too (`in_step` false), outside the step.

    python bench.py [--steps K] [--warmup W] [--no-cpu-baseline]
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
# FP6 methods of Sec. V as (W, X, G_Y) element formats: MicroQonv+ keeps
# activations in E3M2 with FP4 weights and gradients; the "-6" methods use
# E2M3 throughout
FP6_METHODS = {"microqonv_plus": (1, 3, 1), "microqonv_6": (2, 2, 2)}
FP6_SLACK = 16                                     # read slack at the end of an FP6 code buffer


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


PMC_SUMMARY = os.path.join(ROOT, "profiles", "op_traffic_pmc.md")
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


def counter_traffic(op_key):
    """HBM bytes per launch of `op_key` ("layer/format/op") from the committed
    counter summary: FETCH_SIZE and WRITE_SIZE (KiB per dispatch, summed over
    the op's kernels), each scaled by the factor the same counter gives for a
    copy of known size.  None if there is no summary, the op is missing, or the
    sources changed since the counters were taken."""
    if not os.path.exists(PMC_SUMMARY):
        return None
    digest, fetch_f, write_f, rows = None, None, None, {}
    with open(PMC_SUMMARY) as f:
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


def naive_leg(jobs, op_ms, mx, synth, dev, stream, reps=3):
    """Run the naive comparator once per (layer, format) on the same inputs
    (outside the timed region) and report its time, algorithmic bytes and
    quantized elements beside the method's.  The method's bytes are its
    quantize x3 + fwd + dgrad + wgrad (the GEMMs take the im2col implicitly)."""
    import torch
    res = {}
    shared = {}
    for j in jobs:
        cv, fmt = j["cv"], j["fmt"]
        ho, wo = synth.out_hw(cv)
        P, K, co = cv["n"] * ho * wo, cv["kh"] * cv["kw"] * cv["cin"], cv["cout"]
        key = j["name"].split("/")[0]
        if key not in shared:
            x = synth.cbf_to_nchw(j["x"].cpu(), cv["n"], cv["cin"], cv["h"], cv["w"], 32)
            gy = synth.cbf_to_nchw(j["gy"].cpu(), cv["n"], co, ho, wo, 32)
            shared = {key: dict(
                x=x.permute(0, 2, 3, 1).contiguous().to(dev),
                gy=gy.permute(0, 2, 3, 1).reshape(P, co).contiguous().to(dev),
                w=j["w"].permute(0, 2, 3, 1).reshape(co, K).contiguous(),
                col=torch.empty((P, K), dtype=torch.float32, device=dev),
                gcol=torch.empty((P, K), dtype=torch.float32, device=dev),
                y=torch.empty((P, co), dtype=torch.float32, device=dev),
                gx=torch.empty((cv["n"], cv["h"], cv["w"], cv["cin"]), dtype=torch.float32, device=dev),
                gw=torch.empty((co, K), dtype=torch.float32, device=dev))}
        b = shared[key]

        def naive_step():
            mx.naive_im2col_f32(cv, b["x"], out=b["col"])
            qc0 = mx.naive_quantize_1d(b["col"], 0, fmt)
            qw0 = mx.naive_quantize_1d(b["w"], 0, fmt)
            mx.naive_fwd(cv, qc0, qw0, out=b["y"])
            qg0 = mx.naive_quantize_1d(b["gy"], 0, fmt)
            qw1 = mx.naive_quantize_1d(b["w"], 1, fmt)
            mx.naive_dgrad(cv, qg0, qw1, gcol=b["gcol"], out=b["gx"])
            qg1 = mx.naive_quantize_1d(b["gy"], 1, fmt)
            qc1 = mx.naive_quantize_1d(b["col"], 1, fmt)
            mx.naive_wgrad(cv, qg1, qc1, out=b["gw"])

        naive_step()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SPIN_CYCLES)
        e0.record(stream)
        for _ in range(reps):
            naive_step()
        e1.record(stream)
        torch.cuda.synchronize()
        ms_naive = e0.elapsed_time(e1) / reps
        nby, nq = naive_numbers(cv, fmt, mx)
        ours_ops = ("quant_xw", "quant_gy", "fwd", "dgrad", "wgrad")
        oby = sum(j["nums"][op][1] for op in ours_ops)
        ms_ours = sum(op_ms[(j["name"], op)] for op in ours_ops)
        nx = cv["n"] * cv["cin"] * cv["h"] * cv["w"]
        oq = nx + co * K + P * co
        res[j["name"]] = {"bytes_naive": round(sum(nby.values())), "bytes_ours": round(oby),
                          "bytes_ratio": round(sum(nby.values()) / oby, 2),
                          "ms_naive": round(ms_naive, 4), "ms_ours": round(ms_ours, 4),
                          "speedup": round(ms_naive / ms_ours, 2),
                          "quantized_naive": nq, "quantized_ours": oq}
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-naive", action="store_true", help="skip the naive comparator leg")
    ap.add_argument("--no-fused", action="store_true", help="skip the fused-epilogue leg")
    ap.add_argument("--no-fp6", action="store_true", help="skip the FP6-method leg")
    ap.add_argument("--no-sr", action="store_true", help="skip the stochastic-rounding leg")
    ap.add_argument("--no-nvfp", action="store_true", help="skip the NVFP4 leg")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="counter-collection pass: every op once in step order, then a copy of known size")
    ap.add_argument("--layers", default="all", help="comma list of layer indices (profiling aid)")
    ap.add_argument("--fmts", default="0,1")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the path has no "
              f"multi-GPU part)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_28358_amd import mxconv as mx
    from paper_2609_28358_amd import synth
    mx.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

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
        # one eager launch per op, separated, then the calibration copy; the
        # counter summary maps dispatches to ops in this order
        for j, op in seq:
            run(j, op)
            torch.cuda.synchronize()
        src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"pmc_pass": [f"{j['name']}/{op}" for j, op in seq], "copy_bytes": COPY_BYTES,
                          "source_digest": source_digest()}))
        return

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
               "traffic": counter_traffic(f"{dom[0]}/{dom[1]}")})
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
        "metric": "conv fwd+bwd TFLOPS (MXFP8/MXFP4) + quantize/im2col HBM GB/s, % of roofline",
        "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "mxfp8+mxfp4 (fp32 accumulate)", "data": "synthetic",
        "config": {"workload": "conv layer sweep, batch 32: 3x3 s1 64->64 56x56, 1x1 64->256 56x56, "
                               "3x3 s2 128->256 28x28; each in MXFP8 and MXFP4; quantize X+W with X's CBF im2col (one "
                               "launch) + quantize G_Y + fwd + dgrad and wgrad in one launch per layer, the six weight "
                               "gradients' split-K reductions in one launch at the end",
                   "global_batch": 32, "layers": [n for n, _ in synth.SWEEP_LAYERS], "formats": ["mxfp8", "mxfp4"],
                   "parallelism": "single GPU"},
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
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline()
    print(json.dumps(out))


if __name__ == "__main__":
    main()
