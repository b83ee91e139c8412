"""GPU parity on the larger workloads at their own full sizes.

* YOLOv8n-shaped network: representative layers (stride-2 stem at 640x640,
  C2f-style 3x3 and 1x1) at batch 16 in MXFP8 and at batch 64 in MXFP4, from
  bf16 master tensors.  Batch 16 is a batch block of 16 (general kernels);
  batch 64 runs the batch-block-32 kernels with CBF outputs.
* Quantized latent replay: the 8192-latent buffer quantized once in MXFP4,
  batches of 128 assembled from 96 replayed latents (whole 32-sample groups of
  the stored codes, no requantization) and 32 fresh ones, and the back stack's
  3x3 convolutions on such a batch.

* Every distinct convolution of the YOLOv8n-shaped network of
  paper_2609_28358_amd.workloads (the benchmark's headline step) at batch 64
  in MXFP4, CBF activations, seeded synthetic operands of the layer's shape.

Codes and scales are compared bit for bit over whole tensors (the buffer: on
sampled groups); GEMM outputs on 4096 seeded samples per GEMM (every element
of a small weight gradient) against the oracle's single-output routines,
within 1e-5 of the sum of absolute products.
"""
import numpy as np
import pytest
import torch

import mx_tolerance as mxt
import oracle
from paper_2609_28358_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
SAMPLES = 4096


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


def _same(q, ref, what):
    codes, scales = ref
    gs = q.scales.cpu().numpy()
    assert np.array_equal(gs, scales), f"{what} scales differ at {np.flatnonzero(gs != scales)[:8]}"
    gc = q.codes.cpu().numpy()[:len(codes)]
    assert np.array_equal(gc, codes), f"{what} codes differ at {np.flatnonzero(gc != codes)[:8]}"


def _gather(t, idx, shape, layout, bn):
    """Values of a logical (n, c, h, w) output at rows idx, read on the GPU."""
    n, c, h, w = (torch.as_tensor(idx[:, i], device=t.device) for i in range(4))
    if layout == "nchw":
        v = t.reshape(shape)[n, c, h, w]
    else:
        N, C, H, W = shape
        v = t.reshape(N // bn, H, W, C, bn)[n // bn, h, w, c, n % bn]
    return v.cpu().numpy()


def _idx(rng, dims, count):
    return np.stack([rng.integers(0, d, count) for d in dims], 1)


def _check_gemms(mx, cv, fmt, q, o, layout, seed):
    """fwd, dgrad and wgrad of the quantized operands q (GPU) against the
    oracle on its own quantized tensors o, on sampled outputs."""
    lay = mx.NCHW if layout == "nchw" else mx.CBF
    bn = synth.batch_block(cv["n"])
    ho, wo = synth.out_hw(cv)
    y = mx.fwd(cv, q["w"], q["x"], layout=lay)
    gx = mx.dgrad(cv, q["w"], q["gy"], layout=lay)
    gw = mx.wgrad(cv, q["gy"], q["x"])
    torch.cuda.synchronize()
    rng = np.random.default_rng(seed)
    errs = {}
    idx = _idx(rng, (cv["n"], cv["cout"], ho, wo), SAMPLES)
    r, s = oracle.fwd_at(cv, fmt, o["w"], o["x"], idx)
    errs["fwd"] = mxt.gemm_err(_gather(y, idx, (cv["n"], cv["cout"], ho, wo), layout, bn), r, s)
    idx = _idx(rng, (cv["n"], cv["cin"], cv["h"], cv["w"]), SAMPLES)
    r, s = oracle.dgrad_at(cv, fmt, o["w"], o["gy"], idx)
    errs["dgrad"] = mxt.gemm_err(_gather(gx, idx, (cv["n"], cv["cin"], cv["h"], cv["w"]), layout, bn), r, s)
    wdims = (cv["cout"], cv["cin"], cv["kh"], cv["kw"])
    if np.prod(wdims) <= SAMPLES:                       # small weights: every element
        idx = np.stack(np.meshgrid(*[np.arange(d) for d in wdims], indexing="ij"), -1).reshape(-1, 4)
    else:
        idx = _idx(rng, wdims, SAMPLES)
    r, s = oracle.wgrad_at(cv, fmt, o["gy"], o["x"], idx)
    errs["wgrad"] = mxt.gemm_err(gw.cpu().numpy()[tuple(idx.T)], r, s)
    assert max(errs.values()) <= 1.0, errs


# ------------------------------------------------------------------ YOLOv8n-shaped layers
YOLO_CASES = [(16, oracle.E4M3, "nchw"), (64, oracle.E2M1, "cbf")]


@pytest.mark.parametrize("n,fmt,layout", YOLO_CASES, ids=["n16_mxfp8", "n64_mxfp4"])
@pytest.mark.parametrize("li", range(3), ids=[name for name, _ in synth.yolo_layers(16)])
def test_yolo_layer_full_size(mx, n, fmt, layout, li):
    name, cv = synth.yolo_layers(n)[li]
    x, w, gy = synth.yolo_inputs(name, cv, 2000 + li)
    print(f"yolo layer {name} n={n} fmt={fmt}", flush=True)
    bn = synth.batch_block(n)
    q = {"x": mx.quantize(x.to(DEV), mx.ACT, fmt),                    # bf16 NCHW source
         "w": mx.quantize(w.to(DEV), mx.WEIGHT, fmt)}
    gsrc = synth.nchw_to_cbf(gy, bn) if layout == "cbf" else gy
    q["gy"] = mx.quantize(gsrc.to(DEV), mx.ACT, fmt, layout=mx.CBF if layout == "cbf" else mx.NCHW,
                          shape=tuple(gy.shape))
    torch.cuda.synchronize()
    o = {}
    for k, t, role in (("x", x, oracle.ACT), ("w", w, oracle.WEIGHT), ("gy", gy, oracle.ACT)):
        o[k] = oracle.quantize(t.float().numpy(), oracle.NCHW, role, fmt, *t.shape)
        _same(q[k], o[k], k)
    _check_gemms(mx, cv, fmt, q, o, layout, 3000 + li)


# ------------------------------------------------------------------ quantized latent replay
def test_latent_replay_buffer_and_back_stack(mx):
    fmt = oracle.E2M1
    C, H, W = synth.QLR_LATENT
    groups = synth.QLR_BUFFER // 32
    lat = synth.qlr_latents(synth.QLR_BUFFER, 4000)
    print(f"latent buffer {tuple(lat.shape)}", flush=True)
    # the buffer, quantized once from CBF fp32 (batch groups of 32)
    buf = mx.quantize(synth.nchw_to_cbf(lat, 32).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(lat.shape))
    torch.cuda.synchronize()
    gcodes = buf.codes.numel() // groups              # codes / scales of one 32-sample group
    gscales = buf.scales.numel() // groups
    assert gcodes * groups == buf.codes.numel() and gscales * groups == buf.scales.numel()
    rng = np.random.default_rng(4001)
    for g in rng.choice(groups, 4, replace=False):   # sampled groups, bit-exact
        ref = oracle.quantize(lat[32 * g:32 * g + 32].numpy(), oracle.NCHW, oracle.ACT, fmt, 32, C, H, W)
        q = mx.MxTensor(buf.codes[g * gcodes:(g + 1) * gcodes], buf.scales[g * gscales:(g + 1) * gscales],
                        mx.ACT, fmt, (32, C, H, W))
        _same(q, ref, f"buffer group {g}")
    # a batch of 128: three replayed groups (stored codes, copied) + 32 fresh latents quantized now
    picks = [int(g) for g in rng.choice(groups, 3, replace=False)]
    fresh = synth.qlr_latents(32, 4002)
    qf = mx.quantize(synth.nchw_to_cbf(fresh, 32).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=(32, C, H, W))
    codes = torch.cat([buf.codes[g * gcodes:(g + 1) * gcodes] for g in picks] + [qf.codes])
    scales = torch.cat([buf.scales[g * gscales:(g + 1) * gscales] for g in picks] + [qf.scales])
    xb = torch.cat([lat[32 * g:32 * g + 32] for g in picks] + [fresh])
    # replay needs no requantization: the assembled batch is the quantized batch
    assert synth.QLR_BATCH == 128
    ref_x = oracle.quantize(xb.numpy(), oracle.NCHW, oracle.ACT, fmt, *xb.shape)
    qx = mx.MxTensor(codes, scales, mx.ACT, fmt, tuple(xb.shape))
    _same(qx, ref_x, "assembled batch")
    # the back stack's first convolution on the assembled batch
    name, cv = synth.QLR_LAYERS[0]
    w = synth.kaiming(cv["cout"], cv["cin"], 3, 3, 4003)
    ho, wo = synth.out_hw(cv)
    gy = synth.normal((cv["n"], cv["cout"], ho, wo), 1e-3, 4004)
    q = {"x": qx, "w": mx.quantize(w.to(DEV), mx.WEIGHT, fmt),
         "gy": mx.quantize(synth.nchw_to_cbf(gy, 32).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(gy.shape))}
    o = {"x": ref_x, "w": oracle.quantize(w.numpy(), oracle.NCHW, oracle.WEIGHT, fmt, *w.shape),
         "gy": oracle.quantize(gy.numpy(), oracle.NCHW, oracle.ACT, fmt, *gy.shape)}
    _same(q["w"], o["w"], "w")
    _same(q["gy"], o["gy"], "gy")
    _check_gemms(mx, cv, fmt, q, o, "cbf", 4005)


def test_latent_back_stack_second_layer(mx):
    """The 256 -> 256 3x3 of the back stack at batch 128, MXFP4, CBF in and out."""
    fmt = oracle.E2M1
    name, cv = synth.QLR_LAYERS[1]
    ho, wo = synth.out_hw(cv)
    x = synth.silu_normal((cv["n"], cv["cin"], cv["h"], cv["w"]), 4010)
    w = synth.kaiming(cv["cout"], cv["cin"], 3, 3, 4011)
    gy = synth.normal((cv["n"], cv["cout"], ho, wo), 1e-3, 4012)
    q = {"x": mx.quantize(synth.nchw_to_cbf(x, 32).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(x.shape)),
         "w": mx.quantize(w.to(DEV), mx.WEIGHT, fmt),
         "gy": mx.quantize(synth.nchw_to_cbf(gy, 32).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(gy.shape))}
    o = {}
    for k, t, role in (("x", x, oracle.ACT), ("w", w, oracle.WEIGHT), ("gy", gy, oracle.ACT)):
        o[k] = oracle.quantize(t.numpy(), oracle.NCHW, role, fmt, *t.shape)
        _same(q[k], o[k], k)
    _check_gemms(mx, cv, fmt, q, o, "cbf", 4013)


# ------------------------------------------------------------------ the network step's layers
def _distinct_net_layers():
    from paper_2609_28358_amd import workloads as wl
    seen, out = set(), []
    for t in wl.yolo_net(640).convs():
        key = (t["cin"], t["cin_real"], t["cout"], t["k"], t["s"], t["src_h"])
        if key not in seen:
            seen.add(key)
            out.append(t)
    return out


NET_LAYERS = _distinct_net_layers()


@pytest.mark.parametrize("t", NET_LAYERS, ids=[t["name"] for t in NET_LAYERS])
def test_network_layer_full_size(mx, t):
    """One convolution of the headline network at batch 64, MXFP4: X from a
    CBF fp32 tensor (the image: bf16 NCHW, U(0, 1)), W bf16, G_Y CBF fp32."""
    from paper_2609_28358_amd import workloads as wl
    fmt, n = oracle.E2M1, 64
    cv = wl.conv_dict(t, n)
    print(f"network layer {t['name']} {cv}", flush=True)
    seed = 6000 + NET_LAYERS.index(t)
    ho, wo = synth.out_hw(cv)
    xs = (n, cv["cin"], cv["h"], cv["w"])
    w = synth.kaiming(cv["cout"], cv["cin"], cv["kh"], cv["kw"], seed * 3 + 1).to(torch.bfloat16)
    gy = synth.normal((n, cv["cout"], ho, wo), 1e-3, seed * 3 + 2)
    if t["src"] == "image":
        x = synth.uniform(xs, seed * 3).to(torch.bfloat16)
        qx = mx.quantize(x.to(DEV), mx.ACT, fmt)
        xo = x.float()
    else:
        xo = synth.silu_normal(xs, seed * 3)
        qx = mx.quantize(synth.nchw_to_cbf(xo, 32).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=xs)
    q = {"x": qx, "w": mx.quantize(w.to(DEV), mx.WEIGHT, fmt),
         "gy": mx.quantize(synth.nchw_to_cbf(gy, 32).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(gy.shape))}
    torch.cuda.synchronize()
    o = {}
    for k, tt, role in (("x", xo, oracle.ACT), ("w", w.float(), oracle.WEIGHT), ("gy", gy, oracle.ACT)):
        o[k] = oracle.quantize(tt.numpy(), oracle.NCHW, role, fmt, *tt.shape)
        _same(q[k], o[k], k)
    _check_gemms(mx, cv, fmt, q, o, "cbf", seed)
