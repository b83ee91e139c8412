"""The layer-sweep step exactly as bench.py launches it, compared with the
oracle element by element at full size.

Sequence (bench.py sweep_leg, per layer and format, then once at the end):
  mxconv_quantize_multi   X (CBF fp32) with its explicit CBF im2col, and W
  mxconv_quantize         G_Y (CBF fp32)
  mxconv_fwd              Y, CBF out
  mxconv_backward         G_X (CBF out) and the weight gradient's split-K
                          partial sums, deferred
  mxconv_wgrad_reduce_multi  every layer's G_W in one launch
on the three sweep layers (3x3 s1 64->64 56x56, 1x1 64->256 56x56, 3x3 s2
128->256 28x28, batch 32) in MXFP8 and MXFP4, seeded inputs.

Every code and scale of X, W, G_Y and of the im2col is compared bit for bit
with the oracle; every element of Y, G_X and G_W with the oracle's fp64
GEMMs (Sec. IV-B) within 1e-5 of the sum of absolute products.
"""
import ctypes

import numpy as np
import pytest
import torch

import mx_tolerance as mxt
import oracle
from paper_2609_28358_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


def test_sweep_step_full_size(mx):
    L = mx.lib()
    jobs = []
    for li, (name, cv) in enumerate(synth.SWEEP_LAYERS):
        x, w, gy = synth.layer_inputs(cv, 1000 + li, kind="sweep")
        ho, wo = synth.out_hw(cv)
        xd, gd, wd = synth.nchw_to_cbf(x, 32).to(DEV), synth.nchw_to_cbf(gy, 32).to(DEV), w.to(DEV)
        for fmt in (0, 1):
            c = mx.conv_struct(cv)
            j = dict(name=f"{name}/{'mxfp8' if fmt == 0 else 'mxfp4'}", cv=cv, fmt=fmt, x=x, w=w, gy=gy,
                     xd=xd, gd=gd, wd=wd,
                     qx=mx.MxTensor.empty(mx.ACT, fmt, tuple(x.shape), DEV),
                     qw=mx.MxTensor.empty(mx.WEIGHT, fmt, tuple(w.shape), DEV),
                     qg=mx.MxTensor.empty(mx.ACT, fmt, tuple(gy.shape), DEV),
                     col=(torch.empty(L.mxconv_im2col_codes_bytes(ctypes.byref(c), fmt), dtype=torch.uint8,
                                      device=DEV),
                          torch.empty(L.mxconv_im2col_scales_bytes(ctypes.byref(c), fmt), dtype=torch.uint8,
                                      device=DEV)),
                     y=torch.full((cv["n"] // 32, ho, wo, cv["cout"], 32), float("nan"), device=DEV),
                     gx=torch.full((cv["n"] // 32, cv["h"], cv["w"], cv["cin"], 32), float("nan"), device=DEV),
                     gw=torch.full(tuple(w.shape), float("nan"), device=DEV),
                     ws=torch.empty(max(1, mx.wgrad_workspace_bytes(cv, fmt)), dtype=torch.uint8, device=DEV))
            j["col"][0].random_(0, 256)
            j["col"][1].random_(0, 256)
            jobs.append(j)
    # the benchmark's step
    for j in jobs:
        cv, fmt = j["cv"], j["fmt"]
        mx.quantize_multi([(j["xd"], mx.ACT, fmt, mx.CBF, tuple(j["x"].shape), j["qx"], (cv, j["col"][0], j["col"][1])),
                           (j["wd"], mx.WEIGHT, fmt, mx.NCHW, tuple(j["w"].shape), j["qw"])])
        mx.quantize(j["gd"], mx.ACT, fmt, layout=mx.CBF, shape=tuple(j["gy"].shape), out=j["qg"])
        mx.fwd(cv, j["qw"], j["qx"], layout=mx.CBF, out=j["y"])
        mx.backward(cv, j["qw"], j["qg"], j["qx"], layout=mx.CBF, gx_out=j["gx"], gw_out=j["gw"],
                    workspace=j["ws"], deferred=True)
    mx.wgrad_reduce_multi([(j["cv"], j["fmt"], j["ws"], j["gw"]) for j in jobs])
    torch.cuda.synchronize()
    for j in jobs:
        cv, fmt, nm = j["cv"], j["fmt"], j["name"]
        print(f"checking {nm}", flush=True)
        ho, wo = synth.out_hw(cv)
        o = {}
        for k, t, role, q in (("x", j["x"], oracle.ACT, j["qx"]), ("w", j["w"], oracle.WEIGHT, j["qw"]),
                              ("gy", j["gy"], oracle.ACT, j["qg"])):
            o[k] = oracle.quantize(t.numpy(), oracle.NCHW, role, fmt, *t.shape)
            assert np.array_equal(q.scales.cpu().numpy(), o[k][1]), f"{nm} {k} scales"
            assert np.array_equal(q.codes.cpu().numpy(), o[k][0]), f"{nm} {k} codes"
        rc, rs = oracle.im2col_cbf(cv, fmt, *o["x"])
        assert np.array_equal(j["col"][1].cpu().numpy(), rs), f"{nm} im2col scales"
        assert np.array_equal(j["col"][0].cpu().numpy(), rc), f"{nm} im2col codes"
        ry, sy = oracle.fwd(cv, fmt, o["w"], o["x"])
        rgx, sgx = oracle.dgrad(cv, fmt, o["w"], o["gy"])
        rgw, sgw = oracle.wgrad(cv, fmt, o["gy"], o["x"])
        y = synth.cbf_to_nchw(j["y"].cpu(), cv["n"], cv["cout"], ho, wo, 32).numpy()
        gx = synth.cbf_to_nchw(j["gx"].cpu(), cv["n"], cv["cin"], cv["h"], cv["w"], 32).numpy()
        gw = j["gw"].cpu().numpy()
        e = (mxt.gemm_err(y, ry, sy), mxt.gemm_err(gx, rgx, sgx), mxt.gemm_err(gw, rgw, sgw))
        r = (mxt.rel_err(y, ry, sy), mxt.rel_err(gx, rgx, sgx), mxt.rel_err(gw, rgw, sgw))
        print(f"  {nm}: max |err| / sum|a b| fwd {r[0]:.2e} dgrad {r[1]:.2e} wgrad {r[2]:.2e}", flush=True)
        assert max(e) <= 1.0, (nm, e)
