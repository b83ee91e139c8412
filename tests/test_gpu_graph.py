"""The hot path captured once in a HIP graph (through torch's stream
capture) and replayed several times -- with eager work and synchronizations
between the replays, and the outputs overwritten before each replay -- must
reproduce the eager results bit for bit on every replay.  This is how the
benchmark launches its step."""
import ctypes

import pytest
import torch

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


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("cv", [synth.conv_dict(32, 64, 64, 12, 10, 3, 1, 1),
                                synth.conv_dict(32, 64, 256, 9, 7, 1, 1, 0),
                                synth.conv_dict(32, 96, 128, 9, 9, 3, 2, 1)],
                         ids=["3x3s1", "1x1", "3x3s2"])
def test_graph_replay_matches_eager(mx, fmt, cv):
    x, w, gy = synth.layer_inputs(cv, 31, kind="sweep")
    ho, wo = synth.out_hw(cv)
    xs, gs = tuple(x.shape), tuple(gy.shape)
    xd = synth.nchw_to_cbf(x, 32).to(DEV)
    gd = synth.nchw_to_cbf(gy, 32).to(DEV)
    wd = w.to(DEV)
    qx = mx.MxTensor.empty(mx.ACT, fmt, xs, DEV)
    qw = mx.MxTensor.empty(mx.WEIGHT, fmt, tuple(w.shape), DEV)
    qg = mx.MxTensor.empty(mx.ACT, fmt, gs, DEV)
    c = mx.conv_struct(cv)
    col = (torch.empty(mx.lib().mxconv_im2col_codes_bytes(ctypes.byref(c), fmt), dtype=torch.uint8, device=DEV),
           torch.empty(mx.lib().mxconv_im2col_scales_bytes(ctypes.byref(c), fmt), dtype=torch.uint8, device=DEV))
    y = torch.empty((cv["n"] // 32, ho, wo, cv["cout"], 32), device=DEV)
    gx = torch.empty((cv["n"] // 32, cv["h"], cv["w"], cv["cin"], 32), device=DEV)
    gw = torch.empty(tuple(w.shape), device=DEV)
    ws = torch.empty(max(1, mx.wgrad_workspace_bytes(cv, fmt)), dtype=torch.uint8, device=DEV)
    outs = [qx.codes, qx.scales, qw.codes, qw.scales, qg.codes, qg.scales, col[0], col[1], y, gx, gw]

    def step():
        # X (with its CBF im2col) and W in one launch, as the benchmark step does
        mx.quantize_multi([(xd, mx.ACT, fmt, mx.CBF, xs, qx, (cv, col[0], col[1])),
                           (wd, mx.WEIGHT, fmt, mx.NCHW, tuple(wd.shape), qw)])
        mx.quantize(gd, mx.ACT, fmt, layout=mx.CBF, shape=gs, out=qg)
        mx.fwd(cv, qw, qx, layout=mx.CBF, out=y)
        mx.dgrad(cv, qw, qg, layout=mx.CBF, out=gx)
        # the weight gradient's split-K reduction as a batched launch, as in the benchmark step
        mx.wgrad(cv, qg, qx, out=gw, workspace=ws, deferred=True)
        mx.wgrad_reduce_multi([(cv, fmt, ws, gw)])

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    other = torch.randn(xd.shape, device=DEV)
    for r in range(3):
        for t in outs:
            t.fill_(0x5A if t.dtype == torch.uint8 else 7.0)
        torch.cuda.synchronize()
        g.replay()
        mx.quantize(other, mx.ACT, fmt, layout=mx.CBF, shape=xs)      # eager work between replays
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(outs, ref)):
            assert torch.equal(a, b), f"replay {r}: output {i} differs from the eager result"
