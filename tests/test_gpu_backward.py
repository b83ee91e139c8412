"""mxconv_backward gives, bit for bit, the input gradient of mxconv_dgrad and
the weight gradient of mxconv_wgrad (or, deferred, the partial sums of
mxconv_wgrad_deferred): on the grouped launch (batch block 32, kernel width
1 or 3, stride 1 and 2, one and two pixels per wave, one split and split-K)
and on the layers that run as two launches (batch block 16, FP6)."""
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


LAYERS = [
    (synth.conv_dict(32, 64, 64, 28, 28, 3, 1, 1), 0),            # 3x3 stride 1, split-K
    (synth.conv_dict(32, 64, 64, 28, 28, 3, 1, 1), 1),
    (synth.conv_dict(32, 64, 128, 14, 14, 1, 1, 0), 1),           # 1x1
    (synth.conv_dict(32, 32, 64, 6, 7, 1, 1, 0), 0),              # few tiles: one pixel per wave
    (synth.conv_dict(64, 96, 64, 13, 11, 3, 2, 1), 0),            # stride 2: the four phases
    (synth.conv_dict(32, 64, 96, 28, 27, 3, 2, 1), 1),
    (synth.conv_dict(32, 128, 64, 20, 20, 1, 2, 0), 0),           # 1x1 stride 2
    (synth.conv_dict(32, 64, 64, 4, 4, 3, 1, 1), 1),              # one split: G_W written directly
    (synth.conv_dict(96, 64, 160, 9, 9, 3, 1, 1), 0),             # three batch groups, ragged channels
    (synth.conv_dict(32, 16, 16, 40, 36, 3, 1, 1), 1),            # one channel block each side: 32 x 32 wgrad tiles
    (synth.conv_dict(64, 16, 32, 40, 40, 3, 2, 1), 0),            # the same at stride 2
    (synth.conv_dict(32, 32, 16, 12, 12, 1, 1, 0), 1),            # 1x1, one block each side, one split
    (synth.conv_dict(32, 16, 16, 64, 64, 3, 1, 1), 1),            # narrow input-gradient tiles (FP4)
    (synth.conv_dict(64, 16, 32, 64, 64, 3, 2, 1), 1),            # the same in stride-2 phases
    (synth.conv_dict(16, 32, 48, 9, 8, 3, 1, 1), 0),              # batch block 16: two launches
    (synth.conv_dict(32, 64, 32, 10, 10, 3, 1, 1), 2),            # FP6: two launches
]


def _ops(mx, cv, fmt, seed):
    x, w, gy = synth.layer_inputs(cv, seed, kind="sweep")
    bn = synth.batch_block(cv["n"])
    qx = mx.quantize(synth.nchw_to_cbf(x, bn).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(x.shape))
    qw = mx.quantize(w.to(DEV), mx.WEIGHT, fmt)
    qg = mx.quantize(synth.nchw_to_cbf(gy, bn).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(gy.shape))
    return qw, qg, qx


@pytest.mark.parametrize("layout", ["cbf", "nchw"])
@pytest.mark.parametrize("i", range(len(LAYERS)))
def test_backward_matches_separate_calls(mx, i, layout):
    cv, fmt = LAYERS[i]
    lay = mx.CBF if layout == "cbf" else mx.NCHW
    qw, qg, qx = _ops(mx, cv, fmt, 800 + i)
    gx_ref = mx.dgrad(cv, qw, qg, layout=lay)
    gw_ref = mx.wgrad(cv, qg, qx)
    gx, gw = mx.backward(cv, qw, qg, qx, layout=lay)
    torch.cuda.synchronize()
    assert torch.equal(gx, gx_ref)
    assert torch.equal(gw, gw_ref)
    # again into the same outputs, poisoned first
    gx.fill_(float("nan")); gw.fill_(float("nan"))
    mx.backward(cv, qw, qg, qx, layout=lay, gx_out=gx, gw_out=gw)
    torch.cuda.synchronize()
    assert torch.equal(gx, gx_ref)
    assert torch.equal(gw, gw_ref)


@pytest.mark.parametrize("i", [0, 4, 7, 9])
def test_backward_deferred_matches_wgrad_deferred(mx, i):
    cv, fmt = LAYERS[i]
    qw, qg, qx = _ops(mx, cv, fmt, 900 + i)
    need = mx.wgrad_workspace_bytes(cv, fmt)
    ws_ref = torch.zeros(max(need, 16), dtype=torch.uint8, device=DEV)
    ws = torch.full_like(ws_ref, 0x7F)
    gw_ref = torch.zeros((cv["cout"], cv["cin"], cv["kh"], cv["kw"]), dtype=torch.float32, device=DEV)
    gw = torch.zeros_like(gw_ref)
    mx.wgrad(cv, qg, qx, out=gw_ref, workspace=ws_ref, deferred=True)
    gx_ref = mx.dgrad(cv, qw, qg, layout=mx.CBF)
    gx, _ = mx.backward(cv, qw, qg, qx, layout=mx.CBF, gw_out=gw, workspace=ws, deferred=True)
    if need:
        mx.wgrad_reduce_multi([(cv, fmt, ws_ref, gw_ref)])
        mx.wgrad_reduce_multi([(cv, fmt, ws, gw)])
    torch.cuda.synchronize()
    assert torch.equal(gx, gx_ref)
    if need:
        assert torch.equal(ws[:need], ws_ref[:need])
    assert torch.equal(gw, gw_ref)
    assert torch.equal(gw, mx.wgrad(cv, qg, qx))


@pytest.mark.parametrize("fmt", [0, 1])
def test_backward_benchmark_layers(mx, fmt):
    for k, (name, cv) in enumerate(synth.SWEEP_LAYERS):
        qw, qg, qx = _ops(mx, cv, fmt, 950 + k)
        gx, gw = mx.backward(cv, qw, qg, qx, layout=mx.CBF)
        torch.cuda.synchronize()
        assert torch.equal(gx, mx.dgrad(cv, qw, qg, layout=mx.CBF)), name
        assert torch.equal(gw, mx.wgrad(cv, qg, qx)), name
