"""mxconv_wgrad_noalloc (the weight gradient with its split-K partial sums in
the library's own per-GPU device array, for callers that cannot allocate)
against mxconv_wgrad with a caller workspace: bit for bit on two calls in a
row, the second on a smaller layer, and the host-side refusal of a layer
whose partial sums do not fit."""
import ctypes

import pytest
import torch

from paper_2609_28358_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
NOALLOC_WS_MAX = 16 << 20          # MXC_NOALLOC_WS_MAX


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


def _operands(mx, cv, fmt, seed):
    x, w, gy = synth.layer_inputs(cv, seed, kind="sweep")
    bn = synth.batch_block(cv["n"])
    qx = mx.quantize(synth.nchw_to_cbf(x, bn).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(x.shape))
    qg = mx.quantize(synth.nchw_to_cbf(gy, bn).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(gy.shape))
    return qg, qx, tuple(w.shape)


def _noalloc(mx, cv, fmt, qg, qx, gw):
    return mx.lib().mxconv_wgrad_noalloc(ctypes.byref(mx.conv_struct(cv)), fmt, mx._ptr(qg.codes),
                                         mx._ptr(qg.scales), mx._ptr(qx.codes), mx._ptr(qx.scales),
                                         mx._ptr(gw), mx._stream(None))


@pytest.mark.parametrize("fmt", [0, 1], ids=["mxfp8", "mxfp4"])
def test_noalloc_matches_wgrad(mx, fmt):
    layers = [synth.conv_dict(32, 64, 64, 28, 28, 3, 1, 1),      # split-K: partial sums in the array
              synth.conv_dict(32, 32, 32, 14, 14, 3, 1, 1)]      # then a smaller layer
    for i, cv in enumerate(layers):
        need = mx.wgrad_workspace_bytes(cv, fmt)
        assert 0 < need <= NOALLOC_WS_MAX
        qg, qx, wshape = _operands(mx, cv, fmt, 900 + i)
        ref = mx.wgrad(cv, qg, qx)
        gw = torch.full(wshape, float("nan"), device=DEV)
        assert _noalloc(mx, cv, fmt, qg, qx, gw) == 0
        torch.cuda.synchronize()
        assert torch.equal(gw, ref), i


def test_noalloc_refuses_oversized_layer(mx):
    cv = synth.conv_dict(16, 256, 256, 56, 56, 3, 1, 1)
    assert mx.wgrad_workspace_bytes(cv, 0) > NOALLOC_WS_MAX
    t = torch.zeros(64, dtype=torch.uint8, device=DEV)
    dummy = mx.MxTensor(t, t, mx.ACT, 0, (16, 256, 56, 56))
    gw = torch.zeros(16, device=DEV)
    assert _noalloc(mx, cv, 0, dummy, dummy, gw) == -6          # MXC_ERR_WORKSPACE, nothing launched
