"""mxconv_quantize_multi: several quantizations in one call give exactly the
codes and scales of the single calls (and of the oracle), whatever mix of
source kinds, formats and source types the jobs have; a job outside the
one-launch kinds (an NCHW activation) is quantized by its own launch."""
import numpy as np
import pytest
import torch

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


def _jobs(mx):
    x = synth.silu_normal((32, 70, 9, 7), 3)
    x2 = synth.silu_normal((64, 32, 5, 5), 4)
    w = synth.kaiming(64, 70, 3, 3, seed=5)
    w2 = synth.kaiming(20, 48, 1, 1, seed=6)
    xn = synth.normal((16, 40, 4, 6), 1.0, 7)
    return [
        (synth.nchw_to_cbf(x, 32).to(DEV), mx.ACT, 0, mx.CBF, tuple(x.shape), x),
        (w.to(DEV), mx.WEIGHT, 0, mx.NCHW, tuple(w.shape), w),
        (synth.nchw_to_cbf(x2, 32).to(DEV).to(torch.bfloat16), mx.ACT, 3, mx.CBF, tuple(x2.shape),
         x2.to(torch.bfloat16).float()),
        (w2.to(DEV), mx.WEIGHT, 1, mx.NCHW, tuple(w2.shape), w2),
        (xn.to(DEV), mx.ACT, 2, mx.NCHW, tuple(xn.shape), xn),            # its own launch
        (w2.to(DEV).to(torch.bfloat16), mx.WEIGHT, 2, mx.NCHW, tuple(w2.shape), w2.to(torch.bfloat16).float()),
    ]


def test_multi_matches_single_calls_and_oracle(mx):
    jobs = _jobs(mx)
    outs = mx.quantize_multi([(s, r, f, l, sh, None) for s, r, f, l, sh, _ in jobs])
    singles = [mx.quantize(s, r, f, layout=l, shape=sh) for s, r, f, l, sh, _ in jobs]
    torch.cuda.synchronize()
    for (s, r, f, l, sh, ref), o, one in zip(jobs, outs, singles):
        assert torch.equal(o.codes, one.codes) and torch.equal(o.scales, one.scales)
        rc, rs = oracle.quantize(ref.numpy(), oracle.NCHW, r, f, *sh)
        assert np.array_equal(o.scales.cpu().numpy(), rs)
        assert np.array_equal(o.codes.cpu().numpy()[:len(rc)], rc)


def test_multi_layer_operands_full_size(mx):
    """X and W of each benchmark layer, one call per layer, both formats."""
    for li, (name, cv) in enumerate(synth.SWEEP_LAYERS):
        x, w, _ = synth.layer_inputs(cv, 1000 + li, kind="sweep")
        xd, wd = synth.nchw_to_cbf(x, 32).to(DEV), w.to(DEV)
        for fmt in (0, 1):
            qx, qw = mx.quantize_multi([(xd, mx.ACT, fmt, mx.CBF, tuple(x.shape), None),
                                        (wd, mx.WEIGHT, fmt, mx.NCHW, tuple(w.shape), None)])
            sx = mx.quantize(xd, mx.ACT, fmt, layout=mx.CBF, shape=tuple(x.shape))
            sw = mx.quantize(wd, mx.WEIGHT, fmt)
            torch.cuda.synchronize()
            assert torch.equal(qx.codes, sx.codes) and torch.equal(qx.scales, sx.scales)
            assert torch.equal(qw.codes, sw.codes) and torch.equal(qw.scales, sw.scales)
