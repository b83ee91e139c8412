"""Calls from several host threads, each on its own stream, give the same
results as the same calls made one after another (the kernels are
deterministic, so bit for bit).  One layer uses more than 64 KB of LDS per
workgroup, so the per-device launch attribute is raised under concurrency."""
import threading

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


def _layer_outputs(mx, cv, fmt, x, w, gy):
    qx = mx.quantize(synth.nchw_to_cbf(x, 32).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(x.shape))
    qw = mx.quantize(w.to(DEV), mx.WEIGHT, fmt)
    qg = mx.quantize(synth.nchw_to_cbf(gy, 32).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(gy.shape))
    return [qx.codes, qx.scales, mx.fwd(cv, qw, qx, layout=mx.CBF), mx.dgrad(cv, qw, qg, layout=mx.CBF),
            mx.wgrad(cv, qg, qx)]


def test_concurrent_host_threads_match_sequential(mx):
    cases = [(synth.conv_dict(32, 64, 64, 28, 28, 3, 1, 1), 0, 21),      # 3x3 FP8: ring above 64 KB of LDS
             (synth.conv_dict(64, 96, 128, 14, 15, 1, 1, 0), 1, 22)]
    inputs = [(cv, fmt, synth.layer_inputs(cv, seed, kind="sweep")) for cv, fmt, seed in cases]
    ref = [[t.cpu() for t in _layer_outputs(mx, cv, fmt, *xs)] for cv, fmt, xs in inputs]
    torch.cuda.synchronize()
    got = [[None] * 4 for _ in inputs]
    errors = []

    def work(i):
        try:
            cv, fmt, xs = inputs[i]
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                for r in range(4):
                    got[i][r] = [t.cpu() for t in _layer_outputs(mx, cv, fmt, *xs)]
        except Exception as e:          # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(i,)) for i in range(len(inputs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    for i in range(len(inputs)):
        for r in range(4):
            for k, (a, b) in enumerate(zip(ref[i], got[i][r])):
                assert torch.equal(a, b), f"case {i} repetition {r} output {k} differs from the sequential result"
