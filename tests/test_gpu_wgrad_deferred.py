"""The weight gradient in two parts: mxconv_wgrad_deferred per layer, then
mxconv_wgrad_reduce_multi for several layers in one launch, gives exactly
mxconv_wgrad's G_W (the same partial sums, added in the same order) -- for
layers on the split-K lean kernels, a lean layer without split (G_W written
directly), the general kernels (batch block 16), FP6 and mixed operands."""
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
    (synth.conv_dict(32, 64, 64, 28, 28, 3, 1, 1), (0, 0)),          # lean, split-K
    (synth.conv_dict(32, 64, 128, 14, 14, 1, 1, 0), (1, 1)),
    (synth.conv_dict(64, 96, 64, 13, 11, 3, 2, 1), (0, 0)),
    (synth.conv_dict(32, 64, 64, 4, 4, 3, 1, 1), (1, 1)),            # lean, one split: G_W written directly
    (synth.conv_dict(16, 32, 48, 9, 8, 3, 1, 1), (0, 0)),            # batch block 16: general kernels
    (synth.conv_dict(32, 64, 32, 10, 10, 3, 1, 1), (2, 2)),          # FP6 E2M3
    (synth.conv_dict(32, 64, 64, 12, 12, 3, 1, 1), (1, 3)),          # G_Y E2M1 against X E3M2
]


def _operands(mx, cv, fg, fx, seed):
    x, _, gy = synth.layer_inputs(cv, seed, kind="sweep")
    bn = synth.batch_block(cv["n"])
    qx = mx.quantize(synth.nchw_to_cbf(x, bn).to(DEV), mx.ACT, fx, layout=mx.CBF, shape=tuple(x.shape))
    qg = mx.quantize(synth.nchw_to_cbf(gy, bn).to(DEV), mx.ACT, fg, layout=mx.CBF, shape=tuple(gy.shape))
    return qg, qx


def test_deferred_weight_gradients_reduced_together(mx):
    ref, jobs, outs = [], [], []
    for k, (cv, (fg, fx)) in enumerate(LAYERS):
        qg, qx = _operands(mx, cv, fg, fx, 60 + k)
        ref.append(mx.wgrad(cv, qg, qx))
        fmt = mx.pair(fg, fx)
        need = mx.wgrad_workspace_bytes(cv, fmt)
        ws = torch.empty(max(1, need), dtype=torch.uint8, device=DEV) if need else None
        gw = torch.full((cv["cout"], cv["cin"], cv["kh"], cv["kw"]), 7.0, device=DEV)   # overwritten
        mx.wgrad(cv, qg, qx, out=gw, workspace=ws, deferred=True)
        jobs.append((cv, fmt, ws, gw))
        outs.append(gw)
    mx.wgrad_reduce_multi(jobs)
    torch.cuda.synchronize()
    for k, (a, b) in enumerate(zip(ref, outs)):
        assert torch.equal(a, b), f"layer {k}: differs from mxconv_wgrad"
    # twice more over the same buffers, the layers split over two calls
    for gw in outs:
        gw.fill_(-3.0)
    for k, (cv, (fg, fx)) in enumerate(LAYERS):
        qg, qx = _operands(mx, cv, fg, fx, 60 + k)
        mx.wgrad(cv, qg, qx, out=outs[k], workspace=jobs[k][2], deferred=True)
    mx.wgrad_reduce_multi(jobs[:3])
    mx.wgrad_reduce_multi(jobs[3:])
    torch.cuda.synchronize()
    for k, (a, b) in enumerate(zip(ref, outs)):
        assert torch.equal(a, b), f"layer {k}: differs from mxconv_wgrad on the second pass"



def test_reduce_batch_of_the_most_layers(mx):
    """As many layers as one call takes (32; a launch once took 8), split-K
    and direct ones mixed, FP8 and FP4, finished by one call: each equal to
    mxconv_wgrad.  One more layer is refused."""
    shapes = [synth.conv_dict(64, 32 * (1 + k % 3), 32 * (1 + (k + 1) % 2), 12 + k % 5, 13 + k % 4,
                              3 if k % 2 else 1, 1 + (k % 3 == 2)) for k in range(mx.WREDUCE_MAX)]
    ref, jobs, split = [], [], 0
    for k, cv in enumerate(shapes):
        fmt = k % 2
        qg, qx = _operands(mx, cv, fmt, fmt, 200 + k)
        ref.append(mx.wgrad(cv, qg, qx))
        need = mx.wgrad_workspace_bytes(cv, fmt)
        split += need > 0
        ws = torch.empty(max(1, need), dtype=torch.uint8, device=DEV) if need else None
        gw = torch.full((cv["cout"], cv["cin"], cv["kh"], cv["kw"]), 5.0, device=DEV)   # overwritten
        mx.wgrad(cv, qg, qx, out=gw, workspace=ws, deferred=True)
        jobs.append((cv, fmt, ws, gw))
    assert split >= mx.WREDUCE_MAX // 2                   # most of them leave partial sums
    mx.wgrad_reduce_multi(jobs)
    torch.cuda.synchronize()
    for k, (a, j) in enumerate(zip(ref, jobs)):
        assert torch.equal(a, j[3]), f"layer {k}: differs from mxconv_wgrad"
    with pytest.raises(mx.MxconvError):
        mx.wgrad_reduce_multi(jobs + jobs[:1])
