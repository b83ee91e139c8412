"""GPU: the image quantize with MXC_KEEP_PAD (mxconv_quantize's layout flag).

With the flag the few-channel NCHW path writes only the code rows of the
real channels; the caller vouches that the padding rows already hold +0
codes.  Checked against the oracle's quantization: into a zero-filled
buffer the result is byte-equal to it; into a buffer of garbage the real
rows and every scale are equal to it and each padding byte is left as it
was; a second call into the same buffer gives the same bytes; and a path
that does not skip padding (more than four channels) still writes
everything."""
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


def _rows(codes, fmt, c):
    """Codes as [block][32 rows][row bytes] and a mask of the real rows."""
    rb = 32 if fmt == 0 else 16
    v = codes.reshape(-1, 32, rb)
    real = np.zeros((1, 32, 1), dtype=bool)
    real[:, :c] = True
    return v, np.broadcast_to(real, v.shape)


SHAPES = [(32, 3, 17, 19), (64, 3, 40, 40), (96, 4, 5, 13), (32, 1, 8, 8), (64, 2, 1, 130)]


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_keep_pad_image(mx, fmt, bf16, shape):
    t = synth.uniform(shape, 23 + shape[1] + shape[3])
    if bf16:
        t = t.to(torch.bfloat16).float()
    src = (t.to(torch.bfloat16) if bf16 else t).to(DEV)
    ref_c, ref_s = oracle.quantize(t.numpy(), oracle.NCHW, mx.ACT, fmt, *shape)
    # zero-filled buffer: byte-equal to the oracle, also on a second call
    out = mx.MxTensor.empty(mx.ACT, fmt, shape, DEV)
    out.codes.zero_()
    for _ in range(2):
        mx.quantize(src, mx.ACT, fmt, out=out, keep_pad=True)
        torch.cuda.synchronize()
        assert np.array_equal(out.scales.cpu().numpy(), ref_s)
        assert np.array_equal(out.codes.cpu().numpy(), ref_c)
    # garbage: real rows and scales as the oracle's, padding bytes untouched
    out.codes.fill_(0xA5)
    out.scales.fill_(0x5A)
    mx.quantize(src, mx.ACT, fmt, out=out, keep_pad=True)
    torch.cuda.synchronize()
    assert np.array_equal(out.scales.cpu().numpy(), ref_s)
    got, real = _rows(out.codes.cpu().numpy(), fmt, shape[1])
    want, _ = _rows(ref_c, fmt, shape[1])
    assert np.array_equal(got[real], want[real])
    assert np.all(got[~real] == 0xA5)


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
def test_keep_pad_other_paths_write_everything(mx, fmt):
    """Five or more channels (the general NCHW path) and a weight: the flag
    changes nothing, padding rows included."""
    for role, shape in ((mx.ACT, (32, 5, 6, 7)), (mx.ACT, (32, 40, 3, 3)), (mx.WEIGHT, (20, 3, 3, 3))):
        t = synth.normal(shape, 1.0, 31 + shape[1])
        ref_c, ref_s = oracle.quantize(t.numpy(), oracle.NCHW, role, fmt, *shape)
        out = mx.MxTensor.empty(role, fmt, shape, DEV)
        out.codes.fill_(0xA5)
        mx.quantize(t.to(DEV), role, fmt, out=out, keep_pad=True)
        torch.cuda.synchronize()
        assert np.array_equal(out.scales.cpu().numpy(), ref_s)
        assert np.array_equal(out.codes.cpu().numpy(), ref_c)
