"""The whole-network steps the benchmark times (paper_2609_28358_amd.workloads),
at reduced image size, checked GPU against GPU: every call of a step is an
oracle-checked library operation (test_gpu_parity, test_gpu_netops,
test_gpu_fused, test_gpu_configs at these layer shapes), and these tests pin
how the step strings them together:
  * the step runs and every weight gradient is finite and non-zero;
  * the fused route (a single-consumer gradient quantized in its consumer's
    input-gradient epilogue) gives bit for bit the weight gradients of the
    unfused route (input gradient stored, then mxconv_quantize_sum): both
    take every rounding decision on the same values, with fp32 and with
    bf16 master tensors (the GEMM result rounded to bf16 on both routes);
  * the step replayed from a HIP graph, with eager work between replays,
    reproduces the eager step bit for bit on every replay;
  * latent replay: the replayed groups are the stored codes and scales, and
    the fresh group is the front stack's output quantized once.
"""
import pytest
import torch

from paper_2609_28358_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


def _run(calls):
    for c in calls:
        c[1]()
    torch.cuda.synchronize()


@pytest.mark.parametrize("master", [torch.bfloat16, torch.float32], ids=["bf16", "fp32"])
@pytest.mark.parametrize("fmt", [0, 1], ids=["mxfp8", "mxfp4"])
def test_yolo_step_fused_equals_unfused(mx, fmt, master):
    net = wl.yolo_net(128)
    a = wl.NetStep(net, 32, fmt, DEV, fused_dgrad=True, master=master)
    b = wl.NetStep(net, 32, fmt, DEV, fused_dgrad=False, master=master)
    ca, cb = a.calls(), b.calls()
    assert any(c[0].startswith("dgrad_quant") for c in ca) and not any(c[0].startswith("dgrad_quant") for c in cb)
    _run(ca)
    _run(cb)
    for nm in a.gw:
        assert torch.isfinite(a.gw[nm]).all(), nm
        assert a.gw[nm].abs().max() > 0, nm
        assert torch.equal(a.gw[nm], b.gw[nm]), nm
        assert torch.equal(a.gy[nm].codes, b.gy[nm].codes) and torch.equal(a.gy[nm].scales, b.gy[nm].scales), nm


def test_yolo_step_graph_replay(mx):
    st = wl.NetStep(wl.yolo_net(128), 32, mx.E2M1, DEV)
    calls = st.calls()
    _run(calls)
    ref = {k: v.clone() for k, v in st.gw.items()}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for c in calls:
            c[1]()
    for it in range(3):
        for v in st.gw.values():
            v.fill_(float("nan"))             # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in ref:
            assert torch.equal(st.gw[k], ref[k]), (it, k)


@pytest.mark.parametrize("master", [torch.bfloat16, torch.float32], ids=["bf16", "fp32"])
def test_latent_replay_step(mx, master):
    a = wl.QlrStep(DEV, buffer=256, fused_dgrad=True, master=master)
    b = wl.QlrStep(DEV, buffer=256, fused_dgrad=False, master=master)
    _run(a.calls())
    _run(b.calls())
    for i in range(len(a.gw)):
        assert torch.isfinite(a.gw[i]).all() and a.gw[i].abs().max() > 0
        assert torch.equal(a.gw[i], b.gw[i]), i
    x0 = a.x[0]
    for slot, k in enumerate(a.replay):
        assert torch.equal(x0.codes[slot * a.lc:(slot + 1) * a.lc], a.buf_codes[k * a.lc:(k + 1) * a.lc])
        assert torch.equal(x0.scales[slot * a.ls:(slot + 1) * a.ls], a.buf_scales[k * a.ls:(k + 1) * a.ls])
    # the fresh group: the front stack run on its own into a separate tensor
    fresh = mx.MxTensor.empty(mx.ACT, a.fmt, (32,) + a.lat, DEV)
    a._front(a.fresh, fresh)
    torch.cuda.synchronize()
    last = a.batch // 32 - 1
    assert torch.equal(x0.codes[last * a.lc:(last + 1) * a.lc], fresh.codes)
    assert torch.equal(x0.scales[last * a.ls:(last + 1) * a.ls], fresh.scales)
