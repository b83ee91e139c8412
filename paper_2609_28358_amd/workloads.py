"""Whole-network training steps on the MX path: the workloads the paper trains
(Sec. VI: YOLO-nano-class detectors; Sec. VII: quantized latent replay),
with synthetic, seeded tensors of their shapes.

Every step is a fixed sequence of library calls on preallocated device
buffers (so it can be captured once into a HIP graph); every arithmetic step
runs in the library's kernels.  Each tensor is quantized exactly once per
step (Sec. IV-C):
  * weights: their bf16 master copies, quantized at the start of the step
    (several per launch);
  * activations: by the producing convolution's epilogue, after SiLU, which
    also returns the fp32 pre-activation for the backward pass;
  * gradients: each layer's G_Y once, from the sum of what its consumers
    hand back times SiLU' (mxconv_quantize_sum);
  * concatenation and 2x upsampling move whole MX blocks
    (mxconv_concat_cbf).
Weight gradients run with their split-K partial sums deferred and are
finished by batched reductions at the end of the backward pass.

The network below is this project's own YOLOv8n-shaped reading (stride-2 3x3
downsampling convolutions at widths 16/32/64/128/256, C2f-style blocks of
1x1 and 3x3 convolutions, SiLU, a top-down and bottom-up neck with nearest
upsampling and concatenation); it is not the reference implementation's
model definition, and there is no detection head or loss: the three neck
outputs receive an upstream gradient ~ N(0, 1e-3).
"""
import math

import torch

from . import mxconv as mx
from . import synth


# ---------------------------------------------------------------- network description
class Net:
    """A feed-forward graph of convolutions (with SiLU) and concatenations.
    nodes: dicts with kind "input" | "conv" | "concat"; every conv has a
    batch-independent description (cin is the channel count of its source
    tensor as stored, padding channels of a concatenation included)."""

    def __init__(self):
        self.nodes = []
        self.index = {}
        self.outputs = []

    def _add(self, node):
        self.index[node["name"]] = len(self.nodes)
        self.nodes.append(node)
        return node["name"]

    def node(self, name):
        return self.nodes[self.index[name]]

    def input(self, name, c, h, w):
        return self._add(dict(kind="input", name=name, c=c, real=c, h=h, w=w))

    def conv(self, name, src, cout, k, s):
        t = self.node(src)
        p = (k - 1) // 2
        ho, wo = (t["h"] + 2 * p - k) // s + 1, (t["w"] + 2 * p - k) // s + 1
        return self._add(dict(kind="conv", name=name, src=src, cin=t["c"], cin_real=t["real"], cout=cout, k=k, s=s,
                              p=p, c=cout, real=cout, h=ho, w=wo, src_h=t["h"], src_w=t["w"]))

    def concat(self, name, parts):
        """parts: names, or (name, 1) for a part upsampled 2x first."""
        ps = [(p, 0) if isinstance(p, str) else p for p in parts]
        t0 = self.node(ps[0][0])
        h, w = (t0["h"] * 2, t0["w"] * 2) if ps[0][1] else (t0["h"], t0["w"])
        blocks, offs, reals = 0, [], []
        for p, up in ps:
            t = self.node(p)
            assert (t["h"] * (2 if up else 1), t["w"] * (2 if up else 1)) == (h, w), (name, p)
            offs.append(32 * blocks)
            blocks += -(-t["c"] // 32)
            reals.append(t["real"])
        return self._add(dict(kind="concat", name=name, parts=ps, offs=offs, part_real=reals, c=32 * blocks,
                              real=sum(reals), h=h, w=w))

    def c2f(self, prefix, src, cout, n):
        """C2f-style block: two 1x1 convolutions to c = cout/2 channels each
        (the two halves of one 1x1 convolution), n bottlenecks of two 3x3
        convolutions at c channels (no shortcut), the concatenation of both
        halves and every bottleneck output, and a 1x1 convolution to cout."""
        c = cout // 2
        a = self.conv(prefix + ".cv1a", src, c, 1, 1)
        b = self.conv(prefix + ".cv1b", src, c, 1, 1)
        parts, last = [a, b], b
        for i in range(n):
            m = self.conv(f"{prefix}.m{i}a", last, c, 3, 1)
            last = self.conv(f"{prefix}.m{i}b", m, c, 3, 1)
            parts.append(last)
        cat = self.concat(prefix + ".cat", parts)
        return self.conv(prefix + ".cv2", cat, cout, 1, 1)

    def convs(self):
        return [n for n in self.nodes if n["kind"] == "conv"]


def yolo_net(size=640):
    """YOLOv8n-shaped backbone and neck for a 3 x size x size image."""
    g = Net()
    x = g.input("image", 3, size, size)
    b0 = g.conv("b0", x, 16, 3, 2)
    b1 = g.conv("b1", b0, 32, 3, 2)
    b2 = g.c2f("b2", b1, 32, 1)
    b3 = g.conv("b3", b2, 64, 3, 2)
    b4 = g.c2f("b4", b3, 64, 2)               # stride 8
    b5 = g.conv("b5", b4, 128, 3, 2)
    b6 = g.c2f("b6", b5, 128, 2)              # stride 16
    b7 = g.conv("b7", b6, 256, 3, 2)
    b8 = g.c2f("b8", b7, 256, 1)              # stride 32
    n0 = g.concat("n0", [(b8, 1), b6])
    n1 = g.c2f("n1", n0, 128, 1)
    n2 = g.concat("n2", [(n1, 1), b4])
    n3 = g.c2f("n3", n2, 64, 1)               # output, stride 8
    n4 = g.conv("n4", n3, 64, 3, 2)
    n5 = g.concat("n5", [n4, n1])
    n6 = g.c2f("n6", n5, 128, 1)              # output, stride 16
    n7 = g.conv("n7", n6, 128, 3, 2)
    n8 = g.concat("n8", [n7, b8])
    n9 = g.c2f("n9", n8, 256, 1)              # output, stride 32
    g.outputs = [n3, n6, n9]
    return g


def conv_dict(node, n):
    """The mxc_conv of a conv node at batch n."""
    t = node
    return dict(n=n, cin=t["cin"], cout=t["cout"], h=t["src_h"], w=t["src_w"], kh=t["k"], kw=t["k"], sh=t["s"],
                sw=t["s"], ph=t["p"], pw=t["p"])


def mxb(role, fmt, shape):
    """Bytes of an MX tensor's codes and scales."""
    return mx.codes_bytes(role, fmt, *shape) + mx.scales_bytes(role, fmt, *shape)


def mxb_in(role, fmt, shape):
    """Bytes a GEMM reads of an MX operand (or the image quantize writes with
    keep_pad): an activation with a single channel block contributes the
    code rows of its real channels only (its padding rows are known +0
    codes, never fetched or rewritten); otherwise every stored byte, as
    mxb."""
    n, c, h, w = shape
    if role == mx.ACT and c < 32:
        return mx.codes_bytes(role, fmt, *shape) * c / 32.0 + mx.scales_bytes(role, fmt, *shape)
    return mxb(role, fmt, shape)


def real_flops(node, n):
    """2 N Cout Ho Wo Cin Kh Kw with real channels only (no padding)."""
    return 2.0 * n * node["cout"] * node["h"] * node["w"] * node["cin_real"] * node["k"] * node["k"]


# ---------------------------------------------------------------- the step
class NetStep:
    """Buffers and the call sequence of one fwd+bwd training step of `net`
    at batch n (a multiple of 32) in MX format fmt (MXC_E4M3 or MXC_E2M1).

    Inputs (seeded): the image ~ U(0, 1) as bf16 NCHW; bf16 master weights,
    Kaiming-normal over the real input channels (zero on a concatenation's
    padding channels); the upstream gradient of each output ~ N(0, 1e-3) as
    a CBF tensor of the master dtype.

    Full-precision tensors between layers (pre-activations, input gradients,
    upstream gradients) are kept in `master`: bf16 by default, each GEMM
    result rounded to bf16 before it is activated, multiplied or quantized
    (the library's MXC_FN_BF16 / MXC_CBF_BF16 mode), or fp32."""

    def __init__(self, net, n, fmt, device, seed=3000, fused_dgrad=True, master=torch.bfloat16):
        if n % 32:
            raise ValueError("the network step runs batch blocks of 32")
        if master not in (torch.bfloat16, torch.float32):
            raise ValueError("master tensors are bf16 or fp32")
        self.net, self.n, self.fmt, self.dev = net, n, fmt, device
        self.fused = fused_dgrad
        self.master = master
        bf = master == torch.bfloat16
        self.es = 2.0 if bf else 4.0                       # bytes per full-precision element
        self.fbf = mx.FN_BF16 if bf else 0                 # fn flag of the fused calls
        self.gx_layout = mx.CBF_BF16 if bf else mx.CBF
        self.convs = net.convs()
        img = net.nodes[0]
        self.image = synth.uniform((n, img["c"], img["h"], img["w"]), seed).to(torch.bfloat16).to(device)
        self.t = {}      # tensor name -> MxTensor (activations as stored)
        self.y = {}      # conv name -> CBF pre-activation (master dtype)
        self.w = {}      # conv name -> (bf16 master, MxTensor)
        self.gx = {}     # conv name -> CBF input gradient (master dtype)
        self.gy = {}     # conv name -> MxTensor G_Y
        self.ws = {}     # conv name -> split-K workspace
        self.gw = {}     # conv name -> fp32 G_W
        self.cv = {}
        for i, t in enumerate(net.nodes):
            shape = (n, t["c"], t["h"], t["w"])
            if t["kind"] == "input":
                # zero-filled once: the image quantize leaves its padding
                # channels' codes (+0) unwritten on every step
                self.t[t["name"]] = mx.MxTensor.empty(mx.ACT, fmt, shape, device)
                self.t[t["name"]].codes.zero_()
            elif t["kind"] == "concat":
                self.t[t["name"]] = mx.MxTensor.empty(mx.ACT, fmt, shape, device)
            else:
                nm = t["name"]
                cv = conv_dict(t, n)
                self.cv[nm] = cv
                self.t[nm] = mx.MxTensor.empty(mx.ACT, fmt, shape, device)
                self.y[nm] = torch.empty((n // 32, t["h"], t["w"], t["c"], 32), dtype=master, device=device)
                wm = synth.kaiming(t["cout"], t["cin_real"], t["k"], t["k"], seed + 7 * i + 1)
                if t["cin"] != t["cin_real"]:
                    wm = self._spread(wm, net.node(t["src"]))
                wm = wm.to(torch.bfloat16).to(device)
                self.w[nm] = (wm, mx.MxTensor.empty(mx.WEIGHT, fmt, tuple(wm.shape), device))
                self.gy[nm] = mx.MxTensor.empty(mx.ACT, fmt, shape, device)
                if net.node(t["src"])["kind"] != "input":
                    self.gx[nm] = torch.empty((n // 32, cv["h"], cv["w"], cv["cin"], 32), dtype=master,
                                              device=device)
                self.ws[nm] = torch.empty(max(16, mx.wgrad_workspace_bytes(cv, fmt)), dtype=torch.uint8, device=device)
                self.gw[nm] = torch.empty(tuple(wm.shape), dtype=torch.float32, device=device)
        self.ext = {}
        for k, o in enumerate(net.outputs):
            t = net.node(o)
            g = synth.normal((n, t["c"], t["h"], t["w"]), 1e-3, seed + 1000 + k)
            self.ext[o] = synth.nchw_to_cbf(g, 32).to(master).to(device)
        self._plan_backward()

    @staticmethod
    def _spread(wm, cat):
        """Weights over a concatenation's real channels -> its stored channels
        (each part's channels at its block offset, zero on the padding)."""
        cout, _, kh, kw = wm.shape
        full = torch.zeros((cout, cat["c"], kh, kw), dtype=wm.dtype)
        r = 0
        for off, c in zip(cat["offs"], cat["part_real"]):
            full[:, off:off + c] = wm[:, r:r + c]
            r += c
        return full

    def _fusable(self, t):
        """Conv t's input is another conv's output that only t reads and that
        is no network output: t's input-gradient epilogue can quantize it."""
        src = self.net.node(t["src"])
        return (src["kind"] == "conv" and self.consumers[src["name"]] == [("conv", t["name"])]
                and src["name"] not in self.ext)

    # consumers of every tensor: ("conv", conv name) or ("concat", concat name, part index)
    def _plan_backward(self):
        net = self.net
        cons = {t["name"]: [] for t in net.nodes}
        for t in net.nodes:
            if t["kind"] == "conv":
                cons[t["src"]].append(("conv", t["name"]))
            elif t["kind"] == "concat":
                for k, (p, _) in enumerate(t["parts"]):
                    cons[p].append(("concat", t["name"], k))
        self.consumers = cons

    def grad_terms(self, name):
        """Terms (src, c_src, c_off, down) of the gradient of tensor `name`
        (master-dtype CBF tensors)."""
        net = self.net
        terms = []
        for c in self.consumers[name]:
            if c[0] == "conv":
                terms.append((self.gx[c[1]], net.node(c[1])["cin"], 0, 0))
            else:
                cat = net.node(c[1])
                up = cat["parts"][c[2]][1]
                off = cat["offs"][c[2]]
                for cc in self.consumers[cat["name"]]:
                    assert cc[0] == "conv", "a concatenation feeds convolutions only"
                    terms.append((self.gx[cc[1]], cat["c"], off, up))
        if name in self.ext:
            terms.append((self.ext[name], net.node(name)["c"], 0, 0))
        return terms

    def calls(self):
        """The step as a list of (label, callable, algorithmic flops, algorithmic
        bytes): flops of a GEMM with real channels only; bytes = every operand
        read once and every result written once (codes + scales of MX
        tensors, 4 bytes per fp32 element, 2 per bf16 element)."""
        net, n, fmt, es, fbf = self.net, self.n, self.fmt, self.es, self.fbf
        A, W = mx.ACT, mx.WEIGHT
        seq = []
        img = net.nodes[0]
        ishape = (n, img["c"], img["h"], img["w"])
        seq.append(("quant_image", lambda: mx.quantize(self.image, A, fmt, out=self.t[img["name"]], keep_pad=True),
                    0.0, 2.0 * math.prod(ishape) + mxb_in(A, fmt, ishape)))
        names = [t["name"] for t in self.convs]
        for i in range(0, len(names), mx.QMULTI_MAX):
            grp = names[i:i + mx.QMULTI_MAX]
            items = [(self.w[nm][0], W, fmt, mx.NCHW, tuple(self.w[nm][0].shape), self.w[nm][1]) for nm in grp]
            by = sum(2.0 * self.w[nm][0].numel() + mxb(W, fmt, tuple(self.w[nm][0].shape)) for nm in grp)
            seq.append((f"quant_w{i // mx.QMULTI_MAX}", lambda items=items: mx.quantize_multi(items), 0.0, by))
        # forward
        for t in net.nodes[1:]:
            nm = t["name"]
            oshape = (n, t["c"], t["h"], t["w"])
            if t["kind"] == "conv":
                src = net.node(t["src"])
                by = (mxb(W, fmt, tuple(self.w[nm][0].shape)) + mxb_in(A, fmt, (n, src["c"], src["h"], src["w"])) +
                      mxb(A, fmt, oshape) + es * math.prod(oshape))
                seq.append((f"fwd {nm}", lambda nm=nm, t=t: mx.fwd_quant(
                    self.cv[nm], self.w[nm][1], self.t[t["src"]], fn=mx.FN_SILU | mx.FN_PRE_OUT | fbf, out=self.t[nm],
                    act_out=self.y[nm]), real_flops(t, n), by))
            else:
                parts = [(self.t[p], up) for p, up in t["parts"]]
                by = sum(mxb(A, fmt, self.t[p].shape) for p, _ in t["parts"]) + mxb(A, fmt, oshape)
                seq.append((f"concat {nm}", lambda parts=parts, nm=nm: mx.concat_cbf(parts, out=self.t[nm]), 0.0, by))
        # backward, in reverse order: quantize a conv's G_Y once its consumers
        # have handed back their gradients, then its input and weight
        # gradients.  A conv whose input is read by it alone (and is no
        # output) quantizes that input's gradient in its input-gradient
        # epilogue (times SiLU' at the producer's pre-activation), so the
        # producer's G_Y never exists in fp32.
        fused_in = {t["src"] for t in self.convs if self.fused and self._fusable(t)}
        for t in reversed(self.convs):
            nm = t["name"]
            shape = (n, t["c"], t["h"], t["w"])
            if nm not in fused_in:
                terms = self.grad_terms(nm)
                el = math.prod(shape)
                by = sum(es * el * (4 if d else 1) for _, _, _, d in terms) + es * el + mxb(A, fmt, shape)
                seq.append((f"quant_gy {nm}", lambda terms=terms, shape=shape, nm=nm: mx.quantize_sum(
                    terms, shape, fmt, fn=mx.FN_SILU | fbf, z=self.y[nm], out=self.gy[nm]), 0.0, by))
            src = net.node(t["src"])
            sshape = (n, src["c"], src["h"], src["w"])
            xb = mxb_in(A, fmt, sshape)
            gb = mxb_in(A, fmt, shape)
            wb = mxb(W, fmt, tuple(self.w[nm][0].shape))
            gwb = 4.0 * self.gw[nm].numel()
            f = real_flops(t, n)
            if t["src"] in fused_in:
                sn = t["src"]
                seq.append((f"dgrad_quant {nm}", lambda nm=nm, sn=sn: mx.dgrad_quant(
                    self.cv[nm], self.w[nm][1], self.gy[nm], fn=mx.FN_SILU | fbf, z=self.y[sn], out=self.gy[sn]),
                    f, wb + gb + es * math.prod(sshape) + mxb(A, fmt, sshape)))
                seq.append((f"wgrad {nm}", lambda nm=nm, t=t: mx.wgrad(
                    self.cv[nm], self.gy[nm], self.t[t["src"]], out=self.gw[nm], workspace=self.ws[nm],
                    deferred=True), f, gb + xb + gwb))
            elif nm in self.gx:
                seq.append((f"bwd {nm}", lambda nm=nm, t=t: mx.backward(
                    self.cv[nm], self.w[nm][1], self.gy[nm], self.t[t["src"]], layout=self.gx_layout,
                    gx_out=self.gx[nm], gw_out=self.gw[nm], workspace=self.ws[nm], deferred=True),
                    2.0 * f, wb + gb + xb + es * self.gx[nm].numel() + gwb))
            else:
                seq.append((f"wgrad {nm}", lambda nm=nm, t=t: mx.wgrad(
                    self.cv[nm], self.gy[nm], self.t[t["src"]], out=self.gw[nm], workspace=self.ws[nm],
                    deferred=True), f, gb + xb + gwb))
        items = [(self.cv[nm], fmt, self.ws[nm], self.gw[nm]) for nm in names]
        for i in range(0, len(items), mx.WREDUCE_MAX):
            grp = items[i:i + mx.WREDUCE_MAX]
            by = sum((mx.wgrad_workspace_bytes(cv, fmt) + 4.0 * gw.numel()) if mx.wgrad_workspace_bytes(cv, fmt) else 0.0
                     for cv, _, _, gw in grp)
            seq.append((f"wgrad_reduce{i // mx.WREDUCE_MAX}", lambda grp=grp: mx.wgrad_reduce_multi(grp), 0.0, by))
        return seq

    def flops(self):
        """Algorithmic flops of the step's GEMMs (real channels): forward,
        input gradient (not for the first layer, whose input is the image)
        and weight gradient of every convolution."""
        tot = 0.0
        for t in self.convs:
            f = real_flops(t, self.n)
            tot += f * (3 if t["name"] in self.gx else 2)
        return tot


# ---------------------------------------------------------------- quantized latent replay
class QlrStep:
    """Quantized latent replay (Sec. VII): a frozen front stack of three
    stride-2 3x3 convolutions (3 -> 32 -> 64 -> 128 channels, SiLU) maps
    3 x 128 x 128 inputs to 128 x 16 x 16 latents; a buffer of `buffer`
    latents is kept as MX codes and E8M0 scales (built once, outside the
    step, by running the front stack over seeded U(0, 1) inputs); the
    trainable back stack of four 3x3 s1 p1 convolutions (128 -> 256, then
    256 -> 256 three times, SiLU) runs fwd + bwd on batches of 128 = three
    replayed 32-sample groups (copied as stored codes, never requantized)
    and 32 fresh inputs (front stack forward, quantized once by its last
    epilogue straight into the batch).  Upstream gradient ~ N(0, 1e-3)."""

    FRONT = ((3, 32), (32, 64), (64, 128))
    BACK = ((128, 256), (256, 256), (256, 256), (256, 256))

    def __init__(self, device, fmt=mx.E2M1, buffer=8192, batch=128, seed=5000, fused_dgrad=True,
                 master=torch.bfloat16):
        if master not in (torch.bfloat16, torch.float32):
            raise ValueError("master tensors are bf16 or fp32")
        self.dev, self.fmt, self.batch = device, fmt, batch
        self.fused = fused_dgrad
        bf = master == torch.bfloat16
        self.es = 2.0 if bf else 4.0
        self.fbf = mx.FN_BF16 if bf else 0
        self.gx_layout = mx.CBF_BF16 if bf else mx.CBF
        g = torch.Generator()
        g.manual_seed(seed)
        self.front_cv = []
        h = 128
        for i, (ci, co) in enumerate(self.FRONT):
            self.front_cv.append(synth.conv_dict(32, ci, co, h, h, 3, 2, 1))
            h //= 2
        self.lat = (128, h, h)
        self.back_cv = [synth.conv_dict(batch, ci, co, h, h, 3, 1, 1) for ci, co in self.BACK]
        self.front_w = [mx.quantize(synth.kaiming(cv["cout"], cv["cin"], 3, 3, seed + 1 + i).to(device), mx.WEIGHT, fmt)
                        for i, cv in enumerate(self.front_cv)]
        self.back_wm = [synth.kaiming(cv["cout"], cv["cin"], 3, 3, seed + 11 + i).to(torch.bfloat16).to(device)
                        for i, cv in enumerate(self.back_cv)]
        self.back_w = [mx.MxTensor.empty(mx.WEIGHT, fmt, tuple(w.shape), device) for w in self.back_wm]
        # front-stack activations for one 32-sample group
        self.front_x = mx.MxTensor.empty(mx.ACT, fmt, (32, 3, 128, 128), device)
        self.front_x.codes.zero_()     # padding channels' codes stay +0 (quantize with keep_pad)
        self.front_t = []
        for cv in self.front_cv[:-1]:
            ho, wo = synth.out_hw(cv)
            self.front_t.append(mx.MxTensor.empty(mx.ACT, fmt, (32, cv["cout"], ho, wo), device))
        # the replay buffer: groups of 32 latents, stored codes and scales
        self.ngroups = buffer // 32
        lc = mx.codes_bytes(mx.ACT, fmt, 32, *self.lat)
        ls = mx.scales_bytes(mx.ACT, fmt, 32, *self.lat)
        self.lc, self.ls = lc, ls
        self.buf_codes = torch.empty(self.ngroups * lc, dtype=torch.uint8, device=device)
        self.buf_scales = torch.empty(self.ngroups * ls, dtype=torch.uint8, device=device)
        for k in range(self.ngroups):
            img = synth.uniform((32, 3, 128, 128), seed + 100 + k).to(device)
            self._front(img, self._group(self.buf_codes, self.buf_scales, k))
        torch.cuda.synchronize()
        # the step's inputs: fresh images and which stored groups to replay
        self.fresh = synth.uniform((32, 3, 128, 128), seed + 99).to(device)
        nrep = batch // 32 - 1
        self.replay = torch.randperm(self.ngroups, generator=g)[:nrep].tolist()
        # back-stack buffers
        n = batch
        self.x = [mx.MxTensor.empty(mx.ACT, fmt, (n, 128) + self.lat[1:], device)]
        self.y, self.gy, self.gx, self.gw, self.ws = [], [], [], [], []
        for i, cv in enumerate(self.back_cv):
            shp = (n, cv["cout"], cv["h"], cv["w"])
            self.y.append(torch.empty((n // 32, cv["h"], cv["w"], cv["cout"], 32), dtype=master, device=device))
            self.x.append(mx.MxTensor.empty(mx.ACT, fmt, shp, device))
            self.gy.append(mx.MxTensor.empty(mx.ACT, fmt, shp, device))
            self.gx.append(torch.empty((n // 32, cv["h"], cv["w"], cv["cin"], 32), dtype=master, device=device)
                           if i > 0 else None)
            self.gw.append(torch.empty((cv["cout"], cv["cin"], 3, 3), dtype=torch.float32, device=device))
            self.ws.append(torch.empty(max(16, mx.wgrad_workspace_bytes(cv, fmt)), dtype=torch.uint8, device=device))
        last = self.back_cv[-1]
        ge = synth.normal((n, last["cout"], last["h"], last["w"]), 1e-3, seed + 98)
        self.ext = synth.nchw_to_cbf(ge, 32).to(master).to(device)

    def _group(self, codes, scales, k):
        return mx.MxTensor(codes[k * self.lc:(k + 1) * self.lc], scales[k * self.ls:(k + 1) * self.ls], mx.ACT,
                           self.fmt, (32,) + self.lat)

    def _front(self, img, out):
        """Front stack forward on 32 images (fp32 NCHW), its last epilogue
        writing the latents' codes into `out`."""
        mx.quantize(img, mx.ACT, self.fmt, out=self.front_x, keep_pad=True)
        src = self.front_x
        for i, cv in enumerate(self.front_cv):
            dst = out if i == len(self.front_cv) - 1 else self.front_t[i]
            mx.fwd_quant(cv, self.front_w[i], src, fn=mx.FN_SILU, out=dst)
            src = dst

    def calls(self):
        """The step as (label, callable, algorithmic flops, algorithmic bytes)
        tuples, with the conventions of NetStep.calls."""
        fmt, n, es, fbf = self.fmt, self.batch, self.es, self.fbf
        A, W = mx.ACT, mx.WEIGHT
        seq = [("quant_w", lambda: mx.quantize_multi(
            [(w, W, fmt, mx.NCHW, tuple(w.shape), q) for w, q in zip(self.back_wm, self.back_w)]), 0.0,
            sum(2.0 * w.numel() + mxb(W, fmt, tuple(w.shape)) for w in self.back_wm))]
        x0 = self.x[0]
        for slot, k in enumerate(self.replay):    # replayed groups: stored codes and scales, copied
            seq.append((f"replay{slot}", lambda slot=slot, k=k: (
                x0.codes[slot * self.lc:(slot + 1) * self.lc].copy_(self.buf_codes[k * self.lc:(k + 1) * self.lc]),
                x0.scales[slot * self.ls:(slot + 1) * self.ls].copy_(self.buf_scales[k * self.ls:(k + 1) * self.ls])),
                0.0, 2.0 * (self.lc + self.ls)))
        last = n // 32 - 1
        ffl, fby = 0.0, 4.0 * self.fresh.numel() + mxb_in(A, fmt, (32, 3, 128, 128))
        for i, cv in enumerate(self.front_cv):
            ho, wo = synth.out_hw(cv)
            ffl += 2.0 * 32 * cv["cout"] * ho * wo * cv["cin"] * 9
            fby += (mxb(W, fmt, (cv["cout"], cv["cin"], 3, 3)) + mxb_in(A, fmt, (32, cv["cin"], cv["h"], cv["w"])) +
                    mxb(A, fmt, (32, cv["cout"], ho, wo)))
        seq.append(("front", lambda: self._front(self.fresh, self._group(x0.codes, x0.scales, last)), ffl, fby))
        for i, cv in enumerate(self.back_cv):
            shp = (n, cv["cout"], cv["h"], cv["w"])
            f = 2.0 * n * cv["cout"] * cv["h"] * cv["w"] * cv["cin"] * 9
            by = (mxb(W, fmt, (cv["cout"], cv["cin"], 3, 3)) + mxb(A, fmt, (n, cv["cin"], cv["h"], cv["w"])) +
                  mxb(A, fmt, shp) + es * math.prod(shp))
            seq.append((f"fwd back{i}", lambda i=i, cv=cv: mx.fwd_quant(
                cv, self.back_w[i], self.x[i], fn=mx.FN_SILU | mx.FN_PRE_OUT | fbf, out=self.x[i + 1],
                act_out=self.y[i]),
                f, by))
        lc = self.back_cv[-1]
        shp = (n, lc["cout"], lc["h"], lc["w"])
        seq.append(("quant_gy back3", lambda: mx.quantize_sum([(self.ext, lc["cout"], 0, 0)], shp, fmt,
                                                             fn=mx.FN_SILU | fbf, z=self.y[-1], out=self.gy[-1]),
                    0.0, 2.0 * es * math.prod(shp) + mxb(A, fmt, shp)))
        for i in range(len(self.back_cv) - 1, -1, -1):
            cv = self.back_cv[i]
            f = 2.0 * n * cv["cout"] * cv["h"] * cv["w"] * cv["cin"] * 9
            gshp = (n, cv["cout"], cv["h"], cv["w"])
            xshp = (n, cv["cin"], cv["h"], cv["w"])
            wb = mxb(W, fmt, (cv["cout"], cv["cin"], 3, 3))
            wgb = mxb(A, fmt, gshp) + mxb(A, fmt, xshp) + 4.0 * cv["cout"] * cv["cin"] * 9
            if i == 0:     # the latents are not trained: weight gradient only
                seq.append(("wgrad back0", lambda cv=cv: mx.wgrad(cv, self.gy[0], self.x[0], out=self.gw[0],
                                                                  workspace=self.ws[0], deferred=True), f, wgb))
            elif self.fused:   # this layer's input gradient, times SiLU', quantized as the layer below's G_Y
                seq.append((f"dgrad_quant back{i}", lambda i=i, cv=cv: mx.dgrad_quant(
                    cv, self.back_w[i], self.gy[i], fn=mx.FN_SILU | fbf, z=self.y[i - 1], out=self.gy[i - 1]),
                    f, wb + mxb(A, fmt, gshp) + es * math.prod(xshp) + mxb(A, fmt, xshp)))
                seq.append((f"wgrad back{i}", lambda i=i, cv=cv: mx.wgrad(
                    cv, self.gy[i], self.x[i], out=self.gw[i], workspace=self.ws[i], deferred=True), f, wgb))
            else:
                seq.append((f"bwd back{i}", lambda i=i, cv=cv: mx.backward(
                    cv, self.back_w[i], self.gy[i], self.x[i], layout=self.gx_layout, gx_out=self.gx[i],
                    gw_out=self.gw[i], workspace=self.ws[i], deferred=True), 2.0 * f, wb + wgb + es * math.prod(xshp)))
                pc = self.back_cv[i - 1]
                pshp = (n, pc["cout"], pc["h"], pc["w"])
                seq.append((f"quant_gy back{i - 1}", lambda i=i, pc=pc, pshp=pshp: mx.quantize_sum(
                    [(self.gx[i], pc["cout"], 0, 0)], pshp, fmt, fn=mx.FN_SILU | fbf, z=self.y[i - 1],
                    out=self.gy[i - 1]), 0.0, 2.0 * es * math.prod(pshp) + mxb(A, fmt, pshp)))
        rb = sum(mx.wgrad_workspace_bytes(cv, fmt) + 4.0 * cv["cout"] * cv["cin"] * 9 for cv in self.back_cv
                 if mx.wgrad_workspace_bytes(cv, fmt))
        seq.append(("wgrad_reduce", lambda: mx.wgrad_reduce_multi(
            [(cv, fmt, self.ws[i], self.gw[i]) for i, cv in enumerate(self.back_cv)]), 0.0, rb))
        return seq

    def flops(self):
        """Back stack: forward, input gradient (not for the first layer) and
        weight gradient; front stack: forward of the 32 fresh inputs (real
        input channels)."""
        tot = 0.0
        for i, cv in enumerate(self.back_cv):
            f = 2.0 * cv["n"] * cv["cout"] * cv["h"] * cv["w"] * cv["cin"] * 9
            tot += f * (2 if i == 0 else 3)
        for cv in self.front_cv:
            ho, wo = synth.out_hw(cv)
            tot += 2.0 * cv["n"] * cv["cout"] * ho * wo * cv["cin"] * 9
        return tot
