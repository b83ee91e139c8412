"""Seeded synthetic inputs shaped like the paper's convolution workloads.

This module holds no arithmetic of the method: it only draws seeded random
tensors (fp32, on the CPU, so every consumer sees identical bits) and
permutes layouts.  Both the GPU path and the oracle take their inputs from
here; nothing else is shared between them.

Distributions (the layer sweep and single-layer cases):
  * activations: SiLU of N(0, 1) (post-activation feature maps), or N(0, 1)
  * weights: Kaiming-normal, sigma = sqrt(2 / (Cin * Kh * Kw)), or N(0, 0.1)
  * upstream gradients: N(0, 1e-3), or N(0, 1)
SiLU is evaluated in fp64 and rounded once to fp32.
"""
import math

import torch


def conv_dict(n, cin, cout, h, w, k, s=1, p=None):
    if p is None:
        p = (k - 1) // 2
    return dict(n=n, cin=cin, cout=cout, h=h, w=w, kh=k, kw=k, sh=s, sw=s, ph=p, pw=p)


def out_hw(cv):
    ho = (cv["h"] + 2 * cv["ph"] - cv["kh"]) // cv["sh"] + 1
    wo = (cv["w"] + 2 * cv["pw"] - cv["kw"]) // cv["sw"] + 1
    return ho, wo


def _gen(seed):
    g = torch.Generator()
    g.manual_seed(int(seed))
    return g


def normal(shape, std, seed):
    return (torch.randn(shape, generator=_gen(seed), dtype=torch.float32) * std).contiguous()


def silu_normal(shape, seed):
    z = torch.randn(shape, generator=_gen(seed), dtype=torch.float32).double()
    return (z * torch.sigmoid(z)).float().contiguous()


def uniform(shape, seed, lo=0.0, hi=1.0):
    return (torch.rand(shape, generator=_gen(seed), dtype=torch.float32) * (hi - lo) + lo).contiguous()


def kaiming(cout, cin, kh, kw, seed):
    return normal((cout, cin, kh, kw), math.sqrt(2.0 / (cin * kh * kw)), seed)


def layer_inputs(cv, seed, kind="sweep"):
    """X (NCHW), W (OIHW) and G_Y (NCHW) fp32 CPU tensors for one conv layer.

    kind "sweep": X = SiLU(N(0,1)), W Kaiming-normal, G_Y ~ N(0, 1e-3).
    kind "unit":  X ~ N(0,1), W ~ N(0,0.1), G_Y ~ N(0,1).
    Three streams derived from one seed."""
    ho, wo = out_hw(cv)
    xs = (cv["n"], cv["cin"], cv["h"], cv["w"])
    gs = (cv["n"], cv["cout"], ho, wo)
    if kind == "sweep":
        x = silu_normal(xs, seed * 3 + 0)
        w = kaiming(cv["cout"], cv["cin"], cv["kh"], cv["kw"], seed * 3 + 1)
        gy = normal(gs, 1e-3, seed * 3 + 2)
    elif kind == "unit":
        x = normal(xs, 1.0, seed * 3 + 0)
        w = normal((cv["cout"], cv["cin"], cv["kh"], cv["kw"]), 0.1, seed * 3 + 1)
        gy = normal(gs, 1.0, seed * 3 + 2)
    else:
        raise ValueError(kind)
    return x, w, gy


def batch_block(n):
    """Samples per block along the batch: 32, or N itself when N < 32."""
    return 32 if n >= 32 else n


def nchw_to_cbf(x, bn):
    """(N, C, H, W) -> [N/bn][H][W][C][bn], a pure permutation."""
    n, c, h, w = x.shape
    return x.reshape(n // bn, bn, c, h, w).permute(0, 3, 4, 2, 1).contiguous()


def cbf_to_nchw(y, n, c, h, w, bn):
    """Inverse of nchw_to_cbf for a flat or shaped [N/bn][H][W][C][bn] tensor."""
    return y.reshape(n // bn, h, w, c, bn).permute(0, 4, 3, 1, 2).reshape(n, c, h, w).contiguous()


# The benchmark workload: the layer sweep (batch 32) in MXFP8 and MXFP4.
SWEEP_LAYERS = (
    ("3x3_s1_64to64_56", conv_dict(32, 64, 64, 56, 56, 3, 1, 1)),
    ("1x1_s1_64to256_56", conv_dict(32, 64, 256, 56, 56, 1, 1, 0)),
    ("3x3_s2_128to256_28", conv_dict(32, 128, 256, 28, 28, 3, 2, 1)),
)

# The small single-layer case: N=2, 32->32, 8x8, 3x3 s1 p1, MXFP8, one seed.
UNIT_LAYER = conv_dict(2, 32, 32, 8, 8, 3, 1, 1)


# YOLOv8n-shaped backbone + neck (batch 16 in MXFP8, batch 64 in MXFP4; a
# 3x640x640 input, bf16 master tensors).  Representative layers at their full
# sizes: the stride-2 3x3 stem (3 -> 16 channels, 640x640 -> 320x320), a
# C2f-style 3x3 at half the stage width (16 channels, 160x160) and a C2f-style
# 1x1 merging 3c/2 -> c at the deepest stage (384 -> 256, 20x20).
def yolo_layers(n):
    return (
        ("stem_3to16_s2_640", conv_dict(n, 3, 16, 640, 640, 3, 2, 1)),
        ("c2f_3x3_16_160", conv_dict(n, 16, 16, 160, 160, 3, 1, 1)),
        ("c2f_1x1_384to256_20", conv_dict(n, 384, 256, 20, 20, 1, 1, 0)),
    )


def yolo_inputs(name, cv, seed):
    """X and W as bf16 (the master tensors), G_Y fp32.  The stem reads the
    image, U(0, 1); deeper layers read SiLU feature maps; W Kaiming-normal;
    G_Y ~ N(0, 1e-3)."""
    ho, wo = out_hw(cv)
    xs = (cv["n"], cv["cin"], cv["h"], cv["w"])
    x = uniform(xs, seed * 3) if name.startswith("stem") else silu_normal(xs, seed * 3)
    w = kaiming(cv["cout"], cv["cin"], cv["kh"], cv["kw"], seed * 3 + 1)
    gy = normal((cv["n"], cv["cout"], ho, wo), 1e-3, seed * 3 + 2)
    return x.to(torch.bfloat16), w.to(torch.bfloat16), gy


# Quantized latent replay: a buffer of 8192 latents of 128 x 16 x 16 (the
# output of a frozen front stack, SiLU-activated; drawn here as SiLU of
# N(0, 1)), kept as MX codes in groups of 32 samples; the trainable back stack
# of 3x3 s1 p1 convolutions (128 -> 256, then 256 -> 256 at 16x16) runs on
# batches of 128 = 96 replayed + 32 fresh latents.
QLR_BUFFER = 8192
QLR_LATENT = (128, 16, 16)
QLR_BATCH = 128
QLR_LAYERS = (
    ("back_3x3_128to256_16", conv_dict(QLR_BATCH, 128, 256, 16, 16, 3, 1, 1)),
    ("back_3x3_256to256_16", conv_dict(QLR_BATCH, 256, 256, 16, 16, 3, 1, 1)),
)


def qlr_latents(count, seed):
    """`count` latents (count, 128, 16, 16), fp32."""
    return silu_normal((count,) + QLR_LATENT, seed)
