"""Seeded synthetic inputs for the derived-operator workloads.

This module only draws random tensors and describes workload shapes. It holds
none of the operators' arithmetic, so both the CPU oracle and the HIP path can
take their inputs from it without sharing any computation.

Layouts (all row-major, contiguous):
  X   [n][h][w][c]      activation, NHWC (the paper's A[h,w,c] of the convolution
                        expression in section 4.2, with a batch dimension added)
  Wt  [r][s][k][c]      weight (the paper's K[r,s,f,c]; f is the output channel k)
  Q,K,V [b][l][d]       banded batched matmul operands

Every tensor is drawn in float32 on the CPU from
``torch.Generator().manual_seed(1000 * cfg + tensor_id)`` (X=0, Wt=1; Q=0, K=1,
V=2) and, for bf16 workloads, rounded to bfloat16 with round-to-nearest-even.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch


@dataclass(frozen=True)
class ConvWorkload:
    """One convolution-family workload (conv2d, dilated conv2d or conv_transpose2d)."""
    cfg: int
    name: str
    kind: str                      # "conv2d" | "dilated_conv2d" | "conv_transpose2d"
    n: int
    c: int
    h: int
    w: int
    k: int
    r: int
    s: int
    stride: tuple = (1, 1)
    pad: tuple = (0, 0)
    dil: tuple = (1, 1)
    out_pad: tuple = (0, 0)
    dtype: str = "bf16"            # input dtype: "f32" | "bf16"
    x_dist: str = "normal"         # "uniform" | "normal" | "relu_normal"
    w_std: float = 1.0             # std of the weight normal (ignored for uniform)
    w_dist: str = "normal"         # "uniform" | "normal"

    @property
    def transposed(self) -> bool:
        return self.kind == "conv_transpose2d"


@dataclass(frozen=True)
class BandWorkload:
    """Banded dilated batched matmul (Longformer-style sliding-window attention)."""
    cfg: int
    name: str
    b: int
    l: int
    d: int
    w: int                          # half window; band width is 2w+1
    dilation: int
    scale: float = 1.0
    mask_invalid: bool = False      # False: zero mode (out-of-range scores are 0 and count)
    dtype: str = "bf16"


# The five workloads, sized as the layers they stand in for:
# 1: a tiny 3x3 conv (parity only); 2: a ResNet-18 stage-3 conv3x3 at batch 16;
# 3: a DCGAN generator ConvTranspose2d; 4: a CSRNet back-end dilated conv;
# 5: Longformer-base dilated sliding-window attention (8 sequences x 12 heads);
# 6: an SRCNN 9-5-5 second layer (conv5x5, 64 -> 32 channels, "same" padding) on a
# 512x512 image, the workload of the Conv5x5 -> Conv3x3 derived form.
WORKLOADS = {
    1: ConvWorkload(1, "conv3x3_tiny", "conv2d", n=1, c=16, h=14, w=14, k=16, r=3, s=3,
                    stride=(1, 1), pad=(1, 1), dtype="f32", x_dist="uniform", w_dist="uniform"),
    2: ConvWorkload(2, "resnet_conv3x3_n16_c256_14x14", "conv2d", n=16, c=256, h=14, w=14,
                    k=256, r=3, s=3, stride=(1, 1), pad=(1, 1), dtype="bf16",
                    x_dist="normal", w_std=math.sqrt(2.0 / (9 * 256))),
    3: ConvWorkload(3, "dcgan_convT4x4_s2_n16_c512_k256_8x8", "conv_transpose2d", n=16, c=512,
                    h=8, w=8, k=256, r=4, s=4, stride=(2, 2), pad=(1, 1), dtype="bf16",
                    x_dist="normal", w_std=0.02),
    4: ConvWorkload(4, "csrnet_dilconv3x3_d2_c512_96x128", "dilated_conv2d", n=1, c=512,
                    h=96, w=128, k=512, r=3, s=3, stride=(1, 1), pad=(2, 2), dil=(2, 2),
                    dtype="bf16", x_dist="relu_normal", w_std=math.sqrt(2.0 / (9 * 512))),
    5: BandWorkload(5, "longformer_band_b96_l4096_d64_w256_dil2", b=96, l=4096, d=64, w=256,
                    dilation=2, scale=1.0, mask_invalid=False, dtype="bf16"),
    6: ConvWorkload(6, "srcnn_conv5x5_c64_k32_512x512", "conv2d", n=1, c=64, h=512, w=512,
                    k=32, r=5, s=5, stride=(1, 1), pad=(2, 2), dtype="bf16",
                    x_dist="relu_normal", w_std=math.sqrt(2.0 / (25 * 64))),
}


def _gen(cfg: int, tensor_id: int) -> torch.Generator:
    return torch.Generator().manual_seed(1000 * cfg + tensor_id)


def _round(t: torch.Tensor, dtype: str) -> torch.Tensor:
    """float32 -> the workload dtype (RNE for bf16); returned as that dtype."""
    if dtype == "bf16":
        return t.to(torch.bfloat16)
    return t.contiguous()


def _draw(shape, dist: str, std: float, gen: torch.Generator) -> torch.Tensor:
    if dist == "uniform":
        return torch.rand(shape, generator=gen, dtype=torch.float32) * 2.0 - 1.0
    t = torch.randn(shape, generator=gen, dtype=torch.float32) * std
    if dist == "relu_normal":
        t = torch.relu(t)
    return t


def conv_inputs(wl: ConvWorkload, integer: bool = False, seed_offset: int = 0):
    """Return (X, Wt) on the CPU in the workload dtype.

    integer=True draws small integers in {-3..3} instead (held exactly in fp32 and
    bf16), so that every partial and every sum is an exact small integer.
    """
    xs = (wl.n, wl.h, wl.w, wl.c)
    ws = (wl.r, wl.s, wl.k, wl.c)
    gx = _gen(wl.cfg + seed_offset, 0)
    gw = _gen(wl.cfg + seed_offset, 1)
    if integer:
        x = torch.randint(-3, 4, xs, generator=gx).to(torch.float32)
        wt = torch.randint(-3, 4, ws, generator=gw).to(torch.float32)
    else:
        x = _draw(xs, wl.x_dist, 1.0, gx)
        wt = _draw(ws, wl.w_dist, wl.w_std, gw)
    return _round(x, wl.dtype), _round(wt, wl.dtype)


def band_inputs(wl: BandWorkload, integer: bool = False, seed_offset: int = 0):
    """Return (Q, K, V) [b][l][d] on the CPU in the workload dtype."""
    shape = (wl.b, wl.l, wl.d)
    out = []
    for tid in range(3):
        g = _gen(wl.cfg + seed_offset, tid)
        if integer and tid < 2:
            t = torch.randint(-3, 4, shape, generator=g).to(torch.float32)
        else:
            t = torch.randn(shape, generator=g, dtype=torch.float32)
        out.append(_round(t, wl.dtype))
    return tuple(out)


def random_tensor(shape, seed: int, dtype: str = "f32", integer: bool = False,
                  dist: str = "uniform") -> torch.Tensor:
    """A seeded tensor of any shape, for small randomized cases."""
    g = torch.Generator().manual_seed(seed)
    if integer:
        t = torch.randint(-3, 4, tuple(shape), generator=g).to(torch.float32)
    else:
        t = _draw(tuple(shape), dist, 1.0, g)
    return _round(t, dtype)


def device_integer_tensor(shape, seed: int, device, dtype=torch.bfloat16) -> torch.Tensor:
    """A seeded integer-valued tensor (values in {-3..3}) drawn directly on `device`,
    for operands too large to draw on the CPU and copy over (multi-GiB cases that
    are checked on sampled outputs)."""
    g = torch.Generator(device=device).manual_seed(seed)
    t = torch.randint(-3, 4, tuple(shape), generator=g, device=device, dtype=torch.int8)
    return t.to(dtype)
