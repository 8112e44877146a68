"""Seeded synthetic workloads for the Book-Keeping (BK) clipping path.

This module only describes layer stacks and draws their inputs; it contains
none of the method's arithmetic (no norms, no path choice, no clipping, no
noise).  Both the CPU oracle's tests and the GPU path's tests/bench draw their
inputs from here, so the two sides see bit-identical data.

The stacks stand in for the paper's workloads (GPT-2 on E2E-length text, the
long-sequence regime of Section 3.1, ViT-base at 224x224, GPT-2-large with its
token embedding, the convolutions of ResNet-18 at 224x224 behind the
layerwise decision of Section 3.2, and LoRA on GPT-2 small as in App. E.2);
the datasets and pretrained weights are not used.  Shapes
follow Section 2.1 (a in R^{B x T x d}, dL/ds in R^{B x T x p}) and the
per-layer dimensions of GPT-2 small/large and ViT-base.

Recipe (stated once, used everywhere):
  * tensor k of layer l of workload w is drawn by torch's generator seeded with
    1000*w + 2*l + k (k = 0: activations a, k = 1: output gradients g);
  * values are standard normal in float32, g is multiplied by ``g_scale``,
    then the tensor is rounded (round-to-nearest-even) to the workload dtype;
  * token ids of an embedding layer follow a finite Zipf law,
    P(id = k-1) proportional to k^-s for k = 1..V, drawn with numpy's PCG64
    seeded with 1000*w + 999;
  * a convolution layer draws its input x [B, C_in, H, H] (k = 0) and its
    output gradient [B, C_out, Ho, Ho] (k = 1) in the same way (NCHW); its
    linear-layer view has T = Ho*Ho, d = C_in*k*k rounded up to a multiple of
    8 (zero columns), p = C_out;
  * a LayerNorm affine layer draws its normalized input xhat [B, T, p] (k = 0)
    and output gradient (k = 1) like a linear layer with d = p.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

__all__ = ["Layer", "Workload", "WORKLOADS", "get", "draw_linear", "draw_embedding",
           "draw_layer", "zipf_ids", "make_stack", "workload_from_shapes", "conv_layer", "draw_conv"]


@dataclass(frozen=True)
class Layer:
    """One generalized linear layer: s = a W with W in R^{d x p} (Section 2.1).

    kind == "embed": a is the one-hot encoding of token ids over a vocabulary of
    size V == d, so only ids and g are stored.
    """
    kind: str          # "linear" | "embed" | "conv" | "norm" (affine of a LayerNorm, d = p)
    T: int
    d: int
    p: int
    conv: tuple = ()   # kind == "conv": (C_in, k, stride, pad, H_in)
    bias: bool = False # a bias (linear / conv) or a beta (norm)

    @property
    def V(self) -> int:
        return self.d


@dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    B: int
    dtype: str                   # "f32" | "bf16"
    layers: tuple
    clip: str                    # "abadi" | "auto"
    R: float = 1.0
    gamma: float = 0.01
    sigma: float = 1.0
    g_scale: float = 1.0
    zipf_s: float = 1.1
    description: str = ""

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def noise_std(self) -> float:
        # sigma * R for Abadi clipping; automatic clipping bounds every clipped
        # per-sample gradient norm by 1, so its sensitivity is taken as R = 1.
        return self.sigma * (self.R if self.clip == "abadi" else 1.0)


def _gpt2_block(d: int, T: int) -> List[Layer]:
    # attention qkv (d -> 3d), attention output (d -> d), MLP up (d -> 4d),
    # MLP down (4d -> d)
    return [Layer("linear", T, d, 3 * d), Layer("linear", T, d, d),
            Layer("linear", T, d, 4 * d), Layer("linear", T, 4 * d, d)]


def conv_layer(cin: int, cout: int, k: int, stride: int, pad: int, hin: int) -> Layer:
    """A k x k convolution on an hin x hin input, as the linear layer of its unfolding."""
    ho = (hin + 2 * pad - k) // stride + 1
    d = (cin * k * k + 7) // 8 * 8
    return Layer("conv", ho * ho, d, cout, (cin, k, stride, pad, hin))


def _gpt2_full_block(d: int, T: int) -> List[Layer]:
    # every trainable tensor of a block: ln_1, attention qkv and output,
    # ln_2, MLP up and down, with the biases of the four linear maps
    return [Layer("norm", T, d, d, bias=True), Layer("linear", T, d, 3 * d, bias=True),
            Layer("linear", T, d, d, bias=True), Layer("norm", T, d, d, bias=True),
            Layer("linear", T, d, 4 * d, bias=True), Layer("linear", T, 4 * d, d, bias=True)]


def _lora(d: int, r: int, T: int, blocks: int) -> List[Layer]:
    # App. E.2: each LoRA module x(W + LR) trains two sub-modules, x -> xL
    # (d -> r) and xL -> xLR (r -> d); here on the query and value maps
    return [Layer("linear", T, d_in, d_out) for _ in range(blocks) for _ in ("q", "v")
            for d_in, d_out in ((d, r), (r, d))]


def _resnet18_224() -> List[Layer]:
    L = [conv_layer(3, 64, 7, 2, 3, 224)]
    L += [conv_layer(64, 64, 3, 1, 1, 56) for _ in range(4)]
    for cin, cout, h in ((64, 128, 56), (128, 256, 28), (256, 512, 14)):
        L.append(conv_layer(cin, cout, 3, 2, 1, h))
        L += [conv_layer(cout, cout, 3, 1, 1, h // 2) for _ in range(3)]
        L.append(conv_layer(cin, cout, 1, 2, 0, h))        # downsample
    L.append(Layer("linear", 1, 512, 1000))                # classifier
    return L


def _build() -> dict:
    w = {}
    w[1] = Workload(1, "single-linear-64x64-T16-B4-f32", 4, "f32",
                    (Layer("linear", 16, 64, 64),), "abadi", R=1.0, sigma=1.0,
                    description="single linear layer, fp32, a,g ~ N(0,1)")
    w[2] = Workload(2, "gpt2-small-stack-T128-B32-bf16", 32, "bf16",
                    tuple(l for _ in range(12) for l in _gpt2_block(768, 128)),
                    "auto", gamma=0.01, sigma=1.0, g_scale=1e-2,
                    description="12 GPT-2-small blocks (768->2304, 768->768, 768->3072, 3072->768)")
    w[3] = Workload(3, "long-seq-stack-T1024-B16-bf16", 16, "bf16",
                    tuple(l for _ in range(12) for l in (Layer("linear", 1024, 768, 768),
                                                          Layer("linear", 1024, 768, 3072),
                                                          Layer("linear", 1024, 3072, 768))),
                    "abadi", R=1.0, sigma=1.0, g_scale=1e-2,
                    description="12 x (768->768, 768->3072, 3072->768) at T=1024")
    w[4] = Workload(4, "vit-base-stack-T197-B64-bf16", 64, "bf16",
                    (Layer("linear", 196, 768, 768),) +
                    tuple(l for _ in range(12) for l in _gpt2_block(768, 197)),
                    "auto", gamma=0.01, sigma=1.0, g_scale=1e-2,
                    description="ViT-base: patch embedding (196 patches of 16x16x3) + 12 blocks at T=197")
    w[5] = Workload(5, "gpt2-large-stack-T256-B16-bf16+embed", 16, "bf16",
                    tuple(l for _ in range(36) for l in _gpt2_block(1280, 256)) +
                    (Layer("embed", 256, 50257, 1280),),
                    "abadi", R=1.0, sigma=0.8, g_scale=1e-2, zipf_s=1.1,
                    description="36 GPT-2-large blocks + 50257x1280 token embedding, Zipf(1.1) ids")
    w[6] = Workload(6, "resnet18-conv-stack-224-B16-bf16", 16, "bf16", tuple(_resnet18_224()),
                    "auto", gamma=0.01, sigma=1.0, g_scale=1e-2,
                    description="ResNet-18 at 224x224: 20 convolutions (unfolded) + classifier")
    w[7] = Workload(7, "gpt2-small-lora-r16-qv-T128-B32-bf16", 32, "bf16", tuple(_lora(768, 16, 128, 12)),
                    "auto", gamma=0.01, sigma=1.0, g_scale=1e-2,
                    description="LoRA rank 16 on the query and value projections of 12 GPT-2-small "
                                "blocks: 24 x (768 -> 16, 16 -> 768)")
    w[8] = Workload(8, "gpt2-small-full-T128-B32-bf16+bias+ln", 32, "bf16",
                    tuple(l for _ in range(12) for l in _gpt2_full_block(768, 128)) +
                    (Layer("norm", 128, 768, 768, bias=True),),
                    "auto", gamma=0.01, sigma=1.0, g_scale=1e-2,
                    description="12 GPT-2-small blocks with the biases of their 48 linear maps and "
                                "their 24 LayerNorm affines, plus the final LayerNorm")
    return w


WORKLOADS = _build()


def get(wid: int) -> Workload:
    return WORKLOADS[wid]


def workload_from_shapes(layers, B: int, dtype: str = "bf16", clip: str = "abadi", wid: int = 100,
                         **kw) -> Workload:
    """An ad-hoc workload (tests): layers as Layer objects or (T, d, p) tuples."""
    ls = tuple(l if isinstance(l, Layer) else Layer("linear", *l) for l in layers)
    return Workload(wid, f"adhoc-{wid}", B, dtype, ls, clip, **kw)


def _seed(wid: int, l: int, k: int) -> int:
    return 1000 * wid + 2 * l + k


def _randn(shape, seed: int, device) -> torch.Tensor:
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    return torch.randn(shape, generator=gen, dtype=torch.float32, device=device)


def draw_linear(wl: Workload, l: int, B: Optional[int] = None, device="cpu"):
    """(a [B,T,d], g [B,T,p]) of linear layer l in the workload dtype."""
    L = wl.layers[l]
    B = wl.B if B is None else B
    a = _randn((B, L.T, L.d), _seed(wl.wid, l, 0), device)
    g = _randn((B, L.T, L.p), _seed(wl.wid, l, 1), device)
    if wl.g_scale != 1.0:
        g.mul_(wl.g_scale)
    return a.to(wl.torch_dtype), g.to(wl.torch_dtype)


def zipf_ids(n: int, V: int, s: float, seed: int) -> np.ndarray:
    """n token ids in [0, V) with P(id = k-1) proportional to k^-s."""
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    w /= w.sum()
    rng = np.random.default_rng(seed)
    return rng.choice(V, size=n, p=w).astype(np.int64)


def draw_embedding(wl: Workload, l: int, B: Optional[int] = None, device="cpu"):
    """(ids [B,T] int64, g [B,T,p]) of embedding layer l."""
    L = wl.layers[l]
    B = wl.B if B is None else B
    ids = torch.from_numpy(zipf_ids(B * L.T, L.V, wl.zipf_s, 1000 * wl.wid + 999)).view(B, L.T)
    g = _randn((B, L.T, L.p), _seed(wl.wid, l, 1), device)
    if wl.g_scale != 1.0:
        g.mul_(wl.g_scale)
    return ids.to(device), g.to(wl.torch_dtype)


def draw_conv(wl: Workload, l: int, B: Optional[int] = None, device="cpu"):
    """(x [B, C_in, H, H], dL/ds [B, C_out, Ho, Ho]) of convolution layer l (NCHW)."""
    L = wl.layers[l]
    cin, k, stride, pad, hin = L.conv
    B = wl.B if B is None else B
    ho = (hin + 2 * pad - k) // stride + 1
    x = _randn((B, cin, hin, hin), _seed(wl.wid, l, 0), device)
    dy = _randn((B, L.p, ho, ho), _seed(wl.wid, l, 1), device)
    if wl.g_scale != 1.0:
        dy.mul_(wl.g_scale)
    return x.to(wl.torch_dtype), dy.to(wl.torch_dtype)


def draw_layer(wl: Workload, l: int, B: Optional[int] = None, device="cpu"):
    """(a or ids or xhat, g) of layer l; for a convolution the raw (x, dL/ds) in NCHW."""
    if wl.layers[l].kind == "embed":
        return draw_embedding(wl, l, B, device)
    if wl.layers[l].kind == "conv":
        return draw_conv(wl, l, B, device)
    return draw_linear(wl, l, B, device)


def make_stack(wl: Workload, B: Optional[int] = None, device="cpu"):
    """All layers' inputs, as a list of (x, g) with x = a or ids."""
    return [draw_layer(wl, l, B, device) for l in range(len(wl.layers))]
