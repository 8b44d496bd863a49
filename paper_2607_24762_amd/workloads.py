"""Seeded synthetic inputs shaped like the paper's workloads.

The paper measures its operators inside real models fed real data (Table I:
ResNet-50 on ImageNetV2, SD3.5 Medium on T2I-CompBench prompts, Gemma 4 E2B
and Qwen 3.5 35B-A3B on MT-Bench / ShareGPT / LongBench prompts).  None of
those checkpoints or datasets is used here: these generators stand in for
them with seeded tensors of the operator shapes and value distributions
listed below.

This module holds none of the operators' arithmetic.  It only draws random
numbers (numpy PCG64, one generator per workload, float64 draws in C order)
and casts them (float64 -> float32 by numpy, float32 -> bfloat16 / float16
by torch, round-to-nearest-even).  The oracle and the HIP path receive the
identical bits.
"""
from __future__ import annotations

import numpy as np
import torch

_TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


def cast(a64: np.ndarray, dtype: str) -> torch.Tensor:
    """float64 array -> CPU tensor of `dtype` ("f32", "bf16", "f16")."""
    t = torch.from_numpy(np.ascontiguousarray(a64, dtype=np.float64).astype(np.float32))
    return t if dtype == "f32" else t.to(_TORCH[dtype])


def randn(shape, dtype: str, seed: int, mean: float = 0.0, std: float = 1.0) -> torch.Tensor:
    """mean + std * N(0, 1), seeded, cast to dtype."""
    rng = np.random.default_rng(seed)
    return cast(mean + std * rng.standard_normal(tuple(shape)), dtype)


def randn_device(shape, dtype: str, seed: int, device="cuda", mean: float = 0.0, std: float = 1.0) -> torch.Tensor:
    """mean + std * N(0, 1) drawn on the device from a seeded torch generator
    (for tensors too large to draw on the host), cast to dtype."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    t = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if mean != 0.0 or std != 1.0:
        t.mul_(std).add_(mean)
    return t.to({"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype])


def sha256(t: torch.Tensor) -> str:
    """SHA-256 of a CPU tensor's bytes in C order (the exact input bits)."""
    import hashlib

    return hashlib.sha256(t.contiguous().view(torch.uint8).numpy().tobytes()).hexdigest()


def causal_mask_(s: torch.Tensor) -> torch.Tensor:
    """Set the strict upper triangle (key j > query i) of the last two dims
    to -inf, in place; the diagonal stays, so every row keeps an entry."""
    q, k = s.shape[-2], s.shape[-1]
    mask = torch.ones(q, k, dtype=torch.bool).triu_(1)
    s.masked_fill_(mask, float("-inf"))
    return s


# --- the six operator workloads -------------------------------------------

def softmax_square_f32(seed: int = 1) -> dict:
    """Row softmax, fp32 [1024, 1024], x = 2 z."""
    rng = np.random.default_rng(seed)
    x = cast(2.0 * rng.standard_normal((1024, 1024)), "f32")
    return {"op": "softmax", "x": x, "dim": -1, "out_dtype": "f32"}


def avgpool_resnet_head_f32(seed: int = 2) -> dict:
    """ResNet-50 head pooling: fp32 [32, 2048, 7, 7] NCHW, ReLU(z) (about
    half exact zeros), pooled to 1x1."""
    rng = np.random.default_rng(seed)
    x = cast(np.maximum(rng.standard_normal((32, 2048, 7, 7)), 0.0), "f32")
    return {"op": "adaptive_avgpool2d", "x": x, "output_size": (1, 1)}


def avgpool_general_f32(seed: int = 10, shape=(32, 512, 14, 14), output_size=(7, 7)) -> dict:
    """Adaptive average pooling to a general output size, fp32 NCHW,
    ReLU(z) like the head input: by default a VGG-style 7x7 head on a 14x14
    map (2x2 windows); (32, 256, 13, 13) -> (6, 6) gives overlapping 3x3
    windows (an AlexNet-style head)."""
    rng = np.random.default_rng(seed)
    x = cast(np.maximum(rng.standard_normal(shape), 0.0), "f32")
    return {"op": "adaptive_avgpool2d", "x": x, "output_size": tuple(output_size)}


def groupnorm_vae_bf16(seed: int = 3) -> dict:
    """SD3.5 VAE-style GroupNorm: bf16 [1, 512, 128, 128], 32 groups,
    eps 1e-6; x ~ N(0.3, 1.5^2), weight ~ N(1, 0.1^2), bias ~ N(0, 0.1^2),
    all bf16, drawn in that order from one generator."""
    rng = np.random.default_rng(seed)
    x = cast(0.3 + 1.5 * rng.standard_normal((1, 512, 128, 128)), "bf16")
    w = cast(1.0 + 0.1 * rng.standard_normal(512), "bf16")
    b = cast(0.1 * rng.standard_normal(512), "bf16")
    return {"op": "group_norm", "x": x, "num_groups": 32, "weight": w, "bias": b, "eps": 1e-6}


def attn_softmax_causal_bf16(seed: int = 4, heads: int = 8, seq: int = 4096) -> dict:
    """Eager-attention score softmax: bf16 [1, heads, seq, seq], scores
    (3 z) / 16 (N(0, 3^2) scaled by 1/sqrt(256)), strict upper triangle
    -inf (causal), softmax over the key axis, bf16 out."""
    rng = np.random.default_rng(seed)
    s = cast((3.0 * rng.standard_normal((1, heads, seq, seq))) / 16.0, "bf16")
    causal_mask_(s)
    return {"op": "softmax", "x": s, "dim": -1, "out_dtype": "bf16"}


def attn_scores_raw_bf16(seed: int = 4, heads: int = 8, seq: int = 4096) -> dict:
    """The same score draws as attn_softmax_causal_bf16 before scaling and
    masking: bf16 [1, heads, seq, seq] = bf16(3 z), for the fused scaled
    causal softmax with scale 1/16 (= 1/sqrt(256))."""
    rng = np.random.default_rng(seed)
    s = cast(3.0 * rng.standard_normal((1, heads, seq, seq)), "bf16")
    return {"op": "softmax_causal", "x": s, "scale": 1.0 / 16.0, "out_dtype": "bf16"}


def attn_decode_bf16(seed: int = 8, batch: int = 1, heads: int = 8, kv: int = 32768,
                     out_dtype: str = "f32") -> dict:
    """One greedy decode step of eager attention with a KV cache: the single
    new query of each head against kv cached keys, bf16 scores
    [batch, heads, 1, kv] = (3 z) / 16 as in the prefill workload (no mask:
    the newest query sees every cached key), softmax over the key axis with
    fp32 output (the dtype=float32 softmax eager attention calls before
    casting back to bf16)."""
    rng = np.random.default_rng(seed)
    s = cast((3.0 * rng.standard_normal((batch, heads, 1, kv))) / 16.0, "bf16")
    return {"op": "softmax_split", "x": s, "dim": -1, "out_dtype": out_dtype}


def maxpool_resnet_stem_f32(seed: int = 9, batch: int = 32) -> dict:
    """ResNet-50 stem pooling: fp32 [batch, 64, 112, 112] NCHW after the
    stem's BatchNorm + ReLU, so ReLU(z) (about half exact zeros); 3x3 max
    pooling, stride 2, padding 1 -> [batch, 64, 56, 56]."""
    rng = np.random.default_rng(seed)
    x = cast(np.maximum(rng.standard_normal((batch, 64, 112, 112)), 0.0), "f32")
    return {"op": "max_pool2d", "x": x, "kernel_size": 3, "stride": 2, "padding": 1}


def layernorm_sd35_bf16(seed: int = 7, tokens: int = 4096, hidden: int = 1536) -> dict:
    """SD3.5 Medium transformer LayerNorm: bf16 [2, tokens, hidden] (the two
    classifier-free-guidance branches of a 1024x1024 image: 4096 patch
    tokens of width 1536), x ~ N(0, 1), no affine (the adaptive-norm blocks
    apply their own modulation), eps 1e-6."""
    rng = np.random.default_rng(seed)
    x = cast(rng.standard_normal((2, tokens, hidden)), "bf16")
    return {"op": "layer_norm", "x": x, "normalized_shape": (hidden,), "weight": None, "bias": None, "eps": 1e-6}


def router_softmax_f32(seed: int = 5, experts: int = 256, tokens: int = 16384) -> dict:
    """MoE router logits: fp32 [tokens, experts], z ~ N(0, 1) plus +4 on an
    i.i.d. 5% of entries (u ~ U[0, 1) drawn after z, outlier where u < 0.05)."""
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((tokens, experts))
    u = rng.random((tokens, experts))
    outlier = u < 0.05
    x = cast(z + 4.0 * outlier, "f32")
    return {"op": "softmax", "x": x, "dim": -1, "out_dtype": "f32", "outliers": int(outlier.sum())}


WORKLOADS = {
    "softmax_f32_1024x1024": softmax_square_f32,
    "avgpool_f32_32x2048x7x7_to_1x1": avgpool_resnet_head_f32,
    "groupnorm_bf16_1x512x128x128_g32": groupnorm_vae_bf16,
    "attn_softmax_bf16_1x8x4096x4096_causal": attn_softmax_causal_bf16,
    "router_softmax_f32_16384x256": lambda: router_softmax_f32(5, 256),
    "router_softmax_f32_16384x257": lambda: router_softmax_f32(6, 257),
}
