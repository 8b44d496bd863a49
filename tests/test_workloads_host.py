"""The seeded input generators: the structure each workload recipe promises
(shapes, dtypes, masks, outlier rate, ReLU zeros), and that a seed always
gives the same bits.  CPU only."""
import math

import numpy as np
import torch

from paper_2607_24762_amd import workloads as W


def test_same_seed_same_bits():
    a, b = W.router_softmax_f32(5, 64, 256), W.router_softmax_f32(5, 64, 256)
    assert W.sha256(a["x"]) == W.sha256(b["x"])
    assert W.sha256(W.router_softmax_f32(6, 64, 256)["x"]) != W.sha256(a["x"])


def test_router_outliers_are_a_plus_four_shift_at_five_percent():
    for seed, experts in ((5, 256), (6, 257)):
        w = W.WORKLOADS[f"router_softmax_f32_16384x{experts}"]()
        x = w["x"]
        assert x.shape == (16384, experts) and x.dtype == torch.float32
        n = x.numel()
        # Binomial(n, 0.05): the realised count lies within 5 standard deviations.
        sd = math.sqrt(n * 0.05 * 0.95)
        assert abs(w["outliers"] - 0.05 * n) < 5 * sd, w["outliers"]
        # Redraw the recipe: selected entries are z + 4, the rest z.
        rng = np.random.default_rng(seed)
        z = rng.standard_normal((16384, experts))
        u = rng.random((16384, experts))
        sel = u < 0.05
        assert int(sel.sum()) == w["outliers"]
        xd = x.double().numpy()
        assert np.array_equal(xd[sel], (z[sel] + 4.0).astype(np.float32).astype(np.float64))
        assert np.array_equal(xd[~sel], z[~sel].astype(np.float32).astype(np.float64))


def test_causal_scores_mask_the_strict_upper_triangle():
    w = W.attn_softmax_causal_bf16(heads=2, seq=64)
    s = w["x"]
    assert s.dtype == torch.bfloat16 and s.shape == (1, 2, 64, 64)
    upper = torch.ones(64, 64, dtype=torch.bool).triu_(1)
    assert torch.isneginf(s[..., upper].float()).all()
    assert torch.isfinite(s[..., ~upper].float()).all()


def test_relu_inputs_are_half_exact_zeros():
    x = W.avgpool_resnet_head_f32()["x"]
    assert x.shape == (32, 2048, 7, 7) and (x >= 0).all()
    frac = (x == 0).double().mean().item()
    assert abs(frac - 0.5) < 0.002, frac
    # ReLU writes +0.0, never -0.0.
    assert not torch.signbit(x[x == 0]).any()


def test_group_norm_workload_recipe():
    w = W.groupnorm_vae_bf16()
    x, wt, b = w["x"].double(), w["weight"].double(), w["bias"].double()
    assert w["x"].dtype == torch.bfloat16 and w["x"].shape == (1, 512, 128, 128)
    assert w["num_groups"] == 32 and w["eps"] == 1e-6
    assert abs(x.mean().item() - 0.3) < 0.01 and abs(x.std().item() - 1.5) < 0.01
    assert abs(wt.mean().item() - 1.0) < 0.03 and abs(b.mean().item()) < 0.03
