"""GPU parity of kf_max_pool2d against the float64 oracle: bit-exact
values and indices (max pooling selects an input element, so there is no
rounding and the tolerance is zero), for the ResNet-50 stem at full size in
NCHW and channels last, a sweep of window shapes, strides, paddings,
dilations and ceil mode over every kernel variant (the register tiles of 3x3
stride-2 windows, masked and exact, LDS bands with vector and element
staging, the direct fallback for wide planes, channels last with vector and
element channel access), every dtype, special values (NaN, -inf, ties), 3-D
inputs and empty batches.  Every case runs twice: with indices
(the kernels that track the winning position) and without (the value-only
kernels, which keep a running max and a NaN flag); the values must agree
with the oracle either way, with NaN at the same places and signed zeros
compared by value, since a value-only call may return +0 for a window whose
first maximum is -0."""
import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from compare import note
from oracle import oracle
from paper_2607_24762_amd import kf355
from paper_2607_24762_amd import workloads as W
from paper_2607_24762_amd.workloads import randn

pytestmark = pytest.mark.gpu
TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    kf355.lib()


def same_values(y, ref, variant):
    got = y.float().cpu().numpy().astype(np.float64)
    nan_r, nan_g = np.isnan(ref), np.isnan(got)
    assert np.array_equal(nan_r, nan_g), variant
    assert np.array_equal(got[~nan_g], ref[~nan_r]), (variant, float(np.abs(got[~nan_g] - ref[~nan_r]).max()))


def check(x_cpu, x_gpu, k, s, p, d, ceil):
    y, idx = kf355.kf_max_pool2d(x_gpu, k, s, p, d, ceil, return_indices=True)
    torch.cuda.synchronize()
    variant = kf355.last_variant()
    y_only = kf355.kf_max_pool2d(x_gpu, k, s, p, d, ceil)
    torch.cuda.synchronize()
    variant_only = kf355.last_variant()
    ref, ref_idx = oracle.max_pool2d(x_cpu, k, s, p, d, ceil)
    same_values(y, ref, variant)
    same_values(y_only, ref, variant_only)
    assert np.array_equal(idx.cpu().numpy(), ref_idx), variant
    assert (variant == variant_only == "mp_direct" or variant == variant_only + "_idx" or
            (variant == "mp_tile_idx" and variant_only == "mp_tile_exact")), (variant, variant_only)
    assert y.is_contiguous(memory_format=torch.channels_last) == x_gpu.is_contiguous(
        memory_format=torch.channels_last) or x_gpu.is_contiguous()
    return y, idx, variant


@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
def test_resnet_stem(layout):
    w = W.maxpool_resnet_stem_f32()
    note(f"max_pool2d resnet stem {layout}")
    x = w["x"].cuda()
    if layout == "nhwc":
        x = x.contiguous(memory_format=torch.channels_last)
    y, idx, variant = check(w["x"], x, 3, 2, 1, 1, False)
    assert variant == ("mp_tile_idx" if layout == "nchw" else "mp_nhwc_vec_k3_idx"), variant
    kf355.kf_max_pool2d(x, 3, 2, 1)
    assert kf355.last_variant() == ("mp_tile_exact" if layout == "nchw" else "mp_nhwc_vec_k3")
    # Informational second reference: torch eager on the same GPU agrees bit for bit.
    ty, ti = F.max_pool2d(x, 3, 2, 1, return_indices=True)
    assert torch.equal(ty, y) and torch.equal(ti, idx)


WINDOWS = [(k, s, p, d, c) for k in (1, 2, 3, 5) for s in (1, 2, 3) for p in sorted({0, k // 2}) for d in (1, 2)
           for c in (False, True)]


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("hw", [(16, 16), (13, 21), (7, 8), (33, 40)])
def test_window_sweep_nchw(dt, hw):
    x_cpu = randn((2, 3) + hw, dt, seed=hw[0] * 100 + hw[1], std=2.0)
    x = x_cpu.cuda()
    seen = set()
    for k, s, p, d, c in WINDOWS:
        if oracle.pool_out_size(hw[0], k, s, p, d, c) < 1 or oracle.pool_out_size(hw[1], k, s, p, d, c) < 1:
            continue
        note(f"max_pool2d nchw {dt} {hw} k={k} s={s} p={p} d={d} ceil={c}")
        variant = check(x_cpu, x, k, s, p, d, c)[2]
        seen.add(variant)
        tile = k == 3 and s == 2 and d == 1 and hw[1] % (16 // x_cpu.element_size()) == 0
        assert variant == "mp_tile_idx" if tile else variant.startswith("mp_band_"), (k, s, p, d, c, variant)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("c", [64, 24, 5])
def test_window_sweep_nhwc(dt, c):
    x_cpu = randn((2, c, 13, 18), dt, seed=c, std=2.0)
    x = x_cpu.cuda().contiguous(memory_format=torch.channels_last)
    for k, s, p, d, cm in WINDOWS[::3]:
        if oracle.pool_out_size(13, k, s, p, d, cm) < 1 or oracle.pool_out_size(18, k, s, p, d, cm) < 1:
            continue
        note(f"max_pool2d nhwc {dt} c={c} k={k} s={s} p={p} d={d} ceil={cm}")
        _, _, variant = check(x_cpu, x, k, s, p, d, cm)
        vec = 4 if dt == "f32" else 8
        assert variant.startswith("mp_nhwc_vec" if c % vec == 0 else "mp_nhwc_scalar"), variant


def test_wide_planes_take_the_direct_kernel():
    note("max_pool2d direct")
    x_cpu = randn((2, 5, 9001), "f32", seed=4)          # [C, H, W]: a 36 KB row exceeds the band tile
    _, _, variant = check(x_cpu, x_cpu.cuda(), (3, 3), (2, 2), (1, 1), 1, True)
    assert variant == "mp_direct"


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
def test_special_values(dt, layout):
    note(f"max_pool2d special values {dt} {layout}")
    x = randn((2, 8, 12, 12), "f32", seed=8)
    x[0, 0] = float("-inf")                             # all -inf planes
    x[0, 1, 3, 4] = float("nan")
    x[0, 1, 5, 5] = float("nan")                        # two NaN in overlapping windows
    x[0, 2] = 0.5                                       # ties everywhere: first position wins
    x[1, 3, ::2, ::2] = float("inf")
    x[1, 4] = -1.0                                      # padding must not win over negatives
    xt = x.to(TORCH[dt])
    xg = xt.cuda()
    if layout == "nhwc":
        xg = xg.contiguous(memory_format=torch.channels_last)
    check(xt, xg, 3, 2, 1, 1, False)     # register tile (fp32: 12 is whole vectors), else strip scan
    check(xt, xg, 3, 1, 1, 1, False)     # strip scan, stride 1
    check(xt, xg, 2, 2, 0, 1, True)      # 2x2 strip scan
    check(xt, xg, 2, 1, 1, 2, True)      # generic scan (dilation)


def test_three_d_input_and_empty_batch():
    note("max_pool2d 3-D and empty")
    x_cpu = randn((6, 17, 19), "bf16", seed=12)
    check(x_cpu, x_cpu.cuda(), 3, 2, 1, 1, True)
    e = torch.empty(0, 3, 8, 8, device="cuda")
    y = kf355.kf_max_pool2d(e, 2)
    torch.cuda.synchronize()
    assert y.shape == (0, 3, 4, 4)


def test_without_indices_matches_with():
    note("max_pool2d no indices")
    x = randn((4, 16, 30, 30), "f32", seed=13).cuda()
    a = kf355.kf_max_pool2d(x, 3, 2, 1)
    b, _ = kf355.kf_max_pool2d(x, 3, 2, 1, return_indices=True)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("hw", [6, 8])
@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
def test_signed_zero_and_nan_without_indices(layout, hw):
    """Value-only windows: -0 and +0 compare equal, so a window of zeros gives
    a zero (either sign); a window holding NaN gives NaN whatever its
    position among the other elements.  An 8-wide fp32 NCHW plane takes the
    exact register tile (maximum3 folds), a 6-wide one the LDS band."""
    note(f"max_pool2d value-only zeros/NaN {layout} {hw}x{hw}")
    x = torch.full((1, 4, hw, hw), -1.0)
    x[0, 0] = -0.0
    x[0, 1, ::2] = -0.0
    x[0, 1, 1::2] = 0.0
    x[0, 2, 0, 0] = float("nan")
    x[0, 3, 5, 5] = float("nan")
    xg = x.cuda()
    if layout == "nhwc":
        xg = xg.contiguous(memory_format=torch.channels_last)
    y = kf355.kf_max_pool2d(xg, 3, 2, 1)
    torch.cuda.synchronize()
    if layout == "nchw":
        assert kf355.last_variant() == ("mp_tile_exact" if hw == 8 else "mp_band_scalar_k3_strip_s2"), kf355.last_variant()
    ref, _ = oracle.max_pool2d(x.numpy().astype(np.float64), 3, 2, 1)
    same_values(y, ref, kf355.last_variant())
    assert torch.all(y[0, :2] == 0) and torch.isnan(y[0, 2, 0, 0]) and torch.isnan(y[0, 3, 2, 2])


TILE_CASES = [
    # (shape, padding, ceil): exact and masked value-only folds, both paddings, odd output heights (a
    # thread's second row masked), output widths that are not whole vectors (element stores), a plane
    # wider than any band tile, and 1-row planes.
    ((2, 3, 112, 112), 1, False),
    ((2, 3, 112, 112), 0, False),
    ((2, 3, 112, 112), 0, True),
    ((1, 4, 15, 24), 1, False),
    ((1, 4, 15, 24), 0, True),
    ((3, 2, 9, 8), 1, True),
    ((1, 2, 6, 9000), 1, False),
    ((2, 2, 1, 16), 1, False),
    ((2, 2, 2, 32), 0, True),
]


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape,p,ceil", TILE_CASES)
def test_register_tiles(dt, shape, p, ceil):
    note(f"max_pool2d tile {dt} {shape} p={p} ceil={ceil}")
    x_cpu = randn(shape, dt, seed=shape[2] * 7 + shape[3] + p, std=2.0)
    x = x_cpu.cuda()
    e = 16 // x_cpu.element_size()
    _, _, variant = check(x_cpu, x, 3, 2, p, 1, ceil)
    assert variant == ("mp_tile_idx" if shape[3] % e == 0 else variant), variant
    if shape[3] % e == 0:
        kf355.kf_max_pool2d(x, 3, 2, p, 1, ceil)
        ow = oracle.pool_out_size(shape[3], 3, 2, p, 1, ceil)
        exact = 2 * e * -(-ow // e) <= shape[3]
        assert kf355.last_variant() == ("mp_tile_exact" if exact else "mp_tile")
