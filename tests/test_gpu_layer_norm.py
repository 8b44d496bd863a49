"""GPU parity of kf_layer_norm against the float64 oracle: the SD3.5
transformer shape, row widths across the lane-group, workgroup and
streaming kernels, every dtype and affine combination, several normalised
ranks, unaligned rows, in-place use and determinism.  Tolerances as for
GroupNorm: bf16 / fp16 within 1 unit in the last place of the oracle rounded
once (plus |error| <= 2^-22 where |oracle| < 2^-19: fp32 statistics cannot
resolve a bf16 ulp that small); fp32 outputs max abs error <= 1e-6."""
import pytest
import torch

from compare import assert_close, compare, note
from oracle import oracle
from paper_2607_24762_amd import kf355
from paper_2607_24762_amd import workloads as W
from paper_2607_24762_amd.workloads import randn

pytestmark = pytest.mark.gpu
FLOOR = (2.0 ** -19, 2.0 ** -22)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    kf355.lib()


def check(y, ref, dt):
    if dt == "f32":
        r = assert_close(y, ref, "f32")
        print(f"[parity] fp32 layer_norm max_abs {r['max_abs']:.3e}", flush=True)
        return
    assert_close(y, ref, dt, floor=FLOOR)


def run(shape, nd, dt, affine="same", eps=1e-6, seed=0, in_place=False):
    ns = shape[len(shape) - nd:]
    x_cpu = randn(shape, dt, seed=seed, mean=0.3, std=1.5)
    adt = dt if affine == "same" else "f32"
    w_cpu = randn(ns, adt, seed=seed + 1, mean=1.0, std=0.1) if affine in ("same", "f32", "w") else None
    b_cpu = randn(ns, adt, seed=seed + 2, std=0.1) if affine in ("same", "f32", "b") else None
    x = x_cpu.cuda()
    y = kf355.kf_layer_norm(x, ns, w_cpu.cuda() if w_cpu is not None else None,
                            b_cpu.cuda() if b_cpu is not None else None, eps, out=x if in_place else None)
    torch.cuda.synchronize()
    variant = kf355.last_variant()
    check(y, oracle.layer_norm(x_cpu, nd, w_cpu, b_cpu, eps), dt)
    return y, variant


def test_sd35_transformer_workload():
    note("layer_norm [2,4096,1536] bf16")
    w = W.layernorm_sd35_bf16()
    y = kf355.kf_layer_norm(w["x"].cuda(), w["normalized_shape"], None, None, w["eps"])
    torch.cuda.synchronize()
    r = compare(y, oracle.layer_norm(w["x"], 1, None, None, w["eps"]), "bf16", floor=FLOOR)
    print("[parity] layer_norm sd35:", r, kf355.last_variant(), flush=True)
    assert r["ok"], r


WIDTHS = [1, 7, 8, 64, 256, 320, 768, 1024, 1536, 2048, 3072, 4096, 5120, 8192, 16384, 65536, 100000]


@pytest.mark.parametrize("dt", ["bf16", "f32", "f16"])
@pytest.mark.parametrize("d", WIDTHS)
def test_widths(d, dt):
    rows = 37 if d <= 8192 else 3
    note(f"layer_norm rows={rows} d={d} {dt}")
    _, variant = run((rows, d), 1, dt, seed=d)
    assert variant.startswith("ln_"), variant


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("d", [8, 256, 1000, 1024, 1536, 1544, 2048, 4096, 16384, 65536])
def test_widths_without_affine(d, dt):
    # No weight and no bias select the kernels that hold no affine registers
    # (and, for rows of 129-192 slots, two rows per wave).
    rows = 37 if d <= 8192 else 3
    note(f"layer_norm no affine rows={rows} d={d} {dt}")
    _, variant = run((rows, d), 1, dt, affine="none", seed=d + 1)
    assert variant.startswith("ln_"), variant
    if d == 1536 and dt == "bf16":
        assert variant == "ln_wave_vec_lpr32_nv6", variant


@pytest.mark.parametrize("affine", ["f32", "w", "b", "none"])
def test_affine_variants(affine):
    note(f"layer_norm affine={affine}")
    run((64, 1536), 1, "bf16", affine=affine, seed=3)


@pytest.mark.parametrize("shape,nd", [((2, 4, 6, 8), 2), ((3, 2, 5, 5), 3), ((2, 77, 768), 1), ((5,), 1)])
def test_normalised_ranks(shape, nd):
    note(f"layer_norm {shape} nd={nd}")
    run(shape, nd, "bf16", seed=4)


def test_unaligned_rows():
    note("layer_norm unaligned")
    rows, d = 21, 1536
    big = randn((rows * d + 1,), "bf16", seed=6, mean=0.3, std=1.5)
    x_cpu = big[1:].view(rows, d)
    y = kf355.kf_layer_norm(big.cuda()[1:].view(rows, d), d, None, None, 1e-6)
    torch.cuda.synchronize()
    assert "scalar" in kf355.last_variant()
    check(y, oracle.layer_norm(x_cpu, 1, None, None, 1e-6), "bf16")


def test_in_place_and_determinism():
    note("layer_norm in place / repeat")
    run((128, 1536), 1, "bf16", in_place=True, seed=9)
    x = randn((512, 1536), "bf16", seed=10).cuda()
    a = kf355.kf_layer_norm(x, 1536)
    b = kf355.kf_layer_norm(x, 1536)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
