"""GPU parity of kf_softmax_causal (scale + causal mask + softmax in one
pass) against the float64 oracle: the attention workload shape, query /
key lengths that differ (mask aligned to the end of the key axis), every
dtype pair, row lengths across the kernel table, rows that are not whole
vectors, misaligned bases, garbage in
the masked triangle, rows with no visible key, and in-place use.
Tolerances as for kf_softmax: fp32 max abs error <= 1e-6, bf16 / fp16
within 1 unit in the last place of the oracle rounded once."""
import numpy as np
import pytest
import torch

from compare import assert_close, compare, gpu_bits, note, ordered
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


def run(x_cpu, scale, out):
    y = kf355.kf_softmax_causal(x_cpu.cuda(), scale, out_dtype=TORCH[out])
    torch.cuda.synchronize()
    variant = kf355.last_variant()
    assert_close(y, oracle.softmax_causal(x_cpu, scale), out)
    return y, variant


def test_attention_workload_matches_oracle_and_unfused_path():
    note("softmax_causal attention workload [1,8,4096,4096] bf16, scale 1/16")
    w = W.attn_scores_raw_bf16()
    x = w["x"].cuda()
    y = kf355.kf_softmax_causal(x, w["scale"])
    torch.cuda.synchronize()
    assert kf355.last_variant() == "sm_causal_vec_nt128_nv4"
    r = compare(y.cpu(), oracle.softmax_causal(w["x"], w["scale"]), "bf16")
    print("[parity] softmax_causal attention:", r, flush=True)
    assert r["ok"], r
    # Scaling by 1/16 is exact, so the fused result agrees with the unfused
    # softmax of the pre-scaled, pre-masked scores to within the rounding of
    # their fp32 sums, which the two kernels accumulate in different orders
    # (128 threads x 4 vectors per row against 256 x 2): at most 1 bf16 ulp,
    # and the masked entries are +0 in both.
    ref = kf355.kf_softmax(W.attn_softmax_causal_bf16()["x"].cuda(), -1)
    torch.cuda.synchronize()
    a, b = ordered(gpu_bits(y)), ordered(gpu_bits(ref))
    assert int(np.abs(a - b).max()) <= 1
    assert np.array_equal(a == 0, b == 0)


@pytest.mark.parametrize("pair", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32"), ("f16", "f16"), ("f16", "f32")],
                         ids=lambda p: f"{p[0]}-{p[1]}")
@pytest.mark.parametrize("qk", [(1, 1), (4, 4), (7, 7), (16, 64), (64, 64), (33, 257), (128, 1024), (5, 2048),
                                (300, 4096), (64, 8192), (2, 16384), (1, 65536)])
def test_lengths_and_dtypes(pair, qk):
    q, k = qk
    note(f"softmax_causal {pair} q={q} k={k}")
    x = randn((2, q, k), pair[0], seed=q + k, std=3.0)
    _, variant = run(x, 0.125, pair[1])
    # fp32 rows above 32768 keys leave the register-resident table for the
    # two-pass stream.
    expect = "sm_causal_stream_vec" if pair[0] == "f32" and k > 32768 else "sm_causal_"
    assert variant.startswith(expect), variant


@pytest.mark.parametrize("scale", [1.0, 0.0625, 0.37, -0.5])
def test_scales(scale):
    note(f"softmax_causal scale {scale}")
    run(randn((3, 40, 40), "f32", seed=3, std=2.0), scale, "f32")


def test_unaligned_rows_use_element_access():
    note("softmax_causal unaligned")
    q, k = 9, 257
    big = randn((2 * q * k + 1,), "bf16", seed=5, std=2.0)
    x_cpu = big[1:].view(2, q, k)
    y = kf355.kf_softmax_causal(big.cuda()[1:].view(2, q, k), 0.5)
    torch.cuda.synchronize()
    assert "scalar" in kf355.last_variant()
    assert_close(y, oracle.softmax_causal(x_cpu, 0.5), "bf16")


PAIRS = [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32"), ("f16", "f16"), ("f16", "f32")]


@pytest.mark.parametrize("pair", PAIRS, ids=lambda p: f"{p[0]}-{p[1]}")
@pytest.mark.parametrize("qk", [(3, 9), (9, 9), (33, 257), (40, 1001), (8, 2001), (12, 4097), (3, 12001),
                                (2, 30001), (1, 40001)])
def test_rows_that_are_not_whole_vectors(pair, qk):
    """Aligned bases, k not a multiple of the 16-byte vector: masked vectors
    covering each row (q < k puts the visible boundary mid-row; two batches
    so rows share end vectors across the batch boundary too)."""
    q, k = qk
    note(f"softmax_causal masked-vector rows {pair} q={q} k={k}")
    x = randn((2, q, k), pair[0], seed=q * k, std=3.0)
    _, variant = run(x, 0.37, pair[1])
    # fp32 rows above 36864 keys leave the masked-vector table for the
    # two-pass stream over the same masked vectors.
    expect = "sm_causal_stream_edge" if pair[0] == "f32" and k > 36864 else "sm_causal_edge"
    assert variant.startswith(expect), variant


def test_rows_that_are_not_whole_vectors_ignore_the_masked_triangle_in_place():
    note("softmax_causal masked-vector rows: NaN in the masked triangle, in place")
    q = k = 515
    x = randn((2, q, k), "bf16", seed=18, std=2.0)
    poisoned = x.clone()
    poisoned[:, torch.ones(q, k, dtype=torch.bool).triu(1)] = float("nan")
    a = kf355.kf_softmax_causal(x.cuda(), 0.25)
    pd = poisoned.cuda()
    b = kf355.kf_softmax_causal(pd, 0.25, out=pd)
    torch.cuda.synchronize()
    assert kf355.last_variant().startswith("sm_causal_edge")
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert_close(b, oracle.softmax_causal(x, 0.25), "bf16")


@pytest.mark.parametrize("dt,qk,variant", [
    ("bf16", (3, 40961), "sm_causal_stream_edge"),     # just past the masked-vector table
    ("f32", (3, 36865), "sm_causal_stream_edge"),
    ("f16", (3, 131071), "sm_causal_stream_edge"),     # four or five STEP-sized passes
    ("bf16", (5, 65543), "sm_causal_stream_edge"),     # two whole passes and a few keys
    ("f32", (4, 100003), "sm_causal_stream_edge"),
    ("bf16", (2, 65544), "sm_causal_stream_vec"),      # whole vectors past the resident table
    ("f16", (3, 131072), "sm_causal_stream_vec"),
    ("f32", (5, 100000), "sm_causal_stream_vec"),      # several STEP-sized passes, ragged last one
    ("f32", (4, 3), "sm_causal_scalar_nt64_nv1"),      # (a resident case beside them)
])
def test_rows_beyond_the_tables_stream(dt, qk, variant):
    """Rows too long for the register-resident and masked-vector kernels are
    read twice by sm_causal_stream: against the oracle, with q > 1 so the
    visible prefix ends mid-row and the masked tail is never read."""
    q, k = qk
    note(f"softmax_causal stream {dt} q={q} k={k}")
    x = randn((2, q, k), dt, seed=k % 1009, std=3.0)
    _, got = run(x, 0.37, dt)
    assert got == variant, got


@pytest.mark.parametrize("pair", PAIRS, ids=lambda p: f"{p[0]}-{p[1]}")
def test_masked_vector_stream_every_dtype_pair(pair):
    """The masked-vector stream for every dtype pair: two batches of rows
    that are not whole vectors, so rows share end vectors across the batch
    boundary and the tensor's last vector is partial (read element by
    element)."""
    q, k = 3, 40961
    note(f"softmax_causal masked-vector stream {pair} q={q} k={k}")
    x = randn((2, q, k), pair[0], seed=77, std=3.0)
    _, variant = run(x, 0.37, pair[1])
    assert variant == "sm_causal_stream_edge", variant


def test_masked_vector_stream_in_place_ignores_the_masked_triangle():
    note("softmax_causal masked-vector stream: NaN in the masked triangle, in place, aligned base")
    q, k = 4, 40963
    x = randn((2, q, k), "bf16", seed=23, std=2.0)
    poisoned = x.clone()
    poisoned[:, torch.ones(q, k, dtype=torch.bool).triu(k - q + 1)] = float("nan")
    a = kf355.kf_softmax_causal(x.cuda(), 0.25)
    assert kf355.last_variant() == "sm_causal_stream_edge"
    pd = poisoned.cuda()
    b = kf355.kf_softmax_causal(pd, 0.25, out=pd)
    torch.cuda.synchronize()
    assert kf355.last_variant() == "sm_causal_stream_edge"
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert_close(b, oracle.softmax_causal(x, 0.25), "bf16")
    masked = b.cpu()[:, torch.ones(q, k, dtype=torch.bool).triu(k - q + 1)]
    assert (masked.view(torch.int16) == 0).all()   # exact +0


def test_stream_in_place_ignores_the_masked_triangle():
    note("softmax_causal stream: NaN in the masked triangle, in place, unaligned base")
    q, k = 3, 40001
    big = randn((q * k + 1,), "bf16", seed=21, std=2.0)
    x = big[1:].view(1, q, k)
    poisoned = big.clone()
    poisoned[1:].view(1, q, k)[0, torch.ones(q, k, dtype=torch.bool).triu(k - q + 1)] = float("nan")
    a = kf355.kf_softmax_causal(big.cuda()[1:].view(1, q, k), 0.25)
    assert kf355.last_variant() == "sm_causal_stream_scalar"
    pd = poisoned.cuda()[1:].view(1, q, k)            # 2 bytes past an aligned base
    b = kf355.kf_softmax_causal(pd, 0.25, out=pd)
    torch.cuda.synchronize()
    assert kf355.last_variant() == "sm_causal_stream_scalar"
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert_close(b, oracle.softmax_causal(x, 0.25), "bf16")


def test_masked_triangle_is_never_used():
    note("softmax_causal NaN in the masked triangle")
    q = k = 512
    x = randn((2, q, k), "bf16", seed=8, std=2.0)
    poisoned = x.clone()
    poisoned[:, torch.ones(q, k, dtype=torch.bool).triu(1)] = float("nan")
    a = kf355.kf_softmax_causal(x.cuda(), 0.25)
    b = kf355.kf_softmax_causal(poisoned.cuda(), 0.25)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    masked = b.cpu()[:, torch.ones(q, k, dtype=torch.bool).triu(1)]
    assert (masked.view(torch.int16) == 0).all()   # exact +0


def test_rows_without_visible_keys_are_nan():
    note("softmax_causal q > k")
    x = randn((1, 6, 4), "f32", seed=1)
    y, _ = run(x, 1.0, "f32")
    yc = y.cpu()
    assert torch.isnan(yc[0, :2]).all() and torch.isfinite(yc[0, 2:]).all()


def test_in_place():
    note("softmax_causal in place")
    x_cpu = randn((2, 64, 1000), "bf16", seed=9)
    x = x_cpu.cuda()
    kf355.kf_softmax_causal(x, 0.3, out=x)
    torch.cuda.synchronize()
    assert_close(x, oracle.softmax_causal(x_cpu, 0.3), "bf16")
