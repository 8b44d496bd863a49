"""GPU parity beyond 2^31 elements: each operator on a tensor whose element
count, and so some element offsets, exceed the 32-bit range, checked against
the float64 oracle on sampled units (rows, groups, planes, samples) at the
start, on both sides of element 2^31 and at the end.  Inputs are drawn on the
device from a seeded generator (workloads.randn_device: 2^31 draws would not
fit a host-side float64 buffer comfortably); the sampled slices are copied to
the host for the oracle.  Tolerances as in the other parity tests: fp32 max
abs error <= 1e-6, bf16 within 1 unit in the last place, max_pool2d exact."""
import numpy as np
import pytest
import torch

from compare import compare, note
from oracle import oracle
from paper_2607_24762_amd import kf355
from paper_2607_24762_amd.workloads import randn_device

pytestmark = pytest.mark.gpu
BIG = 1 << 31


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    kf355.lib()
    yield
    torch.cuda.empty_cache()


@pytest.fixture(autouse=True)
def release():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def samples(units: int, per_unit: int) -> list:
    """Unit indices at the start, around the unit holding element 2^31, and at the end."""
    b = BIG // per_unit
    return sorted({0, 1, b - 1, b, min(b + 1, units - 1), units - 1})


def check(name, got, ref, fmt):
    r = compare(got, ref, fmt)
    print(f"[parity] {name}: {r}", flush=True)
    assert r["ok"], (name, r)


def test_softmax_rows():
    rows, length = BIG // 4096 + 3, 4096
    note(f"large softmax bf16 [{rows}, {length}]")
    x = randn_device((rows, length), "bf16", seed=31, std=2.0)
    y = kf355.kf_softmax(x, -1)
    torch.cuda.synchronize()
    for r in samples(rows, length):
        check(f"softmax row {r}", y[r], oracle.softmax(x[r].cpu(), -1), "bf16")


def test_causal_softmax_rows():
    heads, n = 33, 8192                          # 33 * 8192 * 8192 > 2^31
    note(f"large causal softmax bf16 [1, {heads}, {n}, {n}]")
    x = randn_device((1, heads, n, n), "bf16", seed=32, std=3.0)
    y = kf355.kf_softmax_causal(x, 1.0 / 16)
    torch.cuda.synchronize()
    flat_x, flat_y = x.view(-1, n), y.view(-1, n)
    for r in samples(heads * n, n):
        i = r % n
        # Query i of a square head sees keys 0..i: the oracle's causal softmax
        # of that prefix as a one-query row, then zeros.
        head = oracle.softmax_causal(flat_x[r, :i + 1].cpu()[None, :], 1.0 / 16)[0]
        ref = np.concatenate([head, np.zeros(n - i - 1)])
        check(f"causal row {r} (query {i})", flat_y[r], ref, "bf16")


def test_layer_norm_rows():
    rows, d = BIG // 1536 + 5, 1536
    note(f"large layer_norm bf16 [{rows}, {d}]")
    x = randn_device((rows, d), "bf16", seed=33)
    y = kf355.kf_layer_norm(x, (d,), eps=1e-6)
    torch.cuda.synchronize()
    for r in samples(rows, d):
        check(f"layer_norm row {r}", y[r], oracle.layer_norm(x[r].cpu()[None], 1, None, None, 1e-6)[0], "bf16")


def test_group_norm_groups():
    n, c, h, w, g = 2, 512, 1536, 1536, 32      # 2.4e9 elements; every group spans 2304 chunks
    note(f"large group_norm bf16 [{n}, {c}, {h}, {w}] G={g}")
    x = randn_device((n, c, h, w), "bf16", seed=34, mean=0.3, std=1.5)
    wt = randn_device((c,), "bf16", seed=35, mean=1.0, std=0.1)
    bs = randn_device((c,), "bf16", seed=36, std=0.1)
    y = kf355.kf_group_norm(x, g, wt, bs, 1e-6)
    torch.cuda.synchronize()
    cpg = c // g
    for s, gi in ((0, 0), (0, g - 1), (1, 0), (1, g - 1)):
        sl = slice(gi * cpg, (gi + 1) * cpg)
        ref = oracle.group_norm(x[s:s + 1, sl].cpu(), 1, wt[sl].cpu(), bs[sl].cpu(), 1e-6)
        r = compare(y[s:s + 1, sl], ref, "bf16", floor=(2.0 ** -19, 2.0 ** -22))
        print(f"[parity] group_norm sample {s} group {gi}: {r}", flush=True)
        assert r["ok"], r


def test_adaptive_avgpool_planes():
    n, c = 21400, 2048                            # 21400 * 2048 * 49 > 2^31
    note(f"large adaptive_avgpool2d fp32 [{n}, {c}, 7, 7]")
    x = torch.relu(randn_device((n, c, 7, 7), "f32", seed=37))
    y = kf355.kf_adaptive_avgpool2d(x, 1)
    torch.cuda.synchronize()
    xp, yp = x.view(-1, 7, 7), y.view(-1)
    for p in samples(n * c, 49):
        check(f"avgpool plane {p}", yp[p:p + 1], oracle.adaptive_avg_pool2d(xp[p:p + 1].cpu(), 1).reshape(-1),
              "f32")


@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
def test_max_pool_planes(layout):
    n, c = 2675, 64                               # 2675 * 64 * 112 * 112 > 2^31
    note(f"large max_pool2d fp32 [{n}, {c}, 112, 112] {layout}")
    x = torch.relu(randn_device((n, c, 112, 112), "f32", seed=38))
    if layout == "nhwc":
        x = x.contiguous(memory_format=torch.channels_last)
    y = kf355.kf_max_pool2d(x, 3, 2, 1)
    torch.cuda.synchronize()
    for s in sorted({0, BIG // (c * 112 * 112), n - 1}):
        ref, _ = oracle.max_pool2d(x[s].cpu(), 3, 2, 1)
        got = y[s].cpu().numpy().astype(np.float64)
        assert np.array_equal(got, ref), (layout, s, kf355.last_variant())
