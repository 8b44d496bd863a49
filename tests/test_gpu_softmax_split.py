"""GPU parity of kf_softmax_split (rows split over several workgroups that
exchange partial (max, sum) states) against the float64 oracle: the decode
attention workload at full size, row counts and lengths across the split
plans (ragged lengths whose rows start off a 16-byte boundary, the tensor's
last partial vector, parts that hold no element of the row), every dtype
pair, special rows, the views that are not split (in place, misaligned
base, many rows), determinism, workspace hygiene, concurrent streams and the
recompute fallback when a workgroup gives up waiting.  Tolerances as for
kf_softmax: fp32 outputs max abs error <= 1e-6; bf16 / fp16 outputs within
1 unit in the last place of the oracle rounded once to the format."""

import numpy as np
import pytest
import torch

from compare import assert_close, note
from exchange_child import spawn
from oracle import oracle
from paper_2607_24762_amd import kf355
from paper_2607_24762_amd import workloads as W
from paper_2607_24762_amd.workloads import randn

pytestmark = pytest.mark.gpu

PAIRS = [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32"), ("f16", "f16"), ("f16", "f32")]
TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    kf355.lib()


def run(x_cpu, out, **kw):
    x = x_cpu.cuda()
    y = kf355.kf_softmax_split(x, -1, out_dtype=TORCH[out])
    torch.cuda.synchronize()
    variant = kf355.last_variant()
    assert_close(y, oracle.softmax(x_cpu, -1), out, **kw)
    return y, variant


@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_decode_workload(out):
    w = W.attn_decode_bf16(out_dtype=out)
    note(f"softmax_split decode workload {tuple(w['x'].shape)} -> {out}")
    _, variant = run(w["x"], out)
    # fp32 output: 192 KiB per row, split; bf16 output: 128 KiB, one workgroup per row.
    assert variant.startswith("sm_split") == (out == "f32"), variant


SHAPES = [(1, 40000), (3, 40001), (8, 32768), (1, 16385), (16, 65539), (5, 12345), (127, 70000), (1, 1 << 20),
          (2, 300001), (100, 100000)]


def planned_split(shape, pair):
    import ctypes
    arr = (ctypes.c_int64 * len(shape))(*shape)
    n = ctypes.c_size_t(0)
    code = {"f32": 0, "bf16": 1, "f16": 2}
    assert kf355.lib().kf_softmax_split_workspace_bytes(code[pair[0]], code[pair[1]], len(shape), arr, -1,
                                                        ctypes.byref(n)) == 0
    return n.value > 0


@pytest.mark.parametrize("pair", PAIRS, ids=lambda p: f"{p[0]}-{p[1]}")
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_split_sweep(pair, shape):
    note(f"softmax_split sweep {pair} {shape}")
    x = randn(shape, pair[0], seed=shape[1] % 1000, std=3.0)
    _, variant = run(x, pair[1])
    planned = planned_split(shape, pair)
    print(f"[variant] {pair} {shape} planned={planned} {variant}")
    if planned and shape[0] <= 16:
        assert variant.startswith("sm_split"), variant     # a grid this small is always resident
    if not planned:
        assert not variant.startswith("sm_split"), variant


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
def test_special_rows(dt):
    length = 65536 + 5
    note(f"softmax_split special rows {dt} len={length}")
    x = randn((9, length), "f32", seed=5, std=2.0)
    x[0] = float("-inf")                      # fully masked -> NaN row
    x[1, length - 3] = float("nan")           # NaN in the last part -> NaN row
    x[2, 7] = float("inf")                    # +inf in the first part -> NaN row
    x[3] = float("-inf")
    x[3, 50000] = 0.5                         # one finite entry -> exact one-hot
    x[4, :20000] = float("-inf")              # whole parts of -inf -> exact +0 there
    x[5] *= 40.0                              # large logits
    x[6] = 1.25                               # uniform row
    x[7, ::3] = float("-inf")
    xt = x.to(TORCH[dt])
    y, variant = run(xt, dt)
    assert variant.startswith("sm_split"), variant
    yc = y.float().cpu()
    assert torch.isnan(yc[:3]).all()
    assert yc[3, 50000].item() == 1.0 and (yc[3, :50000] == 0).all() and (yc[3, 50001:] == 0).all()
    assert (yc[4, :20000] == 0).all() and not torch.signbit(yc[4]).any()
    assert (yc[7, ::3] == 0).all()


def test_uniform_power_of_two_rows_are_exact():
    note("softmax_split uniform rows")
    for dt in ("f32", "bf16"):
        x = torch.full((4, 65536), 0.75).to(TORCH[dt])
        y, variant = run(x, dt)
        assert variant.startswith("sm_split")
        assert (y.float().cpu() == 1.0 / 65536).all()


def test_views_that_are_not_split():
    note("softmax_split unsplit views")
    # In place: the recompute fallback could not re-read x, so the plain path runs.
    x_cpu = randn((4, 131072), "bf16", seed=21)
    x = x_cpu.cuda()
    kf355.kf_softmax_split(x, -1, out=x)
    torch.cuda.synchronize()
    assert not kf355.last_variant().startswith("sm_split")
    assert_close(x, oracle.softmax(x_cpu, -1), "bf16")
    # A base pointer off a 16-byte boundary.
    big = randn((4 * 131072 + 1,), "bf16", seed=22)
    xv = big.cuda()[1:].view(4, 131072)
    y = kf355.kf_softmax_split(xv, -1)
    torch.cuda.synchronize()
    assert not kf355.last_variant().startswith("sm_split")
    assert_close(y, oracle.softmax(big[1:].view(4, 131072), -1), "bf16")
    # Many rows, short rows, a non-last axis: no workspace is needed at all.
    for shape, dim in (((512, 4096), -1), ((64, 1024), -1), ((3, 9000, 4), 1)):
        xc = randn(shape, "f32", seed=23)
        assert kf355.softmax_split_workspace(xc.cuda(), dim).numel() >= 0
        y = kf355.kf_softmax_split(xc.cuda(), dim, workspace=torch.empty(0, dtype=torch.uint8, device="cuda"))
        torch.cuda.synchronize()
        assert not kf355.last_variant().startswith("sm_split")
        assert_close(y, oracle.softmax(xc, dim), "f32")


def test_repeat_calls_are_bitwise_identical_and_leave_the_workspace_zero():
    note("softmax_split determinism + workspace")
    x = W.attn_decode_bf16()["x"].cuda()
    ws = torch.zeros(1 << 16, dtype=torch.uint8, device="cuda")
    first = kf355.kf_softmax_split(x, -1, out_dtype=torch.float32, workspace=ws)
    outs = [kf355.kf_softmax_split(x, -1, out_dtype=torch.float32, workspace=ws) for _ in range(500)]
    torch.cuda.synchronize()
    assert kf355.last_variant().startswith("sm_split")
    for o in outs:
        assert torch.equal(o.view(torch.int32), first.view(torch.int32))
    assert ws.count_nonzero().item() == 0


def test_concurrent_calls_on_two_streams():
    note("softmax_split two streams")
    x = W.attn_decode_bf16(kv=65536)["x"].cuda()
    ref = kf355.kf_softmax_split(x, -1, out_dtype=torch.float32)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for _ in range(20):
        with torch.cuda.stream(s1):
            outs.append(kf355.kf_softmax_split(x, -1, out_dtype=torch.float32))
        with torch.cuda.stream(s2):
            outs.append(kf355.kf_softmax_split(x, -1, out_dtype=torch.float32))
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o.view(torch.int32), ref.view(torch.int32))


def test_gave_up_waiting_recomputes_bit_identically(tmp_path):
    note("softmax_split forced recompute (child process)")
    x = W.attn_decode_bf16()["x"].cuda()
    y = kf355.kf_softmax_split(x, -1, out_dtype=torch.float32)
    torch.cuda.synchronize()
    got = spawn(tmp_path, ["softmax_split"], KF355_SM_WAIT_TICKS="0")
    assert str(got["variant0"]).startswith("sm_split")
    assert int(got["give_ups"]) >= 1
    assert int(got["rest"]) == 0
    assert np.array_equal(got["bits0"], y.view(torch.int32).cpu().numpy())
