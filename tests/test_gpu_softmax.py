"""GPU parity of kf_softmax against the float64 oracle: row-length sweep
across every kernel variant (one-row-per-lane-group, workgroup, streaming,
strided axis, staged spans and masked vectors for rows that are not whole
vectors), every dtype
pair, misaligned rows, special values and in-place use.  Tolerances: fp32 outputs max abs error <= 1e-6; bf16 / fp16 outputs
within 1 unit in the last place of the oracle rounded once to the format."""
import math

import numpy as np
import pytest
import torch

from compare import assert_close, note
from oracle import oracle
from paper_2607_24762_amd import kf355
from paper_2607_24762_amd.workloads import randn

pytestmark = pytest.mark.gpu

PAIRS = [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32"), ("f16", "f16"), ("f16", "f32")]
TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    kf355.lib()  # raises if the library is missing


def run_case(x_cpu, dim, out, **kw):
    x = x_cpu.cuda()
    y = kf355.kf_softmax(x, dim, out_dtype=TORCH[out])
    torch.cuda.synchronize()
    variant = kf355.last_variant()
    ref = oracle.softmax(x_cpu, dim)
    r = assert_close(y, ref, out, **kw)
    return y, variant, r


LENGTHS = [1, 2, 3, 7, 8, 63, 64, 65, 127, 255, 256, 257, 511, 1023, 1024, 1025, 2047, 2048, 4095, 4096,
           4097, 8192, 16384, 32768, 65537]


@pytest.mark.parametrize("pair", PAIRS, ids=lambda p: f"{p[0]}-{p[1]}")
@pytest.mark.parametrize("length", LENGTHS)
def test_row_length_sweep(pair, length):
    rows = 37 if length <= 8192 else 3
    note(f"softmax sweep {pair} rows={rows} len={length}")
    x = randn((rows, length), pair[0], seed=length, std=3.0)
    _, variant, _ = run_case(x, -1, pair[1])
    assert variant.startswith("sm_"), variant


@pytest.mark.parametrize("length", [256, 257, 1024, 4096])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_misaligned_base_pointer(length, dt):
    # A view starting one element into its buffer: rows are no longer
    # 16-byte aligned, so the scalar-access variants must take over.
    rows = 33
    note(f"softmax misaligned {dt} len={length}")
    big = randn((rows * length + 1,), dt, seed=11)
    x_cpu = big[1:].view(rows, length)
    x = big.cuda()[1:].view(rows, length)
    y = kf355.kf_softmax(x, -1)
    torch.cuda.synchronize()
    assert "scalar" in kf355.last_variant()
    assert_close(y, oracle.softmax(x_cpu, -1), dt)


@pytest.mark.parametrize("shape,dim", [((4, 37, 5), 1), ((3, 8, 16, 16), 1), ((6, 5), 0), ((2, 3, 300), 0),
                                       ((2, 2, 3, 4097), 2)])
@pytest.mark.parametrize("pair", [("f32", "f32"), ("bf16", "bf16")], ids=lambda p: p[0])
def test_non_last_dim(shape, dim, pair):
    note(f"softmax dim={dim} shape={shape} {pair}")
    x = randn(shape, pair[0], seed=3, std=2.0)
    _, variant, _ = run_case(x, dim, pair[1])
    assert variant == "sm_cols"


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("length", [5, 256, 257, 4096, 70000])
def test_special_rows(dt, length):
    note(f"softmax special rows {dt} len={length}")
    x = randn((8, length), "f32", seed=5, std=2.0)
    x[0] = float("-inf")                      # fully masked -> NaN row
    x[1, length // 2] = float("nan")          # NaN -> NaN row
    x[2, 0] = float("inf")                    # +inf -> NaN row
    x[3] = float("-inf")
    x[3, length - 1] = 0.5                    # one finite entry -> exact one-hot
    x[4, ::2] = float("-inf")                 # masked entries -> exact +0
    x[5] *= 40.0                              # large logits
    x[6] = 1.25                               # uniform row
    xt = x.to(TORCH[dt])
    y, _, _ = run_case(xt, -1, dt)
    yc = y.float().cpu()
    assert torch.isnan(yc[:3]).all()
    assert yc[3, length - 1].item() == 1.0 and (yc[3, :-1] == 0).all()
    assert not torch.signbit(yc[3]).any() and not torch.signbit(yc[4]).any()
    assert (yc[4, ::2] == 0).all()
    if length in (256, 4096):
        assert (yc[6] == 1.0 / length).all()  # a power-of-two uniform row is exact


@pytest.mark.parametrize("length", [1000, 257])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_in_place(dt, length):
    note(f"softmax in place {dt} len={length}")
    x_cpu = randn((64, length), dt, seed=9)
    x = x_cpu.cuda()
    y = kf355.kf_softmax(x, -1, out=x)
    torch.cuda.synchronize()
    assert y.data_ptr() == x.data_ptr()
    assert_close(x, oracle.softmax(x_cpu, -1), dt)


def span_rows(length, pair):
    """Rows per workgroup of the staged-span kernel for rows that are not
    whole 16-byte vectors, or 0 when it does not apply: the fewest rows whose
    span is whole input and output vectors, times as many as fit 4096 fp32."""
    vin, vout = (4 if pair[0] == "f32" else 8), (4 if pair[1] == "f32" else 8)
    if length % vin == 0 and length % vout == 0:
        return 0
    align = max(v // math.gcd(length, v) for v in (vin, vout))
    r = min(256, 4096 // length)
    r -= r % align
    return r if r >= align else 0


@pytest.mark.parametrize("pair", PAIRS, ids=lambda p: f"{p[0]}-{p[1]}")
@pytest.mark.parametrize("length", [1, 3, 5, 127, 129, 257, 385, 511, 513, 1023, 1025, 4095])
def test_ragged_rows_take_staged_spans(pair, length):
    """Rows of 129-512 elements take the 16-row plan (16 lanes per row,
    ceil(L / 16) elements per lane, up to 32 KiB of staging); the rest as
    many rows as fit 4096 floats."""
    rows = 1000                                   # not a multiple of any span's rows: a partial last workgroup
    note(f"softmax staged spans {pair} len={length}")
    x = randn((rows, length), pair[0], seed=length + 7, std=3.0)
    _, variant, _ = run_case(x, -1, pair[1])
    assert variant.startswith("sm_span") == (span_rows(length, pair) > 0), variant
    if variant.startswith("sm_span") and 128 < length <= 512:
        per_lane = -(-length // 16)
        assert variant == f"sm_span_lpr16_npl{max(per_lane, 8)}", variant


# Rows that are not whole 16-byte vectors, too long for staged spans: the
# aligned vectors covering each row with the neighbours' elements masked.
# Lengths reach every lane-group and workgroup configuration for 16-bit
# inputs (ceil((L - 1) / 8) + 1 slots) and the fp32 ones past the
# element-wise kernels' 16384; row counts leave a partial last workgroup and
# a tensor that ends inside a vector.
EDGE_16 = [515, 701, 1001, 1201, 1501, 2001, 3001, 4097, 8001, 12001, 16001, 24001, 32001, 40001]
EDGE_32 = [16385, 20001, 30001]


def edge_rows(length):
    return 37 if length <= 8192 else 5


@pytest.mark.parametrize("pair", [p for p in PAIRS if p[0] != "f32"], ids=lambda p: f"{p[0]}-{p[1]}")
@pytest.mark.parametrize("length", EDGE_16)
def test_masked_vector_rows_16bit(pair, length):
    rows = edge_rows(length)
    note(f"softmax masked-vector rows {pair} rows={rows} len={length}")
    x = randn((rows, length), pair[0], seed=length + 3, std=3.0)
    _, variant, _ = run_case(x, -1, pair[1])
    assert variant.startswith(("sm_wave_edge", "sm_block_edge")), variant


@pytest.mark.parametrize("length", EDGE_32)
def test_masked_vector_rows_fp32(length):
    note(f"softmax masked-vector rows f32 len={length}")
    x = randn((5, length), "f32", seed=length + 3, std=3.0)
    _, variant, _ = run_case(x, -1, "f32")
    assert variant.startswith("sm_block_edge"), variant


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_masked_vector_rows_special_and_in_place(dt):
    note(f"softmax masked-vector rows special values in place {dt}")
    length = 4097
    x = randn((9, length), "f32", seed=21, std=2.0)
    x[0] = float("-inf")                      # fully masked -> NaN row
    x[1, 7] = float("nan")                    # NaN in the row's first vector
    x[2, length - 1] = float("inf")           # +inf in the row's last vector
    x[3] = float("-inf")
    x[3, 0] = 0.5                             # one finite entry -> exact one-hot
    x[4, 1::2] = float("-inf")                # masked entries -> exact +0
    x[5] = 1.25                               # uniform row
    x_cpu = x.to(TORCH[dt])
    xd = x_cpu.cuda()
    y = kf355.kf_softmax(xd, -1, out=xd)
    torch.cuda.synchronize()
    assert y.data_ptr() == xd.data_ptr() and kf355.last_variant().startswith("sm_block_edge")
    assert_close(y, oracle.softmax(x_cpu, -1), dt)
    yc = y.float().cpu()
    assert torch.isnan(yc[:3]).all() and not torch.isnan(yc[3:]).any()
    assert yc[3, 0].item() == 1.0 and (yc[3, 1:] == 0).all() and not torch.signbit(yc[3]).any()
    assert (yc[4, 1::2] == 0).all()


def test_zero_d_and_empty():
    note("softmax 0-d and empty")
    y = kf355.kf_softmax(torch.tensor(3.0, device="cuda"), 0)
    e = kf355.kf_softmax(torch.empty(0, 5, device="cuda"), -1)
    torch.cuda.synchronize()
    assert y.item() == 1.0 and e.shape == (0, 5)


def test_repeat_calls_are_bitwise_identical():
    note("softmax determinism")
    x = randn((512, 4096), "bf16", seed=13).cuda()
    a = kf355.kf_softmax(x, -1)
    b = kf355.kf_softmax(x, -1)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
