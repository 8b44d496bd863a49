"""GPU parity of kf_adaptive_avgpool2d against the float64 oracle: 1x1
outputs over plane sizes that select each LDS tiling (1, 4, 16 and 64
threads per plane) and the plane-per-workgroup kernel, ragged plane counts,
misaligned inputs, generic output sizes (staged planes, vector and element
staging, and a thread per cell for large planes) and 3-D inputs, in fp32 / bf16 /
fp16.  Tolerances: fp32 max abs error <= 1e-6; bf16 / fp16 within 1 unit in
the last place of the oracle rounded once."""
import pytest
import torch

from compare import assert_close, note
from oracle import oracle
from paper_2607_24762_amd import kf355
from paper_2607_24762_amd.workloads import randn

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    kf355.lib()


def relu_input(shape, dt, seed):
    return torch.relu(randn(shape, "f32", seed=seed)).to({"f32": torch.float32, "bf16": torch.bfloat16,
                                                           "f16": torch.float16}[dt])


def run(x_cpu, out, dt, x_gpu=None):
    x = x_gpu if x_gpu is not None else x_cpu.cuda()
    y = kf355.kf_adaptive_avgpool2d(x, out)
    torch.cuda.synchronize()
    variant = kf355.last_variant()
    assert_close(y, oracle.adaptive_avg_pool2d(x_cpu, out), dt)
    return variant


ONE_BY_ONE = [
    ((2, 3, 7, 7), "ap_flat_tps4"),         # 49-element planes: 64 per workgroup
    ((4, 100, 7, 7), "ap_flat_tps4"),       # 400 planes: ragged last workgroup
    ((32, 2048, 7, 7), "ap_flat_tps4"),     # the ResNet-50 head
    ((3, 5, 1, 1), "ap_flat_tps1"),
    ((1, 7, 3, 3), "ap_flat_tps1"),
    ((2, 8, 4, 5), "ap_flat_tps2"),
    ((2, 64, 8, 8), "ap_flat_tps4"),        # even plane size
    ((2, 40, 10, 10), "ap_flat_tps8"),
    ((2, 64, 14, 14), "ap_flat_tps16"),
    ((1, 16, 20, 20), "ap_flat_tps32"),
    ((2, 16, 28, 28), "ap_flat_tps64"),
    ((1, 8, 56, 56), "ap_plane"),
    ((1, 3, 224, 224), "ap_plane"),
    ((1, 2, 37, 41), "ap_plane"),           # odd plane: scalar loads
]


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape,variant", ONE_BY_ONE, ids=lambda v: str(v))
def test_one_by_one(shape, variant, dt):
    note(f"avgpool 1x1 {shape} {dt}")
    assert run(relu_input(shape, dt, 1), (1, 1), dt) == variant


GENERIC = [
    ((2, 3, 7, 7), (3, 3)), ((1, 2, 13, 17), (5, 7)), ((1, 1, 4, 6), (8, 9)), ((3, 10, 9), (4, 2)),
    ((2, 4, 7, 7), (7, 7)), ((1, 2, 5, 5), (1, 3)),
    ((2, 512, 14, 14), (7, 7)),      # 2x2 windows (a VGG-style head at twice the resolution)
    ((2, 256, 13, 13), (6, 6)),      # overlapping 3x3 windows (AlexNet-style)
    ((3, 7, 9, 11), (4, 5)),         # 21 planes, odd spans: ragged workgroups
    ((1, 5, 64, 64), (3, 3)),        # one plane per workgroup
    ((1, 3, 1, 1), (5, 6)),          # one element spread over a larger output
    ((1, 2, 70, 70), (5, 5)),        # planes beyond the staging tile
]


def staged_variant(shape, out, dt, x):
    """The kernel the host picks: staged planes when a plane fits the 4096-element tile (vector staging when the
    planes per workgroup make whole 16-byte spans and x is aligned; a fixed k x k window read when no window
    is more than k <= 4 rows or columns), else a thread per output cell."""
    h, w = shape[-2], shape[-1]
    s = h * w
    if s > 4096:
        return "ap_window"
    vec = 4 if dt == "f32" else 8
    planes = 1
    for d in shape[:-2]:
        planes *= d
    p = max(1, min(4096 // s, planes // 2048))
    while p > 1 and (p * s) % vec:
        p -= 1
    name = "ap_staged_vec" if (p * s) % vec == 0 and x.data_ptr() % 16 == 0 else "ap_staged_scalar"

    def extent(n, m):
        return max(((k + 1) * n + m - 1) // m - (k * n) // m for k in range(m))
    e = max(extent(h, out[0]), extent(w, out[1]))
    return name + (f"_k{e if e > 1 else 2}" if e <= 4 else "")


@pytest.mark.parametrize("shape,out", GENERIC, ids=lambda v: str(v))
@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
def test_generic_sizes(shape, out, dt):
    note(f"avgpool {shape}->{out} {dt}")
    x_cpu = relu_input(shape, dt, 2)
    x = x_cpu.cuda()
    assert run(x_cpu, out, dt, x_gpu=x) == staged_variant(shape, out, dt, x)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_misaligned_input(dt):
    note(f"avgpool misaligned {dt}")
    planes, s = 300, 49
    big = relu_input((planes * s + 1,), dt, 3)
    x_cpu = big[1:].view(3, 100, 7, 7)
    x = big.cuda()[1:].view(3, 100, 7, 7)
    run(x_cpu, (1, 1), dt, x_gpu=x)
    assert run(x_cpu, (3, 3), dt, x_gpu=x) == "ap_staged_scalar_k3"


def test_constant_input_is_exact():
    note("avgpool constant")
    x = torch.full((4, 96, 7, 7), 0.375, device="cuda")
    y = kf355.kf_adaptive_avgpool2d(x, 1)
    torch.cuda.synchronize()
    assert (y == 0.375).all()


CHANNELS_LAST = [
    ((32, 2048, 7, 7), 1),          # the ResNet-50 head, channels last
    ((2, 64, 14, 14), 7),           # divisible windows
    ((2, 48, 7, 7), (3, 5)),        # overlapping adaptive windows
    ((1, 24, 5, 9), (8, 4)),        # output taller than the input
    ((3, 5, 6, 6), 2),              # channels not whole 16-byte vectors: scalar path
    ((2, 200, 9, 11), (1, 3)),      # channels beyond one 64-vector block
    ((4, 512, 14, 14), 7),          # 2 x 2 windows, many channel vectors
    ((2, 256, 13, 13), 6),          # overlapping 3 x 3 windows
    ((2, 64, 8, 8), 2),             # 4 x 4 windows
    ((2, 64, 10, 10), 2),           # 5 x 5 windows: split over thread groups
    ((2, 6, 10, 10), 1),            # large window, channels not whole vectors: scalar thread groups
    ((2, 32, 12, 12), 1),           # 144-pixel window: three batches of 64 per workgroup
    ((1, 40, 11, 11), 2),           # overlapping 6 x 6 windows (ordinary loads), a partial channel block
]


def window_extent(n, m):
    """Largest adaptive window extent pooling n positions into m."""
    return max(((k + 1) * n + m - 1) // m - (k * n) // m for k in range(m))


def nhwc_variant(shape, out, dt):
    oh, ow = (out, out) if isinstance(out, int) else out
    vec = 4 if dt == "f32" else 8
    kind = "vec" if shape[1] % vec == 0 else "scalar"
    ext = max(window_extent(shape[2], oh), window_extent(shape[3], ow))
    if ext <= 4:
        return f"ap_nhwc_cell_{kind}_k{max(ext, 2)}"
    return f"ap_nhwc_{kind}"


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape,out", CHANNELS_LAST, ids=lambda v: str(v))
def test_channels_last(shape, out, dt):
    note(f"avgpool channels last {shape} -> {out} {dt}")
    x_cpu = relu_input(shape, dt, seed=shape[1])
    x = x_cpu.cuda().contiguous(memory_format=torch.channels_last)
    variant = run(x_cpu, out, dt, x_gpu=x)
    assert variant == nhwc_variant(shape, out, dt), variant


def test_channels_last_output_keeps_the_layout():
    note("avgpool channels last layout")
    x_cpu = relu_input((2, 16, 9, 9), "f32", seed=3)
    x = x_cpu.cuda().contiguous(memory_format=torch.channels_last)
    y = kf355.kf_adaptive_avgpool2d(x, (3, 3))
    torch.cuda.synchronize()
    assert y.is_contiguous(memory_format=torch.channels_last)
    assert_close(y, oracle.adaptive_avg_pool2d(x_cpu, (3, 3)), "f32")
