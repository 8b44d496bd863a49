"""GPU check of the calibration copy and read (kf_stream_copy and
kf_stream_read, measurement aids): byte-exact copies, and the XOR of every
4 KiB block, at sizes that are whole waves, ragged tails and a single
16-byte vector."""
import pytest
import torch

from compare import note
from paper_2607_24762_amd import kf355

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    kf355.lib()


@pytest.mark.parametrize("nbytes", [16, 4096, 4096 * 3 + 16, 1 << 20, (256 << 20) + 4080])
def test_copy_is_exact(nbytes):
    note(f"stream_copy {nbytes} bytes")
    g = torch.Generator(device="cuda")
    g.manual_seed(nbytes % 1000)
    src = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device="cuda", generator=g)
    dst = torch.zeros_like(src)
    kf355.stream_copy(src, dst)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
    assert kf355.last_variant() == "stream_copy"


@pytest.mark.parametrize("nbytes", [16, 4096, 4096 * 3 + 16, 1 << 20, (12 << 20) + 4080])
def test_read_xors_every_block(nbytes):
    note(f"stream_read {nbytes} bytes")
    g = torch.Generator(device="cuda")
    g.manual_seed(nbytes % 997)
    src = torch.randint(-2 ** 31, 2 ** 31 - 1, (nbytes // 4,), dtype=torch.int32, device="cuda", generator=g)
    blocks = -(-nbytes // 4096)
    dst = torch.full((blocks * 4,), -1, dtype=torch.int32, device="cuda")
    kf355.stream_read(src, dst)
    torch.cuda.synchronize()
    assert kf355.last_variant() == "stream_read"
    words = torch.zeros(blocks * 1024, dtype=torch.int32)
    words[: nbytes // 4] = src.cpu()
    ref = words.view(blocks, 256, 4).numpy()
    import numpy as np
    expect = np.bitwise_xor.reduce(ref, axis=1)
    assert np.array_equal(dst.cpu().view(blocks, 4).numpy(), expect)
