"""GPU check of the calibration copy and read (kf_stream_copy and
kf_stream_read, measurement aids): byte-exact copies, and the parity bits of
every 2 KiB block, at sizes that are whole waves, ragged tails and a single
16-byte vector."""
import numpy as np
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


@pytest.mark.parametrize("nbytes", [16, 1024 + 16, 4096, 4096 * 3 + 16, 1 << 20, (8 << 20) - 16, (8 << 20) + 16,
                                    (256 << 20) + 4080])
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


@pytest.mark.parametrize("nbytes", [16, 2048, 2048 * 3 + 16, 4096, 1 << 20, (12 << 20) + 4080])
def test_read_parity_of_every_block(nbytes):
    note(f"stream_read {nbytes} bytes")
    g = torch.Generator(device="cuda")
    g.manual_seed(nbytes % 997)
    src = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device="cuda", generator=g)
    blocks = -(-nbytes // 2048)
    dst = torch.full((blocks,), -1, dtype=torch.int64, device="cuda")
    kf355.stream_read(src, dst)
    torch.cuda.synchronize()
    assert kf355.last_variant() == "stream_read"
    data = np.zeros(blocks * 2048, dtype=np.uint8)
    data[:nbytes] = src.cpu().numpy()
    # Block b, vector k (16 bytes), lane L = k % 64: bit L of word b is the
    # parity of the set bits of vectors L and 64 + L.
    ones = np.unpackbits(data).reshape(blocks, 2, 64, 128).sum(axis=(1, 3))
    expect = ((ones & 1).astype(np.uint64) << np.arange(64, dtype=np.uint64)).sum(axis=1, dtype=np.uint64)
    got = dst.cpu().numpy().view(np.uint64)
    assert np.array_equal(got, expect)
