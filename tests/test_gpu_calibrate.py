"""GPU check of the calibration copy (kf_stream_copy, a measurement aid):
byte-exact copies at sizes that are whole waves, ragged tails and a single
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
