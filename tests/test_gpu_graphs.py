"""libkf355 calls captured in HIP graphs (torch.cuda.CUDAGraph) and replayed:
every operator, including the two that exchange partial results between
workgroups through a workspace (fused GroupNorm, split softmax), captured with
preallocated outputs and workspaces, replayed several times with fresh input
copied in and the program's own eager work and synchronisations between the
replays.  Every replay must equal, bit for bit, the same call made outside the
graph on the same input (the kernels are deterministic), and the exchange
workspaces must be all zero after every replay (the kernels leave them so; no
memset is recorded in any graph)."""
import pytest
import torch

from compare import note
from paper_2607_24762_amd import kf355
from paper_2607_24762_amd.workloads import randn_device

pytestmark = pytest.mark.gpu
REPLAYS = 5


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    kf355.lib()


NAMES = ["softmax", "softmax_causal", "softmax_split", "group_norm", "group_norm_nhwc", "layer_norm",
         "adaptive_avgpool2d", "max_pool2d"]


def case(name):
    """(input shape, dtype, call(x, out, ws) -> None, output factory, workspace factory) for one operator;
    built inside the test, so collecting this module on a host without a GPU allocates nothing."""
    def ws_gn(x):
        return torch.zeros(kf355.kf_group_norm_workspace_bytes(x, 32), dtype=torch.uint8, device="cuda")

    def ws_split(x):
        return torch.zeros(kf355.softmax_split_workspace(x, -1, torch.float32).numel(), dtype=torch.uint8,
                           device="cuda")

    if name == "softmax":
        return (8, 1024, 1024), "bf16", lambda x, y, ws: kf355.kf_softmax(x, -1, out=y), torch.empty_like, None
    if name == "softmax_causal":
        return ((2, 8, 512, 512), "bf16", lambda x, y, ws: kf355.kf_softmax_causal(x, 0.125, out=y),
                torch.empty_like, None)
    if name == "softmax_split":
        return ((1, 8, 1, 32768), "bf16",
                lambda x, y, ws: kf355.kf_softmax_split(x, -1, out_dtype=torch.float32, out=y, workspace=ws),
                lambda x: torch.empty(x.shape, dtype=torch.float32, device="cuda"), ws_split)
    if name in ("group_norm", "group_norm_nhwc"):      # the nhwc input is made channels last below
        w = torch.full((512,), 1.25, device="cuda", dtype=torch.bfloat16)
        b = torch.full((512,), -0.5, device="cuda", dtype=torch.bfloat16)
        return ((1, 512, 128, 128), "bf16",
                lambda x, y, ws: kf355.kf_group_norm(x, 32, w, b, 1e-6, out=y, workspace=ws), torch.empty_like,
                ws_gn)
    if name == "layer_norm":
        return ((2, 4096, 1536), "bf16", lambda x, y, ws: kf355.kf_layer_norm(x, (1536,), eps=1e-6, out=y),
                torch.empty_like, None)
    if name == "adaptive_avgpool2d":
        return ((32, 2048, 7, 7), "f32", lambda x, y, ws: kf355.kf_adaptive_avgpool2d(x, 1, out=y),
                lambda x: torch.empty(32, 2048, 1, 1, device="cuda"), None)
    return ((8, 64, 112, 112), "f32", lambda x, y, ws: kf355.kf_max_pool2d(x, 3, 2, 1, out=y),
            lambda x: torch.empty(8, 64, 56, 56, device="cuda"), None)


@pytest.mark.parametrize("name", NAMES)
def test_capture_and_replay(name):
    shape, dt, call, make_out, make_ws = case(name)
    note(f"graph {name} {shape} {dt}")
    x = randn_device(shape, dt, seed=41)
    if name.endswith("_nhwc"):
        x = x.contiguous(memory_format=torch.channels_last)
    y = make_out(x)
    ws = make_ws(x) if make_ws else None
    call(x, y, ws)                                   # warm up outside the capture
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        call(x, y, ws)
    torch.cuda.synchronize()
    ref_out = make_out(x)
    for i in range(REPLAYS):
        x.copy_(randn_device(shape, dt, seed=100 + i, std=1.0 + i))     # fresh input, eager work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = y.contiguous().clone()                 # dense copy: byte views need a unit last stride
        call(x, ref_out, ws)                         # the same call outside the graph
        torch.cuda.synchronize()
        ref = ref_out.contiguous()
        assert torch.equal(got.view(torch.uint8) if got.dtype != torch.float32 else got.view(torch.int32),
                           ref.view(torch.uint8) if ref.dtype != torch.float32 else ref.view(torch.int32)), \
            (name, i)
        if ws is not None:
            assert int(ws.count_nonzero().item()) == 0, (name, i)
