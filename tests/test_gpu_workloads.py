"""GPU parity at the full workload shapes (the tensors the benchmark times),
every element against the float64 oracle, in the launch configuration the
benchmark uses.  Tolerances: fp32 outputs max abs error <= 1e-6; bf16 outputs
within 1 unit in the last place of the oracle rounded once to bf16 (GroupNorm
also accepts |error| <= 2^-22 where |oracle| < 2^-19, see
test_gpu_group_norm.py; strict counts are printed)."""
import numpy as np
import pytest
import torch

from compare import compare, note
from oracle import oracle
from paper_2607_24762_amd import kf355
from paper_2607_24762_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    kf355.lib()


def report(name, r):
    print(f"[parity] {name}: {r}", flush=True)
    assert r["ok"], r


@pytest.mark.parametrize("name", ["softmax_f32_1024x1024", "router_softmax_f32_16384x256",
                                  "router_softmax_f32_16384x257"])
def test_fp32_softmax_workloads(name):
    note(name)
    w = W.WORKLOADS[name]()
    y = kf355.kf_softmax(w["x"].cuda(), -1)
    torch.cuda.synchronize()
    report(name, compare(y, oracle.softmax(w["x"], -1), "f32"))


def test_attention_softmax_causal_bf16():
    name = "attn_softmax_bf16_1x8x4096x4096_causal"
    note(name)
    w = W.WORKLOADS[name]()
    x = w["x"].cuda()
    y = kf355.kf_softmax(x, -1)
    torch.cuda.synchronize()
    yc = y.cpu()
    # Causal structure: row 0 is exactly one-hot, every masked entry +0.0.
    assert (yc[..., 0, 0] == 1.0).all()
    mask = torch.ones(4096, 4096, dtype=torch.bool).triu_(1)
    masked = yc[..., mask]
    assert (masked.view(torch.int16) == 0).all()
    del masked
    report(name, compare(yc, oracle.softmax(w["x"], -1), "bf16"))


def test_groupnorm_vae_bf16():
    name = "groupnorm_bf16_1x512x128x128_g32"
    note(name)
    w = W.WORKLOADS[name]()
    y = kf355.kf_group_norm(w["x"].cuda(), w["num_groups"], w["weight"].cuda(), w["bias"].cuda(), w["eps"])
    torch.cuda.synchronize()
    ref = oracle.group_norm(w["x"], w["num_groups"], w["weight"], w["bias"], w["eps"])
    report(name, compare(y, ref, "bf16", floor=(2.0 ** -19, 2.0 ** -22)))


def test_avgpool_resnet_head_f32():
    name = "avgpool_f32_32x2048x7x7_to_1x1"
    note(name)
    w = W.WORKLOADS[name]()
    y = kf355.kf_adaptive_avgpool2d(w["x"].cuda(), w["output_size"])
    torch.cuda.synchronize()
    report(name, compare(y, oracle.adaptive_avg_pool2d(w["x"], w["output_size"]), "f32"))


@pytest.mark.parametrize("shape,out", [((32, 512, 14, 14), (7, 7)), ((32, 256, 13, 13), (6, 6))])
def test_avgpool_general_sizes_f32(shape, out):
    """The general-size pooling rows at the shapes the benchmark times."""
    name = f"avgpool_f32_{'x'.join(map(str, shape))}_to_{out[0]}x{out[1]}"
    note(name)
    w = W.avgpool_general_f32(shape=shape, output_size=out)
    x = w["x"].cuda()
    y = torch.empty(shape[0], shape[1], *out, device="cuda")
    kf355.prepare_adaptive_avgpool2d(x, y)()
    torch.cuda.synchronize()
    assert kf355.last_variant().startswith("ap_staged_vec_k"), kf355.last_variant()
    report(name, compare(y, oracle.adaptive_avg_pool2d(w["x"], out), "f32"))
