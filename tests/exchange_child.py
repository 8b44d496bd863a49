"""Child process for the exchange-fallback tests: runs one or more workloads
of the kernels that exchange partials between workgroups (GroupNorm's fused
path, the split-row softmax) in order, on ONE shared zero-filled workspace,
with the environment it was started with (KF355_GN_WAIT_TICKS=0 or
KF355_SM_WAIT_TICKS=0 makes every waiting workgroup of that operator give up
at once and recompute the partials itself), and saves each output's bits and
variant, the workspace's give-up count (the first word of its status block)
and the count of non-zero bytes after the status block.

usage: exchange_child.py OUT.npz OP [OP ...]
OP: group_norm | group_norm_nhwc | group_norm_small | group_norm_parts | group_norm_tiles_small |
    group_norm_split | softmax_split

Further environment knobs the tests use: KF355_GN_MODE=fused (GroupNorm
without gn_pipe), KF355_GN_PARTS=k (gn_pipe with k workgroups per group) and
KF355_GN_STAGGER_TICKS=0 (gn_pipe without its staggered issue) and
KF355_GN_SPLIT_RECOMPUTE=1 (gn_split recomputing every part)."""
import os
import sys

import numpy as np
import torch

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from paper_2607_24762_amd import kf355  # noqa: E402
from paper_2607_24762_amd import workloads as W  # noqa: E402


def inputs(op: str) -> dict:
    """The inputs of each op, on the host (the parent draws the same ones)."""
    if op in ("group_norm", "group_norm_nhwc"):
        w = W.groupnorm_vae_bf16()
        return {"x": w["x"], "groups": 32, "weight": w["weight"], "bias": w["bias"], "eps": w["eps"]}
    if op == "group_norm_small":
        # 24 channels per group over 32 x 32: two parts per group, eight groups.
        return {"x": W.randn((2, 96, 32, 32), "bf16", seed=31, mean=-0.2, std=2.0), "groups": 4,
                "weight": W.randn((96,), "bf16", seed=32, mean=1.0, std=0.1),
                "bias": W.randn((96,), "bf16", seed=33, std=0.1), "eps": 1e-5}
    if op == "group_norm_parts":
        # 4 channels of 64 x 64 per group: 16384 elements, one 16384-element
        # chunk, two of 8192 or four of 4096.
        return {"x": W.randn((2, 32, 64, 64), "bf16", seed=41, mean=0.5, std=1.2), "groups": 8,
                "weight": W.randn((32,), "bf16", seed=42, mean=1.0, std=0.1),
                "bias": W.randn((32,), "bf16", seed=43, std=0.1), "eps": 1e-6}
    if op == "group_norm_tiles_small":
        # Channels last, 64-channel tiles: 192 channels, 64 per group, 1024
        # pixels: 4 parts per group.
        return {"x": W.randn((1, 192, 32, 32), "bf16", seed=54, mean=-0.4, std=1.1), "groups": 3,
                "weight": W.randn((192,), "bf16", seed=55, mean=1.0, std=0.1),
                "bias": W.randn((192,), "bf16", seed=56, std=0.1), "eps": 1e-6}
    if op == "group_norm_split":
        # 16 channels of 512 x 512 per group: 256 chunks of 16384, gn_split.
        return {"x": W.randn((1, 32, 512, 512), "bf16", seed=61, mean=0.8, std=1.3), "groups": 2,
                "weight": W.randn((32,), "bf16", seed=62, mean=1.0, std=0.1),
                "bias": W.randn((32,), "bf16", seed=63, std=0.1), "eps": 1e-6}
    if op == "softmax_split":
        return {"x": W.attn_decode_bf16()["x"]}
    raise SystemExit(f"unknown op {op}")


def run(op: str, ws: torch.Tensor) -> torch.Tensor:
    a = inputs(op)
    x = a["x"].cuda()
    if op == "softmax_split":
        return kf355.kf_softmax_split(x, -1, out_dtype=torch.float32, workspace=ws)
    if op in ("group_norm_nhwc", "group_norm_tiles_small"):
        x = x.contiguous(memory_format=torch.channels_last)
    return kf355.kf_group_norm(x, a["groups"], a["weight"].cuda(), a["bias"].cuda(), a["eps"], workspace=ws)


def spawn(tmp_path, ops, **env) -> dict:
    """Runs this file in a child process with `env` added to the environment
    (the wait bounds are read once per process) and returns what it saved."""
    import subprocess
    out = str(tmp_path / ("child_" + "_".join(ops) + ".npz"))
    r = subprocess.run([sys.executable, "-u", os.path.abspath(__file__), out, *ops],
                       env=dict(os.environ, **env), timeout=300, capture_output=True, text=True)
    print(r.stdout, r.stderr[-2000:])
    assert r.returncode == 0, r.returncode
    got = np.load(out)
    return {k: got[k] for k in got.files}


def main():
    out_path, ops = sys.argv[1], sys.argv[2:]
    knobs = ("KF355_GN_WAIT_TICKS", "KF355_SM_WAIT_TICKS", "KF355_GN_MODE", "KF355_GN_PARTS", "KF355_GN_STAGGER_TICKS",
             "KF355_GN_SPLIT_RECOMPUTE")
    print(f"[child] ops={ops} " + " ".join(f"{k}={os.environ.get(k)}" for k in knobs), flush=True)
    ws = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    saved = {}
    for i, op in enumerate(ops):
        y = run(op, ws)
        torch.cuda.synchronize()
        saved[f"variant{i}"] = kf355.last_variant()
        y = y.contiguous()
        saved[f"bits{i}"] = y.view(torch.int16 if y.element_size() == 2 else torch.int32).cpu().numpy()
        print(f"[child] {op}: variant={saved[f'variant{i}']} give_ups={kf355.workspace_give_ups(ws)}", flush=True)
    saved["give_ups"] = kf355.workspace_give_ups(ws)
    saved["rest"] = int(ws[256:].count_nonzero().item())
    np.savez(out_path, **saved)
    print(f"[child] give_ups={saved['give_ups']} nonzero_after_status={saved['rest']}", flush=True)


if __name__ == "__main__":
    main()
