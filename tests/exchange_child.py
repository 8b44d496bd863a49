"""Child process for the exchange-fallback tests: runs one workload of a
kernel that exchanges partials between workgroups (GroupNorm's fused path,
the split-row softmax) once, with the environment it was started with
(KF355_GN_WAIT_TICKS=0 or KF355_SM_WAIT_TICKS=0 makes every waiting
workgroup give up at once and recompute the partials itself), and saves the
output bits, the workspace's give-up word and the count of other non-zero
workspace bytes.

usage: exchange_child.py group_norm|group_norm_nhwc|softmax_split OUT.npz"""
import ctypes
import os
import sys

import numpy as np
import torch

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from paper_2607_24762_amd import kf355  # noqa: E402
from paper_2607_24762_amd import workloads as W  # noqa: E402

op, out_path = sys.argv[1], sys.argv[2]
print(f"[child] op={op} KF355_GN_WAIT_TICKS={os.environ.get('KF355_GN_WAIT_TICKS')} "
      f"KF355_SM_WAIT_TICKS={os.environ.get('KF355_SM_WAIT_TICKS')}", flush=True)
ws = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
nb = ctypes.c_size_t(0)
if op in ("group_norm", "group_norm_nhwc"):
    w = W.groupnorm_vae_bf16()
    x = w["x"].cuda()
    if op == "group_norm_nhwc":
        x = x.contiguous(memory_format=torch.channels_last)
    y = kf355.kf_group_norm(x, 32, w["weight"].cuda(), w["bias"].cuda(), w["eps"], workspace=ws)
    shape = (ctypes.c_int64 * 4)(1, 512, 128, 128)
    kf355.lib().kf_group_norm_workspace_bytes(1, 4, shape, 32, ctypes.byref(nb))
elif op == "softmax_split":
    w = W.attn_decode_bf16()
    x = w["x"].cuda()
    y = kf355.kf_softmax_split(x, -1, out_dtype=torch.float32, workspace=ws)
    shape = (ctypes.c_int64 * 4)(*x.shape)
    kf355.lib().kf_softmax_split_workspace_bytes(1, 0, 4, shape, -1, ctypes.byref(nb))
else:
    raise SystemExit(f"unknown op {op}")
torch.cuda.synchronize()
variant = kf355.last_variant()
flag = int(ws[nb.value - 256:nb.value - 252].cpu().view(torch.int32).item())
rest = int(ws[: nb.value - 256].count_nonzero().item())
bits = y.contiguous().view(torch.int16 if y.element_size() == 2 else torch.int32).cpu().numpy()
np.savez(out_path, bits=bits, flag=flag, rest=rest, variant=variant)
print(f"[child] variant={variant} flag={flag} nonzero_before_flag={rest}", flush=True)
