"""Child process for test_gpu_group_norm: runs the SD3.5 GroupNorm workload
once with the environment it was started with (e.g. KF355_GN_WAIT_TICKS=0,
which makes every fused workgroup recompute its group's statistics) and
saves the output bits and the workspace's give-up word."""
import os
import sys

import numpy as np
import torch

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from paper_2607_24762_amd import kf355  # noqa: E402
from paper_2607_24762_amd import workloads as W  # noqa: E402

out_path = sys.argv[1]
print(f"[child] KF355_GN_WAIT_TICKS={os.environ.get('KF355_GN_WAIT_TICKS')}", flush=True)
w = W.groupnorm_vae_bf16()
ws = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
y = kf355.kf_group_norm(w["x"].cuda(), 32, w["weight"].cuda(), w["bias"].cuda(), w["eps"], workspace=ws)
torch.cuda.synchronize()
variant = kf355.last_variant()
import ctypes  # noqa: E402
shape = (ctypes.c_int64 * 4)(1, 512, 128, 128)
nb = ctypes.c_size_t(0)
kf355.lib().kf_group_norm_workspace_bytes(1, 4, shape, 32, ctypes.byref(nb))
flag = int(ws[nb.value - 256:nb.value - 252].cpu().view(torch.int32).item())
rest = int(ws[: nb.value - 256].count_nonzero().item())
np.savez(out_path, bits=y.view(torch.int16).cpu().numpy(), flag=flag, rest=rest, variant=variant)
print(f"[child] variant={variant} flag={flag} nonzero_before_flag={rest}", flush=True)
