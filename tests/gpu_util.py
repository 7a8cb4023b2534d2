"""Helpers shared by the GPU tests: device transfer, bf16 rounding, relative L2."""

import numpy as np
import torch

from paper_2511_06724_amd import dn

DEV = torch.device("cuda:0") if torch.cuda.is_available() else None


def tdtype(dtype):
    return torch.bfloat16 if dtype == dn.DN_BF16 else torch.float32


def to_dev(a, dtype=dn.DN_FP32):
    """numpy fp32 -> device tensor of the kernel dtype; returns (tensor, the values it holds as fp64)."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(tdtype(dtype)).contiguous()
    return t, t.float().cpu().numpy().astype(np.float64)


def f32_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def rel_l2(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


def announce(msg):
    print(msg, flush=True)
