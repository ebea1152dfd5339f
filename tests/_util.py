"""Helpers shared by the GPU tests: host arrays <-> device tensors, error metrics."""
import sys

import numpy as np
import torch


def say(*args):
    """Print and flush, so that a GPU run names its case before each step."""
    print(*args, flush=True)
    sys.stdout.flush()


def dev(x: np.ndarray, device="cuda") -> torch.Tensor:
    """Upload a synth array: uint16 arrays are bf16 bit patterns."""
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(x).to(device)


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def row_rel_l2(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per-row ||got - ref|| / ||ref|| (0/0 counts as 0)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.linalg.norm(got - ref, axis=1)
    den = np.linalg.norm(ref, axis=1)
    out = np.where(den > 0, num / np.where(den > 0, den, 1.0), num)
    return out
