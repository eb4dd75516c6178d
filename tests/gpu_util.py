"""Helpers shared by the GPU parity tests (device transfers and comparisons).

Nothing here computes any part of the method: expected values come from the
CPU oracle, device results from libpcs through its C ABI.
"""
import numpy as np
import torch


def dev(a: np.ndarray) -> torch.Tensor:
    """Host uint8 bytes -> device uint8 tensor."""
    return torch.from_numpy(np.ascontiguousarray(a).reshape(-1).view(np.uint8).copy()).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> host uint8 bytes."""
    torch.cuda.synchronize()
    return t.detach().contiguous().view(torch.uint8).cpu().numpy().reshape(-1)


def u64(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.detach().cpu().numpy().view(np.uint64).reshape(-1)


def zeros_u64(n: int) -> torch.Tensor:
    return torch.zeros(max(n, 1), dtype=torch.int64, device="cuda")


def arena(nbytes: int) -> torch.Tensor:
    return torch.empty(nbytes, dtype=torch.uint8, device="cuda")


def log(*a):
    print(*a, flush=True)
