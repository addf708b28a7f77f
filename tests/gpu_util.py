"""Shared helpers of the GPU parity tests (host <-> device copies only)."""
import numpy as np
import torch


def dev():
    return torch.device("cuda:0")


def to_gpu(a: np.ndarray, dtype: str = None) -> torch.Tensor:
    """Upload a storage array; bf16 bit patterns (uint16) become torch.bfloat16."""
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype == "bf16":
        t = t.view(torch.bfloat16)
    return t.to(dev())


def to_np(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def bits(a: np.ndarray) -> np.ndarray:
    """Bit patterns of a 16-bit float storage array for bitwise comparison."""
    return np.ascontiguousarray(a).view(np.uint16)


def first_mismatch(got: np.ndarray, ref: np.ndarray):
    bad = np.argwhere(got != ref)
    if bad.size == 0:
        return None
    i = tuple(bad[0])
    return f"{len(bad)} mismatches, first at {i}: got {got[i]} ref {ref[i]}"
