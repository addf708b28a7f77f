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


CANARY_BYTES = 4096          # guard bytes on each side of an output buffer
CANARY_BYTE = 0xA5


class Guarded:
    """A device output buffer with canary bytes on both sides.

    `t` is a contiguous tensor of the requested shape and dtype in the middle
    of a larger allocation whose first and last CANARY_BYTES bytes hold
    CANARY_BYTE; the interior starts filled with it too.  `check()` asserts
    that a call wrote nothing outside its output (an out-of-bounds store
    that stays inside the allocation would otherwise go unnoticed)."""

    def __init__(self, shape, dtype, name="output"):
        shape = tuple(int(s) for s in shape)
        elt = torch.empty((), dtype=dtype).element_size()
        n = 1
        for s in shape:
            n *= s
        self.name = name
        self.raw = torch.full((n * elt + 2 * CANARY_BYTES,), CANARY_BYTE, dtype=torch.uint8,
                              device=dev())
        self.t = self.raw[CANARY_BYTES:CANARY_BYTES + n * elt].view(dtype).view(shape)

    def check(self):
        head = self.raw[:CANARY_BYTES]
        tail = self.raw[self.raw.numel() - CANARY_BYTES:]
        for part, where in ((head, "before"), (tail, "after")):
            bad = torch.nonzero(part != CANARY_BYTE)
            assert bad.numel() == 0, (f"{self.name}: {bad.numel()} canary bytes {where} the "
                                      f"buffer overwritten (first at offset {int(bad[0])})")
        return self.t


def check_canaries(*guards):
    for g in guards:
        g.check()
