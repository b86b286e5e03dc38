"""Helpers for the GPU tests: guarded device buffers and host conversions."""

import numpy as np
import torch

PAD = 256  # guard band on each side of every output buffer
CANARY = 0xA5


def to_device(a):
    """numpy (float32 / uint16 / int32) -> contiguous device tensor with the same bits."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to("cuda")
    return torch.from_numpy(a).to("cuda")


def to_host(t, dtype):
    """device tensor -> numpy array of the given dtype (bit reinterpretation)."""
    return t.detach().contiguous().view(torch.uint8).cpu().numpy().view(dtype)


class Guarded:
    """A device buffer with canary bytes before and after it."""

    def __init__(self, nbytes, torch_dtype):
        self.nbytes = nbytes
        self.raw = torch.full((PAD + nbytes + PAD,), CANARY, dtype=torch.uint8, device="cuda")
        self.t = self.raw[PAD:PAD + nbytes].view(torch_dtype)

    def intact(self):
        head = self.raw[:PAD]
        tail = self.raw[PAD + self.nbytes:]
        return bool(torch.all(head == CANARY).item()) and bool(torch.all(tail == CANARY).item())


def torch_dtype(dtype):
    return torch.float32 if dtype == "fp32" else torch.int16


def np_dtype(dtype):
    return np.float32 if dtype == "fp32" else np.uint16


def bits(a, dtype):
    return a.view(np.uint32) if dtype == "fp32" else a


def assert_bits_equal(got, want, dtype, what=""):
    g, w = bits(np.asarray(got), dtype), bits(np.asarray(want), dtype)
    if not np.array_equal(g, w):
        bad = np.flatnonzero(g != w)
        i = int(bad[0])
        raise AssertionError(f"{what}: {bad.size} mismatches, first at {i}: got {int(g[i]):#x} want {int(w[i]):#x}")
