"""Helpers for GPU parity tests: host<->device copies with exact bit
patterns, and mismatch reports that name the first differing element."""
import numpy as np
import torch

DEV = "cuda:0"
_TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
_NP_BITS = {"f32": np.uint32, "f16": np.uint16, "bf16": np.uint16}


def to_dev(a, dtype=None):
    """numpy -> GPU tensor, bit-exact.  bf16 arrays are uint16 bit patterns."""
    a = np.ascontiguousarray(a)
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)
    if a.dtype == np.uint16 and dtype == "f16":
        return torch.from_numpy(a.view(np.float16)).to(DEV)
    return torch.from_numpy(a).to(DEV)


def from_dev(t):
    """GPU tensor -> numpy with the same bits (bf16 -> uint16 patterns)."""
    t = t.detach()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def bits(a):
    a = np.asarray(a)
    if a.dtype in (np.float32, np.int32, np.uint32):
        return a.view(np.uint32)
    if a.dtype in (np.float16, np.uint16, np.int16):
        return a.view(np.uint16)
    return a.view(np.uint8)


def empty(n, dtype):
    return poisoned(n, _TORCH[dtype])


def poisoned(n, dtype):
    """Output buffer filled with 0xA5 bytes: a region a kernel fails to write
    cannot match the expected values by accident."""
    t = torch.empty(n, dtype=dtype, device=DEV)
    if n:
        t.view(torch.uint8).fill_(0xA5)
    return t


def assert_bits_equal(got, want, what, block=None):
    g, w = bits(got).reshape(-1), bits(want).reshape(-1)
    assert g.shape == w.shape, f"{what}: shape {g.shape} vs {w.shape}"
    if not np.array_equal(g, w):
        i = int(np.flatnonzero(g != w)[0])
        nbad = int(np.count_nonzero(g != w))
        loc = f" (block {i // block})" if block else ""
        raise AssertionError(f"{what}: {nbad} of {g.size} differ; first at {i}{loc}: "
                             f"got {g[i]:#x} want {w[i]:#x}")


def sync():
    torch.cuda.synchronize()
