"""Helpers for the GPU parity tests: move numpy bit patterns to and from the
device through PyTorch, and compare results to the oracle element by element."""
from __future__ import annotations

import numpy as np

NP_BITS = {"f32": np.uint32, "bf16": np.uint16, "i32": np.uint32, "u32": np.uint32}


def torch_dtype(dtype: str):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16, "i32": torch.int32,
            "u32": torch.int32}[dtype]


def to_dev(a: np.ndarray, dtype: str, device="cuda"):
    """Upload a numpy element array (bf16 as uint16 bits, u32 as uint32) unchanged."""
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    elif dtype == "f32":
        t = torch.from_numpy(np.ascontiguousarray(a, np.float32))
    else:
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int32))
    return t.to(device)


def bits(t_or_a, dtype: str) -> np.ndarray:
    """Raw bit patterns of a tensor or numpy array of `dtype` elements."""
    import torch
    if isinstance(t_or_a, torch.Tensor):
        t = t_or_a.detach().cpu().contiguous()
        if dtype == "bf16":
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.view(torch.int32).numpy().view(np.uint32)
    a = np.ascontiguousarray(t_or_a)
    return a.view(NP_BITS[dtype])


def nan_mask(b: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return ((b & 0x7F80) == 0x7F80) & ((b & 0x7F) != 0)
    if dtype == "f32":
        return ((b & 0x7F800000) == 0x7F800000) & ((b & 0x7FFFFF) != 0)
    return np.zeros(b.shape, bool)


def assert_parity(got, exp, dtype: str, op: str, what: str = "") -> None:
    """Bit-exact equality; for float sum/prod a NaN matches any NaN (payloads
    are not specified by the definition)."""
    g = bits(got, dtype)
    e = bits(exp, dtype)
    assert g.shape == e.shape, (what, g.shape, e.shape)
    if dtype in ("f32", "bf16") and op in ("sum", "prod"):
        en, gn = nan_mask(e, dtype), nan_mask(g, dtype)
        ok = (g == e) | (en & gn)
    else:
        ok = g == e
    if not ok.all():
        bad = np.flatnonzero(~ok)
        i = int(bad[0])
        raise AssertionError(f"{what}: {bad.size} of {g.size} elements differ; first at {i}: "
                             f"got {int(g[i]):#x} expected {int(e[i]):#x}")
