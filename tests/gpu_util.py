"""Helpers for the GPU parity tests: move numpy bit patterns to and from the
device through PyTorch, and compare results to the oracle element by element."""
from __future__ import annotations

import numpy as np

NP_BITS = {"f32": np.uint32, "bf16": np.uint16, "i32": np.uint32, "u32": np.uint32,
           "f16": np.uint16, "e4m3": np.uint8, "e5m2": np.uint8, "i64": np.uint64,
           "u64": np.uint64, "f64": np.uint64, "i8": np.uint8, "u8": np.uint8}


FLOATS = ("f32", "bf16", "f16", "e4m3", "e5m2", "f64")


def torch_dtype(dtype: str):
    """Storage dtype of a device tensor holding `dtype` elements (fp8 kept as
    uint8 bytes, 64-bit integers as int64; calls pass dtype= explicitly)."""
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16, "i32": torch.int32,
            "u32": torch.int32, "f16": torch.float16, "e4m3": torch.uint8,
            "e5m2": torch.uint8, "i64": torch.int64, "u64": torch.int64,
            "f64": torch.float64, "i8": torch.int8, "u8": torch.uint8}[dtype]


def to_dev(a: np.ndarray, dtype: str, device="cuda"):
    """Upload a numpy element array (bit patterns for bf16/f16/fp8) unchanged."""
    import torch
    a = np.ascontiguousarray(a)
    if dtype == "bf16":
        t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    elif dtype == "f16":
        t = torch.from_numpy(a.view(np.int16)).view(torch.float16)
    elif dtype == "f32":
        t = torch.from_numpy(a.astype(np.float32, copy=False))
    elif dtype in ("e4m3", "e5m2", "u8"):
        t = torch.from_numpy(a.view(np.uint8))
    elif dtype == "i8":
        t = torch.from_numpy(a.view(np.int8))
    elif dtype == "f64":
        t = torch.from_numpy(a.view(np.float64))
    elif dtype in ("i64", "u64"):
        t = torch.from_numpy(a.view(np.int64))
    else:
        t = torch.from_numpy(a.view(np.int32))
    return t.to(device)


def bits(t_or_a, dtype: str) -> np.ndarray:
    """Raw bit patterns of a tensor or numpy array of `dtype` elements."""
    import torch
    if isinstance(t_or_a, torch.Tensor):
        t = t_or_a.detach().cpu().contiguous()
        es = t.element_size()
        view = {1: torch.uint8, 2: torch.int16, 4: torch.int32, 8: torch.int64}[es]
        return t.view(view).numpy().view(NP_BITS[dtype])
    a = np.ascontiguousarray(t_or_a)
    return a.view(NP_BITS[dtype])


def nan_mask(b: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return ((b & 0x7F80) == 0x7F80) & ((b & 0x7F) != 0)
    if dtype == "f32":
        return ((b & 0x7F800000) == 0x7F800000) & ((b & 0x7FFFFF) != 0)
    if dtype == "f16":
        return ((b & 0x7C00) == 0x7C00) & ((b & 0x3FF) != 0)
    if dtype == "e5m2":
        return ((b & 0x7C) == 0x7C) & ((b & 0x3) != 0)
    if dtype == "e4m3":
        return (b & 0x7F) == 0x7F
    if dtype == "f64":
        return ((b & 0x7FF0000000000000) == 0x7FF0000000000000) & ((b & 0xFFFFFFFFFFFFF) != 0)
    return np.zeros(b.shape, bool)


def assert_parity(got, exp, dtype: str, op: str, what: str = "") -> None:
    """Bit-exact equality; for float sum/prod a NaN matches any NaN (payloads
    are not specified by the definition)."""
    g = bits(got, dtype)
    e = bits(exp, dtype)
    assert g.shape == e.shape, (what, g.shape, e.shape)
    if dtype in FLOATS and op in ("sum", "prod", "avg"):
        en, gn = nan_mask(e, dtype), nan_mask(g, dtype)
        ok = (g == e) | (en & gn)
    else:
        ok = g == e
    if not ok.all():
        bad = np.flatnonzero(~ok)
        i = int(bad[0])
        raise AssertionError(f"{what}: {bad.size} of {g.size} elements differ; first at {i}: "
                             f"got {int(g[i]):#x} expected {int(e[i]):#x}")
