"""The CPU oracle against what arithmetic fixes independently of it.

See tests/pins.py for what each pin checks and why it is independent.
"""
import os

import pytest

import pins


@pytest.mark.parametrize("pin", pins.FAST_PINS, ids=lambda f: f.__name__)
def test_pin(orc, pin):
    pin(orc)


def test_bruteforce_wide(orc):
    """More columns and larger P against the exact rational brute force."""
    pins.pin_bruteforce(orc, seed=101, ncols=64, nsrc_list=(4, 16, 33))


def test_narrow_formats_vs_torch_wide(orc):
    """fp16 / e4m3 / e5m2 conversions against PyTorch on 2 x 2^21 random patterns."""
    pins.pin_narrow_vs_torch(orc, n_random=1 << 21, seed=43)


def test_more_types_bruteforce_wide(orc):
    pins.pin_more_types_bruteforce(orc, seed=47, ncols=48, nsrc_list=(4, 16, 33))


def test_bf16_down_vs_torch(orc):
    """Every sign/exponent/high-mantissa half with each class of dropped bits,
    plus 2^20 random patterns, against PyTorch's CPU conversion."""
    pins.pin_bf16_vs_torch(orc)


@pytest.mark.skipif(not os.environ.get("XRED_EXHAUSTIVE"), reason="set XRED_EXHAUSTIVE=1")
def test_bf16_down_exhaustive(orc):
    """All 2^32 binary32 patterns (minutes; opt-in)."""
    import numpy as np
    import torch
    step = 1 << 26
    for start in range(0, 1 << 32, step):
        bits = np.arange(start, start + step, dtype=np.uint64).astype(np.uint32)
        got = orc.f32_bits_to_bf16(bits)
        exp = torch.from_numpy(bits.view(np.float32)).to(torch.bfloat16).view(torch.int16)
        exp = exp.numpy().view(np.uint16)
        nan_in = ((bits & 0x7F800000) == 0x7F800000) & ((bits & 0x7FFFFF) != 0)
        assert np.array_equal(got[~nan_in], exp[~nan_in]), start
        assert np.all((got[nan_in] & 0x7FFF) == 0x7FC0), start


def test_closed_form_at_scale(orc):
    """Integer-valued bf16 gradients at 2^22 elements x 8 sources: exact int64 sum."""
    pins.pin_integer_closed_form(orc, n=1 << 22, P=8, seed=21)


def test_multithreaded_identical(orc):
    """Splitting elements over threads leaves every element's fold unchanged."""
    import numpy as np
    import workloads
    w = workloads.WORKLOADS["c2"]
    srcs = workloads.sources(w, count=1 << 18)
    a = orc.allreduce_local(srcs, "bf16", "sum", nthreads=1)
    b = orc.allreduce_local(srcs, "bf16", "sum", nthreads=max(2, orc.max_threads()))
    assert np.array_equal(a, b)
