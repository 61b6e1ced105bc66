"""Checks that pin the CPU oracle to something other than itself.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises AssertionError
on a mismatch.  They are run against the real oracle (test_oracle_pins.py)
and against copies of it with planted mistakes (test_oracle_mutants.py),
which must each fail at least one pin.

What pins what:
  - exact rational brute force (tests/brute.py) on tiny random and special
    inputs, every dtype x op: single-rounding correctness and fold order;
  - hand-derived IEEE 754 closed forms (tests/golden/);
  - PyTorch's CPU binary32 -> bf16 conversion over every sign/exponent/
    high-mantissa pattern with each class of dropped bits;
  - closed forms at scale: integer-valued inputs make every binary32 partial
    sum exact, so the result is the int64 sum;
  - integer sums and products against numpy int64 modulo 2^32;
  - invariants: all-ones columns sum to P, a -0.0 buffer is the bitwise
    identity for sum, P=1 is a copy, max/min are permutation invariant,
    integer sums are permutation invariant, ReduceScatter shards concatenate
    to the AllReduce, the step-wise sequence equals the fused left fold, a
    batch equals its items.
"""
from __future__ import annotations

import json
from pathlib import Path

import numpy as np

import brute

GOLDEN = Path(__file__).resolve().parent / "golden"
NP = {"f32": np.float32, "bf16": np.uint16, "i32": np.int32, "u32": np.uint32,
      "f16": np.uint16, "e4m3": np.uint8, "e5m2": np.uint8, "i64": np.int64, "u64": np.uint64,
      "f64": np.float64, "i8": np.int8, "u8": np.uint8}
DTYPES = ("f32", "bf16", "i32", "u32")
OPS = ("sum", "prod", "max", "min")
# the further element types and AVG (float types only)
MORE_DTYPES = ("f16", "e4m3", "e5m2", "i64", "u64")
# the rest of the usual collective element types: binary64, 8-bit integers
WIDE_NARROW_DTYPES = ("f64", "i8", "u8")
FLOATS = ("f32", "bf16", "f16", "e4m3", "e5m2", "f64")


def ops_for(dtype: str):
    return OPS + ("avg",) if dtype in FLOATS else OPS

F32_SPECIALS = [
    0x00000000, 0x80000000, 0x7F800000, 0xFF800000, 0x7F7FFFFF, 0xFF7FFFFF,
    0x00000001, 0x80000001, 0x007FFFFF, 0x807FFFFF, 0x00800000, 0x80800000,
    0x3F800000, 0xBF800000, 0x3F800001, 0x33800000, 0x33800001, 0xB3800000,
    0x4B800000, 0x3F000000, 0x7FC00000, 0x7F800001, 0xFFC00000, 0x00400000,
]
BF16_SPECIALS = [
    0x0000, 0x8000, 0x7F80, 0xFF80, 0x7F7F, 0xFF7F, 0x0001, 0x8001, 0x007F, 0x0080,
    0x3F80, 0xBF80, 0x3F81, 0x3B80, 0x3B00, 0x4B80, 0x7FC0, 0x7F81, 0xFFC0, 0x3F00,
]


def _bits(a: np.ndarray) -> np.ndarray:
    return a.view({1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}[a.dtype.itemsize])


def _is_nan_bits(b: int, dtype: str) -> bool:
    if dtype == "bf16":
        return (b & 0x7F80) == 0x7F80 and (b & 0x7F) != 0
    if dtype == "f32":
        return brute.is_nan32(b)
    if dtype == "f16":
        return (b & 0x7C00) == 0x7C00 and (b & 0x3FF) != 0
    if dtype == "e5m2":
        return (b & 0x7C) == 0x7C and (b & 0x3) != 0
    if dtype == "e4m3":
        return (b & 0x7F) == 0x7F
    if dtype == "f64":
        return brute.is_nan64(b)
    return False


def _same(got: int, exp: int, dtype: str, op: str) -> bool:
    """Bitwise equality, except that NaN payloads of sum/prod/avg are unpinned."""
    if dtype in FLOATS and op in ("sum", "prod", "avg") and _is_nan_bits(exp, dtype):
        return _is_nan_bits(got, dtype)
    return got == exp


def random_column_values(rng, dtype: str, n: int) -> np.ndarray:
    """Random bit patterns mixing specials, random bits and nearby magnitudes."""
    if dtype == "f32":
        pool = np.array(F32_SPECIALS, np.uint32)
        rb = rng.integers(0, 2**32, size=n, dtype=np.uint64).astype(np.uint32)
        near = (rng.standard_normal(n).astype(np.float32)).view(np.uint32)
        tiny = rng.integers(0, 1 << 24, size=n, dtype=np.uint32)   # subnormal / tiny normal
        pick = rng.integers(0, 4, size=n)
        out = np.where(pick == 0, pool[rng.integers(0, pool.size, n)],
                       np.where(pick == 1, rb, np.where(pick == 2, near, tiny)))
        return out.astype(np.uint32).view(np.float32)
    if dtype == "bf16":
        pool = np.array(BF16_SPECIALS, np.uint16)
        rb = rng.integers(0, 2**16, size=n, dtype=np.uint32).astype(np.uint16)
        near = (rng.standard_normal(n).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        tiny = rng.integers(0, 0x0100, size=n, dtype=np.uint32).astype(np.uint16)
        pick = rng.integers(0, 4, size=n)
        return np.where(pick == 0, pool[rng.integers(0, pool.size, n)],
                        np.where(pick == 1, rb, np.where(pick == 2, near, tiny))).astype(np.uint16)
    if dtype == "f16":
        pool = np.array([0x0000, 0x8000, 0x7C00, 0xFC00, 0x7BFF, 0xFBFF, 0x0001, 0x8001, 0x03FF,
                         0x0400, 0x3C00, 0xBC00, 0x3C01, 0x1400, 0x7E00, 0x7C01, 0x3800], np.uint16)
        rb = rng.integers(0, 2**16, size=n, dtype=np.uint32).astype(np.uint16)
        near = rng.standard_normal(n).astype(np.float16).view(np.uint16)
        tiny = rng.integers(0, 0x0800, size=n, dtype=np.uint32).astype(np.uint16)
        pick = rng.integers(0, 4, size=n)
        return np.where(pick == 0, pool[rng.integers(0, pool.size, n)],
                        np.where(pick == 1, rb, np.where(pick == 2, near, tiny))).astype(np.uint16)
    if dtype in ("e4m3", "e5m2"):
        # every byte is a value; weight small magnitudes so sums stay in range
        rb = rng.integers(0, 256, size=n, dtype=np.uint32).astype(np.uint8)
        mid = (rng.integers(0x20, 0x48, size=n, dtype=np.uint32).astype(np.uint8)
               | (rng.integers(0, 2, size=n, dtype=np.uint32).astype(np.uint8) << 7))
        return np.where(rng.integers(0, 2, size=n) == 0, rb, mid).astype(np.uint8)
    if dtype == "f64":
        pool = np.array([0x0, 0x8000000000000000, 0x7FF0000000000000, 0xFFF0000000000000,
                         0x7FEFFFFFFFFFFFFF, 0xFFEFFFFFFFFFFFFF, 0x1, 0x8000000000000001,
                         0x000FFFFFFFFFFFFF, 0x0010000000000000, 0x3FF0000000000000,
                         0xBFF0000000000000, 0x3FF0000000000001, 0x3CA0000000000000,
                         0x3CA0000000000001, 0x7FF8000000000000, 0x7FF0000000000001,
                         0xFFF8000000000000, 0x4330000000000000], np.uint64)
        rb = rng.integers(0, 2**64, size=n, dtype=np.uint64)
        near = rng.standard_normal(n).view(np.uint64)
        tiny = rng.integers(0, 1 << 53, size=n, dtype=np.uint64)
        pick = rng.integers(0, 4, size=n)
        out = np.where(pick == 0, pool[rng.integers(0, pool.size, n)],
                       np.where(pick == 1, rb, np.where(pick == 2, near, tiny)))
        return out.astype(np.uint64).view(np.float64)
    if dtype in ("i8", "u8"):
        sp = np.array([0, 1, 0xFF, 0x7F, 0x80, 2, 0x10], np.uint8)
        rb = rng.integers(0, 256, size=n, dtype=np.uint32).astype(np.uint8)
        small = rng.integers(0, 8, size=n, dtype=np.uint32).astype(np.uint8)
        pick = rng.integers(0, 3, size=n)
        out = np.where(pick == 0, sp[rng.integers(0, sp.size, n)],
                       np.where(pick == 1, rb, small)).astype(np.uint8)
        return out.view(np.int8) if dtype == "i8" else out
    if dtype in ("i64", "u64"):
        sp = np.array([0, 1, 2**64 - 1, 2**63 - 1, 2**63, 2, 2**32, 2**32 - 1], np.uint64)
        rb = rng.integers(0, 2**64, size=n, dtype=np.uint64)
        small = rng.integers(0, 8, size=n, dtype=np.uint64)
        pick = rng.integers(0, 3, size=n)
        out = np.where(pick == 0, sp[rng.integers(0, sp.size, n)],
                       np.where(pick == 1, rb, small)).astype(np.uint64)
        return out.view(np.int64) if dtype == "i64" else out
    specials = np.array([0, 1, 0xFFFFFFFF, 0x7FFFFFFF, 0x80000000, 2, 0x10000], np.uint32)
    rb = rng.integers(0, 2**32, size=n, dtype=np.uint64).astype(np.uint32)
    small = rng.integers(0, 8, size=n, dtype=np.uint32)
    pick = rng.integers(0, 3, size=n)
    out = np.where(pick == 0, specials[rng.integers(0, specials.size, n)],
                   np.where(pick == 1, rb, small)).astype(np.uint32)
    return out.view(np.int32) if dtype == "i32" else out


def pin_bruteforce(orc, seed: int = 7, ncols: int = 48, nsrc_list=(1, 2, 3, 5, 8)) -> None:
    """Oracle == exact rational brute force, every dtype x op, tiny inputs."""
    rng = np.random.default_rng(seed)
    for dtype in DTYPES:
        for op in OPS:
            for P in nsrc_list:
                srcs = [random_column_values(rng, dtype, ncols) for _ in range(P)]
                got = _bits(orc.allreduce_local(srcs, dtype, op))
                sb = [_bits(s) for s in srcs]
                for i in range(ncols):
                    col = [int(s[i]) for s in sb]
                    exp = brute.reduce_column(col, dtype, op)
                    assert _same(int(got[i]), exp, dtype, op), (
                        f"{dtype} {op} P={P} col={[hex(c) for c in col]} "
                        f"got={int(got[i]):#x} exp={exp:#x}")


def pin_golden_reduce(orc) -> None:
    """Oracle == hand-derived IEEE 754 closed forms (tests/golden/reduce_cases.json)."""
    cases = json.loads((GOLDEN / "reduce_cases.json").read_text())
    for c in cases:
        dtype, op = c["dtype"], c["op"]
        srcs = [np.array([int(h, 16)], np.uint16 if dtype == "bf16" else np.uint32)
                .view(NP[dtype]) for h in c["column"]]
        got = int(_bits(orc.allreduce_local(srcs, dtype, op))[0])
        if c["expect"] == "NAN":
            assert _is_nan_bits(got, dtype), f"{c}: got {got:#x}"
        else:
            assert got == int(c["expect"], 16), f"{c}: got {got:#x}"


def pin_golden_bf16(orc) -> None:
    """down() == hand-derived roundTiesToEven cases (tests/golden/bf16_rne_cases.txt)."""
    ins, exps = [], []
    for line in (GOLDEN / "bf16_rne_cases.txt").read_text().splitlines():
        if not line.strip() or line.startswith("#"):
            continue
        f, b = line.split()[:2]
        ins.append(int(f, 16))
        exps.append(int(b, 16))
    got = orc.f32_bits_to_bf16(np.array(ins, np.uint32))
    for x, g, e in zip(ins, got, exps):
        assert int(g) == e, f"{x:#010x}: got {int(g):#06x} expected {e:#06x}"


def _golden_rows(name):
    for line in (GOLDEN / name).read_text().splitlines():
        if line.strip() and not line.startswith("#"):
            yield line.split()[:3]


def pin_golden_narrow(orc) -> None:
    """fp16 / fp8 down() and up() == the cases the formats' definitions fix
    (tests/golden/narrow_cases.txt, tests/golden/widen_cases.txt)."""
    rows = list(_golden_rows("narrow_cases.txt"))
    for dt in ("f16", "e4m3", "e5m2"):
        mine = [(int(f, 16), int(b, 16)) for d, f, b in rows if d == dt]
        got = orc.f32_bits_to_small(np.array([f for f, _ in mine], np.uint32), dt)
        for (f, e), g in zip(mine, got.tolist()):
            assert g == e, f"{dt} down({f:#010x}): got {g:#x} expected {e:#x}"
    rows = list(_golden_rows("widen_cases.txt"))
    for dt in ("f16", "e4m3", "e5m2"):
        mine = [(int(b, 16), w) for d, b, w in rows if d == dt]
        got = orc.small_to_f32_bits(np.array([b for b, _ in mine]), dt)
        for (b, e), g in zip(mine, got.tolist()):
            if e == "nan":
                ok = (g & 0x7F800000) == 0x7F800000 and (g & 0x7FFFFF) != 0
            else:
                ok = g == int(e, 16)
            assert ok, f"{dt} up({b:#x}): got {g:#010x} expected {e}"


def pin_bf16_vs_brute(orc, seed: int = 3, n: int = 4000) -> None:
    """down() == exact rational rounding on random and boundary patterns."""
    rng = np.random.default_rng(seed)
    hi = rng.integers(0, 1 << 16, size=n, dtype=np.uint32)
    lo = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], np.uint32)[rng.integers(0, 6, n)]
    bits = (hi << 16) | lo
    got = orc.f32_bits_to_bf16(bits)
    for b, g in zip(bits.tolist(), got.tolist()):
        e = brute.f32_to_bf16(b)
        assert g == e, f"{b:#010x}: got {g:#06x} expected {e:#06x}"


def pin_bf16_vs_torch(orc, lows=(0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF), extra_random=1 << 20,
                      seed: int = 11) -> None:
    """down() == PyTorch CPU float32 -> bfloat16 for every high half and each class of
    dropped bits, plus a random sample; NaNs compared by class only."""
    import torch
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    parts = [hi | np.uint32(l) for l in lows]
    if extra_random:
        parts.append(np.random.default_rng(seed).integers(0, 2**32, size=extra_random,
                                                          dtype=np.uint64).astype(np.uint32))
    bits = np.concatenate(parts)
    got = orc.f32_bits_to_bf16(bits)
    exp = torch.from_numpy(bits.view(np.float32)).to(torch.bfloat16).view(torch.int16)
    exp = exp.numpy().view(np.uint16)
    nan_in = ((bits & 0x7F800000) == 0x7F800000) & ((bits & 0x7FFFFF) != 0)
    got_nan = ((got & 0x7F80) == 0x7F80) & ((got & 0x7F) != 0)
    assert np.array_equal(got_nan, nan_in), "NaN class differs"
    ok = nan_in | (got == exp)
    if not ok.all():
        i = int(np.flatnonzero(~ok)[0])
        raise AssertionError(f"{int(bits[i]):#010x}: got {int(got[i]):#06x} torch {int(exp[i]):#06x}")


def pin_up_bf16(orc) -> None:
    """up() of every bf16 pattern is the exact binary32 whose top half it is."""
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = orc.bf16_to_f32_bits(h)
    assert np.array_equal(got, h.astype(np.uint32) << 16)


def pin_integer_closed_form(orc, n: int = 1 << 16, P: int = 8, seed: int = 5) -> None:
    """Integer-valued inputs in [-128,128]: every partial sum is exact in binary32,
    so the result equals the int64 sum (bf16 output: PyTorch's rounding of it)."""
    import torch
    rng = np.random.default_rng(seed)
    ints = [rng.integers(-128, 129, size=n) for _ in range(P)]
    exact = np.sum(np.stack(ints), axis=0)
    srcs32 = [x.astype(np.float32) for x in ints]
    got32 = orc.allreduce_local(srcs32, "f32", "sum")
    assert np.array_equal(got32, exact.astype(np.float32)), "f32 integer closed form"
    srcs16 = [torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16)
              .numpy().view(np.uint16) for x in ints]
    got16 = orc.allreduce_local(srcs16, "bf16", "sum")
    exp16 = torch.from_numpy(exact.astype(np.float32)).to(torch.bfloat16).view(torch.int16)
    assert np.array_equal(got16, exp16.numpy().view(np.uint16)), "bf16 integer closed form"
    prod_src = [rng.integers(-2, 3, size=n).astype(np.float32) for _ in range(P)]
    exp_prod = np.prod(np.stack(prod_src).astype(np.int64), axis=0).astype(np.float32)
    assert np.array_equal(orc.allreduce_local(prod_src, "f32", "prod"), exp_prod)


def pin_int_mod32(orc, n: int = 1 << 14, P: int = 32, seed: int = 9) -> None:
    """int32/uint32 sum and product == numpy int64 arithmetic reduced modulo 2^32;
    max/min == numpy's signed/unsigned extrema."""
    rng = np.random.default_rng(seed)
    raw = [rng.integers(0, 2**32, size=n, dtype=np.uint64) for _ in range(P)]
    u = [r.astype(np.uint32) for r in raw]
    i = [x.view(np.int32) for x in u]
    mask = np.uint64(0xFFFFFFFF)
    s = np.zeros(n, np.uint64)
    pr = np.ones(n, np.uint64)
    for r in raw:
        s = (s + r) & mask
        pr = (pr * r) & mask     # exact: both factors < 2^32, product < 2^64
    for dt, srcs in (("i32", i), ("u32", u)):
        assert np.array_equal(_bits(orc.allreduce_local(srcs, dt, "sum")), s.astype(np.uint32))
        assert np.array_equal(_bits(orc.allreduce_local(srcs, dt, "prod")), pr.astype(np.uint32))
    st = np.stack(i)
    assert np.array_equal(orc.allreduce_local(i, "i32", "max"), st.max(axis=0))
    assert np.array_equal(orc.allreduce_local(i, "i32", "min"), st.min(axis=0))
    ut = np.stack(u)
    assert np.array_equal(orc.allreduce_local(u, "u32", "max"), ut.max(axis=0))
    assert np.array_equal(orc.allreduce_local(u, "u32", "min"), ut.min(axis=0))


def pin_invariants(orc, n: int = 4099, seed: int = 13) -> None:
    """All-ones -> P; -0 buffer identity; P=1 copy; permutation invariance of
    max/min and integer sum."""
    rng = np.random.default_rng(seed)
    for P in (1, 2, 7, 64):
        ones32 = [np.ones(n, np.float32)] * P
        assert np.all(orc.allreduce_local(ones32, "f32", "sum") == np.float32(P))
        ones16 = [np.full(n, 0x3F80, np.uint16)] * P
        got = orc.allreduce_local(ones16, "bf16", "sum")
        assert np.all(got.astype(np.uint32) << 16 == np.float32(P).view(np.uint32)), P
    # -0.0 is the bitwise identity for sum (keeps -0 elements as -0)
    x = random_column_values(rng, "f32", n)
    x[::5] = np.float32(-0.0)
    nz = np.full(n, -0.0, np.float32)
    for srcs in ([x, nz], [nz, x], [x, nz, nz]):
        got = _bits(orc.allreduce_local(srcs, "f32", "sum"))
        xb = _bits(x)
        nan = ((xb & 0x7F800000) == 0x7F800000) & ((xb & 0x7FFFFF) != 0)
        assert np.array_equal(got[~nan], xb[~nan])
    # +0.0 is the identity by value, and turns -0 into +0
    pz = np.zeros(n, np.float32)
    got = _bits(orc.allreduce_local([x, pz], "f32", "sum"))
    negz = _bits(x) == 0x80000000
    assert np.all(got[negz] == 0)
    # P = 1 is a copy of the source (non-NaN), in every dtype
    for dt in DTYPES:
        s = random_column_values(rng, dt, n)
        sb = _bits(s)
        for op in OPS:
            got = _bits(orc.allreduce_local([s], dt, op))
            if dt in ("f32", "bf16"):
                nan = np.array([_is_nan_bits(int(v), dt) for v in sb])
                assert np.array_equal(got[~nan], sb[~nan]), (dt, op)
            else:
                assert np.array_equal(got, sb), (dt, op)
    # max/min over a random permutation of sources: identical bits
    for dt in ("f32", "bf16", "i32", "u32"):
        srcs = [random_column_values(rng, dt, n) for _ in range(9)]
        perm = [srcs[j] for j in rng.permutation(9)]
        for op in ("max", "min"):
            a = _bits(orc.allreduce_local(srcs, dt, op))
            b = _bits(orc.allreduce_local(perm, dt, op))
            assert np.array_equal(a, b), (dt, op)
        if dt in ("i32", "u32"):
            for op in ("sum", "prod"):
                assert np.array_equal(_bits(orc.allreduce_local(srcs, dt, op)),
                                      _bits(orc.allreduce_local(perm, dt, op)))


def pin_composition(orc, seed: int = 17) -> None:
    """ReduceScatter shards concatenate to the AllReduce; the step-wise sequence
    equals the fused left fold; a batch equals its items."""
    rng = np.random.default_rng(seed)
    for dt in DTYPES:
        for op in OPS:
            P, rc = 5, 37
            srcs = [random_column_values(rng, dt, P * rc) for _ in range(P)]
            full = _bits(orc.allreduce_local(srcs, dt, op))
            for r in range(P):
                sh = _bits(orc.reduce_scatter_local(srcs, r, dt, op))
                exp = full[r * rc:(r + 1) * rc]
                if dt in ("f32", "bf16") and op in ("sum", "prod"):
                    both_nan = np.array([_is_nan_bits(int(a), dt) and _is_nan_bits(int(b), dt)
                                         for a, b in zip(sh, exp)], bool)
                    assert np.array_equal(sh[~both_nan], exp[~both_nan]), (dt, op, r)
                else:
                    assert np.array_equal(sh, exp), (dt, op, r)
            # step-wise: INIT with chunk 0, add chunks 1..P-2, FINAL with chunk P-1;
            # and INIT + adds + acc_cast; both equal the fused fold over the P chunks
            chunks = [random_column_values(rng, dt, 53) for _ in range(P)]
            fused = _bits(orc.allreduce_local(chunks, dt, op))
            acc = orc.reduce_copy_step(chunks[0], None, dt, op, init=True)
            for c in chunks[1:-1]:
                acc = orc.reduce_copy_step(c, acc, dt, op)
            acc_copy = acc.copy()
            fin = _bits(orc.reduce_copy_step(chunks[-1], acc, dt, op, final=True))
            assert np.array_equal(_bits(acc), _bits(acc_copy)), "FINAL must not write acc"
            acc2 = orc.reduce_copy_step(chunks[-1], acc_copy, dt, op)
            cast = _bits(orc.acc_cast(acc2, dt))
            for got in (fin, cast):
                if dt in ("f32", "bf16") and op in ("sum", "prod"):
                    mask = np.array([not (_is_nan_bits(int(a), dt) and _is_nan_bits(int(b), dt))
                                     for a, b in zip(got, fused)], bool)
                    assert np.array_equal(got[mask], fused[mask]), (dt, op)
                else:
                    assert np.array_equal(got, fused), (dt, op)
            one = _bits(orc.reduce_copy_step(chunks[0], None, dt, op, init=True, final=True))
            assert np.array_equal(one, _bits(orc.allreduce_local([chunks[0]], dt, op)))
    # batch == items
    items = []
    for k in range(6):
        P = int(rng.integers(1, 9))
        n = int(rng.integers(1, 300))
        items.append([random_column_values(rng, "bf16", n) for _ in range(P)])
    outs = orc.batched_reduce(items, "bf16", "sum")
    for srcs, out in zip(items, outs):
        exp = orc.allreduce_local(srcs, "bf16", "sum")
        nan = np.array([_is_nan_bits(int(v), "bf16") for v in exp], bool)
        assert np.array_equal(out[~nan], exp[~nan])


# ------------------------------------------------ simulated schedules --

def sim_chunk_len(count: int, nranks: int) -> int:
    """The schedules' chunk length: ceil(count / G) rounded up to 64 elements."""
    m = -(-count // nranks)
    return -(-m // 64) * 64


def brute_ring_element(col, c: int, dtype: str, op: str) -> int:
    """One element of chunk c after a ring AllReduce over len(col) ranks: the
    partial starts as rank c+1's value and travels c+2, ..., c+G-1, c, each hop
    being a two-source reduce (received, own) rounded to the I/O dtype."""
    G = len(col)
    if G == 1:
        return col[0]
    v = col[(c + 1) % G]
    for j in range(2, G + 1):
        v = brute.reduce_column([v, col[(c + j) % G]], dtype, op)
    return v


def brute_rhd_element(col, b: int, dtype: str, op: str) -> int:
    """One element of block b after recursive halving: at distance d every
    rank combines its partner's value (received) with its own; block b ends at
    rank b."""
    G = len(col)
    w = list(col)
    d = G // 2
    while d >= 1:
        w = [brute.reduce_column([w[r ^ d], w[r]], dtype, op) for r in range(G)]
        d //= 2
    return w[b]


def pin_sim_bruteforce(orc, seed: int = 23, per_case: int = 12) -> None:
    """Every rank's output of the simulated ring / halving-doubling AllReduce
    equals the exact rational chain of hops, element by element, on ragged
    sizes whose trailing chunks are short or empty; all ranks hold the same bits."""
    rng = np.random.default_rng(seed)
    for algo, sizes, brute_el in (("ring", (1, 2, 3, 5, 8), brute_ring_element),
                                  ("rhd", (1, 2, 4, 8), brute_rhd_element)):
        for dtype in DTYPES:
            for op in OPS:
                for G in sizes:
                    n = 64 * G + 70 if G > 1 else 37
                    sends = [random_column_values(rng, dtype, n) for _ in range(G)]
                    outs = [_bits(o) for o in orc.allreduce_sim(sends, dtype, op, algo)]
                    for r in range(1, G):
                        assert np.array_equal(outs[r], outs[0]), f"{algo} G={G}: ranks differ"
                    M = sim_chunk_len(n, G)
                    idx = {0, n - 1} | {min(n - 1, k * M + e) for k in range(1, G) for e in (-1, 0)}
                    idx |= set(rng.integers(0, n, per_case).tolist())
                    sb = [_bits(s) for s in sends]
                    for i in sorted(idx):
                        col = [int(x[i]) for x in sb]
                        exp = brute_el(col, i // M, dtype, op)
                        assert _same(int(outs[0][i]), exp, dtype, op), (
                            f"{algo} {dtype} {op} G={G} i={i} got={int(outs[0][i]):#x} exp={exp:#x}")


def pin_sim_closed_forms(orc, n: int = 5003, seed: int = 29) -> None:
    """Closed forms and invariants of the simulated schedules: integer-valued
    inputs whose every partial is exact give the int64 sum at every rank
    (bf16 too, as |partials| <= 128 are exact there); int32 sums wrap to the
    numpy int64 sum mod 2^32; max/min equal the order-free fused reduce; one
    rank copies its buffer bit for bit; with two ranks the ring and the
    halving-doubling schedules perform the same single hop per element."""
    import torch
    rng = np.random.default_rng(seed)
    for algo, G in (("ring", 8), ("ring", 7), ("rhd", 8)):
        ints = [rng.integers(-16, 17, size=n) for _ in range(G)]
        exact = np.sum(np.stack(ints), axis=0)
        f32 = orc.allreduce_sim([x.astype(np.float32) for x in ints], "f32", "sum", algo)
        bf = orc.allreduce_sim([torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16)
                                .view(torch.int16).numpy().view(np.uint16) for x in ints],
                               "bf16", "sum", algo)
        exp16 = torch.from_numpy(exact.astype(np.float32)).to(torch.bfloat16).view(torch.int16)
        for r in range(G):
            assert np.array_equal(f32[r], exact.astype(np.float32)), f"{algo} f32 closed form"
            assert np.array_equal(bf[r], exp16.numpy().view(np.uint16)), f"{algo} bf16 closed form"
        wide = [rng.integers(-2**31, 2**31, size=n).astype(np.int32) for _ in range(G)]
        wsum = (np.sum(np.stack(wide).astype(np.int64), axis=0) & 0xFFFFFFFF).astype(np.uint32)
        for o in orc.allreduce_sim(wide, "i32", "sum", algo):
            assert np.array_equal(o.view(np.uint32), wsum), f"{algo} int32 wrap"
        for op in ("max", "min"):
            vals = [random_column_values(rng, "f32", n) for _ in range(G)]
            fused = _bits(orc.allreduce_local(vals, "f32", op))
            for o in orc.allreduce_sim(vals, "f32", op, algo):
                assert np.array_equal(_bits(o), fused), f"{algo} {op} order-free"
    one = random_column_values(rng, "bf16", 1000)
    one[:4] = [0x7F81, 0xFF81, 0x8000, 0x0001]           # NaN payloads and -0 survive a copy
    for algo in ("ring", "rhd"):
        assert np.array_equal(orc.allreduce_sim([one], "bf16", "sum", algo)[0], one)
    two = [random_column_values(rng, "bf16", 777) for _ in range(2)]
    a = orc.allreduce_sim(two, "bf16", "sum", "ring")
    b = orc.allreduce_sim(two, "bf16", "sum", "rhd")
    for x, y in zip(a, b):
        nan = np.array([_is_nan_bits(int(v), "bf16") for v in x], bool)
        assert np.array_equal(x[~nan], y[~nan]) and np.all(
            [_is_nan_bits(int(v), "bf16") for v in y[nan]]), "G=2 ring vs rhd"


# ------------------------------------------- further types and AVG --

def pin_more_types_bruteforce(orc, seed: int = 31, ncols: int = 32,
                              nsrc_list=(1, 2, 3, 5, 8)) -> None:
    """fp16, fp8 e4m3/e5m2, int64, uint64 with every op, and AVG on every float
    type, against the exact rational brute force."""
    rng = np.random.default_rng(seed)
    cases = [(d, o) for d in MORE_DTYPES for o in ops_for(d)] + [("f32", "avg"), ("bf16", "avg")]
    for dtype, op in cases:
        for P in nsrc_list:
            srcs = [random_column_values(rng, dtype, ncols) for _ in range(P)]
            got = _bits(orc.allreduce_local(srcs, dtype, op))
            sb = [_bits(s) for s in srcs]
            for i in range(ncols):
                col = [int(s[i]) for s in sb]
                exp = brute.reduce_column(col, dtype, op)
                assert _same(int(got[i]), exp, dtype, op), (
                    f"{dtype} {op} P={P} col={[hex(c) for c in col]} "
                    f"got={int(got[i]):#x} exp={exp:#x}")


def pin_narrow_vs_torch(orc, n_random: int = 1 << 16, seed: int = 37) -> None:
    """Widening of every f16 / e4m3 / e5m2 pattern and narrowing of random and
    boundary binary32 patterns against PyTorch's CPU conversions.  They agree
    everywhere except e4m3 overflow, where PyTorch gives NaN and the definition
    saturates at +-448 (checked separately: every |x| >= 448 gives 448)."""
    import torch
    tt = {"f16": torch.float16, "e4m3": torch.float8_e4m3fn, "e5m2": torch.float8_e5m2}
    rng = np.random.default_rng(seed)
    bits = np.concatenate([
        rng.integers(0, 2**32, n_random, dtype=np.uint64).astype(np.uint32),
        rng.integers(0x30000000, 0x48000000, n_random, dtype=np.uint64).astype(np.uint32),
        np.arange(0, 1 << 16, dtype=np.uint32) << 16 | 0x8000,      # exact ties
        np.arange(0, 1 << 16, dtype=np.uint32) << 16]).astype(np.uint32)
    f = bits.view(np.float32)
    for dt, t in tt.items():
        itemsize = 2 if dt == "f16" else 1
        pats = np.arange(1 << (8 * itemsize), dtype=np.uint64).astype(NP[dt])
        wide = orc.small_to_f32_bits(pats, dt)
        ref = torch.from_numpy(pats.view(np.int16) if itemsize == 2 else pats).view(t)
        ref = ref.float().numpy().view(np.uint32)
        nan = np.isnan(ref.view(np.float32))
        assert np.array_equal(np.isnan(wide.view(np.float32)), nan), f"{dt} widening NaN set"
        assert np.array_equal(wide[~nan], ref[~nan]), f"{dt} widening"
        got = orc.f32_bits_to_small(bits, dt)
        tr = torch.from_numpy(f.copy()).to(t)
        exp = (tr.view(torch.int16).numpy().view(np.uint16) if itemsize == 2
               else tr.view(torch.uint8).numpy())
        keep = ~np.isnan(f)
        if dt == "e4m3":
            over = np.abs(f) >= 448.0
            assert np.all(got[over & keep] == np.where(np.signbit(f[over & keep]), 0xFE, 0x7E)), \
                "e4m3 saturation"
            keep &= ~over
        assert np.array_equal(got[keep], exp[keep]), f"{dt} narrowing"
        gn = got[np.isnan(f)]
        assert all(_is_nan_bits(int(v), dt) for v in gn), f"{dt} NaN stays NaN"


def pin_more_types_closed_forms(orc, n: int = 1 << 15, seed: int = 41) -> None:
    """AVG of integer-valued inputs over a power-of-two P is the exact mean;
    fp8 and fp16 sums of small integers are exact before the final rounding,
    so they equal PyTorch's conversion of the int64 sum; int64/uint64 sums
    and products wrap like numpy's 64-bit arithmetic; max/min are permutation
    invariant."""
    import torch
    rng = np.random.default_rng(seed)
    for P in (2, 4, 8):
        ints = [rng.integers(-64, 65, size=n) for _ in range(P)]
        tot = np.sum(np.stack(ints), axis=0)
        got = orc.allreduce_local([x.astype(np.float32) for x in ints], "f32", "avg")
        assert np.array_equal(got, (tot / P).astype(np.float32)), f"avg closed form P={P}"
    for dt, t in (("f16", torch.float16), ("e4m3", torch.float8_e4m3fn),
                  ("e5m2", torch.float8_e5m2)):
        ints = [rng.integers(-8, 9, size=n) for _ in range(8)]
        srcs = []
        for x in ints:
            tx = torch.from_numpy(x.astype(np.float32)).to(t)
            srcs.append(tx.view(torch.int16).numpy().view(np.uint16) if dt == "f16"
                        else tx.view(torch.uint8).numpy())
        tot = torch.from_numpy(np.sum(np.stack(ints), axis=0).astype(np.float32)).to(t)
        exp = (tot.view(torch.int16).numpy().view(np.uint16) if dt == "f16"
               else tot.view(torch.uint8).numpy())
        assert np.array_equal(orc.allreduce_local(srcs, dt, "sum"), exp), f"{dt} integer sums"
    a = [rng.integers(-2**63, 2**63, size=n, dtype=np.int64) for _ in range(5)]
    with np.errstate(over="ignore"):
        assert np.array_equal(orc.allreduce_local(a, "i64", "sum"), np.sum(np.stack(a), axis=0))
        assert np.array_equal(orc.allreduce_local(a, "i64", "prod"), np.prod(np.stack(a), axis=0))
        u = [x.view(np.uint64) for x in a]
        assert np.array_equal(orc.allreduce_local(u, "u64", "sum"), np.sum(np.stack(u), axis=0))
    assert np.array_equal(orc.allreduce_local(a, "i64", "max"), np.max(np.stack(a), axis=0))
    assert np.array_equal(orc.allreduce_local([x.view(np.uint64) for x in a], "u64", "min"),
                          np.min(np.stack([x.view(np.uint64) for x in a]), axis=0))
    for dt in ("f16", "e4m3", "e5m2"):
        srcs = [random_column_values(rng, dt, 4096) for _ in range(6)]
        for op in ("max", "min"):
            ref = orc.allreduce_local(srcs, dt, op)
            perm = [srcs[k] for k in rng.permutation(6)]
            assert np.array_equal(orc.allreduce_local(perm, dt, op), ref), f"{dt} {op} order"


# ------------------------------------------- binary64 and 8-bit integers --

def pin_wide_narrow_bruteforce(orc, seed: int = 61, ncols: int = 32,
                               nsrc_list=(1, 2, 3, 5, 8)) -> None:
    """fp64 (exact rational arithmetic rounded to binary64) and int8 / uint8
    (byte arithmetic modulo 2^8, compared signed or unsigned on the bytes:
    not the oracle's widen-then-truncate route) with every op, AVG on fp64."""
    rng = np.random.default_rng(seed)
    for dtype in WIDE_NARROW_DTYPES:
        for op in ops_for(dtype):
            for P in nsrc_list:
                srcs = [random_column_values(rng, dtype, ncols) for _ in range(P)]
                got = _bits(orc.allreduce_local(srcs, dtype, op))
                sb = [_bits(s) for s in srcs]
                for i in range(ncols):
                    col = [int(s[i]) for s in sb]
                    exp = brute.reduce_column(col, dtype, op)
                    assert _same(int(got[i]), exp, dtype, op), (
                        f"{dtype} {op} P={P} col={[hex(c) for c in col]} "
                        f"got={int(got[i]):#x} exp={exp:#x}")


def pin_wide_narrow_closed_forms(orc, n: int = 1 << 15, seed: int = 67) -> None:
    """fp64 sums and products of integer-valued inputs are exact below 2^53,
    so they equal numpy's int64 results; AVG over a power-of-two P is the exact
    mean; fp64 max/min of finite nonzero values equal numpy's; int8 / uint8
    sums and products equal numpy's own 8-bit wrapping arithmetic, max/min
    numpy's; the step-wise sequence (INIT, adds, FINAL or the closing cast)
    equals the fused fold; ReduceScatter shards concatenate to the AllReduce;
    max/min are permutation invariant."""
    rng = np.random.default_rng(seed)
    ints = [rng.integers(-1000, 1001, size=n) for _ in range(8)]
    f = [x.astype(np.float64) for x in ints]
    tot = np.sum(np.stack(ints), axis=0)
    assert np.array_equal(orc.allreduce_local(f, "f64", "sum"), tot.astype(np.float64))
    small = [rng.integers(-9, 10, size=n) for _ in range(6)]
    prod = np.prod(np.stack(small), axis=0)
    assert np.array_equal(orc.allreduce_local([x.astype(np.float64) for x in small], "f64",
                                              "prod"), prod.astype(np.float64))
    for P in (2, 4, 8):
        got = orc.allreduce_local(f[:P], "f64", "avg")
        assert np.array_equal(got, np.sum(np.stack(ints[:P]), axis=0) / P), f"f64 avg P={P}"
    # signed zeros in every order: the total order puts -0 below +0
    pz, nz = np.zeros(4, np.float64), np.full(4, -0.0)
    for srcs in ([pz, nz], [nz, pz], [pz, pz, nz], [nz, pz, pz], [pz, nz, pz]):
        hi = _bits(orc.allreduce_local(srcs, "f64", "max"))
        lo = _bits(orc.allreduce_local(srcs, "f64", "min"))
        assert np.all(hi == 0) and np.all(lo == 0x8000000000000000), "f64 max/min of +-0"
    g = [rng.standard_normal(n) + 0.5 for _ in range(7)]
    assert np.array_equal(orc.allreduce_local(g, "f64", "max"), np.max(np.stack(g), axis=0))
    assert np.array_equal(orc.allreduce_local(g, "f64", "min"), np.min(np.stack(g), axis=0))
    for dt, t in (("i8", np.int8), ("u8", np.uint8)):
        a = [random_column_values(rng, dt, n) for _ in range(9)]
        st = np.stack(a)
        assert np.array_equal(orc.allreduce_local(a, dt, "sum"), np.sum(st, axis=0, dtype=t))
        assert np.array_equal(orc.allreduce_local(a, dt, "prod"), np.prod(st, axis=0, dtype=t))
        assert np.array_equal(orc.allreduce_local(a, dt, "max"), np.max(st, axis=0))
        assert np.array_equal(orc.allreduce_local(a, dt, "min"), np.min(st, axis=0))
    for dt in WIDE_NARROW_DTYPES:
        for op in OPS:
            P, rc = 5, 41
            srcs = [random_column_values(rng, dt, P * rc) for _ in range(P)]
            full = _bits(orc.allreduce_local(srcs, dt, op))
            for r in range(P):
                sh = _bits(orc.reduce_scatter_local(srcs, r, dt, op))
                exp = full[r * rc:(r + 1) * rc]
                ok = [_same(int(x), int(y), dt, op) for x, y in zip(sh, exp)]
                assert all(ok), (dt, op, r)
            chunks = [random_column_values(rng, dt, 53) for _ in range(P)]
            fused = _bits(orc.allreduce_local(chunks, dt, op))
            acc = orc.reduce_copy_step(chunks[0], None, dt, op, init=True)
            for c in chunks[1:-1]:
                acc = orc.reduce_copy_step(c, acc, dt, op)
            acc_copy = acc.copy()
            fin = _bits(orc.reduce_copy_step(chunks[-1], acc, dt, op, final=True))
            cast = _bits(orc.acc_cast(orc.reduce_copy_step(chunks[-1], acc_copy, dt, op), dt))
            for got in (fin, cast):
                assert all(_same(int(x), int(y), dt, op) for x, y in zip(got, fused)), (dt, op)
            if op in ("max", "min"):
                perm = [srcs[k] for k in rng.permutation(P)]
                assert np.array_equal(_bits(orc.allreduce_local(perm, dt, op)), full), (dt, op)


def pin_wide_narrow_sim(orc, seed: int = 71) -> None:
    """The simulated ring and halving-doubling schedules on fp64 and int8 /
    uint8 against the chain of hops computed by the brute force."""
    rng = np.random.default_rng(seed)
    for algo, sizes, brute_el in (("ring", (2, 3, 5), brute_ring_element),
                                  ("rhd", (2, 4, 8), brute_rhd_element)):
        for dtype in WIDE_NARROW_DTYPES:
            for op in OPS:
                for G in sizes:
                    n = 64 * G + 70
                    sends = [random_column_values(rng, dtype, n) for _ in range(G)]
                    outs = [_bits(o) for o in orc.allreduce_sim(sends, dtype, op, algo)]
                    M = sim_chunk_len(n, G)
                    sb = [_bits(x) for x in sends]
                    for i in sorted({0, n - 1, M - 1, M, n // 2}):
                        col = [int(x[i]) for x in sb]
                        exp = brute_el(col, i // M, dtype, op)
                        for r in range(G):
                            assert _same(int(outs[r][i]), exp, dtype, op), (
                                f"{algo} {dtype} {op} G={G} rank {r} i={i}")


def pin_selfcheck(orc) -> None:
    assert orc.selfcheck() == 0, "floating-point environment"


FAST_PINS = [pin_selfcheck, pin_golden_reduce, pin_golden_bf16, pin_bf16_vs_brute,
             pin_up_bf16, pin_integer_closed_form, pin_int_mod32, pin_invariants,
             pin_composition, pin_bruteforce, pin_sim_closed_forms, pin_sim_bruteforce,
             pin_narrow_vs_torch, pin_more_types_closed_forms, pin_more_types_bruteforce,
             pin_golden_narrow, pin_wide_narrow_bruteforce, pin_wide_narrow_closed_forms,
             pin_wide_narrow_sim]
