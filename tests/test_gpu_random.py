"""Seeded random sweep over every entry point, against the CPU oracle.

Each case draws, from a fixed seed, an entry point, an element type, an op
valid for both, a source / chunk / rank count, sizes biased to the vector and
tile boundaries (one element, k vectors +- 1, k 512-vector tiles +- 1, or
anything up to a few hundred thousand elements), 16-byte or element-only
alignment and, where allowed, an in-place output.  Inputs mix random bit
patterns with the special values of each type (pins.random_column_values).
Results must match the oracle bit for bit (NaN payloads of float
sum/prod/avg by NaN-ness only).  The case is printed before it runs.
"""
import os

import numpy as np
import pytest

import gpu_util as gu
import pins

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

DTYPES = ("f32", "bf16", "f16", "e4m3", "e5m2", "i32", "u32", "i64", "u64", "f64", "i8",
          "u8")
ES = {"f32": 4, "bf16": 2, "f16": 2, "e4m3": 1, "e5m2": 1, "i32": 4, "u32": 4, "i64": 8,
      "u64": 8, "f64": 8, "i8": 1, "u8": 1}
CASES = 40
CORES = min(16, len(os.sched_getaffinity(0)))


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()
    return xr


def _size(rng, dtype, cap=300_000):
    vec = 16 // ES[dtype]
    kind = rng.integers(0, 4)
    if kind == 0:
        n = int(rng.integers(1, 100))
    elif kind == 1:
        n = vec * int(rng.integers(1, 64)) + int(rng.integers(-1, 2))
    elif kind == 2:
        n = 512 * vec * int(rng.integers(1, 4)) + int(rng.integers(-1, 2))
    else:
        n = int(rng.integers(1, cap))
    return max(1, min(n, cap))


def _op(rng, dtype, avg_ok=True):
    ops = pins.ops_for(dtype) if avg_ok else pins.OPS
    return str(ops[rng.integers(0, len(ops))])


def _dev(arrs, dtype, offset):
    """Device copies of the arrays, each starting `offset` elements into its
    own allocation (offset 1 breaks 16-byte alignment)."""
    out = []
    for a in arrs:
        pad = np.concatenate([np.zeros(offset, a.dtype), a]) if offset else a
        out.append(gu.to_dev(pad, dtype)[offset:])
    return out


def _empty(n, dtype, offset):
    return torch.empty(n + offset, dtype=gu.torch_dtype(dtype), device="cuda")[offset:]


def _say(case, what):
    print(f"case {case}: {what}", flush=True)


@pytest.mark.parametrize("seed", range(8))
def test_random_fused_and_reduce_scatter(xr, orc, seed):
    rng = np.random.default_rng(9000 + seed)
    for case in range(CASES):
        dtype = DTYPES[rng.integers(0, len(DTYPES))]
        op = _op(rng, dtype)
        P = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 9, 12, 16, 17, 31, 32, 33, 63, 64]))
        off = int(rng.integers(0, 2))
        if rng.random() < 0.6:
            n = _size(rng, dtype, cap=max(1, (1 << 21) // P))
            in_place = rng.random() < 0.25
            _say(case, f"allreduce_local {dtype} {op} P={P} n={n} offset={off} "
                       f"in_place={in_place}")
            srcs_np = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
            exp = orc.allreduce_local(srcs_np, dtype, op)
            srcs = _dev(srcs_np, dtype, off)
            out = srcs[int(rng.integers(0, P))] if in_place else _empty(n, dtype, off)
            xr.allreduce_local(srcs, out, op, dtype=dtype)
            torch.cuda.synchronize()
            gu.assert_parity(out, exp, dtype, op, f"case {case}")
        else:
            rc = _size(rng, dtype, cap=max(1, (1 << 20) // (P * P)))
            rank = int(rng.integers(0, P))
            _say(case, f"reduce_scatter_local {dtype} {op} P={P} rank={rank} recvcount={rc} "
                       f"offset={off}")
            srcs_np = [pins.random_column_values(rng, dtype, P * rc) for _ in range(P)]
            exp = orc.reduce_scatter_local(srcs_np, rank, dtype, op)
            srcs = _dev(srcs_np, dtype, off)
            out = _empty(rc, dtype, off)
            xr.reduce_scatter_local(srcs, rank, out, op, dtype=dtype)
            torch.cuda.synchronize()
            gu.assert_parity(out, exp, dtype, op, f"case {case}")


@pytest.mark.parametrize("seed", range(6))
def test_random_stepwise_and_ring(xr, orc, seed):
    rng = np.random.default_rng(9100 + seed)
    for case in range(CASES):
        dtype = DTYPES[rng.integers(0, len(DTYPES))]
        op = _op(rng, dtype, avg_ok=False)
        C = int(rng.integers(1, 18))
        if rng.random() < 0.5:
            n = _size(rng, dtype, cap=200_000)
            off = int(rng.integers(0, 2))
            closing = "final" if rng.random() < 0.5 else "cast"
            _say(case, f"step-wise {dtype} {op} chunks={C} n={n} offset={off} close={closing}")
            chunks_np = [pins.random_column_values(rng, dtype, n) for _ in range(C)]
            exp = orc.allreduce_local(chunks_np, dtype, op)
            d = _dev(chunks_np, dtype, off)
            acc_t = torch.int64 if ES[dtype] == 8 else torch.float32
            acc = torch.empty(n + off, dtype=acc_t, device="cuda")[off:]
            out = _empty(n, dtype, off)
            if C == 1:
                xr.reduce_copy_step(d[0], None, out, op, init=True, final=True, dtype=dtype)
            else:
                xr.reduce_copy_step(d[0], acc, None, op, init=True, dtype=dtype)
                for c in d[1:-1]:
                    xr.reduce_copy_step(c, acc, None, op, dtype=dtype)
                if closing == "final":
                    xr.reduce_copy_step(d[-1], acc, out, op, final=True, dtype=dtype)
                else:
                    xr.reduce_copy_step(d[-1], acc, None, op, dtype=dtype)
                    xr.acc_cast(acc, out, dtype=dtype)
            torch.cuda.synchronize()
            gu.assert_parity(out, exp, dtype, op, f"case {case}")
        else:
            n = min(_size(rng, dtype, cap=300_000), xr.ring_max_count(dtype))
            _say(case, f"ring_reduce {dtype} {op} chunks={C} n={n}")
            chunks_np = [pins.random_column_values(rng, dtype, n) for _ in range(C)]
            exp = orc.allreduce_local(chunks_np, dtype, op)
            d = _dev(chunks_np, dtype, 0)
            out = _empty(n, dtype, 0)
            xr.ring_reduce(d, out, op, dtype=dtype)
            torch.cuda.synchronize()
            gu.assert_parity(out, exp, dtype, op, f"case {case}")


@pytest.mark.parametrize("seed", range(6))
def test_random_batched(xr, orc, seed):
    rng = np.random.default_rng(9200 + seed)
    for case in range(CASES // 2):
        dtype = DTYPES[rng.integers(0, len(DTYPES))]
        op = _op(rng, dtype)
        K = int(rng.integers(1, 24))
        on_device = rng.random() < 0.5
        off = int(rng.integers(0, 2))
        shapes = [(int(rng.integers(1, 13)), _size(rng, dtype, cap=60_000)) for _ in range(K)]
        _say(case, f"batched_reduce {dtype} {op} items={shapes} offset={off} "
                   f"device_descriptors={on_device}")
        items_np = [[pins.random_column_values(rng, dtype, n) for _ in range(P)]
                    for P, n in shapes]
        exps = [orc.allreduce_local(srcs, dtype, op) for srcs in items_np]
        items = [(_dev(srcs, dtype, off), _empty(n, dtype, off))
                 for srcs, (P, n) in zip(items_np, shapes)]
        if on_device:
            keep, rows = [], []
            for srcs, out in items:
                pa = torch.tensor([s.data_ptr() for s in srcs], dtype=torch.int64, device="cuda")
                keep.append(pa)
                rows.append((pa.data_ptr(), out.data_ptr(), out.numel(), len(srcs), 0))
            arr = np.zeros(len(rows), xr.ITEM_DTYPE)
            for k, r in enumerate(rows):
                arr[k] = r
            desc = torch.from_numpy(arr.view(np.uint8).copy()).to("cuda")
            xr.batched_reduce(desc, op, dtype=dtype)
        else:
            xr.batched_reduce(items, op, dtype=dtype)
        torch.cuda.synchronize()
        for k, ((_, out), exp) in enumerate(zip(items, exps)):
            gu.assert_parity(out, exp, dtype, op, f"case {case} item {k}")


@pytest.mark.parametrize("seed", range(6))
def test_random_sim(xr, orc, seed):
    rng = np.random.default_rng(9300 + seed)
    for case in range(CASES):
        dtype = DTYPES[rng.integers(0, len(DTYPES))]
        op = _op(rng, dtype, avg_ok=False)
        schedule = ("ring", "rhd", "ring1", "rhd1")[rng.integers(0, 4)]
        G = int(rng.integers(1, 21)) if schedule.startswith("ring") else 1 << int(rng.integers(0, 6))
        n = _size(rng, dtype, cap=max(1, (1 << 20) // G))
        off = int(rng.integers(0, 2))
        in_place = rng.random() < 0.3
        _say(case, f"allreduce_sim {schedule} {dtype} {op} G={G} n={n} offset={off} "
                   f"in_place={in_place}")
        sends_np = [pins.random_column_values(rng, dtype, n) for _ in range(G)]
        exp = orc.allreduce_sim(sends_np, dtype, op, schedule.rstrip("1"))
        sends = _dev(sends_np, dtype, off)
        recvs = sends if in_place else [_empty(n, dtype, off) for _ in range(G)]
        xr.allreduce_sim(sends, recvs, op, schedule=schedule, dtype=dtype)
        torch.cuda.synchronize()
        for r in range(G):
            gu.assert_parity(recvs[r], exp[r], dtype, op, f"case {case} rank {r}")


@pytest.mark.parametrize("seed", range(2))
def test_random_sim_one_launch_large(xr, orc, seed):
    """The one-launch schedules around and past 8 MiB per rank, where their
    workgroup shapes change: random type, op, rank count, alignment and
    in-place output, lengths within a few vectors of the switch or up to
    1.5 times past it."""
    rng = np.random.default_rng(9400 + seed)
    for case in range(6):
        dtype = DTYPES[rng.integers(0, len(DTYPES))]
        op = _op(rng, dtype, avg_ok=False)
        schedule = ("ring1", "rhd1")[rng.integers(0, 2)]
        G = int(rng.integers(2, 9)) if schedule == "ring1" else 1 << int(rng.integers(1, 4))
        edge = (8 << 20) // ES[dtype]
        vec = 16 // ES[dtype]
        if rng.random() < 0.5:
            n = edge + vec * int(rng.integers(-2, 3)) + int(rng.integers(-1, 2))
        else:
            n = edge + int(rng.integers(0, edge // 2))
        off = int(rng.integers(0, 2))
        in_place = rng.random() < 0.3
        _say(case, f"allreduce_sim {schedule} {dtype} {op} G={G} n={n} offset={off} "
                   f"in_place={in_place}")
        sends_np = [pins.random_column_values(rng, dtype, n) for _ in range(G)]
        exp = orc.allreduce_sim(sends_np, dtype, op, schedule.rstrip("1"), nthreads=CORES)
        sends = _dev(sends_np, dtype, off)
        recvs = sends if in_place else [_empty(n, dtype, off) for _ in range(G)]
        xr.allreduce_sim(sends, recvs, op, schedule=schedule, dtype=dtype)
        torch.cuda.synchronize()
        for r in range(G):
            gu.assert_parity(recvs[r], exp[r], dtype, op, f"case {case} rank {r}")
        del sends, recvs
        torch.cuda.empty_cache()
