"""GPU parity of xred_allreduce_sim: a whole ring or halving-doubling
AllReduce over G simulated ranks on one GPU, against the oracle's
message-by-message simulation of the same schedule.

Every rank's output must equal the oracle's bit for bit (NaN payloads of
float sum/prod compare by NaN-ness only), and all ranks must hold the same
bits.  Covered: every dtype x op; ring G = 1, 2, 3, 5, 8, 13 and
halving-doubling G = 1, 2, 4, 8, 16, and G = 32, 64 (the maximum) for three
dtype x op pairs; sizes from one element to several tiles
per chunk with short and empty trailing chunks; in place; element-aligned
(not 16-byte aligned) buffers; a CU budget; the full G=8 x 2^26 bf16 bucket
the benchmark times, for both schedules.  Each schedule also runs with all of
its steps in one launch ("ring1", "rhd1"), which must give the same bits as
the oracle's simulation of that schedule.
"""
import os

import numpy as np
import pytest

import gpu_util as gu
import pins
import workloads as wl

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

DTYPES = ("f32", "bf16", "i32", "u32")
OPS = ("sum", "prod", "max", "min")
CORES = min(16, len(os.sched_getaffinity(0)))


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()
    yield xr
    xr.set_max_workgroups(0)


def _check(outs, exp, dtype, op, what):
    b0 = gu.bits(outs[0], dtype)
    for r, o in enumerate(outs):
        assert np.array_equal(gu.bits(o, dtype), b0), f"{what}: rank {r} differs from rank 0"
        gu.assert_parity(o, exp[r], dtype, op, f"{what} rank {r}")


def _oracle_schedule(schedule):
    return schedule.rstrip("1")


def _run(xr, sends_np, dtype, op, schedule, in_place=False):
    sends = [gu.to_dev(s, dtype) for s in sends_np]
    recvs = sends if in_place else [torch.empty_like(s) for s in sends]
    xr.allreduce_sim(sends, recvs, op, schedule=schedule, dtype=dtype)
    torch.cuda.synchronize()
    return recvs


def _sizes(G):
    return (1, 37, 64 * G + 70, 4096 * 5 + 3, (1 << 17) + 5)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("op", OPS)
def test_ring_and_rhd_parity(xr, orc, dtype, op):
    rng = np.random.default_rng(61 + 10 * DTYPES.index(dtype) + OPS.index(op))
    for schedule, ranks in (("ring", (1, 2, 3, 5, 8, 13)), ("rhd", (1, 2, 4, 8, 16))):
        for G in ranks:
            for n in _sizes(G):
                if G * n > (1 << 21):
                    continue
                sends = [pins.random_column_values(rng, dtype, n) for _ in range(G)]
                exp = orc.allreduce_sim(sends, dtype, op, schedule)
                for variant in (schedule, schedule + "1"):
                    outs = _run(xr, sends, dtype, op, variant)
                    _check(outs, exp, dtype, op, f"{variant} {dtype} {op} G={G} n={n}")


@pytest.mark.parametrize("schedule", ["ring", "rhd", "ring1", "rhd1"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_in_place(xr, orc, schedule, dtype):
    rng = np.random.default_rng(7)
    for G, n in ((2, 999), (4, 64 * 4 + 70), (8, (1 << 16) + 3)):
        sends = [pins.random_column_values(rng, dtype, n) for _ in range(G)]
        outs = _run(xr, sends, dtype, "sum", schedule, in_place=True)
        _check(outs, orc.allreduce_sim(sends, dtype, "sum", _oracle_schedule(schedule)), dtype,
               "sum", f"in place {schedule} G={G}")


@pytest.mark.parametrize("schedule", ["ring", "rhd", "ring1", "rhd1"])
def test_element_aligned_buffers(xr, orc, schedule):
    """Buffers one element off 16-byte alignment take the scalar path."""
    rng = np.random.default_rng(8)
    G, n = 4, 64 * 4 * 3 + 11
    for dtype in ("bf16", "f32", "i32"):
        sends_np = [pins.random_column_values(rng, dtype, n) for _ in range(G)]
        big = [gu.to_dev(np.concatenate([np.zeros(1, s.dtype), s]), dtype) for s in sends_np]
        sends = [b[1:] for b in big]
        rbig = [torch.empty_like(b) for b in big]
        recvs = [b[1:] for b in rbig]
        xr.allreduce_sim(sends, recvs, "max", schedule=schedule, dtype=dtype)
        torch.cuda.synchronize()
        _check(recvs, orc.allreduce_sim(sends_np, dtype, "max", _oracle_schedule(schedule)),
               dtype, "max", f"element-aligned {schedule} {dtype}")


def test_budget_does_not_change_results(xr, orc):
    rng = np.random.default_rng(9)
    G, n = 8, (1 << 15) + 77
    sends = [pins.random_column_values(rng, "bf16", n) for _ in range(G)]
    exp = orc.allreduce_sim(sends, "bf16", "sum", "ring")
    for budget in (1, 7, 0):
        for schedule in ("ring", "ring1"):
            prev = xr.set_max_workgroups(budget)
            try:
                outs = _run(xr, sends, "bf16", "sum", schedule)
            finally:
                xr.set_max_workgroups(prev)
            _check(outs, exp, "bf16", "sum", f"{schedule} budget {budget}")


@pytest.mark.parametrize("schedule", ["ring", "rhd"])
def test_full_bucket(xr, orc, schedule):
    """The benchmark's workload: 8 ranks x 2^26 bf16, both schedules, step by
    step and in one launch."""
    w = wl.WORKLOADS["sim"]
    sends = wl.sources(w)
    exp = orc.allreduce_sim(sends, w.dtype, w.op, schedule, nthreads=CORES)
    for variant in (schedule, schedule + "1"):
        outs = _run(xr, sends, w.dtype, w.op, variant)
        _check(outs, exp, w.dtype, w.op, f"sim {variant}")
        del outs
        torch.cuda.empty_cache()


@pytest.mark.parametrize("G", [32, 64])
def test_most_ranks(xr, orc, G):
    """G = 32 and the maximum 64 (every tree level of the one-launch
    halving-doubling, leaves loaded in 4 or 8 batches), all four schedules,
    with a ragged last chunk and empty trailing chunks."""
    rng = np.random.default_rng(70 + G)
    for dtype, op in (("bf16", "sum"), ("f32", "max"), ("i32", "prod")):
        for n in (64 * G + 70, 64 * (G - 3) + 1, 4096 * G + 3):
            sends = [pins.random_column_values(rng, dtype, n) for _ in range(G)]
            for schedule in ("ring", "rhd"):
                exp = orc.allreduce_sim(sends, dtype, op, schedule)
                for variant in (schedule, schedule + "1"):
                    outs = _run(xr, sends, dtype, op, variant)
                    _check(outs, exp, dtype, op, f"{variant} {dtype} {op} G={G} n={n}")


@pytest.mark.parametrize("dtype,op,G,n", [
    ("bf16", "sum", 8, (8 << 20) // 2 - 1),        # one element below 8 MiB per rank
    ("bf16", "max", 3, (8 << 20) // 2 + 37),       # past it: the large workgroup shapes
    ("f32", "prod", 5, (8 << 20) // 4 + 5),
    ("u8", "sum", 16, (8 << 20) + 3),
    ("i8", "min", 4, (8 << 20) + 64 * 4 + 1),
    ("f64", "sum", 8, (8 << 20) // 8 + 9),
])
def test_one_launch_shapes_by_size(xr, orc, dtype, op, G, n):
    """The one-launch schedules pick their workgroup shape by bytes per rank
    (8 MiB): both sides of the switch, ragged chunks, 1- to 8-byte elements,
    and halving-doubling where G is a power of two."""
    rng = np.random.default_rng(90 + G)
    sends = [pins.random_column_values(rng, dtype, n) for _ in range(G)]
    for schedule in ("ring", "rhd") if G & (G - 1) == 0 else ("ring",):
        exp = orc.allreduce_sim(sends, dtype, op, schedule, nthreads=CORES)
        outs = _run(xr, sends, dtype, op, schedule + "1")
        _check(outs, exp, dtype, op, f"{schedule}1 {dtype} {op} G={G} n={n}")
        del outs
        torch.cuda.empty_cache()


@pytest.mark.parametrize("schedule", ["ring1", "rhd1"])
def test_one_launch_large_element_aligned(xr, orc, schedule):
    """Past 8 MiB per rank with buffers one element off 16-byte alignment:
    the scalar path of the large shapes."""
    rng = np.random.default_rng(95)
    G, n = 4, (8 << 20) // 2 + 3
    sends_np = [pins.random_column_values(rng, "bf16", n) for _ in range(G)]
    big = [gu.to_dev(np.concatenate([np.zeros(1, s.dtype), s]), "bf16") for s in sends_np]
    rbig = [torch.empty_like(b) for b in big]
    recvs = [b[1:] for b in rbig]
    xr.allreduce_sim([b[1:] for b in big], recvs, "sum", schedule=schedule, dtype="bf16")
    torch.cuda.synchronize()
    _check(recvs, orc.allreduce_sim(sends_np, "bf16", "sum", _oracle_schedule(schedule),
                                    nthreads=CORES), "bf16", "sum", f"element-aligned {schedule}")
