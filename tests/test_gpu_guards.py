"""Guard bands around every output the library writes, for the entry points
other than xred_allreduce_local (which test_gpu_parity covers): each output
sits between two bands of canary bytes that must be untouched after the call,
at a 16-byte aligned offset (vector paths) and one element off (scalar
paths), with ragged lengths.  Results are also checked against the oracle.
"""
import numpy as np
import pytest

import gpu_util as gu
import pins

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

G = 4096        # guard elements on each side
CANARY = 0x5A


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()
    return xr


class Guarded:
    """n elements of `tdtype` at element offset G + shift of a canary-filled store."""

    def __init__(self, n, tdtype, shift):
        self.n, self.shift = n, shift
        self.store = torch.zeros(n + 2 * G + shift, dtype=tdtype, device="cuda")
        self.store.view(torch.uint8).fill_(CANARY)
        self.t = self.store[G + shift:G + shift + n]

    def check(self, what):
        raw = self.store.view(torch.uint8).cpu().numpy()
        es = self.store.element_size()
        lo, hi = (G + self.shift) * es, (G + self.shift + self.n) * es
        assert np.all(raw[:lo] == CANARY), f"{what}: bytes before the output were written"
        assert np.all(raw[hi:] == CANARY), f"{what}: bytes after the output were written"


def _dev(arrs, dtype, shift):
    return [gu.to_dev(np.concatenate([np.zeros(shift, a.dtype), a]), dtype)[shift:] for a in arrs]


@pytest.mark.parametrize("dtype", ["bf16", "f32", "e4m3", "i64"])
@pytest.mark.parametrize("shift", [0, 1])
def test_reduce_scatter_guards(xr, orc, dtype, shift):
    rng = np.random.default_rng(3)
    P, rc = 5, 3 * 4096 + 37
    srcs = [pins.random_column_values(rng, dtype, P * rc) for _ in range(P)]
    d = _dev(srcs, dtype, shift)
    out = Guarded(rc, gu.torch_dtype(dtype), shift)
    xr.reduce_scatter_local(d, 3, out.t, "sum", dtype=dtype)
    torch.cuda.synchronize()
    gu.assert_parity(out.t, orc.reduce_scatter_local(srcs, 3, dtype, "sum"), dtype, "sum", "rs")
    out.check(f"reduce_scatter {dtype} shift={shift}")


@pytest.mark.parametrize("dtype", ["bf16", "e5m2", "u64"])
@pytest.mark.parametrize("shift", [0, 1])
def test_step_and_cast_guards(xr, orc, dtype, shift):
    rng = np.random.default_rng(4)
    n = 2 * 4096 * 8 + 13
    chunks = [pins.random_column_values(rng, dtype, n) for _ in range(4)]
    d = _dev(chunks, dtype, shift)
    acc_t = torch.int64 if dtype in ("i64", "u64") else torch.float32
    acc = Guarded(n, acc_t, shift)
    out = Guarded(n, gu.torch_dtype(dtype), shift)
    out2 = Guarded(n, gu.torch_dtype(dtype), shift)
    xr.reduce_copy_step(d[0], acc.t, None, "max", init=True, dtype=dtype)
    for c in d[1:-1]:
        xr.reduce_copy_step(c, acc.t, None, "max", dtype=dtype)
    xr.reduce_copy_step(d[-1], acc.t, out.t, "max", final=True, dtype=dtype)
    xr.reduce_copy_step(d[-1], acc.t, None, "max", dtype=dtype)
    xr.acc_cast(acc.t, out2.t, dtype=dtype)
    torch.cuda.synchronize()
    exp = orc.allreduce_local(chunks, dtype, "max")
    gu.assert_parity(out.t, exp, dtype, "max", "step final")
    gu.assert_parity(out2.t, exp, dtype, "max", "cast")
    for g, what in ((acc, "acc"), (out, "final"), (out2, "cast")):
        g.check(f"step {what} {dtype} shift={shift}")


@pytest.mark.parametrize("dtype", ["bf16", "f16", "i32"])
def test_ring_guards(xr, orc, dtype):
    rng = np.random.default_rng(6)
    n = 5 * 512 * 8 + 21     # several tiles, ragged (the ring needs 16-byte alignment)
    chunks = [pins.random_column_values(rng, dtype, n) for _ in range(7)]
    out = Guarded(n, gu.torch_dtype(dtype), 0)
    xr.ring_reduce(_dev(chunks, dtype, 0), out.t, "sum", dtype=dtype)
    torch.cuda.synchronize()
    gu.assert_parity(out.t, orc.allreduce_local(chunks, dtype, "sum"), dtype, "sum", "ring")
    out.check(f"ring {dtype}")


@pytest.mark.parametrize("shift", [0, 1])
def test_batched_guards(xr, orc, shift):
    rng = np.random.default_rng(8)
    dtype = "bf16"
    sizes = [1, 9, 4095, 8192 + 3, 3 * 8192, 70001]
    items_np = [[pins.random_column_values(rng, dtype, n) for _ in range(1 + k % 8)]
                for k, n in enumerate(sizes)]
    outs = [Guarded(n, torch.bfloat16, shift) for n in sizes]
    xr.batched_reduce([(_dev(s, dtype, shift), o.t) for s, o in zip(items_np, outs)], "sum",
                      dtype=dtype)
    torch.cuda.synchronize()
    for k, (s, o) in enumerate(zip(items_np, outs)):
        gu.assert_parity(o.t, orc.allreduce_local(s, dtype, "sum"), dtype, "sum", f"item {k}")
        o.check(f"batched item {k} shift={shift}")


@pytest.mark.parametrize("schedule", ["ring", "rhd", "ring1", "rhd1"])
@pytest.mark.parametrize("shift", [0, 1])
def test_sim_guards(xr, orc, schedule, shift):
    rng = np.random.default_rng(10)
    dtype = "bf16"
    for Gr, n in ((8, 8 * 4096 + 77), (4, 64 * 4 + 5)):
        sends = [pins.random_column_values(rng, dtype, n) for _ in range(Gr)]
        recvs = [Guarded(n, torch.bfloat16, shift) for _ in range(Gr)]
        xr.allreduce_sim(_dev(sends, dtype, shift), [r.t for r in recvs], "sum",
                         schedule=schedule, dtype=dtype)
        torch.cuda.synchronize()
        exp = orc.allreduce_sim(sends, dtype, "sum", schedule.rstrip("1"))
        for r, (g, e) in enumerate(zip(recvs, exp)):
            gu.assert_parity(g.t, e, dtype, "sum", f"{schedule} rank {r}")
            g.check(f"sim {schedule} G={Gr} rank {r} shift={shift}")
