"""Entry points called from several host threads at once, each thread
enqueueing on its own stream: the fused reduce, host-descriptor batches
(whose staging slots the threads share), device-descriptor batches on the
queue kernel (tile counters bound to each stream) and the ring with host
flags (relay word bound to each stream), while one thread keeps changing the
process-wide CU budget.  Every output is then compared with the oracle:
the header's claim that every call is thread-safe and that results never
depend on the budget."""
import threading

import numpy as np
import pytest

import gpu_util as gu
import pins

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

THREADS = 4
ROUNDS = 12
DT = "bf16"


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()
    return xr


def _cols(rng, P, n):
    return [pins.random_column_values(rng, DT, n) for _ in range(P)]


def _dev(cols):
    return [gu.to_dev(c, DT) for c in cols]


class Job:
    """One round of one thread: inputs on the device, outputs, expectations."""

    def __init__(self, xr, rng):
        # fused
        P, n = int(rng.integers(1, 9)), int(rng.integers(1, 100_000))
        self.fused_host = _cols(rng, P, n)
        self.fused_src = _dev(self.fused_host)
        self.fused_out = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
        # host-descriptor batch
        K = int(rng.integers(20, 81))
        self.hb_host, self.hb_items = [], []
        for _ in range(K):
            cols = _cols(rng, int(rng.integers(1, 9)), int(rng.integers(1, 4_000)))
            self.hb_host.append(cols)
            self.hb_items.append((_dev(cols), torch.zeros(cols[0].size, dtype=torch.bfloat16,
                                                          device="cuda")))
        # device-descriptor batch (65..150 items: the queue kernel)
        K = int(rng.integers(65, 151))
        self.db_host, self.db_outs, self.db_keep = [], [], []
        rows = np.zeros(K, xr.ITEM_DTYPE)
        for k in range(K):
            cols = _cols(rng, int(rng.integers(1, 9)), int(rng.integers(1, 6_000)))
            dev = _dev(cols)
            out = torch.zeros(cols[0].size, dtype=torch.bfloat16, device="cuda")
            pa = torch.tensor([d.data_ptr() for d in dev], dtype=torch.int64, device="cuda")
            self.db_keep += dev + [pa]
            self.db_host.append(cols)
            self.db_outs.append(out)
            rows[k] = (pa.data_ptr(), out.data_ptr(), cols[0].size, len(cols), 0)
        self.db_items = torch.from_numpy(rows.view(np.uint8).copy()).to("cuda")
        # ring of 16 chunks with every flag preset in pinned host memory
        self.ring_host = _cols(rng, 16, 16384)
        self.ring_src = _dev(self.ring_host)
        self.ring_out = torch.zeros(16384, dtype=torch.bfloat16, device="cuda")
        self.ready = torch.full((16,), 1, dtype=torch.int32).pin_memory()
        self.status = torch.zeros(1, dtype=torch.int32).pin_memory()

    def enqueue(self, xr, stream):
        with torch.cuda.stream(stream):
            xr.allreduce_local(self.fused_src, self.fused_out)
            xr.batched_reduce(self.hb_items, "sum", dtype=DT)
            xr.batched_reduce(self.db_items, "sum", dtype=DT)
            xr.ring_reduce(self.ring_src, self.ring_out, ready=self.ready, epoch=1,
                           status=self.status)

    def check(self, orc, what):
        gu.assert_parity(self.fused_out, orc.allreduce_local(self.fused_host, DT, "sum"), DT,
                         "sum", f"{what} fused")
        for k, (cols, (_, out)) in enumerate(zip(self.hb_host, self.hb_items)):
            gu.assert_parity(out, orc.allreduce_local(cols, DT, "sum"), DT, "sum",
                             f"{what} host batch item {k}")
        for k, (cols, out) in enumerate(zip(self.db_host, self.db_outs)):
            gu.assert_parity(out, orc.allreduce_local(cols, DT, "sum"), DT, "sum",
                             f"{what} device batch item {k}")
        assert int(self.status[0]) == 0, f"{what} ring timed out"
        gu.assert_parity(self.ring_out, orc.allreduce_local(self.ring_host, DT, "sum"), DT,
                         "sum", f"{what} ring")


def test_threads_on_their_own_streams(xr, orc):
    rng = np.random.default_rng(9100)
    jobs = [[Job(xr, rng) for _ in range(ROUNDS)] for _ in range(THREADS)]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(THREADS)]
    errors = []
    start = threading.Barrier(THREADS + 1)
    stop_budget = threading.Event()

    def worker(t):
        try:
            start.wait()
            for job in jobs[t]:
                job.enqueue(xr, streams[t])
        except Exception as e:   # re-raised below, in the test's thread
            errors.append((t, e))

    def budgets():
        r = np.random.default_rng(9101)
        start.wait()
        while not stop_budget.is_set():
            xr.set_max_workgroups(int(r.choice([0, 0, 1, 7, 64, 300])))

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(THREADS)]
    knob = threading.Thread(target=budgets)
    prev = xr.set_max_workgroups(0)
    try:
        for th in threads + [knob]:
            th.start()
        for th in threads:
            th.join(timeout=300)
        stop_budget.set()
        knob.join(timeout=60)
    finally:
        stop_budget.set()
        xr.set_max_workgroups(prev)
    assert not any(th.is_alive() for th in threads), "a worker thread did not finish"
    assert not errors, errors
    for s in streams:
        s.synchronize()
    print(f"{THREADS} threads x {ROUNDS} rounds enqueued; checking", flush=True)
    for t in range(THREADS):
        for r, job in enumerate(jobs[t]):
            job.check(orc, f"thread {t} round {r}")
