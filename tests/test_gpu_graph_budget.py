"""Workgroup budgets and HIP graph capture.

- xred_set_max_workgroups only changes how many workgroups share the work:
  results must be bit-identical under budgets of 1, 3, 64 and none (this
  runs every kernel's grid-stride path with very small grids).
- Paths documented as capturable (fused / reduce-scatter calls, device-
  resident batches, the one-launch ring without flags) are captured into a
  graph once and replayed several times with eager work and synchronisation
  between replays; every replay must equal the eager result of the same
  inputs.  No library call inside the capture records a memset.
"""
import numpy as np
import pytest

import gpu_util as gu
import pins

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()
    yield xr
    xr.set_max_workgroups(0)


def _device_items(xr, items):
    keep, rows = [], []
    for srcs, out in items:
        pa = torch.tensor([s.data_ptr() for s in srcs], dtype=torch.int64, device="cuda")
        keep.append(pa)
        rows.append((pa.data_ptr(), out.data_ptr(), out.numel(), len(srcs), 0))
    arr = np.zeros(len(rows), xr.ITEM_DTYPE)
    for k, r in enumerate(rows):
        arr[k] = r
    return torch.from_numpy(arr.view(np.uint8).copy()).to("cuda"), keep


def test_budget_does_not_change_results(xr, orc):
    rng = np.random.default_rng(12)
    n = 3 * 4096 * 8 + 5
    srcs_np = [pins.random_column_values(rng, "bf16", n) for _ in range(8)]
    exp = orc.allreduce_local(srcs_np, "bf16", "sum")
    srcs = [gu.to_dev(s, "bf16") for s in srcs_np]
    acc = torch.empty(n, dtype=torch.float32, device="cuda")
    items = [(srcs[:3], torch.empty(n, dtype=torch.bfloat16, device="cuda")),
             (srcs[2:8], torch.empty(1000, dtype=torch.bfloat16, device="cuda"))]
    items[1] = ([s[:1000] for s in srcs[2:8]], items[1][1])
    exp_items = [orc.allreduce_local(srcs_np[:3], "bf16", "sum"),
                 orc.allreduce_local([s[:1000] for s in srcs_np[2:8]], "bf16", "sum")]
    for budget in (1, 3, 64, 0):
        prev = xr.set_max_workgroups(budget)
        try:
            out = torch.empty_like(srcs[0])
            xr.allreduce_local(srcs, out)
            step_out = torch.empty_like(srcs[0])
            xr.reduce_copy_step(srcs[0], acc, None, init=True)
            for s in srcs[1:-1]:
                xr.reduce_copy_step(s, acc, None)
            xr.reduce_copy_step(srcs[-1], acc, step_out, final=True)
            for _, o in items:
                o.zero_()
            xr.batched_reduce(items, dtype="bf16")
            torch.cuda.synchronize()
        finally:
            xr.set_max_workgroups(prev)
        gu.assert_parity(out, exp, "bf16", "sum", f"fused, budget {budget}")
        gu.assert_parity(step_out, exp, "bf16", "sum", f"step-wise, budget {budget}")
        for (_, o), e in zip(items, exp_items):
            gu.assert_parity(o, e, "bf16", "sum", f"batched, budget {budget}")


def test_graph_capture_and_replay(xr):
    torch.manual_seed(3)
    n = (1 << 18) + 3
    srcs = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(6)]
    out_fused = torch.empty_like(srcs[0])
    out_ring = torch.empty_like(srcs[0])
    aligned = [s[:1 << 18] for s in srcs]          # the ring path needs whole vectors
    out_ring = torch.empty(1 << 18, dtype=torch.bfloat16, device="cuda")
    b_outs = [torch.empty(5000, dtype=torch.bfloat16, device="cuda") for _ in range(3)]
    b_items = [([s[:5000] for s in srcs[k:k + 3]], b_outs[k]) for k in range(3)]
    dev_items, keep = _device_items(xr, b_items)

    def work():
        xr.allreduce_local(srcs, out_fused)
        xr.ring_reduce(aligned, out_ring)
        xr.batched_reduce(dev_items, dtype="bf16")

    # warm up on a side stream, then capture
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        work()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    torch.cuda.synchronize()

    for r in range(4):
        # eager work between replays: change the inputs in place
        for s in srcs:
            s.mul_(0.5).add_(float(r))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (out_fused.clone(), out_ring.clone(), [o.clone() for o in b_outs])
        # eager reference of the same inputs
        ref_fused = torch.empty_like(out_fused)
        xr.allreduce_local(srcs, ref_fused)
        ref_ring = torch.empty_like(out_ring)
        xr.ring_reduce(aligned, ref_ring)
        ref_b = [torch.empty_like(o) for o in b_outs]
        xr.batched_reduce([(i[0], o) for i, o in zip(b_items, ref_b)], dtype="bf16")
        torch.cuda.synchronize()
        assert torch.equal(got[0].view(torch.int16), ref_fused.view(torch.int16)), r
        assert torch.equal(got[1].view(torch.int16), ref_ring.view(torch.int16)), r
        for a, b in zip(got[2], ref_b):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), r
    del keep


def test_graph_capture_more_paths(xr):
    """fp8 fused, fp16 AVG batched and the simulated ring (one launch per step)
    captured once and replayed with eager input changes between replays."""
    g_torch = torch.Generator(device="cuda")
    g_torch.manual_seed(11)
    n = (1 << 16) + 37
    e4 = [torch.randint(0, 0x40, (n,), generator=g_torch, dtype=torch.uint8, device="cuda")
          for _ in range(5)]
    h = [torch.randn(n, device="cuda").to(torch.float16) for _ in range(4)]
    sim_s = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(4)]
    out_e4 = torch.empty_like(e4[0])
    out_h = torch.empty_like(h[0])
    sim_r = [torch.empty_like(x) for x in sim_s]
    h_items, keep = _device_items(xr, [(h, out_h)])

    def work():
        xr.allreduce_local(e4, out_e4, "sum", dtype="e4m3")
        xr.batched_reduce(h_items, "avg", dtype="f16")
        xr.allreduce_sim(sim_s, sim_r, schedule="ring")

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        work()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    torch.cuda.synchronize()
    for r in range(4):
        for x in e4:
            x.add_(1).bitwise_and_(0x3F)
        for x in h + sim_s:
            x.mul_(0.5).add_(float(r))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (out_e4.clone(), out_h.clone(), [x.clone() for x in sim_r])
        ref_e4 = torch.empty_like(out_e4)
        xr.allreduce_local(e4, ref_e4, "sum", dtype="e4m3")
        ref_h = torch.empty_like(out_h)
        xr.batched_reduce([(h, ref_h)], "avg", dtype="f16")
        ref_r = [torch.empty_like(x) for x in sim_s]
        xr.allreduce_sim(sim_s, ref_r, schedule="ring")
        torch.cuda.synchronize()
        assert torch.equal(got[0], ref_e4), r
        assert torch.equal(got[1].view(torch.int16), ref_h.view(torch.int16)), r
        for a, b in zip(got[2], ref_r):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), r
    del keep


# the refused call enqueues nothing, so the captured graph is empty by design
@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")
def test_host_descriptors_refuse_capture(xr):
    """Host-mode batches are staged through reused slots, so capturing one is
    refused before anything is enqueued; the same call works eagerly after."""
    srcs = [torch.randn(3000, device="cuda").to(torch.bfloat16) for _ in range(3)]
    out = torch.empty_like(srcs[0])
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        xr.batched_reduce([(srcs, out)], dtype="bf16")
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with pytest.raises(xr.XredError) as e:
        with torch.cuda.graph(g):
            xr.batched_reduce([(srcs, out)], dtype="bf16")
    assert e.value.name == "XRED_UNSUPPORTED", e.value
    torch.cuda.synchronize()
    ref = torch.empty_like(out)
    xr.allreduce_local(srcs, ref)
    out.zero_()
    xr.batched_reduce([(srcs, out)], dtype="bf16")
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))

