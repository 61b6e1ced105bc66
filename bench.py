#!/usr/bin/env python3
"""Benchmark of libxred on one MI355X.

The headline step is one xred_allreduce_local call on the gradient-bucket
workload: P=8 source buffers x 64M bf16 (128 MiB each), binary32
accumulation in rank order, bf16 output.  Throughput counts algorithmic bytes
(P+1)*N*sizeof per call, with inputs resident in HBM before timing starts.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-secondary] [--no-cpu-baseline]

Prints ONE JSON line on stdout.  Timing: W untimed calls, then K calls
bracketed by a synchronisation and HIP events recorded on the stream the
kernels are launched on; ms_per_step = event time / K.  The roofline object
uses the same events; `traffic` comes from the committed rocprofv3 counter
summary of the same kernel and is null when the kernel sources changed since.
The cpu_baseline object times the CPU oracle on a bounded sample on this
host.  Secondary workloads (the other configurations) are reported under
"secondary" and are not part of `value`.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time
from pathlib import Path

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

METRIC = "reduce-copy GB/s (read+write) and % HBM peak at 1 GPU; small-msg µs/call"
HBM_PEAK_GBS = 8000.0     # MI355X HBM3E, published
# workloads --workload can time; the variants reuse another workload's inputs
WORKLOAD_NAMES = ("c1", "c2", "c3", "c3ring", "c3ringflags", "c4", "c4dev", "c5a", "c5b", "c2fp8",
                  "sim", "sim1")
WORKLOAD_OF = {"c3ring": "c3", "c3ringflags": "c3", "c4dev": "c4"}
CSRC = "paper_2510_20171_amd/csrc/"
_COMMON = [CSRC + "xred_device.hpp", CSRC + "xred_kernels.hpp", CSRC + "xred_dispatch.hpp"]
KERNEL_SOURCES = {
    "reduce": _COMMON + [CSRC + f for f in ("xred_reduce.hpp", "xred_reduce.hip",
                                           "xred_reduce_float.hip", "xred_reduce_fp8.hip",
                                           "xred_reduce_int.hip", "xred_reduce_ext.hip")],
    "step": _COMMON + [CSRC + "xred_step.hip"],
    "batched": _COMMON + [CSRC + f for f in ("xred_batched.hpp", "xred_batched.hip",
                                            "xred_batched_float.hip", "xred_batched_fp8.hip",
                                            "xred_batched_int.hip", "xred_batched_ext.hip")],
    "ring": _COMMON + [CSRC + "xred_ring.hip"],
    "sim": _COMMON + [CSRC + "xred_sim.hip"],
}


def kernel_source_sha(family: str = "reduce") -> str:
    """Hash of a kernel family's sources with comments and blank space
    removed, so that editing a comment keeps its counter profile current."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[family]:
        text = (ROOT / f).read_text()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def committed_traffic(profile: Path, family: str):
    """HBM bytes per launch from a committed counter summary, if it still
    describes the current kernel sources."""
    if not profile.exists():
        return None
    text = profile.read_text()
    sha = re.search(r"kernel_source_sha:\s*([0-9a-f]+)", text)
    tb = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not sha or not tb or sha.group(1) != kernel_source_sha(family):
        return None
    return float(tb.group(1))


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Timer:
    """HIP events on the current stream (the stream every call is launched on)."""

    def __init__(self, torch):
        self.torch = torch
        self.e0 = torch.cuda.Event(enable_timing=True)
        self.e1 = torch.cuda.Event(enable_timing=True)

    def loop_ms(self, fn, reps: int, warm: int = 3) -> float:
        for _ in range(warm):
            fn()
        self.torch.cuda.synchronize()
        self.e0.record()
        for _ in range(reps):
            fn()
        self.e1.record()
        self.e1.synchronize()
        return self.e0.elapsed_time(self.e1) / reps

    def single_ms(self, fn, reps: int) -> list:
        out = []
        for _ in range(reps):
            self.e0.record()
            fn()
            self.e1.record()
            self.e1.synchronize()
            out.append(self.e0.elapsed_time(self.e1))
        return out

    def cold_ms(self, fn, reps: int, flush) -> list:
        """Each call after evicting L2 and the 256 MB MALL: 1 GiB is written and then
        read, so the caches end up holding clean lines of the flush buffer only (a
        write alone would leave dirty lines whose write-back the timed call pays)."""
        out = []
        sink = getattr(self, "_sink", None)
        if sink is None:
            sink = self._sink = self.torch.empty((), dtype=flush.dtype, device=flush.device)
        for _ in range(reps):
            flush.zero_()
            self.torch.sum(flush, dim=0, out=sink)
            self.e0.record()
            fn()
            self.e1.record()
            self.e1.synchronize()
            out.append(self.e0.elapsed_time(self.e1))
        return out


class PinnedWords:
    """n uint32 words of hipHostMalloc'd host memory, with their device address."""

    def __init__(self, n: int):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipHostMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t,
                                           ctypes.c_uint]
        self.hip.hipHostGetDevicePointer.argtypes = [ctypes.POINTER(ctypes.c_void_p),
                                                     ctypes.c_void_p, ctypes.c_uint]
        self.hip.hipHostFree.argtypes = [ctypes.c_void_p]
        self.host, self.dev = ctypes.c_void_p(), ctypes.c_void_p()
        if self.hip.hipHostMalloc(ctypes.byref(self.host), 4 * n, 0) != 0:
            raise RuntimeError("hipHostMalloc failed")
        if self.hip.hipHostGetDevicePointer(ctypes.byref(self.dev), self.host, 0) != 0:
            raise RuntimeError("hipHostGetDevicePointer failed")
        self.words = (ctypes.c_uint32 * n).from_address(self.host.value)
        for i in range(n):
            self.words[i] = 0

    def free(self):
        if self.host:
            self.hip.hipHostFree(self.host)
            self.host = None


def call_sync_us(torch, fn, reps: int) -> list:
    """Wall-clock µs of one call followed by a synchronisation of its stream."""
    stream = torch.cuda.current_stream()
    fn()
    stream.synchronize()
    out = []
    for _ in range(reps):
        t0 = time.perf_counter()
        fn()
        stream.synchronize()
        out.append((time.perf_counter() - t0) * 1e6)
    return out


def median(xs):
    xs = sorted(xs)
    return xs[len(xs) // 2]


def dev_bf16(torch, a):
    import numpy as np
    return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to("cuda")


def dev_any(torch, a, dtype):
    import numpy as np
    if dtype == "bf16":
        return dev_bf16(torch, a)
    if dtype == "f32":
        return torch.from_numpy(a).to("cuda")
    if dtype == "e4m3":
        return torch.from_numpy(a).to("cuda")
    return torch.from_numpy(a.view(np.int32)).to("cuda")


def reduce_call(L, xr, srcs, out, dtype, op):
    """A prebuilt C-ABI call (no per-call Python marshalling in the timed loop)."""
    arr = xr._lib.ptr_array([s.data_ptr() for s in srcs])
    n, P = out.numel(), len(srcs)
    dptr = ctypes.c_void_p(out.data_ptr())
    dt, o = xr.DTYPE[dtype], xr.OP[op]
    import torch
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)

    def fn():
        st = L.xred_allreduce_local(arr, P, dptr, n, dt, o, stream)
        if st:
            xr._lib.check(st)
    fn._keep = arr
    return fn


def cpu_baseline(srcs_np, dtype, op, P, es, target_s=10.0):
    import oracle
    orc = oracle.load()
    cores = min(16, oracle.host_cores())
    n = srcs_np[0].size
    t0 = time.perf_counter()
    orc.allreduce_local(srcs_np, dtype, op, nthreads=cores)
    t1 = time.perf_counter() - t0
    reps = max(1, int(target_s / max(t1, 1e-3)))
    t0 = time.perf_counter()
    for _ in range(reps):
        orc.allreduce_local(srcs_np, dtype, op, nthreads=cores)
    el = time.perf_counter() - t0
    gbs = (P + 1) * n * es * reps / el / 1e9
    # the same oracle on one core, for about 3 s
    t0 = time.perf_counter()
    reps1 = 0
    while time.perf_counter() - t0 < 3.0:
        orc.allreduce_local(srcs_np, dtype, op, nthreads=1)
        reps1 += 1
    el1 = time.perf_counter() - t0
    return {"value": round(gbs, 3), "unit": "GB/s", "cores": cores, "kind": "oracle",
            "sample": f"first {n} elements of each of the P={P} sources, {reps} reps, "
                      f"{el:.1f} s, OpenMP over elements",
            "one_core_value": round((P + 1) * n * es * reps1 / el1 / 1e9, 3),
            "host_cores_available": oracle.host_cores(), "cpu_model": cpu_model()}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def secondary(torch, xr, L, timer, wl, flush, res):
    """The figures besides the headline, filled into `res` as they are taken
    (so a failure part-way keeps the ones already measured)."""
    import numpy as np
    # copy ceiling (torch's device copy kernel), 1 GiB -> 1 GiB
    a = torch.empty(1 << 29, dtype=torch.int16, device="cuda")
    b = torch.empty_like(a)
    ms = timer.loop_ms(lambda: b.copy_(a), 10)
    res["copy_ceiling_GBs"] = round(2 * a.numel() * 2 / (ms * 1e-3) / 1e9, 1)
    del a, b

    # c1: P=4 x 1M f32 (20 MiB: cache resident); warm and cold
    w = wl.WORKLOADS["c1"]
    d = [dev_any(torch, s, "f32") for s in wl.sources(w)]
    out = torch.empty_like(d[0])
    fn = reduce_call(L, xr, d, out, "f32", "sum")
    ab = w.alg_bytes()
    warm = timer.loop_ms(fn, 1000)
    cold = median(timer.cold_ms(fn, 30, flush))
    wall_us = median(call_sync_us(torch, fn, 200))
    res["c1"] = {"us_per_call_warm": round(warm * 1e3, 2), "GBs_warm": round(ab / warm / 1e6, 1),
                 "us_cold": round(cold * 1e3, 2), "GBs_cold": round(ab / cold / 1e6, 1),
                 "us_call_and_sync_p50": round(wall_us, 1)}
    del d, out

    # c3: step-wise ring, 16 chunks x 1M bf16 into a binary32 accumulator
    w = wl.WORKLOADS["c3"]
    chunks = [dev_bf16(torch, c.copy()) for c in wl.stepwise_chunks(w)]
    acc = torch.empty(w.count, dtype=torch.float32, device="cuda")
    out = torch.empty_like(chunks[0])
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    cp = [ctypes.c_void_p(c.data_ptr()) for c in chunks]
    ap, op_ = ctypes.c_void_p(acc.data_ptr()), ctypes.c_void_p(out.data_ptr())

    def seq():
        L.xred_reduce_copy_step(cp[0], ap, None, w.count, 1, 0, 1, stream)
        for c in cp[1:]:
            L.xred_reduce_copy_step(c, ap, None, w.count, 1, 0, 0, stream)
        L.xred_acc_cast(ap, op_, w.count, 1, stream)

    def steps15():
        for c in cp[1:]:
            L.xred_reduce_copy_step(c, ap, None, w.count, 1, 0, 0, stream)
    seq_ms = timer.loop_ms(seq, 50)
    st_ms = timer.loop_ms(steps15, 50) / 15
    # the same sequence captured once in a HIP graph (17 kernel nodes) and
    # replayed; its output is checked against the eager sequence's
    seq()
    eager = out.clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        cs = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        L.xred_reduce_copy_step(cp[0], ap, None, w.count, 1, 0, 1, cs)
        for c in cp[1:]:
            L.xred_reduce_copy_step(c, ap, None, w.count, 1, 0, 0, cs)
        L.xred_acc_cast(ap, op_, w.count, 1, cs)
    out.zero_()
    graph_ms = timer.loop_ms(graph.replay, 50)
    torch.cuda.synchronize()
    graph_ok = bool(torch.equal(out.view(torch.int16), eager.view(torch.int16)))
    del graph
    fused = torch.empty_like(out)
    ffn = reduce_call(L, xr, chunks, fused, "bf16", "sum")
    fused_ms = timer.loop_ms(ffn, 50)
    ring_arr = xr._lib.ptr_array([c.data_ptr() for c in chunks])
    ring_out = ctypes.c_void_p(fused.data_ptr())
    ring_ms = timer.loop_ms(lambda: L.xred_ring_reduce(ring_arr, 16, ring_out, w.count, 1, 0, None,
                                                       1, 0, None, stream), 50)
    flags = PinnedWords(16)
    for i in range(16):
        flags.words[i] = 1
    ring_flag_ms = timer.loop_ms(lambda: L.xred_ring_reduce(ring_arr, 16, ring_out, w.count, 1, 0,
                                                            flags.dev, 1, 0, None, stream), 50)
    # per-step cost of observing an already-set host flag: 64 steps on one tile
    tiny = [torch.ones(4096, dtype=torch.bfloat16, device="cuda") for _ in range(64)]
    tiny_arr = xr._lib.ptr_array([c.data_ptr() for c in tiny])
    tiny_out = torch.empty_like(tiny[0])
    flags64 = PinnedWords(64)
    for i in range(64):
        flags64.words[i] = 1
    t_none = timer.loop_ms(lambda: L.xred_ring_reduce(tiny_arr, 64, ctypes.c_void_p(tiny_out.data_ptr()),
                                                      4096, 1, 0, None, 1, 0, None, stream), 50)
    t_flag = timer.loop_ms(lambda: L.xred_ring_reduce(tiny_arr, 64, ctypes.c_void_p(tiny_out.data_ptr()),
                                                      4096, 1, 0, flags64.dev, 1, 0, None, stream), 50)
    torch.cuda.synchronize()
    flags.free()
    flags64.free()
    moved = 16 * w.count * 2 + 15 * w.count * 8 + w.count * 4 + w.count * 4 + w.count * 2
    res["c3"] = {"us_per_step": round(st_ms * 1e3, 2),
                 "step_GBs_moved": round(w.count * 10 / st_ms / 1e6, 1),
                 "us_sequence": round(seq_ms * 1e3, 2),
                 "us_sequence_graph_replay": round(graph_ms * 1e3, 2),
                 "graph_replay_matches_eager": graph_ok,
                 "sequence_GBs_alg": round(17 * w.count * 2 / seq_ms / 1e6, 1),
                 "sequence_GBs_moved": round(moved / seq_ms / 1e6, 1),
                 "fused_16src_us": round(fused_ms * 1e3, 2),
                 "fused_16src_GBs": round(17 * w.count * 2 / fused_ms / 1e6, 1),
                 "ring_one_launch_us": round(ring_ms * 1e3, 2),
                 "ring_one_launch_GBs": round(17 * w.count * 2 / ring_ms / 1e6, 1),
                 "ring_host_flags_preset_us": round(ring_flag_ms * 1e3, 2),
                 "ring_64_steps_1_tile_us": round(t_none * 1e3, 2),
                 "ring_64_steps_1_tile_host_flags_us": round(t_flag * 1e3, 2),
                 "host_flag_poll_us_per_step": round((t_flag - t_none) * 1e3 / 64, 3)}
    del chunks, acc, out, fused

    # c5a / c5b: P=32 x 8M
    for name in ("c5a", "c5b"):
        w = wl.WORKLOADS[name]
        d = [dev_any(torch, s, w.dtype) for s in wl.sources(w)]
        out = torch.empty_like(d[0])
        fn = reduce_call(L, xr, d, out, w.dtype, w.op)
        ms = timer.loop_ms(fn, 20)
        gbs = w.alg_bytes() / ms / 1e6
        res[name] = {"us": round(ms * 1e3, 1), "GBs": round(gbs, 1),
                     "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 1)}
        del d, out

    # c4: 4096 small reductions in one launch (host and device descriptors)
    w = wl.WORKLOADS["c4"]
    sizes = wl.batched_sizes(w)
    arena, offs = wl.batched_arena(w, sizes)
    arena_d = dev_bf16(torch, arena)
    del arena
    base = arena_d.data_ptr()
    # outputs packed at 128-element (256 B) boundaries: item k at opos[k]
    ends = np.cumsum((sizes + 127) // 128 * 128)
    opos = np.concatenate([[0], ends[:-1]]).astype(np.int64)
    outs = torch.empty(int(ends[-1]), dtype=torch.bfloat16, device="cuda")
    assert int(opos[-1]) + int(sizes[-1]) <= outs.numel()
    P = offs.shape[1]
    ptr_rows = [(ctypes.c_void_p * P)(*[base + int(o) * 2 for o in offs[k]]) for k in range(len(sizes))]
    items = xr.pack_items([(ctypes.addressof(ptr_rows[k]), outs.data_ptr() + int(opos[k]) * 2,
                            int(sizes[k]), P) for k in range(len(sizes))])
    K = len(sizes)
    host_fn = lambda: L.xred_batched_reduce(items, K, 1, 0, 0, stream)  # noqa: E731
    ptrs_d = torch.tensor((base + offs * 2).reshape(-1).astype(np.int64), device="cuda")
    arr = np.zeros(K, xr.ITEM_DTYPE)
    arr["srcs"] = ptrs_d.data_ptr() + 8 * P * np.arange(K, dtype=np.uint64)
    arr["dst"] = outs.data_ptr() + opos.astype(np.uint64) * 2
    arr["count"] = sizes
    arr["nsrc"] = P
    items_d = torch.from_numpy(arr.view(np.uint8).copy()).to("cuda")
    dev_fn = lambda: L.xred_batched_reduce(ctypes.c_void_p(items_d.data_ptr()), K, 1, 0, 1,  # noqa
                                           stream)
    noalloc_fn = lambda: L.xred_batched_reduce_noalloc(  # noqa: E731
        ctypes.c_void_p(items_d.data_ptr()), K, 1, 0, stream)
    ab = w.alg_bytes(sizes)
    # 30 calls after 5: the first call's host plan, built while the GPU is
    # idle, weighs on the average of a short loop
    host_ms = timer.loop_ms(host_fn, 30, warm=5)
    dev_ms = timer.loop_ms(dev_fn, 30, warm=5)
    noalloc_ms = timer.loop_ms(noalloc_fn, 30, warm=5)
    singles = [reduce_call(L, xr, [arena_d[int(o):int(o) + int(sizes[k])] for o in offs[k]],
                           outs[int(opos[k]):int(opos[k]) + int(sizes[k])], "bf16", "sum")
               for k in range(K)]

    def all_singles():
        for f in singles:
            f()
    sep_ms = timer.loop_ms(all_singles, 3, warm=1)
    res["c4"] = {"alg_bytes": ab, "items": K,
                 "host_desc_us": round(host_ms * 1e3, 1), "host_desc_GBs": round(ab / host_ms / 1e6, 1),
                 "device_desc_us": round(dev_ms * 1e3, 1),
                 "device_desc_GBs": round(ab / dev_ms / 1e6, 1),
                 "device_desc_noalloc_us": round(noalloc_ms * 1e3, 1),
                 "us_per_item": round(host_ms * 1e3 / K, 3),
                 "separate_calls_us": round(sep_ms * 1e3, 1),
                 "separate_calls_GBs": round(ab / sep_ms / 1e6, 1)}
    del arena_d, outs, items_d, ptrs_d, singles

    res["stream_mix_ceiling"] = stream_mix_ceiling(torch, xr, L, timer)
    res["small_calls"] = small_calls(torch, xr, L)
    res["flag_handoff"] = flag_handoff(torch)

    # CU budget: GB/s of the P=8 bf16 reduce on FTAR-sized 8 MiB chunks
    # (4M elements per source) as the workgroup budget grows
    n = 4 << 20
    d = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(8)]
    out = torch.empty_like(d[0])
    fn = reduce_call(L, xr, d, out, "bf16", "sum")
    curve = {}
    for cap in (1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 0):
        prev = L.xred_set_max_workgroups(cap)
        try:
            ms = timer.loop_ms(fn, 20 if cap == 0 or cap >= 8 else 5, warm=1)
        finally:
            L.xred_set_max_workgroups(prev)
        curve[str(cap) if cap else "all"] = round(9 * n * 2 / ms / 1e6, 1)
    res["cu_budget_p8_bf16_8MiB_GBs"] = curve
    del d, out

    # further element types and AVG at the gradient-bucket footprint: P=8
    # sources of 128 MiB each (random bytes; float bytes masked to finite values)
    more = {}
    for dt, es, op in (("f16", 2, "sum"), ("e4m3", 1, "sum"), ("e5m2", 1, "sum"),
                       ("i64", 8, "sum"), ("bf16", 2, "avg"), ("f32", 4, "avg"),
                       ("f64", 8, "sum"), ("i8", 1, "sum"), ("u8", 1, "max")):
        n = (128 << 20) // es
        d = []
        for _ in range(8):
            x = torch.randint(0, 256, (n * es,), dtype=torch.uint8, device="cuda")
            if dt in ("e4m3", "e5m2"):
                x &= 0x3F if dt == "e4m3" else 0x3B     # finite magnitudes below 1
            elif dt in ("f16", "bf16", "f32"):
                x.view(torch.int16 if es == 2 else torch.int32).bitwise_and_(
                    0x3BFF if dt == "f16" else (0x3F7F if dt == "bf16" else 0x3F7FFFFF))
            elif dt == "f64":
                x.view(torch.int64).bitwise_and_(0x3FEFFFFFFFFFFFFF)   # finite, below 1
            d.append(x)
        out = torch.empty_like(d[0])
        arr = xr._lib.ptr_array([x.data_ptr() for x in d])
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        fn = (lambda a=arr, o=out, nn=n, t=xr.DTYPE[dt], oo=xr.OP[op]:
              L.xred_allreduce_local(a, 8, ctypes.c_void_p(o.data_ptr()), nn, t, oo, stream))
        ms = timer.loop_ms(fn, 20)
        more[f"{dt}_{op}_p8_128MiB"] = {"us": round(ms * 1e3, 2),
                                        "GBs": round(9 * n * es / ms / 1e6, 1)}
        del d, out
    res["more_types"] = more

    # simulated AllReduce schedules on one GPU: 8 ranks, ring and halving-doubling,
    # one launch per step and all steps in one launch ("ring1", "rhd1"), at the
    # bucket size and at 1 MiB per rank; GB/s counts each form's own algorithmic
    # bytes (5 (G-1) N per step schedule, 2 G N in one launch)
    sim = {}
    for label, n in (("64M", 64 << 20), ("512K", 512 << 10)):
        sends = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(8)]
        recvs = [torch.empty_like(x) for x in sends]
        arr_s = xr._lib.ptr_array([x.data_ptr() for x in sends])
        arr_r = xr._lib.ptr_array([x.data_ptr() for x in recvs])
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        for sched in ("ring", "rhd", "ring1", "rhd1"):
            fn = (lambda sc=xr.SCHEDULE[sched]:
                  L.xred_allreduce_sim(arr_s, arr_r, 8, n, 1, 0, sc, stream))
            ms = timer.loop_ms(fn, 20 if n > (1 << 20) else 200)
            ab = (2 * 8 if sched.endswith("1") else 5 * 7) * n * 2
            sim[f"{sched}_{label}"] = {"us": round(ms * 1e3, 2), "GBs": round(ab / ms / 1e6, 1)}
        del sends, recvs
    res["sim_g8_bf16"] = sim

    # small-message latency: P=8 bf16, back-to-back and single call
    lat = {}
    # 16 MiB per source is one GPU's share of a c2 bucket reduce-scattered over 8 GPUs
    for kib in (8, 64, 1024, 8192, 16384, 32768, 131072):
        n = kib * 1024 // 2
        d = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(8)]
        out = torch.empty_like(d[0])
        fn = reduce_call(L, xr, d, out, "bf16", "sum")
        ms = timer.loop_ms(fn, 1000 if kib <= 1024 else 200 if kib <= 16384 else 50)
        lat[f"{kib}KiB"] = {"us_per_call": round(ms * 1e3, 2),
                            "GBs": round(9 * n * 2 / ms / 1e6, 1)}
        if kib <= 1024:
            one = median(call_sync_us(torch, fn, 200))
            lat[f"{kib}KiB"]["us_call_and_sync_p50"] = round(one, 1)
        del d, out
    res["latency_p8_bf16"] = lat

    # reduce-scatter over the same share (P=8 bf16, 8 ranks, shards of 2^23
    # and 2^23 + 1 elements): with the odd length rank 1's shard starts 2
    # bytes past a 16-byte boundary in every send buffer while its output is
    # aligned (the realigned stores); rank 0's is aligned either way
    rs = {}
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for rc in (1 << 23, (1 << 23) + 1):
        sends = [torch.empty(8 * rc, dtype=torch.bfloat16, device="cuda").uniform_(-1, 1)
                 for _ in range(8)]
        out = torch.empty(rc, dtype=torch.bfloat16, device="cuda")
        arr = xr._lib.ptr_array([t.data_ptr() for t in sends])
        for rank in (0, 1):
            ms = timer.loop_ms(lambda: L.xred_reduce_scatter_local(
                arr, 8, rank, ctypes.c_void_p(out.data_ptr()), rc, 1, 0, stream), 200)
            rs[f"recvcount_{rc}_rank{rank}"] = {"us_per_call": round(ms * 1e3, 2),
                                                "GBs": round(9 * rc * 2 / ms / 1e6, 1)}
        del sends, out, arr
        torch.cuda.empty_cache()
    res["reduce_scatter_p8_bf16_share"] = rs

    # messages larger than the bucket: 8 bf16 sources of 256 and 512 MiB (the
    # launches whose occupancy cap grows with the bytes per source)
    big = {}
    for mib in (256, 512):
        n = mib << 19
        d = [torch.empty(n, dtype=torch.bfloat16, device="cuda").normal_() for _ in range(8)]
        out = torch.empty_like(d[0])
        ms = timer.loop_ms(reduce_call(L, xr, d, out, "bf16", "sum"), 10)
        big[f"{mib}MiB"] = {"us": round(ms * 1e3, 1), "GBs": round(9 * n * 2 / ms / 1e6, 1)}
        del d, out
        torch.cuda.empty_cache()
    res["large_p8_bf16"] = big

    # co-scheduling: P=8 bf16 x 8 MiB reduces on one stream while bf16 8192^3
    # matrix products run on another (both default priority), on two ordinary
    # streams (per workgroup budget) and on the two streams of a CU partition
    # (the reduce on 16 or 32 CUs, the products on the others); the reduce loop
    # alone lasts about as long as the products
    n = 4 << 20
    d = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(8)]
    out = torch.empty_like(d[0])
    arr = xr._lib.ptr_array([x.data_ptr() for x in d])
    ga = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    gb = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    gc = torch.empty_like(ga)
    reps_g = 20

    def run(sg, sr, g, reps_r):
        """(products' span, reduces' span, span of both) in ms."""
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        torch.cuda.synchronize()
        ev[0].record(sg)
        ev[2].record(sr)
        if g:
            with torch.cuda.stream(sg):
                for _ in range(reps_g):
                    torch.mm(ga, gb, out=gc)
        st = ctypes.c_void_p(sr.cuda_stream)
        for _ in range(reps_r):
            L.xred_allreduce_local(arr, 8, ctypes.c_void_p(out.data_ptr()), n, 1, 0, st)
        ev[1].record(sg)
        ev[3].record(sr)
        torch.cuda.synchronize()
        ends = (ev[0].elapsed_time(ev[1]), ev[0].elapsed_time(ev[3]))
        both = max(ends) - min(0.0, ev[0].elapsed_time(ev[2]))
        return ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[3]), both

    def pair(sg, sr):
        """The two loops alone and together on streams sg (products) and sr."""
        run(sg, sr, True, 10)
        g_alone, _, _ = run(sg, sr, True, 0)
        _, r1, _ = run(sg, sr, False, 100)
        reps = max(10, int(g_alone / (r1 / 100)))
        _, r_alone, _ = run(sg, sr, False, reps)
        g_with, r_with, both = run(sg, sr, True, reps)
        # the two streams overlapped only if both finished well before
        # the sum of their times alone
        overlapped = both < 0.9 * (g_alone + r_alone)
        e = {"gemm_ms_alone": round(g_alone / reps_g, 3),
             "reduce_us_alone": round(r_alone / reps * 1e3, 1),
             "reduce_GBs_alone": round(9 * n * 2 * reps / r_alone / 1e6, 1),
             "reduce_us_with_gemm": round(r_with / reps * 1e3, 1),
             "span_both_ms": round(both, 3), "sum_alone_ms": round(g_alone + r_alone, 3),
             "overlapped": overlapped}
        if overlapped:
            e["gemm_slowdown_pct"] = round(100 * (g_with / g_alone - 1), 1)
        return e, reps

    sg, sr = torch.cuda.Stream(), torch.cuda.Stream()
    run(sg, sr, True, 10)
    g_full, _, _ = run(sg, sr, True, 0)
    co = {"gemm_alone_ms": round(g_full / reps_g, 3),
          "gemm_TFLOPs": round(2 * 8192 ** 3 * reps_g / g_full / 1e9, 0)}
    prev = xr.set_max_workgroups(0)
    try:
        for budget in (16, 0):
            xr.set_max_workgroups(budget)
            co[f"streams_budget_{budget or 'none'}"], _ = pair(sg, sr)
    finally:
        xr.set_max_workgroups(prev)
    # the same work on the whole chip, one loop after the other
    _, r_full, _ = run(sg, sr, False, 200)
    for ncu in (16, 32):
        try:
            a, b = xr.stream_create_partition(ncu)
        except xr.XredError as err:   # the runtime may refuse more hardware queues
            co[f"partition_{ncu}_cus"] = {"error": str(err)}
            continue
        try:
            e, reps = pair(torch.cuda.ExternalStream(b), torch.cuda.ExternalStream(a))
        finally:
            xr.stream_destroy(a)
            xr.stream_destroy(b)
        e["serial_on_all_cus_ms"] = round(g_full + r_full / 200 * reps, 3)
        co[f"partition_{ncu}_cus"] = e
    res["coschedule_gemm_bf16"] = co
    del d, out, ga, gb, gc
    return res


def stream_mix_ceiling(torch, xr, L, timer):
    """The traffic-only ceiling of three stream mixes (libxred_ceiling.so:
    the fused kernel's tiles reading and writing the same streams with no
    fold), best over resident-wave caps, next to libxred on the same buffers:
    8 reads + 1 write of 128 MiB (the bucket), 32 reads + 1 write of 32 MiB
    (the extremum/integer configuration) and 8 reads + 8 writes of 128 MiB
    (a simulated 8-rank AllReduce in one launch)."""
    C = ctypes.CDLL(str(ROOT / "paper_2510_20171_amd" / "libxred_ceiling.so"))
    C.xred_ceiling_mix.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                                   ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    out = {}
    for name, nsrc, ndst, mib in (("c2_8r1w_128MiB", 8, 1, 128), ("c5_32r1w_32MiB", 32, 1, 32),
                                  ("sim1_8r8w_128MiB", 8, 8, 128)):
        n = mib << 20
        srcs = [torch.randint(-2 ** 31, 2 ** 31 - 1, (n // 4,), dtype=torch.int32, device="cuda")
                for _ in range(nsrc)]
        dsts = [torch.empty(n // 4, dtype=torch.int32, device="cuda") for _ in range(ndst)]
        sa = xr._lib.ptr_array([x.data_ptr() for x in srcs])
        da = xr._lib.ptr_array([x.data_ptr() for x in dsts])
        ab = (nsrc + ndst) * n
        caps = {}
        for waves in (4, 6, 8, 12, 16, 24, 0):
            fn = (lambda w_=waves: C.xred_ceiling_mix(sa, nsrc, da, ndst, n, w_, stream))
            if fn() != 0:
                raise RuntimeError("xred_ceiling_mix launch failed")
            ms = timer.loop_ms(fn, 10)
            caps[str(waves) if waves else "none"] = round(ab / ms / 1e6, 1)
        best = max(caps.values())
        if ndst == 1:
            # the bucket's own type for its shape; the integer configuration's for P=32
            dt, tt = ("bf16", torch.bfloat16) if nsrc == 8 else ("i32", torch.int32)
            lib_fn = reduce_call(L, xr, [x.view(tt) for x in srcs], dsts[0].view(tt), dt, "sum")
            what = f"xred_allreduce_local {dt} sum"
        else:
            lib_fn = (lambda: L.xred_allreduce_sim(sa, da, nsrc, n // 2, 1, 0,
                                                   xr.SCHEDULE["ring1"], stream))
            what = "xred_allreduce_sim bf16 sum ring1"
        lib_ms = timer.loop_ms(lib_fn, 10)
        lib = ab / lib_ms / 1e6
        out[name] = {"ceiling_GBs": best, "ceiling_by_waves_per_cu": caps,
                     "library": what, "library_GBs": round(lib, 1),
                     "library_frac_of_ceiling": round(lib / best, 4)}
        del srcs, dsts
        torch.cuda.empty_cache()
    return out


def flag_handoff(torch, rounds: int = 2000, skip: int = 16):
    """The host-to-kernel handoff of a flag in pinned host memory (the
    host-kernel coordinated mode of Section 4.1), as a ping-pong between a
    host thread and one polling lane (libxred_ceiling.so): the host's round
    trip is one handoff each way.  "relayed" passes the flag through a word in
    device memory to a second workgroup first, the hop the ring kernel's
    poller adds.  Per round the polling lane also counts its loads of the
    flag and times them on the device clock, which gives the latency of one
    poll of host memory."""
    import numpy as np
    C = ctypes.CDLL(str(ROOT / "paper_2510_20171_amd" / "libxred_ceiling.so"))
    C.xred_ceiling_handoff.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_uint32),
                                       ctypes.POINTER(ctypes.c_double), ctypes.c_void_p]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    out = {"rounds": rounds - skip}
    for name, relay in (("direct", 0), ("relayed", 1)):
        rtt = (ctypes.c_double * rounds)()
        polls = (ctypes.c_uint32 * rounds)()
        seen = (ctypes.c_double * rounds)()
        rc = C.xred_ceiling_handoff(rounds, relay, 1000, rtt, polls, seen, stream)
        if rc != 0:
            raise RuntimeError(f"xred_ceiling_handoff({name}) returned {rc}")
        r = np.array(rtt[skip:])
        n = np.array(polls[skip:], dtype=np.float64)
        t = np.array(seen[skip:])
        many = n >= 2
        out[name] = {"rtt_p10_us": round(float(np.percentile(r, 10)), 2),
                     "rtt_p50_us": round(float(np.percentile(r, 50)), 2),
                     "rtt_p90_us": round(float(np.percentile(r, 90)), 2),
                     "polls_per_round_p50": float(np.median(n)),
                     "poll_latency_us_p50": (round(float(np.median(t[many] / n[many])), 3)
                                             if many.any() else None)}
    out["one_way_us_est"] = round(out["direct"]["rtt_p50_us"] / 2, 2)
    out["relay_hop_us_p50"] = round(out["relayed"]["rtt_p50_us"] - out["direct"]["rtt_p50_us"], 2)
    return out


def small_calls(torch, xr, L):
    """One call and a synchronisation of its stream, wall clock (median of
    200): latency-bound batched and ring calls."""
    import numpy as np
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    res = {}
    n = 4096                                     # 8 KiB of bf16 per source
    for K in (64, 256):
        srcs = [torch.randn(K * n, device="cuda").to(torch.bfloat16) for _ in range(8)]
        out = torch.empty(K * n, dtype=torch.bfloat16, device="cuda")
        ptrs = torch.tensor([[s.data_ptr() + 2 * n * k for s in srcs] for k in range(K)],
                            dtype=torch.int64, device="cuda")
        arr = np.zeros(K, xr.ITEM_DTYPE)
        arr["srcs"] = ptrs.data_ptr() + 64 * np.arange(K, dtype=np.uint64)
        arr["dst"] = out.data_ptr() + 2 * n * np.arange(K, dtype=np.uint64)
        arr["count"] = n
        arr["nsrc"] = 8
        items_d = torch.from_numpy(arr.view(np.uint8).copy()).to("cuda")
        rows = [(ctypes.c_void_p * 8)(*[s.data_ptr() + 2 * n * k for s in srcs])
                for k in range(K)]
        items_h = xr.pack_items([(ctypes.addressof(rows[k]), out.data_ptr() + 2 * n * k, n, 8)
                                 for k in range(K)])
        dev = ctypes.c_void_p(items_d.data_ptr())
        res[f"batch_{K}x8KiB_device_desc_us"] = round(median(call_sync_us(
            torch, lambda: L.xred_batched_reduce(dev, K, 1, 0, 1, stream), 200)), 1)
        res[f"batch_{K}x8KiB_noalloc_us"] = round(median(call_sync_us(
            torch, lambda: L.xred_batched_reduce_noalloc(dev, K, 1, 0, stream), 200)), 1)
        res[f"batch_{K}x8KiB_host_desc_us"] = round(median(call_sync_us(
            torch, lambda: L.xred_batched_reduce(items_h, K, 1, 0, 0, stream), 200)), 1)
        del srcs, out, ptrs, items_d
    chunks = [torch.randn(1 << 16, device="cuda").to(torch.bfloat16) for _ in range(16)]
    ring_out = torch.empty_like(chunks[0])
    ca = xr._lib.ptr_array([c.data_ptr() for c in chunks])
    ro = ctypes.c_void_p(ring_out.data_ptr())
    flags = PinnedWords(16)
    for i in range(16):
        flags.words[i] = 1
    res["ring_16x64K_bf16_us"] = round(median(call_sync_us(
        torch, lambda: L.xred_ring_reduce(ca, 16, ro, 1 << 16, 1, 0, None, 1, 0, None, stream),
        200)), 1)
    res["ring_16x64K_bf16_host_flags_us"] = round(median(call_sync_us(
        torch, lambda: L.xred_ring_reduce(ca, 16, ro, 1 << 16, 1, 0, flags.dev, 1, 0, None,
                                          stream), 200)), 1)
    torch.cuda.synchronize()
    flags.free()
    return res


def build_workload(name, torch, xr, L, wl):
    """Inputs resident in HBM and one step of workload `name`.

    Returns a dict with the step callable, algorithmic bytes per step, the
    dominant kernel, its source family and committed profile, a config
    description, and a callable timing the CPU oracle on a bounded sample."""
    import numpy as np
    w = wl.WORKLOADS[WORKLOAD_OF.get(name, name)]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if name in ("c3ring", "c3ringflags"):
        log(f"generating c3 inputs for the one-launch ring (16 chunks x {w.count} bf16)")
        chunks_np = [c.copy() for c in wl.stepwise_chunks(w)]
        chunks = [dev_bf16(torch, c) for c in chunks_np]
        out = torch.empty_like(chunks[0])
        arr = xr._lib.ptr_array([c.data_ptr() for c in chunks])
        dptr = ctypes.c_void_p(out.data_ptr())
        flags = None
        if name == "c3ringflags":
            # every chunk's flag already set in pinned host memory: the launch
            # pays the poll and the relay, not a wait
            flags = PinnedWords(16)
            for i in range(16):
                flags.words[i] = 1

        def step():
            st = L.xred_ring_reduce(arr, 16, dptr, w.count, 1, 0,
                                    flags.dev if flags else None, 1, 0, None, stream)
            if st:
                xr._lib.check(st)
        step._keep_inputs = (chunks, out, arr, flags)
        how = ("chunks gated by host-pinned flags, all set" if flags else "all chunks ready")
        res = dict(step=step, alg_bytes=17 * w.count * 2, family="ring",
                   kernel="ring_kernel<bf16, sum>",
                   profile=ROOT / "profiles" / f"ring_bf16_{name}.md",
                   config={"workload": f"{name}: xred_ring_reduce of 16 chunks x "
                                       f"{w.count} bf16 in one launch, accumulator on chip, {how}",
                           "chunks": 16, "N": w.count, "io_dtype": "bf16"})
        res["cpu"] = lambda: cpu_baseline(chunks_np, "bf16", "sum", 16, 2)
        return res
    if w.kind == "allreduce":
        log(f"generating {name} inputs (P={w.nsrc} x {w.count} {w.dtype})")
        srcs_np = wl.sources(w)
        d = [dev_any(torch, s, w.dtype) for s in srcs_np]
        out = torch.empty_like(d[0])
        step = reduce_call(L, xr, d, out, w.dtype, w.op)
        step._keep_inputs = (d, out)
        es = wl.ELEM_SIZE[w.dtype]
        np_ = w.nsrc if w.nsrc <= 8 or w.nsrc in (16, 32, 64) else 0
        res = dict(step=step, alg_bytes=w.alg_bytes(), family="reduce",
                   kernel=f"reduce_vec_kernel<{w.dtype}, {w.op}, NP={np_}>",
                   profile=ROOT / "profiles" / f"reduce_{w.dtype}_{name}.md",
                   config={"workload": f"{name}: allreduce_local P={w.nsrc} x {w.count} {w.dtype}, "
                                       f"{w.op}, fixed rank order", "P": w.nsrc, "N": w.count,
                           "io_dtype": w.dtype})
        sample_n = min(w.count, (1 << 25) // w.nsrc)
        res["cpu"] = lambda: cpu_baseline([s[:sample_n] for s in srcs_np], w.dtype, w.op,
                                          w.nsrc, es)
        return res
    if w.kind == "sim":
        G, N = w.nsrc, w.count
        log(f"generating {name} inputs ({G} ranks x {N} {w.dtype})")
        sends_np = wl.sources(w)
        sends = [dev_bf16(torch, s) for s in sends_np]
        recvs = [torch.empty_like(s) for s in sends]
        arr_s = xr._lib.ptr_array([s.data_ptr() for s in sends])
        arr_r = xr._lib.ptr_array([r.data_ptr() for r in recvs])

        def step():
            st = L.xred_allreduce_sim(arr_s, arr_r, G, N, 1, 0, xr.SCHEDULE[w.schedule], stream)
            if st:
                xr._lib.check(st)
        step._keep_inputs = (sends, recvs, arr_s, arr_r)
        one = w.schedule.endswith("1")
        base = w.schedule.rstrip("1")
        if one:
            kernel = f"sim_all_kernel<bf16, sum, {base}, vec> (every step in one launch)"
            how = "every step in one launch, messages forwarded in registers"
        else:
            kernel = ("whole ring schedule: 7 x sim_step_vec_kernel<bf16, sum, reduce> + "
                      "7 x sim_step_vec_kernel<bf16, sum, copy>")
            how = "2(G-1) steps, zero-copy messages"
        res = dict(step=step, alg_bytes=w.alg_bytes(), family="sim", kernel=kernel,
                   profile=ROOT / "profiles" / f"sim_bf16_{name}.md",
                   config={"workload": f"{name}: {base} AllReduce of {G} simulated ranks x {N} "
                                       f"bf16 on one GPU ({how})",
                           "ranks": G, "N": N, "io_dtype": "bf16", "schedule": w.schedule})
        sample = [s[:1 << 22] for s in sends_np]

        def cpu():
            import oracle
            orc = oracle.load()
            cores = min(16, oracle.host_cores())
            t0 = time.perf_counter()
            reps = 0
            while time.perf_counter() - t0 < 10.0:
                orc.allreduce_sim(sample, "bf16", "sum", base, nthreads=cores)
                reps += 1
            el = time.perf_counter() - t0
            ab = w.alg_bytes() // N * sample[0].size * reps
            return {"value": round(ab / el / 1e9, 3), "unit": "GB/s", "cores": cores,
                    "kind": "oracle",
                    "sample": f"first {sample[0].size} elements of each rank, {reps} reps, "
                              f"{el:.1f} s, OpenMP over elements within each hop"}
        res["cpu"] = cpu
        return res
    if w.kind == "stepwise":
        log(f"generating {name} inputs (16 chunks x {w.count} bf16)")
        chunks_np = wl.stepwise_chunks(w)
        chunks = [dev_bf16(torch, c.copy()) for c in chunks_np]
        acc = torch.empty(w.count, dtype=torch.float32, device="cuda")
        out = torch.empty_like(chunks[0])
        cp = [ctypes.c_void_p(c.data_ptr()) for c in chunks]
        ap, op_ = ctypes.c_void_p(acc.data_ptr()), ctypes.c_void_p(out.data_ptr())

        def step():
            L.xred_reduce_copy_step(cp[0], ap, None, w.count, 1, 0, 1, stream)
            for c in cp[1:]:
                L.xred_reduce_copy_step(c, ap, None, w.count, 1, 0, 0, stream)
            L.xred_acc_cast(ap, op_, w.count, 1, stream)
        step._keep_inputs = (chunks, acc, out)
        res = dict(step=step, alg_bytes=17 * w.count * 2, family="step",
                   kernel="step_kernel<bf16, sum, 0>",
                   profile=ROOT / "profiles" / f"step_bf16_{name}.md",
                   config={"workload": f"{name}: INIT + 15 reduce_copy_step + acc_cast, "
                                       f"16 chunks x {w.count} bf16, fp32 accumulator",
                           "chunks": 16, "N": w.count, "io_dtype": "bf16"})
        res["cpu"] = lambda: cpu_baseline([c.copy() for c in chunks_np], "bf16", "sum", 16, 2)
        return res
    # batched
    sizes = wl.batched_sizes(w)
    log(f"generating {name} inputs ({len(sizes)} items, P={w.nsrc})")
    arena, offs = wl.batched_arena(w, sizes)
    arena_d = dev_bf16(torch, arena)
    base = arena_d.data_ptr()
    ends = np.cumsum((sizes + 127) // 128 * 128)
    opos = np.concatenate([[0], ends[:-1]]).astype(np.int64)
    outs = torch.empty(int(ends[-1]), dtype=torch.bfloat16, device="cuda")
    assert int(opos[-1]) + int(sizes[-1]) <= outs.numel()
    P, K = offs.shape[1], len(sizes)
    rows = [(ctypes.c_void_p * P)(*[base + int(o) * 2 for o in offs[k]]) for k in range(K)]
    items = xr.pack_items([(ctypes.addressof(rows[k]), outs.data_ptr() + int(opos[k]) * 2,
                            int(sizes[k]), P) for k in range(K)])

    if name == "c4dev":
        # the same items with descriptors and source-pointer arrays in device memory
        ptrs_d = torch.tensor((base + offs * 2).reshape(-1).astype(np.int64), device="cuda")
        arr = np.zeros(K, xr.ITEM_DTYPE)
        arr["srcs"] = ptrs_d.data_ptr() + 8 * P * np.arange(K, dtype=np.uint64)
        arr["dst"] = outs.data_ptr() + opos.astype(np.uint64) * 2
        arr["count"] = sizes
        arr["nsrc"] = P
        items_d = torch.from_numpy(arr.view(np.uint8).copy()).to("cuda")
        items_ptr = ctypes.c_void_p(items_d.data_ptr())

        def step():
            st = L.xred_batched_reduce(items_ptr, K, 1, 0, 1, stream)
            if st:
                xr._lib.check(st)
        step._keep_inputs = (arena_d, outs, ptrs_d, items_d)
        kernel, where = "batched_queue_kernel<bf16, sum, 2>", "device descriptors"
    else:
        def step():
            st = L.xred_batched_reduce(items, K, 1, 0, 0, stream)
            if st:
                xr._lib.check(st)
        step._keep_inputs = (arena_d, outs, rows, items)
        kernel, where = "batched_table_kernel<bf16, sum>", "host descriptors"
    res = dict(step=step, alg_bytes=w.alg_bytes(sizes), family="batched", kernel=kernel,
               profile=ROOT / "profiles" / f"batched_bf16_{name}.md",
               config={"workload": f"{name}: batched_reduce of {K} items, P={P} bf16, sizes "
                                   f"log-uniform 8 KiB-1 MiB per source, {where}",
                       "items": K, "P": P, "io_dtype": "bf16"})
    sample = [[arena[o:o + int(sizes[k])] for o in offs[k]] for k in range(64)]

    def cpu():
        import oracle
        orc = oracle.load()
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < 10.0:
            for s in sample:
                orc.allreduce_local(s, "bf16", "sum")
            reps += 1
        el = time.perf_counter() - t0
        ab = sum((P + 1) * s[0].size * 2 for s in sample) * reps
        return {"value": round(ab / el / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
                "sample": f"first 64 items, {reps} reps, {el:.1f} s, one thread"}
    res["cpu"] = cpu
    return res


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c2",
                    choices=WORKLOAD_NAMES,
                    help="which workload one step runs (default: the c2 gradient bucket)")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run 3 plain device copies of 1 GiB (for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: libxred's reduce step runs on a single MI355X "
              "and has no multi-GPU path; run with --gpus 1.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2510_20171_amd as xr
    import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    L = xr.load()
    timer = Timer(torch)
    wk = build_workload(args.workload, torch, xr, L, wl)
    step, ab = wk["step"], wk["alg_bytes"]

    log(f"timing {args.steps} steps after {args.warmup} warmup")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    timer.e0.record()
    for _ in range(args.steps):
        step()
    timer.e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = timer.e0.elapsed_time(timer.e1) / args.steps
    gbs = ab / (ms * 1e-3) / 1e9
    # per-call spread (with the secondary figures only, so that profiled runs
    # hold the timed loop's calls alone): each call between its own events,
    # back to back and after evicting L2 and the MALL
    per_call = None
    if not args.no_secondary:
        flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        single = sorted(timer.single_ms(step, max(10, args.steps)))
        cold = sorted(timer.cold_ms(step, max(10, min(args.steps, 30)), flush))
        pct = lambda xs, q: round(xs[min(len(xs) - 1, int(q * len(xs)))] * 1e3, 2)
        per_call = {"p10_us": pct(single, 0.1), "p50_us": pct(single, 0.5),
                    "p90_us": pct(single, 0.9), "cold_p50_us": pct(cold, 0.5),
                    "cold_p90_us": pct(cold, 0.9)}

    io = wk["config"].get("io_dtype")
    acc = ("f32" if io in ("bf16", "f32", "f16", "e4m3", "e5m2")
           else "u64" if io in ("i64", "u64") else "u32")
    config = dict(wk["config"], accumulate=acc, alg_bytes_per_step=ab, parallelism="single GPU")
    result = {
        "metric": METRIC, "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": config["accumulate"], "data": "synthetic", "config": config,
        "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "wall_s_timed": round(wall, 4),
        "per_call": per_call,
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": committed_traffic(wk["profile"], wk["family"]),
                     "kernel": wk["kernel"],
                     "kernel_source_sha": kernel_source_sha(wk["family"])},
    }
    if args.calibrate_copy:
        a = torch.empty(1 << 29, dtype=torch.int16, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        log("calibration: 3 copies of 1 GiB done")
        del a, b
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample")
        result["cpu_baseline"] = wk["cpu"]()
    del wk, step
    torch.cuda.empty_cache()
    if not args.no_secondary and args.workload == "c2":
        log("secondary workloads")
        flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        result["secondary"] = {}
        try:
            secondary(torch, xr, L, timer, wl, flush, result["secondary"])
        except Exception as e:   # a failed extra figure must not cost the headline line
            result["secondary"]["error"] = f"{type(e).__name__}: {e}"
            log(f"secondary figures stopped: {type(e).__name__}: {e}")
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
