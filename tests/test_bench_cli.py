"""bench.py's contract pieces that need no GPU: it refuses more than one GPU
with a message, and the algorithmic byte counts of the workloads are the
closed forms it reports (CPU)."""
import subprocess
import sys
from pathlib import Path

import workloads as wl

ROOT = Path(__file__).resolve().parents[1]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_bytes():
    M = 1 << 20
    # (P+1) N sizeof for a fused reduce: the bucket is 1,207,959,552 bytes
    assert wl.WORKLOADS["c2"].alg_bytes() == 9 * 64 * M * 2 == 1_207_959_552
    assert wl.WORKLOADS["c5a"].alg_bytes() == 33 * 8 * M * 4
    assert wl.WORKLOADS["c2fp8"].alg_bytes() == 9 * 128 * M
    # a simulated ring over G ranks: 5 (G-1) N per schedule step by step,
    # 2 G N with every step in one launch
    assert wl.WORKLOADS["sim"].alg_bytes() == 5 * 7 * 64 * M * 2
    assert wl.WORKLOADS["sim1"].alg_bytes() == 2 * 8 * 64 * M * 2
    # batched: (P_k + 1) n_k sizeof summed over the items
    assert wl.WORKLOADS["c4"].alg_bytes([10, 20]) == 9 * 30 * 2


def test_c4_batch_bytes_match_the_quoted_figure():
    # the seeded 4096-item batch (host and device descriptors alike) moves the
    # algorithmic byte count the committed profiles and results quote
    w = wl.WORKLOADS["c4"]
    sizes = wl.batched_sizes(w)
    assert len(sizes) == 4096
    assert 4096 <= int(sizes.min()) and int(sizes.max()) <= (1 << 20) // 2
    assert w.alg_bytes(sizes) == 7_801_271_568


def test_every_bench_workload_has_a_definition():
    sys.path.insert(0, str(ROOT))
    import bench
    assert "c4dev" in bench.WORKLOAD_NAMES and "c2" in bench.WORKLOAD_NAMES
    for n in bench.WORKLOAD_NAMES:
        assert bench.WORKLOAD_OF.get(n, n) in wl.WORKLOADS, n
