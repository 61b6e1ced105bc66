"""The Python binding's own checks (CPU, no GPU needed): every tensor handed
to the kernels must be on the output's device, contiguous, of the dtype's
element size and of the expected length, so that no kernel reads or writes
outside a tensor.  A stand-in object with the tensor attributes the binding
reads plays a GPU tensor; every case fails before the library is called.
"""
import pytest

torch = pytest.importorskip("torch")
import paper_2510_20171_amd as xr  # noqa: E402


class FakeGpuTensor:
    def __init__(self, n, dtype=torch.bfloat16, device="cuda:0", contiguous=True, cuda=True,
                 pinned=False):
        self.n, self.dtype, self.device = n, dtype, torch.device(device)
        self.is_cuda, self._contig, self._pinned = cuda, contiguous, pinned

    def numel(self):
        return self.n

    def element_size(self):
        return torch.empty(0, dtype=self.dtype).element_size()

    def is_contiguous(self):
        return self._contig

    def is_pinned(self):
        return self._pinned

    def data_ptr(self):
        return 1 << 40


def _invalid(fn, match):
    with pytest.raises(xr.XredError) as e:
        fn()
    assert e.value.status == xr.INVALID_ARGUMENT
    assert match in str(e.value)


def test_cpu_tensors_are_rejected():
    a = torch.zeros(16, dtype=torch.bfloat16)
    _invalid(lambda: xr.allreduce_local([a, a], torch.zeros_like(a)), "not in GPU")


def test_allreduce_local_checks():
    out = FakeGpuTensor(100)
    _invalid(lambda: xr.allreduce_local([FakeGpuTensor(100), FakeGpuTensor(99)], out),
             "srcs[1] has 99 elements")
    _invalid(lambda: xr.allreduce_local([FakeGpuTensor(100, contiguous=False)], out),
             "not contiguous")
    _invalid(lambda: xr.allreduce_local([FakeGpuTensor(100, device="cuda:1")], out), "cuda:1")
    _invalid(lambda: xr.allreduce_local([FakeGpuTensor(100)], out, dtype="f32"),
             "2-byte elements")
    _invalid(lambda: xr.allreduce_local([FakeGpuTensor(100)], out, dtype="nope"), "unknown dtype")


def test_reduce_scatter_needs_full_send_buffers():
    out = FakeGpuTensor(10)
    _invalid(lambda: xr.reduce_scatter_local([FakeGpuTensor(30)] * 4, 1, out),
             "expected 40")


def test_step_and_cast_check_the_accumulator():
    x = FakeGpuTensor(64, dtype=torch.int64)
    _invalid(lambda: xr.reduce_copy_step(x, FakeGpuTensor(64, dtype=torch.float32)),
             "the dtype needs 8")
    _invalid(lambda: xr.reduce_copy_step(FakeGpuTensor(64), None), "acc is required")
    _invalid(lambda: xr.reduce_copy_step(FakeGpuTensor(64), FakeGpuTensor(64, torch.float32),
                                         None, final=True), "out is required")
    _invalid(lambda: xr.acc_cast(FakeGpuTensor(63, torch.float32), FakeGpuTensor(64)),
             "expected 64")


def test_batched_items_are_checked():
    items = [([FakeGpuTensor(8)], FakeGpuTensor(8)), ([FakeGpuTensor(7)], FakeGpuTensor(8))]
    _invalid(lambda: xr.batched_reduce(items, dtype="bf16"), "items[1].srcs[0]")


def test_ring_flags_must_be_reachable_and_long_enough():
    chunks = [FakeGpuTensor(32)] * 3
    out = FakeGpuTensor(32)
    pageable = FakeGpuTensor(3, dtype=torch.int32, cuda=False)
    _invalid(lambda: xr.ring_reduce(chunks, out, ready=pageable), "pinned host")
    short = FakeGpuTensor(2, dtype=torch.int32, cuda=False, pinned=True)
    _invalid(lambda: xr.ring_reduce(chunks, out, ready=short), "at least 3")
    _invalid(lambda: xr.ring_reduce(chunks, out, status=FakeGpuTensor(1, torch.int16)),
             "the dtype needs 4")


def test_sim_buffers_are_checked():
    sends = [FakeGpuTensor(50)] * 4
    _invalid(lambda: xr.allreduce_sim(sends, [FakeGpuTensor(50)] * 3), "one recv buffer")
    _invalid(lambda: xr.allreduce_sim(sends, [FakeGpuTensor(50)] * 3 + [FakeGpuTensor(51)]),
             "recvs[3] has 51")


def test_library_shares_torchs_hip_runtime():
    """Loading the library with nothing else imported first must not map a
    second HIP runtime beside torch's: torch's device pointers and streams are
    only valid in the runtime that made them."""
    import ast
    import subprocess
    import sys
    from pathlib import Path
    root = Path(__file__).resolve().parents[1]
    code = ("import paper_2510_20171_amd as xr\n"
            "xr.load()\n"
            "import torch\n"
            "print(sorted({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}))\n")
    out = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True,
                         timeout=300, check=True).stdout
    runtimes = ast.literal_eval(out.strip().splitlines()[-1])
    assert len(runtimes) == 1, runtimes
