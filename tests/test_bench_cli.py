"""Host-side checks of bench.py's command line: runs on more than one GPU
are refused with a message before anything touches a device."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""  # no JSON line for a run that did not happen


def test_trace_summary_keeps_only_the_marked_region(tmp_path):
    """--summarize-trace takes the dispatches between the first two marker
    spin kernels of a rocprofv3 kernel trace, per kernel name."""
    rows = [("k_other", 0, 5), ("at::cuda::spin_kernel(long)", 10, 20), ("aqlm::k_a", 30, 40),
            ("aqlm::k_a", 50, 62), ("aqlm::k_b", 70, 71), ("at::cuda::spin_kernel(long)", 80, 90),
            ("aqlm::k_a", 100, 200), ("at::cuda::spin_kernel(long)", 300, 310)]
    path = tmp_path / "kernel_trace.csv"
    with open(path, "w") as f:
        f.write('"Kind","Kernel_Name","Start_Timestamp","End_Timestamp"\n')
        for name, t0, t1 in rows:
            f.write(f'"KERNEL_DISPATCH","{name}",{t0 * 1000},{t1 * 1000}\n')
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--summarize-trace", str(path)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    import json
    out = json.loads(r.stdout)
    assert out["dispatches"] == 3
    assert out["window_us"] == 60.0
    a = out["kernels"]["aqlm::k_a"]
    assert a["calls"] == 2 and a["total_us"] == 22.0 and a["avg_us"] == 11.0
    assert out["kernels"]["aqlm::k_b"]["calls"] == 1


def test_floors_library_exports_and_refuses_bad_arguments():
    """The measurement library behind bench.py --floors is built beside the
    product library, exports its six microbenchmarks, and refuses arguments
    that would put an access out of range before any launch (so no GPU is
    needed here)."""
    import ctypes
    path = os.path.join(ROOT, "paper_2401_06118_amd", "libaqlm_floors.so")
    if not os.path.exists(path):
        import pytest
        pytest.skip("libraries not built (python -m paper_2401_06118_amd.build)")
    lib = ctypes.CDLL(path)
    names = ["floor_empty", "floor_dep_load", "floor_read", "floor_mfma", "floor_lds_gather", "floor_l2_gather"]
    for n in names:
        assert hasattr(lib, n), n
    vp, ci = ctypes.c_void_p, ctypes.c_int
    lib.floor_lds_gather.argtypes = [vp, ci, ci, ci, vp]
    lib.floor_l2_gather.argtypes = [vp, ctypes.c_uint32, vp, ci, ci, vp]
    lib.floor_read.argtypes = [vp, ctypes.c_size_t, vp, ci, vp]
    invalid = 1  # hipErrorInvalidValue
    fake = 0x10000
    assert lib.floor_lds_gather(fake, 1, 1, 17, None) == invalid   # more copies than the table holds
    assert lib.floor_lds_gather(fake, 1, 1, 0, None) == invalid
    assert lib.floor_l2_gather(fake, 3000, fake, 1, 1, None) == invalid  # not a power of two
    assert lib.floor_read(fake, 0, fake, 1, None) == invalid
    assert lib.floor_read(None, 16, fake, 1, None) == invalid
