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
