"""bench.py's command line on the CPU: more than one GPU is refused with a
message before anything touches a device."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_help_lists_the_contract_flags():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--help"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0
    for flag in ("--gpus", "--steps", "--warmup", "--workload", "--sign", "--path"):
        assert flag in r.stdout


def test_committed_traffic_follows_the_kernel_source():
    """The roofline's traffic comes from the committed counter summary only when
    it was taken on the current kernel source, for that workload and kernel."""
    sys.path.insert(0, ROOT)
    import json

    import bench
    h = bench.kernel_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0
    for wl in ("tiny", "small", "medium", "large", "xl"):
        path = os.path.join(ROOT, "profiles", f"hbm_traffic_{wl}.json")
        with open(path) as f:
            rec = json.load(f)
        for name, k in rec["kernels"].items():
            want = k["bytes_per_launch"] if rec["kernel_source_hash"] == h else None
            assert bench.committed_traffic(h, wl, name) == want, (wl, name)
            assert bench.committed_traffic(rec["kernel_source_hash"], wl, name) == \
                k["bytes_per_launch"]
            # within 1% of the algorithmic bytes: the kernels move no extra traffic
            assert abs(k["bytes_per_launch"] / k["algorithmic_bytes"] - 1) < 0.01, (wl, name)
        assert bench.committed_traffic("0" * 16, wl, "local_adamw") is None
    assert bench.committed_traffic(h, "no-such-workload", "local_adamw") is None
    assert bench.committed_traffic(h, "xl", "no_such_kernel") is None
