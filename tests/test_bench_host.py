"""Host-side contract of bench.py (no GPU): the one-GPU limit and the lookup of
measured HBM traffic from the committed rocprofv3 counter summary."""
import importlib.util
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
WORKLOAD = "llama8b-n32-32layer"


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_exits_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""   # no JSON line for a configuration that was not measured


def _recorded(name):
    vals = {}
    for line in open(os.path.join(ROOT, "profiles", f"hbm_traffic_{name}.md")):
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].strip().split(": ", 1)
            vals[k.strip("` ")] = v.strip("` ")
    return vals


def test_traffic_is_reported_only_for_the_kernels_it_was_measured_on(monkeypatch):
    b = _bench()
    rec = _recorded(WORKLOAD)
    value = float(rec["pced_decode_attn HBM bytes per launch"])
    assert 1e8 < value < 1e9   # one layer's K/V pages of the 33 caches plus split states, in bytes
    assert b.measured_traffic("no-such-workload", "pced_decode_attn") is None
    monkeypatch.setattr(b, "kernel_source_sha256", lambda: rec["kernel source sha256"])
    assert b.measured_traffic(WORKLOAD, "pced_decode_attn") == value
    assert b.measured_traffic(WORKLOAD, "no_such_kernel") is None
    monkeypatch.setattr(b, "kernel_source_sha256", lambda: "0" * 64)
    assert b.measured_traffic(WORKLOAD, "pced_decode_attn") is None


def test_kernel_source_hash_is_of_the_kernel_file():
    import hashlib
    b = _bench()
    path = os.path.join(ROOT, "paper_2601_08670_amd", "csrc", "pced_kernels.hip")
    assert b.kernel_source_sha256() == hashlib.sha256(open(path, "rb").read()).hexdigest()
