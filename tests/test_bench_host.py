"""Host-side logic of bench.py: the refusal of several GPUs, the committed HBM
traffic lookup (valid only for the kernel source it was measured on) and the
CPU-oracle baseline's fields.  No GPU needed."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import pam_workloads as wl  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_committed_counters_follow_the_kernel_digest(tmp_path, monkeypatch):
    digest = bench.kernel_source_digest()
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "traffic_wX_fwd.md").write_text(
        f"traffic_bytes_per_launch: 1.5e+09\nsustained_clock_ghz: 2.05\nkernel_source_sha256_16: {digest}\n")
    (prof / "traffic_wX_dX.md").write_text(
        "traffic_bytes_per_launch: 1.5e+09\nkernel_source_sha256_16: 0000000000000000\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.committed_counter("wX", "fwd", "traffic_bytes_per_launch") == 1.5e9
    assert bench.committed_counter("wX", "fwd", "sustained_clock_ghz") == 2.05
    assert bench.committed_counter("wX", "dX", "traffic_bytes_per_launch") is None   # another kernel source
    assert bench.committed_counter("wX", "dW", "traffic_bytes_per_launch") is None   # never measured


def test_cpu_baseline_fields():
    host = wl.workload_inputs(2)
    res = bench.cpu_baseline(2, host, wl.WORKLOADS[2]["forms"], 0.5)
    assert res["kind"] == "oracle" and res["unit"] == "GPAM-MAC/s"
    assert res["cores"] >= 1 and res["value"] > 0
    assert res["one_core"]["value"] > 0
    assert "fwd" in res["sample"] and "dW" in res["sample"]
    from oracle import pam_c
    assert pam_c.num_threads() == res["cores"]              # thread count restored
