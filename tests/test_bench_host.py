"""Host-side pieces of bench.py: the one-GPU contract, the traffic summary
lookup (numbers are used only when taken on the current kernel source) and
the CPU-baseline object, on the tiny workload."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stdout + r.stderr


def test_traffic_summary_needs_the_current_source(tmp_path, monkeypatch):
    src = tmp_path / "kernel.hip"
    src.write_text("// kernel v1\n")
    plan = tmp_path / "plan.cpp"
    plan.write_text("// plan v1\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCES", (str(src), str(plan)))
    monkeypatch.setattr(bench, "PROFILE_DIR", str(tmp_path))
    digest = bench.source_digest()
    f = tmp_path / f"{bench.PARTIAL_KERNEL}_demo_traffic.txt"
    f.write_text("# demo\nhbm_bytes_per_launch: 1234.0\n"
                 f"kernel_source_sha256_16: {digest}\n")
    assert bench.read_traffic("demo") == (1234.0, str(f))
    src.write_text("// kernel v2\n")                 # the kernel changed
    assert bench.read_traffic("demo") == (None, "stale")
    src.write_text("// kernel v1\n")
    assert bench.read_traffic("demo") == (1234.0, str(f))
    plan.write_text("// plan v2\n")                  # the planner changed
    assert bench.read_traffic("demo") == (None, "stale")
    assert bench.read_traffic("absent") == (None, None)


WORKLOADS = ("tiny", "7b_pre_repack", "post_repack", "32b_fp8", "agentic_mix",
             "32b_fp8_tp4", "agentic_mix_tp8")


def test_committed_traffic_summaries_match_the_kernel_source():
    """The committed counters were taken on the kernel and planner sources
    as they are, so the bench line reports them (a stale summary would
    report null)."""
    for w in WORKLOADS:
        value, where = bench.read_traffic(w)
        assert where not in (None, "stale"), w
        assert value > 0


def test_committed_kernel_statistics_match_the_kernel_source():
    """Each workload's rocprofv3 statistics list the attention kernels'
    rows and were taken on the current kernel and planner sources."""
    for w in WORKLOADS:
        path = os.path.join(bench.PROFILE_DIR, f"decode_items_{w}_stats.md")
        text = open(path).read()
        assert f"kernel_source_sha256_16: {bench.source_digest()}" in text, w
        assert "| decode_items<" in text, w


def test_cpu_baseline_object_on_the_tiny_workload():
    pytest.importorskip("threadpoolctl")
    from workloads import get_config, make_workload
    wl = make_workload(get_config("tiny"), seed=None, device="cpu")
    cb = bench.cpu_baseline(wl, budget_s=0.2)
    assert cb["kind"] == "oracle" and cb["unit"] == "TB/s"
    assert cb["value"] > 0 and cb["cores"] >= 1 and cb["seconds"] > 0
    assert "trajectories" in cb["sample"]
