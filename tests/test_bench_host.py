"""Host logic of the benchmark (CPU only): the algorithmic byte count, the
kernel-source hash and the single-GPU guard."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads as wl  # noqa: E402


def test_algorithmic_bytes_by_hand():
    # N = 3 bf16 rows, D = 10, packets of 4 (lengths 4, 4, 2), Adam (3 fp32
    # vectors read and written).
    w = wl.scaled(wl.WORKLOADS["n8_d16m_bf16_adam"], n=3, d=10, packet=4)
    mg = np.array([[1, 0, 1], [1, 1, 0], [0, 1, 1]], np.uint8)
    mb = np.array([[1, 1, 0], [0, 1, 1], [1, 1, 1]], np.uint8)
    lens = np.array([4, 4, 2])
    b = bench.algorithmic_bytes(w, mg, mb, lens, drift=True)
    # grads: packet 0 twice (8 elems), packet 1 twice (8), packet 2 twice (4) -> 20 elems x 2 B
    assert b["grads_read"] == 40
    assert b["state_rw"] == 2 * 4 * 3 * 10
    # replicas written: packet 0 twice, 1 three times, 2 twice -> 8 + 12 + 4 = 24 elems
    assert b["replicas_written"] == 48
    # stale: packet 0 once, packet 2 once -> 4 + 2 = 6 elems
    assert b["stale_read"] == 12
    assert b["total"] == 40 + 240 + 48 + 12
    s = bench.algorithmic_bytes(w, mg, mb, lens, drift=False, estimator="stale_fill",
                                ages=True, reliable=True)
    assert s["stale_read"] == 0
    assert s["g_prev_read"] == (30 - 20) * 2 and s["g_prev_written"] == 20 * 2
    assert s["ages_rw"] == 2 * 2 * 3 * 3 and s["reliable_read"] == 3


def test_kernel_source_hash_ignores_comments(tmp_path, monkeypatch):
    for rel in bench.KERNEL_SOURCES:
        dst = tmp_path / rel
        dst.parent.mkdir(parents=True, exist_ok=True)
        dst.write_text(open(os.path.join(ROOT, rel)).read())
    monkeypatch.setattr(bench, "HERE", str(tmp_path))
    h0 = bench.kernel_source_hash()
    first = tmp_path / bench.KERNEL_SOURCES[0]
    first.write_text(first.read_text() + "\n// a comment\n/* another\n one */\n")
    assert bench.kernel_source_hash() == h0
    first.write_text(first.read_text() + "\nstatic int changed_code = 1;\n")
    assert bench.kernel_source_hash() != h0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_counter_traffic_only_for_its_workload_and_sources(tmp_path, monkeypatch):
    prof = tmp_path / "pmc.txt"
    prof.write_text("# header: comment lines are skipped\nkernel_source_sha256: abc\n"
                    "workload: n64_llama7b_shard_bf16_adam\nhbm_bytes_per_dispatch: 123\n")
    monkeypatch.setattr(bench, "PMC_PROFILE", str(prof))
    assert bench.read_pmc_traffic("abc", "n64_llama7b_shard_bf16_adam") == 123.0
    assert bench.read_pmc_traffic("abd", "n64_llama7b_shard_bf16_adam") is None
    assert bench.read_pmc_traffic("abc", "n8_d16m_bf16_adam") is None
    monkeypatch.setattr(bench, "PMC_PROFILE", str(tmp_path / "missing.txt"))
    assert bench.read_pmc_traffic("abc", "n64_llama7b_shard_bf16_adam") is None
