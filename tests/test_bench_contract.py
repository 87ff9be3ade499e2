"""Host-side parts of the benchmark's contract (no GPU): the one-GPU refusal
and the lookup of the profiled HBM traffic, which must report nothing once
the kernel source differs from the one the counters were taken on."""
import hashlib
import json
import shutil
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
sys.path.insert(0, str(ROOT))
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


@pytest.fixture
def fake_root(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    csrc = tmp_path / "paper_2609_33586_amd" / "csrc"
    csrc.mkdir(parents=True)
    shutil.copy(ROOT / "paper_2609_33586_amd" / "csrc" / "h15attn.hip", csrc / "h15attn.hip")
    monkeypatch.setattr(bench, "ROOT", tmp_path)
    return tmp_path


def write_record(root, sha):
    rec = {"source_sha256_prefix": sha,
           "workloads": {"w": {"h15": {"hbm_read_bytes": 1000, "hbm_write_bytes": 234, "kernel_avg_us": 1.0}}}}
    (root / "profiles" / "hbm_traffic.txt").write_text(json.dumps(rec) + "\n")


def test_traffic_reported_for_the_profiled_source(fake_root):
    src = fake_root / "paper_2609_33586_amd" / "csrc" / "h15attn.hip"
    write_record(fake_root, hashlib.sha256(src.read_bytes()).hexdigest()[:16])
    assert bench.profiled_traffic("w", "h15") == 1234
    assert bench.profiled_traffic("w", "exact") is None
    assert bench.profiled_traffic("other", "h15") is None


def test_traffic_null_once_the_source_changed(fake_root):
    src = fake_root / "paper_2609_33586_amd" / "csrc" / "h15attn.hip"
    write_record(fake_root, hashlib.sha256(src.read_bytes()).hexdigest()[:16])
    src.write_text(src.read_text() + "\n// edited\n")
    assert bench.profiled_traffic("w", "h15") is None


def test_committed_traffic_record_is_well_formed():
    rec = json.loads((ROOT / "profiles" / "hbm_traffic.txt").read_text())
    assert len(rec["source_sha256_prefix"]) == 16
    for wl, modes in rec["workloads"].items():
        for mode, t in modes.items():
            assert t["hbm_read_bytes"] > 0 and t["hbm_write_bytes"] > 0 and t["kernel_avg_us"] > 0, (wl, mode)
