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


class _FakeEvent:
    clock = [0.0]

    def __init__(self, enable_timing=True):
        self.t = None

    def record(self, stream=None):
        self.t = _FakeEvent.clock[0]

    def elapsed_time(self, other):
        return other.t - self.t


class _FakeCuda:
    Event = _FakeEvent

    @staticmethod
    def synchronize():
        pass


class _FakeTorch:
    cuda = _FakeCuda


def test_timed_windows_counts_every_call_and_alternates():
    # Every variant gets exactly `steps` timed calls (after `warmup` untimed
    # ones) in windows of at most `window` calls, and the variants take turns.
    log = []

    def make(name, ms):
        def fn():
            log.append(name)
            _FakeEvent.clock[0] += ms
        return fn
    calls = {"a": make("a", 1.0), "b": make("b", 2.0), "c": make("c", 3.0)}
    res = bench.timed_windows(_FakeTorch, None, calls, steps=12, warmup=4, window=5)
    assert log[:12] == ["a"] * 4 + ["b"] * 4 + ["c"] * 4
    for name, ms in (("a", 1.0), ("b", 2.0), ("c", 3.0)):
        assert sum(n for _, n in res[name]) == 12
        assert [n for _, n in res[name]] == [5, 5, 2]
        assert all(abs(t - ms * n) < 1e-9 for t, n in res[name])
    # turn 0: a b c; turn 1: c b a; turn 2: a b c (the last windows hold 2)
    expect = []
    for names, n in (("abc", 5), ("cba", 5), ("abc", 2)):
        for nm in names:
            expect += [nm] * n
    assert log[12:] == expect
