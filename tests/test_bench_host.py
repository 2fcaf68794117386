"""Host-side logic of bench.py, on the CPU: the one-GPU guard, the timing
plan (which calls get event pairs) and the per-call averaging of group-timed
attention, and the digest that ties a committed counter record to the
kernel sources it was taken on."""
import os
import subprocess
import sys
from types import SimpleNamespace

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


class FakeEvent:
    def __init__(self, t):
        self.t = t

    def elapsed_time(self, other):
        return other.t - self.t


class FakeRunner:
    """Records what step_timers asks for."""

    def __init__(self, L, group, append):
        self.w = SimpleNamespace(L=L, group=group,
                                 groups=[list(range(k, min(L, k + group)))
                                         for k in range(0, L, group)])
        self.kv_new = object() if append else None

    def new_timers(self, layers=None, groups=None, attn_groups=()):
        return {"layers": list(layers), "groups": list(groups or []),
                "attn_groups": list(attn_groups)}


def test_step_timers_rotate_over_groups_without_append():
    r = FakeRunner(L=32, group=4, append=False)
    args = SimpleNamespace(timed_layers=2)
    plans = [bench.step_timers(r, args, k) for k in range(10)]
    assert [p["attn_groups"] for p in plans] == [[k % 8] for k in range(10)]
    assert all(p["layers"] == [] and p["groups"] == p["attn_groups"] for p in plans)


def test_step_timers_time_single_calls_with_append():
    r = FakeRunner(L=32, group=4, append=True)
    args = SimpleNamespace(timed_layers=2)
    plans = [bench.step_timers(r, args, k) for k in range(17)]
    assert plans[0]["layers"] == [0, 1] and plans[16]["layers"] == [0, 1]
    assert plans[3]["layers"] == [6, 7]
    assert all(p["attn_groups"] == [] for p in plans)


def test_group_timed_attention_is_averaged_per_call():
    w = SimpleNamespace(groups=[[0, 1, 2, 3], [4, 5, 6, 7], [8, 9]])
    timers = [
        {"at": {}, "atg": {0: (FakeEvent(0.0), FakeEvent(0.4))}},      # 4 calls, 0.4 ms
        {"at": {}, "atg": {2: (FakeEvent(1.0), FakeEvent(1.3))}},      # 2 calls, 0.3 ms
        {"at": {5: (FakeEvent(2.0), FakeEvent(2.12))}, "atg": {}},     # 1 call
    ]
    per_call, calls = bench.attention_samples(timers, w)
    assert calls == 4 + 2 + 1
    assert np.allclose(per_call, [0.1, 0.15, 0.12])


def test_sources_digest_tracks_content(tmp_path, monkeypatch):
    a = tmp_path / "a.hip"
    b = tmp_path / "b.h"
    a.write_text("kernel one\n")
    b.write_text("header\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    d1 = bench.sources_digest(("a.hip", "b.h"))
    assert d1 == bench.sources_digest(("a.hip", "b.h"))
    a.write_text("kernel two\n")
    assert bench.sources_digest(("a.hip", "b.h")) != d1


def test_committed_counter_records_parse():
    for wl in ("llama3-8b-kv", "llama-70b-tp8-share"):
        rec = bench.counter_record(f"paged_attention_{wl}_counters.md", bench.ATTN_SOURCES)
        if rec is None:
            pytest.skip("counter record does not match the current attention sources")
        assert rec["bytes_per_call"] > 0 and rec["fetch_scale"] > 0 and rec["write_scale"] > 0
