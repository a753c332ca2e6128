"""Host-side checks of bench.py's measurement contract (CPU only): the
algorithmic units the roofline divides by, the counter-traffic table keyed on
the kernel sources, the sampling of event-timed launches, and the refusal of
more than one GPU."""
import json
import os
import subprocess
import sys
from collections import Counter

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from mira_inputs import CONFIGS  # noqa: E402


def test_algorithmic_bytes_mixtral_decode():
    cfg = CONFIGS["mixtral_decode"]
    counts = [0] * cfg.G
    counts[1] = counts[5] = 1            # one token, top-2
    u = bench.algorithmic_units(cfg, counts)
    R, C = cfg.R, cfg.C
    assert u["active"] == 2 and u["pairs"] == 2
    assert u["gu_bytes"] == 234_938_368 == 2 * (2 * R * C + 2 * R)
    assert u["dn_bytes"] == 2 * R * C
    # gate/up + down of one expert is its packed blob without the padding
    assert (u["gu_bytes"] + u["dn_bytes"]) // 2 == 3 * R * C + 2 * R
    assert u["gu_flops"] == 2 * 4.0 * C * R and u["dn_flops"] == 2 * 2.0 * C * R


def test_algorithmic_bytes_int4():
    cfg = CONFIGS["mixtral_decode"]
    counts = [0] * cfg.G
    counts[0] = counts[7] = 1
    u = bench.algorithmic_units(cfg, counts, "int4")
    R, C = cfg.R, cfg.C
    per_matrix = R * C // 2 + R * (C // 64) * 2    # nibbles + one fp16 scale per row and group
    assert u["gu_bytes"] == 124_780_544 == 2 * 2 * per_matrix
    assert u["dn_bytes"] == 2 * per_matrix


def test_prefill_flops_count_every_pair():
    cfg = CONFIGS["fine_grained"]
    counts = [3] * cfg.E + [5] * cfg.S
    u = bench.algorithmic_units(cfg, counts)
    assert u["pairs"] == 3 * cfg.E + 5 * cfg.S
    assert u["gu_flops"] == u["pairs"] * 4.0 * cfg.C * cfg.R


def test_traffic_entries_follow_the_sources(monkeypatch):
    # an entry counts only while the kernel sources hash to the value it was
    # measured on; then it is the scaled counter bytes per launch
    for key, ent in bench.TRAFFIC.items():
        monkeypatch.setattr(bench, "source_hash", lambda sources, sha=ent["sha"]: sha)
        got = bench.traffic_bytes(*key)
        assert got == int((ent["fetch_kib"] * bench.FETCH_SCALE + ent["write_kib"] * bench.WRITE_SCALE) * 1024)
    monkeypatch.setattr(bench, "source_hash", lambda sources: "0" * 16)
    assert all(bench.traffic_bytes(*key) is None for key in bench.TRAFFIC)
    assert bench.traffic_bytes("decode_gateup", "no_such_workload") is None


def test_source_hash_covers_the_shared_headers(tmp_path, monkeypatch):
    h = bench.source_hash(("decode.hip",))
    assert len(h) == 16 and h == bench.source_hash(("decode.hip",))
    assert h != bench.source_hash(("prefill.hip",))


@pytest.mark.parametrize("steps,copies", [(200, 5), (200, 2), (100, 3), (7, 4)])
def test_event_steps_sample_every_copy_equally(steps, copies):
    picked = [i for i in range(steps) if bench.event_step(i, copies)]
    assert picked and picked[0] == 0
    per_copy = Counter(i % copies for i in picked)
    assert len(set(per_copy.values())) == 1 or steps < copies * bench.PROF_EVERY
    if steps % (copies * bench.PROF_EVERY) == 0:
        assert len(picked) == steps // bench.PROF_EVERY


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"] and line["n_gpus"] == 2


def test_source_hash_ignores_comments_but_not_code():
    a = "int f(int x) { return x + 1; }  // one\n/* two\n   lines */\n"
    b = "// another comment\nint   f(int x)\n{ return x + 1; }\n"
    c = "int f(int x) { return x + 2; }\n"
    d = 'const char* s = "// kept";\n'
    assert bench.strip_comments(a) == bench.strip_comments(b)
    assert bench.strip_comments(a) != bench.strip_comments(c)
    assert "// kept" in bench.strip_comments(d)
