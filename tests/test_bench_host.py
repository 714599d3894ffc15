"""Host-side checks of bench.py: the one-GPU contract, the algorithmic byte
models against their parts counted by hand for the production and
delta-rule shapes, and the rule that traffic counters taken on other kernel
sources are not reported."""
import importlib.util
import json
import os
import subprocess
import sys

import numpy as np
import pytest

from synth import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], cwd=ROOT, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_verify_bytes_production(bench):
    # 32 requests x 64 nodes, Hk = 16, Hv = 32, d = 128, bf16 q/k/v
    B, N = 32, 2048
    state = B * 32 * 128 * 128 * 4          # S_pre read once
    out = N * 32 * 128 * 4                  # O written once, fp32
    qk = N * 2 * 16 * 128 * 2
    v = N * 32 * 128 * 2
    gates = N * 32 * 4
    forest = N * 4 + (B + 1) * 4
    want = state + out + qk + v + gates + forest
    assert want == 134_488_196
    assert bench.verify_bytes(W.CONFIGS["production"], N, B) == want


def test_verify_bytes_delta_rule(bench):
    # 16 requests x 128 nodes; beta is read next to the gates
    B, N = 16, 2048
    want = (B * 32 * 128 * 128 * 4 + N * 32 * 128 * 4 + N * 2 * 16 * 128 * 2 + N * 32 * 128 * 2
            + 2 * N * 32 * 4 + N * 4 + (B + 1) * 4)
    assert bench.verify_bytes(W.CONFIGS["gdn"], N, B) == want
    assert abs(want / 1e6 - 101.2) < 0.05


def test_commit_bytes_counts_only_committing_slots(bench):
    cfg = W.CONFIGS["production"]
    slot = 2 * 32 * 128 * 128 * 4            # one request's states, read and written
    row = 16 * 128 * 2 + 32 * 128 * 2 + 32 * 4 + 4   # k, v, g and parent of one path row
    lens = [0, 3, 1, 0]
    assert bench.commit_bytes(cfg, lens) == 2 * slot + 4 * row + 4 * 5
    assert bench.commit_bytes(cfg, [0, 0]) == 4 * 3      # nothing accepted: offsets only


def test_source_hash_ignores_comments_and_whitespace(bench, tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "HASHED_SOURCES", ["k.hip"])
    f = tmp_path / "k.hip"
    f.write_text("int x = 1; // the value\n/* block\n comment */ int y;\n")
    h0 = bench.source_hash()
    f.write_text("int   x = 1;\n\n int y;   // another remark\n")
    assert bench.source_hash() == h0
    f.write_text("int x = 2; int y;\n")
    assert bench.source_hash() != h0


def test_traffic_reported_only_for_matching_sources(bench, tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    stamp = {"src_hash": "0123456789abcdef", "verify": {"bytes_per_launch": 138_000_000}}
    (tmp_path / "profiles" / "traffic_production.json").write_text(json.dumps(stamp))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "source_hash", lambda: "0123456789abcdef")
    assert bench.traffic_for("production", "verify") == 138_000_000
    assert bench.traffic_for("production", "commit") is None       # no counters for that kernel
    assert bench.traffic_for("gdn", "verify") is None              # no stamp for that workload
    monkeypatch.setattr(bench, "source_hash", lambda: "fedcba9876543210")
    assert bench.traffic_for("production", "verify") is None       # kernels changed since


def test_committed_traffic_stamp_is_well_formed():
    d = json.load(open(os.path.join(ROOT, "profiles", "traffic_production.json")))
    assert len(d["src_hash"]) == 16
    for k in ("verify", "commit"):
        e = d[k]
        assert e["bytes_per_launch"] == e["fetch_bytes"] + e["write_bytes"]
        assert np.isclose(e["fetch_bytes"], e["fetch_kib_raw"] * 1024 * d["fetch_scale"], rtol=1e-3)
