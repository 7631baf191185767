"""Host logic of bench.py that needs no GPU: the one-GPU guard, the layer
count of each sweep cell and the staleness rule for the committed traffic
counters."""

import json
import os
import subprocess
import sys

import numpy as np

import bench
from paper_2609_19702_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def layer_bytes(w):
    return w.batch * w.num_kv_heads * (w.prompt_len + w.decode_len) * w.head_dim * 2 * 2


def test_sweep_layers_bounds():
    cells = synth.sweep_workloads()
    assert len(cells) == 36
    seen_cap = False
    for w in cells:
        n, lb = bench.sweep_layers(w), layer_bytes(w)
        assert n >= 2
        assert n * lb <= bench.SWEEP_MAX_BYTES or n == 2, w.name
        if n >= bench.SWEEP_MIN_LAYERS:
            # the smallest count that reaches the byte floor (or the layer floor)
            assert n * lb >= bench.SWEEP_MIN_BYTES or n == bench.SWEEP_MIN_LAYERS, w.name
            if n > bench.SWEEP_MIN_LAYERS:
                assert (n - 1) * lb < bench.SWEEP_MIN_BYTES, w.name
        else:
            seen_cap = True
            assert (n + 1) * lb > bench.SWEEP_MAX_BYTES, w.name
    # the 96x96 grid at batch 256 is over the cap: ~40 GiB per layer
    assert seen_cap


def test_sweep_layers_small_cell_reaches_one_gib():
    w = [c for c in synth.sweep_workloads() if c.name == "sweep_g24_b1_w64"][0]
    n = bench.sweep_layers(w)
    assert n * layer_bytes(w) >= 1 << 30
    assert (n - 1) * layer_bytes(w) < 1 << 30


def test_traffic_only_for_the_current_kernel_source(tmp_path, monkeypatch):
    h = bench.kernel_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0
    f = tmp_path / "traffic.json"
    f.write_text(json.dumps({
        "w_now": {"kernel_hash": h, "hbm_bytes_per_launch": 123.0},
        "w_old": {"kernel_hash": "0" * 16, "hbm_bytes_per_launch": 456.0},
    }))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.traffic_for("w_now", h) == 123.0
    assert bench.traffic_for("w_old", h) is None
    assert bench.traffic_for("absent", h) is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.json"))
    assert bench.traffic_for("w_now", h) is None


def test_step_percentiles_match_numpy():
    rng = np.random.default_rng(3)
    for n in (1, 2, 7, 20, 101):
        xs = rng.exponential(1.0, n).tolist()
        got = bench.percentiles(xs)
        for k, f in (("median", 50), ("p10", 10), ("p90", 90)):
            assert abs(got[k] - float(np.percentile(xs, f))) <= 1e-12 * max(1.0, max(xs)), (n, k)
        assert got["n"] == n
