"""Host-side checks of bench.py's bookkeeping (no GPU): the flop count of the
benchmark workload, the multi-GPU refusal, and the traffic table's guard on
kernel sources."""
import os
import subprocess
import sys

import bench
from paper_2605_15684_amd.inputs import preset

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_flops_of_the_benchmark_workload():
    w = preset("grid64")
    # 16 heads x 4096 image queries x 10 kept blocks x 64 keys x 4 D flops
    assert bench.flops(w) == 16 * 4096 * 640 * 4 * 64
    assert bench.flops(w, dense=True) == 16 * 4096 * 4096 * 4 * 64
    assert abs(bench.flops(w) / 1e9 - 10.737) < 1e-3


def test_flops_with_text_tokens():
    w = preset("grid64_text")
    pairs = w.t_img * (w.keep * 64 + w.n_text) + w.n_text * w.seq_len
    assert bench.pairs_per_bh(w) == pairs
    assert bench.flops(w) == 4.0 * 64 * pairs * w.batch * w.heads


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_only_for_the_measured_sources(monkeypatch):
    key = ("k_attn_mfma<64, 3, false, false>", "grid64")
    entry = {"sha": "", "fetch_kib": 12000.0, "write_kib": 8192.0, "fetch_factor": 2.0, "write_factor": 1.0}
    monkeypatch.setitem(bench.MEASURED_TRAFFIC, key, dict(entry, sha=bench.sources_sha(key[0])))
    t = bench.measured_traffic(*key)
    assert t == entry["fetch_kib"] * 1024 * entry["fetch_factor"] + entry["write_kib"] * 1024 * entry["write_factor"]
    monkeypatch.setitem(bench.MEASURED_TRAFFIC, key, dict(entry, sha="0" * 16))
    assert bench.measured_traffic(*key) is None
    assert bench.measured_traffic(key[0], "grid128") is None
