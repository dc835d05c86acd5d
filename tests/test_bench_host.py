"""Host-side logic of bench.py that needs no GPU: the prefill GEMM's fetch
floor under its tile schedule, the rule that reports recorded HBM traffic
only for the kernel source it was taken on, and the one-GPU guard."""
import json
import os
import subprocess
import sys

import pytest

import bench

# OPT-13B W6A6 step, 4096 tokens: (layer, channels N, K, tile channels x tokens)
OPT13B = [("qkv", 15360, 5120, 320, 256), ("out", 5120, 5120, 320, 256),
          ("fc1", 20480, 5120, 320, 256), ("fc2", 5120, 20480, 320, 256)]


@pytest.mark.parametrize("name,N,K,bn,bm", OPT13B)
def test_fetch_floor_closed_form(name, N, K, bn, bm):
    # whole passes of 256 tiles; on each of the 8 XCDs a pass runs 8 token
    # tiles by 4 channel tiles and fetches those 12 panels over all of K once
    M = 4096
    tiles = (M // bm) * (-(-N // bn))
    assert tiles % 256 == 0
    passes = tiles // 256
    expect = passes * 8 * (8 * bm + 4 * bn) * K
    assert bench.prefill_fetch_floor(M, N, K, bn, bm) == expect


@pytest.mark.parametrize("M,N,K,bn,bm", [(4096, 15360, 5120, 320, 256), (2048, 12288, 4096, 256, 256),
                                         (300, 772, 1040, 256, 256), (8192, 36864, 9216, 256, 256),
                                         (513, 129, 768, 320, 256)])
def test_fetch_floor_bounds(M, N, K, bn, bm):
    # at least every operand panel once, at most every tile fetching its own
    tiles_m, tiles_n = -(-M // bm), -(-N // bn)
    floor = bench.prefill_fetch_floor(M, N, K, bn, bm)
    assert (tiles_m * bm + tiles_n * bn) * K <= floor <= tiles_m * tiles_n * (bm + bn) * K


def test_recorded_floor_matches_the_schedule():
    with open(bench.TRAFFIC_RECORD) as f:
        rec = json.load(f)
    for name, N, K, bn, bm in OPT13B:
        layer = rec["per_layer"][name]
        assert layer["tile"] == f"{bn}x{bm}"
        assert layer["fetch_floor_bytes"] == bench.prefill_fetch_floor(4096, N, K, bn, bm)


def test_traffic_reported_only_for_the_recorded_source(tmp_path, monkeypatch):
    src = tmp_path / "kernel.hip"
    src.write_text("// one version of the kernel\n")
    monkeypatch.setattr(bench, "PREFILL_SOURCES", [str(src)])
    record = tmp_path / "traffic.json"
    record.write_text(json.dumps({"source_sha256": bench.prefill_source_digest(),
                                  "traffic_bytes_per_launch": 123.0}))
    monkeypatch.setattr(bench, "TRAFFIC_RECORD", str(record))
    assert bench.measured_traffic() == 123.0
    src.write_text("// the kernel changed since the counters were taken\n")
    assert bench.measured_traffic() is None
    monkeypatch.setattr(bench, "TRAFFIC_RECORD", str(tmp_path / "missing.json"))
    assert bench.measured_traffic() is None


def test_more_than_one_gpu_is_refused():
    out = subprocess.run([sys.executable, os.path.join(bench.ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=300)
    assert out.returncode != 0
    assert "one GPU" in out.stdout + out.stderr
