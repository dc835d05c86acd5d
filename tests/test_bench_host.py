"""Host-side logic of bench.py that needs no GPU: the prefill GEMM's fetch
floor under its tile schedule, the rule that reports recorded HBM traffic
only for the kernel source it was taken on, the helper kernels' traffic
summary, and the one-GPU guard."""
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


def _counter_csv(path, counter, dispatches):
    """A rocprofv3 counter_collection.csv with one row per (dispatch, kernel,
    value, start, end)."""
    path.mkdir(parents=True)
    lines = ['"Dispatch_Id","Kernel_Name","Grid_Size","Counter_Name","Counter_Value",'
             '"Start_Timestamp","End_Timestamp"']
    for d, name, value, t0, t1 in dispatches:
        lines.append(f'{d},"{name}",1024,"{counter}",{value},{t0},{t1}')
    (path / "p_counter_collection.csv").write_text("\n".join(lines) + "\n")


def test_helper_traffic_table(tmp_path, capsys):
    """The helper probe's summary scales each dispatch's FETCH_SIZE and
    WRITE_SIZE by the copy's factors and sets them against the algorithmic
    bytes of its shape: made-up counters equal to those bytes give ratios of
    exactly 1."""
    gib_kib = (1 << 30) / 1024
    _counter_csv(tmp_path / "copy_fetch", "FETCH_SIZE",
                 [(1, "__amd_rocclr_copyBuffer", gib_kib / 2, 0, 100)])
    _counter_csv(tmp_path / "copy_write", "WRITE_SIZE",
                 [(1, "__amd_rocclr_copyBuffer", gib_kib, 0, 100)])
    fetch, write, d = [], [], 1
    for label, M, K, kern in bench.HELPER_PROBE:
        rd = 2 * M * K + (12 if kern == "ln_quantize_kernel" else 8) * K
        for _ in range(3):
            fetch.append((d, f"ot::detail::{kern}<6>", rd / 1024 / 2, 0, 10_000))
            write.append((d, f"ot::detail::{kern}<6>", M * K / 1024, 0, 10_000))
            d += 1
    _counter_csv(tmp_path / "helper_fetch", "FETCH_SIZE", fetch)
    _counter_csv(tmp_path / "helper_write", "WRITE_SIZE", write)
    bench.helper_traffic(str(tmp_path))
    out = capsys.readouterr().out
    rows = [line for line in out.splitlines() if line.startswith("| ot_")]
    assert len(rows) == 3
    for row in rows:
        cells = [c.strip() for c in row.strip("|").split("|")]
        assert cells[5] == "1.000" and cells[6] == "1.000", row
        assert cells[7] == "10.0", row
