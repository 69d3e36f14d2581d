"""Host-side measurement plumbing (no GPU): the rocprofv3 summary tool and
bench.py's lookup of counted HBM traffic."""
import csv
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2606_21633_amd import profsum  # noqa: E402

ATTN = "void herald::(anonymous namespace)::attn_bf16_kernel<128, 32, 2, 4, false>(args)"
COPY = "void at::native::vectorized_elementwise_kernel<4, mul>(args)"


def _trace(d, durations):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_kernel_trace.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, ["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        t = 1000
        for name, us in durations:
            w.writerow({"Kernel_Name": name, "Start_Timestamp": t,
                        "End_Timestamp": t + int(us * 1000)})
            t += int(us * 1000) + 10


def _counters(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter,
                        "Counter_Value": v})


def test_trace_selects_the_launches_before_the_final_ones(tmp_path, capsys):
    d = str(tmp_path / "t")
    _trace(d, [(ATTN, 100.0)] * 3 + [(ATTN, 30.0)] * 4 + [(ATTN, 50.0)] * 2)
    profsum.main(["trace", d, "--kernel", "attn_bf16_kernel", "--last", "4",
                  "--skip-last", "2"])
    out = capsys.readouterr().out
    assert "attn_bf16_kernel<128, 32, 2, 4, false>" in out
    assert "4 launches" in out and "avg 30.00 us" in out


def test_traffic_scales_each_counter_by_its_copy_calibration(tmp_path, capsys):
    gib = 1 << 30
    _counters(str(tmp_path / "f"), "FETCH_SIZE", [(ATTN, 900.0), (ATTN, 1000.0), (ATTN, 1000.0)])
    _counters(str(tmp_path / "w"), "WRITE_SIZE", [(ATTN, 50.0), (ATTN, 40.0), (ATTN, 40.0)])
    # the copy reads back 1/2 of its bytes as FETCH_SIZE and all as WRITE_SIZE
    _counters(str(tmp_path / "cf"), "FETCH_SIZE", [(COPY, gib / 1024 / 2)])
    _counters(str(tmp_path / "cw"), "WRITE_SIZE", [(COPY, gib / 1024)])
    profsum.main(["traffic", "--fetch", str(tmp_path / "f"), "--write", str(tmp_path / "w"),
                  "--copy-fetch", str(tmp_path / "cf"), "--copy-write", str(tmp_path / "cw"),
                  "--copy-bytes", str(gib), "--kernel", "attn_bf16_kernel", "--last", "2",
                  "--source-sha256", "abc"])
    line = [x for x in capsys.readouterr().out.splitlines() if x.startswith("traffic:")][0]
    kv = dict(tok.split("=") for tok in line.split()[1:])
    assert kv["source_sha256"] == "abc"
    assert float(kv["fetch"]) == pytest.approx(2 * 1000.0 * 1024)
    assert float(kv["write"]) == pytest.approx(40.0 * 1024)
    assert float(kv["bytes_per_launch"]) == pytest.approx(2 * 1000.0 * 1024 + 40.0 * 1024)


def test_traffic_scales_fetch_by_the_read_calibration_when_given(tmp_path, capsys):
    gib = 1 << 30
    red = "void at::native::reduce_kernel<512, 1, op>(args)"
    _counters(str(tmp_path / "f"), "FETCH_SIZE", [(ATTN, 1000.0)])
    _counters(str(tmp_path / "w"), "WRITE_SIZE", [(ATTN, 40.0)])
    _counters(str(tmp_path / "cf"), "FETCH_SIZE", [(COPY, gib / 1024 / 2.4)])
    _counters(str(tmp_path / "cw"), "WRITE_SIZE", [(COPY, gib / 1024)])
    # the plain read counts 1/2 of its bytes; the copy 1/2.4 of its reads
    _counters(str(tmp_path / "rf"), "FETCH_SIZE", [(red, gib / 1024 / 2)])
    profsum.main(["traffic", "--fetch", str(tmp_path / "f"), "--write", str(tmp_path / "w"),
                  "--copy-fetch", str(tmp_path / "cf"), "--copy-write", str(tmp_path / "cw"),
                  "--read-fetch", str(tmp_path / "rf"), "--copy-bytes", str(gib),
                  "--kernel", "attn_bf16_kernel"])
    line = [x for x in capsys.readouterr().out.splitlines() if x.startswith("traffic:")][0]
    kv = dict(tok.split("=") for tok in line.split()[1:])
    assert float(kv["fetch"]) == pytest.approx(2 * 1000.0 * 1024)
    assert float(kv["write"]) == pytest.approx(40.0 * 1024)


def test_bench_reports_traffic_only_for_the_profiled_source(tmp_path, monkeypatch):
    import bench
    from paper_2606_21633_amd import synth
    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bench, "PROFILES", str(prof))
    f = prof / "block_attn_layer32k_traffic.txt"
    f.write_text(f"# header\ntraffic: source_sha256={bench.kernel_source_digest()} "
                 f"bytes_per_launch=123456 fetch=1 write=2\n")
    assert bench.profiled_traffic(synth.LAYER_32K, False) == 123456.0
    assert bench.profiled_traffic(synth.LAYER_32K, True) is None       # dense run
    assert bench.profiled_traffic(synth.LONG_128K, False) is None      # other workload
    f.write_text("traffic: source_sha256=0000 bytes_per_launch=123456\n")
    assert bench.profiled_traffic(synth.LAYER_32K, False) is None      # kernel changed
    f.unlink()
    assert bench.profiled_traffic(synth.LAYER_32K, False) is None      # no profile
