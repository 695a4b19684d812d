"""Host logic of bench.py (no GPU): the refusal of multi-GPU runs, the
algorithmic work it divides by measured times, and the HBM-traffic summary
it builds from two rocprofv3 counter runs."""

import csv
import json
import os

import pytest

import bench
from paper_2306_05420_amd import synthetic as syn


def _wl(name):
    return next(w for w in syn.WORKLOADS if w.name == name)


def test_multi_gpu_request_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU" in capsys.readouterr().err


def test_stage_work_wx256_closed_forms():
    w = _wl("wx256")
    s = bench.stage_work(w)
    # x and the spectrum X, bf16 complex: B S C H W and S (2L-1) B C H values
    assert s["dft_fwd"]["bytes"] == 2 * 2 * 256 * 256 * 256 * 4 + 2 * 255 * 2 * 256 * 256 * 4
    assert s["dft_fwd"]["bytes"] == 535_822_336
    # mixing: spin 1 exists from l = 1 on, so l = 0 mixes 256 x 256 channels
    # and every other degree 512 x 512; 8 real flops per complex product
    want = 8 * 2 * (1 * 256 * 256 + (128 * 128 - 1) * 512 * 512)
    assert s["mix"]["flops"] == want == 68_716_331_008
    # quadrature: 4 flops per (l, m, j, column), sum over m of (L - |m|) = L^2
    # for spin 0 and L^2 - 1 for spin 1 (l >= |s|)
    assert s["lat_fwd"]["flops"] == 4 * 256 * 2 * 256 * (128 * 128 + 128 * 128 - 1)
    # filters, coefficients in and out of the mixing
    assert s["mix"]["bytes"] == (128 * 128 * 2 * 2 * 256 * 4) * 2 + 128 * 2 * 256 * 2 * 256 * 4


def test_stage_work_float_small_grid_has_whole_transform_stages():
    s = bench.stage_work(_wl("mol"))
    w = _wl("mol")
    x_b = w.B * len(w.spins_in) * w.C_in * w.H * w.W * 8
    assert s["small_fwd"]["bytes"] > x_b and s["small_fwd"]["flops"] == s["lat_fwd"]["flops"]


def _counter_csv(path, counter, rows):
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                           "Counter_Value"])
        wr.writeheader()
        for i, (kernel, kib) in enumerate(rows):
            wr.writerow({"Dispatch_Id": i, "Kernel_Name": kernel, "Counter_Name": counter,
                         "Counter_Value": kib})


def test_summarize_counters_scales_by_the_copy(tmp_path):
    gib_kib = (1 << 30) / 1024
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    dft = "void swsft::(anonymous namespace)::dft_fwd_kernel<bf16, bf16, 16, 16, true>(...)"
    mix = "void swsft::(anonymous namespace)::mix_split_kernel<2, 2, 2, false, false>(...)"
    # FETCH reads half of a copy's bytes (scale 2); WRITE reads them all (scale 1)
    _counter_csv(fetch, "FETCH_SIZE", [(bench.COPY_KERNEL + "(...)", gib_kib / 2), (dft, 1000.0),
                                       (dft, 1100.0), (dft, 1200.0), (mix, 10.0)])
    _counter_csv(write, "WRITE_SIZE", [(bench.COPY_KERNEL + "(...)", gib_kib), (dft, 500.0),
                                       (mix, 20.0)])
    out = tmp_path / "traffic.json"
    rec = bench.summarize_counters(str(fetch), str(write), str(out))
    assert json.loads(out.read_text()) == rec
    assert rec["calibration"]["fetch_scale"] == 2.0 and rec["calibration"]["write_scale"] == 1.0
    d = rec["kernels"]["dft_fwd"]  # median of the three dispatches
    assert d["hbm_read_bytes"] == 1100 * 1024 * 2 and d["hbm_write_bytes"] == 500 * 1024
    assert d["hbm_bytes_per_launch"] == d["hbm_read_bytes"] + d["hbm_write_bytes"]
    assert rec["kernels"]["mix"]["hbm_bytes_per_launch"] == 10 * 1024 * 2 + 20 * 1024
    assert rec["source_digest"] == bench.source_digest()


def test_summarize_counters_needs_the_copy(tmp_path):
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    _counter_csv(fetch, "FETCH_SIZE", [("dft_fwd_kernel<>", 1.0)])
    _counter_csv(write, "WRITE_SIZE", [("dft_fwd_kernel<>", 1.0)])
    with pytest.raises(SystemExit):
        bench.summarize_counters(str(fetch), str(write), str(tmp_path / "t.json"))


def test_measured_traffic_only_for_matching_sources(tmp_path, monkeypatch):
    os.makedirs(tmp_path / "profiles")
    rec = {"source_digest": "abc", "kernels": {"dft_fwd": {"hbm_bytes_per_launch": 123}}}
    (tmp_path / "profiles" / "traffic_wx256.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "source_digest", lambda: "abc")
    assert bench.measured_traffic("dft_fwd") == 123
    assert bench.measured_traffic("mix") is None
    monkeypatch.setattr(bench, "source_digest", lambda: "other")
    assert bench.measured_traffic("dft_fwd") is None
