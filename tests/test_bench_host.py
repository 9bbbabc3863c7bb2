"""Host logic of bench.py (no GPU): the one-GPU contract, the calibration of
the HBM byte counters, the guard that drops recorded traffic once the kernel
sources change, and the per-token byte and flop counts behind the roofline."""
import csv
import importlib.util
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def _counter_csv(path, counter, rows):
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        wr.writeheader()
        for name, kib in rows:
            wr.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": kib})


def test_ingest_scales_each_counter_by_the_calibrating_copy(bench, tmp_path):
    copy_kib = bench.COPY_BYTES / 1024
    # FETCH_SIZE reads half the copy's bytes (scale 2), WRITE_SIZE all of them (scale 1);
    # small plan set-up copies must not be taken for the calibrating one
    fetch = [("__amd_rocclr_copyBuffer", 4.0), ("__amd_rocclr_copyBuffer", copy_kib / 2),
             ("void dpb::encode3_kernel<true, 8, 4, false>(...)", 1000.0),
             ("void dpb::encode3_kernel<true, 8, 4, false>(...)", 1002.0),
             ("void dpb::encode3_kernel<true, 8, 4, false>(...)", 1001.0),
             ("void dpb::decode2_kernel<true, 5, false>(...)", 500.0),
             ("void dpb::decode_bwd2_kernel<true, true, 5, false>(...)", 1200.0)]
    write = [("__amd_rocclr_copyBuffer", copy_kib), ("__amd_rocclr_fillBufferAligned", 1.0),
             ("void dpb::encode3_kernel<true, 8, 4, false>(...)", 300.0),
             ("void dpb::decode2_kernel<true, 5, false>(...)", 700.0),
             ("void dpb::decode_bwd2_kernel<true, true, 5, false>(...)", 900.0)]
    fp, wp = tmp_path / "f.csv", tmp_path / "w.csv"
    _counter_csv(fp, "FETCH_SIZE", fetch)
    _counter_csv(wp, "WRITE_SIZE", write)
    rec = bench.ingest_counters(str(fp), str(wp), "train")
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    assert rec["kernel_source_digest"] == bench.kernel_source_digest()
    enc = rec["kernels"]["encode"]
    assert enc["fetch_bytes"] == pytest.approx(1001.0 * 1024 * 2)   # median of the dispatches
    assert enc["write_bytes"] == pytest.approx(300.0 * 1024)
    assert enc["hbm_bytes_per_launch"] == pytest.approx(enc["fetch_bytes"] + enc["write_bytes"])
    assert rec["kernels"]["decode_bwd"]["fetch_bytes"] == pytest.approx(1200.0 * 1024 * 2)
    assert enc["tokens"] == 65536


def test_ingest_without_calibrating_copy_fails(bench, tmp_path):
    fp, wp = tmp_path / "f.csv", tmp_path / "w.csv"
    _counter_csv(fp, "FETCH_SIZE", [("void dpb::encode3_kernel<true, 8, 4, false>(...)", 10.0)])
    _counter_csv(wp, "WRITE_SIZE", [("__amd_rocclr_copyBuffer", 1.0)])
    with pytest.raises(SystemExit):
        bench.ingest_counters(str(fp), str(wp), "train")


def test_recorded_traffic_is_used_only_for_the_current_sources(bench, tmp_path, monkeypatch):
    path = tmp_path / "traffic.json"
    rec = {"kernel_source_digest": bench.kernel_source_digest(),
           "kernels": {"decode_bwd": {"tokens": 65536, "hbm_bytes_per_launch": 123.0}}}
    path.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(path))
    assert bench.load_traffic("decode_bwd", 65536) == 123.0
    assert bench.load_traffic("decode_bwd", 1000) is None       # another workload size
    assert bench.load_traffic("encode", 65536) is None          # not recorded
    rec["kernel_source_digest"] = "0" * 16
    path.write_text(json.dumps(rec))
    assert bench.load_traffic("decode_bwd", 65536) is None      # sources changed since
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.json"))
    assert bench.load_traffic("decode_bwd", 65536) is None


def test_algorithmic_counts_at_the_train_shape(bench):
    from paper_2607_20652_amd import inputs
    w = inputs.workload("train")
    k_tot = 96
    b = bench.algorithmic_bytes_per_token(w, k_tot)
    assert b["encode"] == 768 * 2 + 96 * 8
    assert b["decode"] == 96 * 8 + 768 * 2
    assert b["decode_bwd"] == 2 * (96 * 4 + 768 * 2)
    assert b["forward"] == 3840          # read x, write the code and y
    hier = ([10, 12, 15, 17, 20], [0, 16, 16, 16, 16], [8, 8, 8, 8, 64])
    f = bench.algorithmic_flops_per_token(w, k_tot, hier)
    assert f["encode"] == 2 * 4 * 8 * 16 * 768          # 393,216 multiply-adds of child scoring
    assert f["decode"] == 2 * 88 * 768
    assert f["decode_bwd"] == 4 * 88 * 768
