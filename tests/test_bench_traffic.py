"""The roofline's HBM-traffic bookkeeping in bench.py (CPU only): the
counter summary scales each counter by the calibration copy, and a stored
figure is used only for the kernel source it was measured on."""
import csv
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
          "Start_Timestamp", "End_Timestamp"]


def write_csv(path, counter, copy_kib, attn_kib):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        # the counter is reported per XCD: two rows per dispatch
        for did, name, kib, dur in (("5", "__amd_rocclr_copyBuffer", copy_kib, 400),
                                    ("7", "void scope::attn_kernel<128, true>(int)", attn_kib, 9000)):
            for part in (0.25, 0.75):
                w.writerow(dict(Dispatch_Id=did, Kernel_Name=name, Counter_Name=counter,
                                Counter_Value=kib * part, Start_Timestamp=0, End_Timestamp=dur))


def test_summary_scales_by_the_calibration_copy(tmp_path):
    f, w = tmp_path / "f.csv", tmp_path / "w.csv"
    kib = bench.CALIB_BYTES / 1024
    write_csv(f, "FETCH_SIZE", kib / 2, 1000.0)   # fetch counter reads half
    write_csv(w, "WRITE_SIZE", kib, 10.0)
    text = bench.traffic_summary(str(f), str(w))
    kv = dict(l.split(": ", 1) for l in text.splitlines() if ": " in l and not l.startswith(" "))
    assert float(kv["fetch_bytes_per_launch"]) == pytest.approx(1000.0 * 1024 * 2)
    assert float(kv["write_bytes_per_launch"]) == pytest.approx(10.0 * 1024)
    assert float(kv["hbm_bytes_per_launch"]) == pytest.approx(2000.0 * 1024 + 10.0 * 1024)
    assert kv["attention_source_sha256"] == bench.source_digest()


def test_stored_traffic_only_for_the_measured_source(tmp_path, monkeypatch):
    good = tmp_path / "t.txt"
    good.write_text(f"config: hy720\nattention_source_sha256: {bench.source_digest()}\n"
                    "hbm_bytes_per_launch: 1.5e+11\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(good))
    assert bench.committed_traffic("hy720") == 1.5e11
    assert bench.committed_traffic("wan720") is None
    stale = tmp_path / "s.txt"
    stale.write_text("config: hy720\nattention_source_sha256: 00\nhbm_bytes_per_launch: 1e9\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(stale))
    assert bench.committed_traffic("hy720") is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.txt"))
    assert bench.committed_traffic("hy720") is None
