"""Host logic of the HBM-traffic summaries (no GPU): counter scaling by the
calibration copy and the source stamp that invalidates stale figures."""

import csv

from paper_2205_01435_amd import traffic


def _csv(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, v in rows:
            w.writerow({"Kernel_Name": name, "Grid_Size": 256, "Counter_Name": counter, "Counter_Value": v})


def test_summary_scaling_and_stamp(tmp_path):
    calib_kib = traffic.CALIB_BYTES / 1024
    # the copy shows half its bytes (plus a little) in FETCH_SIZE, all of them in WRITE_SIZE
    fk = calib_kib / 2 + 64
    _csv(tmp_path / "f.csv", "FETCH_SIZE", [("copyBuffer", fk), ("k_persist<2, 4, false>", 100.0),
                                            ("k_persist<2, 4, false>", 300.0), ("k_gates<x>", 7.0)])
    _csv(tmp_path / "w.csv", "WRITE_SIZE", [("copyBuffer", calib_kib), ("k_persist<2, 4, false>", 50.0),
                                            ("k_persist<2, 4, false>", 50.0)])
    out = tmp_path / "s.md"
    res = traffic.summarize(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "k_persist<2, 4, false>",
                            str(out), "cmd")
    f = calib_kib / fk
    assert abs(res["FETCH_SIZE"]["factor"] - f) < 1e-12 and res["WRITE_SIZE"]["factor"] == 1.0
    want = (200.0 * f + 50.0) * 1024
    assert abs(res["traffic_bytes_per_launch"] - want) < 1e-6 * want
    assert abs(traffic.read_summary(str(out)) - want) <= 1.0  # the summary keeps whole bytes
    text = out.read_text()
    assert "kernel_sources: wm_persist.hip," in text
    # a stamp that does not match the current sources reads as no figure
    stale = text.replace("kernel_source_sha256: ", "kernel_source_sha256: 0")
    out.write_text(stale)
    assert traffic.read_summary(str(out)) is None
    assert traffic.read_summary(str(tmp_path / "missing.md")) is None


def test_kernel_sources_by_class():
    assert traffic.kernel_sources("k_persist<1, 2, true>")[0] == "wm_persist.hip"
    assert traffic.kernel_sources("k_gates")[0] == "wm_kernels.hip"
