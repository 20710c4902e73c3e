"""The rocprofv3 summary tool on synthetic counter files (CPU only): calibration from the
fill / copy / sum kernels, the span of one level, and the sums."""
import csv

import pytest

from paper_2608_21131_amd import rocprof_summary as rs

HEAD = ["Correlation_Id", "Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value",
        "Start_Timestamp", "End_Timestamp"]
GIB_KIB = (1 << 30) // 1024


def _write(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(HEAD)
        t = 1000
        for i, (name, grid, val) in enumerate(rows):
            w.writerow([i + 1, i + 1, grid, name, counter, val, t, t + 500])
            t += 1000


def _runs(tmp_path, read_scale, write_scale, level):
    """Calibration kernels, a warm-up level and a timed level; level = [(kernel, read, write)]."""
    fill = "void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<double> >"
    copy = "__amd_rocclr_copyBuffer"
    red = "void at::native::reduce_kernel<512, 1, at::native::ReduceOp<double> >"
    cal_f = [(fill, 1 << 25, 3.0), (copy, 1 << 17, GIB_KIB * read_scale), (red, 1 << 17, GIB_KIB * read_scale)]
    cal_w = [(fill, 1 << 25, GIB_KIB * write_scale), (copy, 1 << 17, GIB_KIB * write_scale), (red, 1 << 17, 0.1)]
    seq = [("k_warm", 64, 1.0, 1.0), ("k_mac_diag3<32>", 3072, 5.0, 5.0)]
    for _ in range(2):
        seq += [(k, 64, r, w_) for k, r, w_ in level]
    fe = [(k, g, r * read_scale / 1024) for k, g, r, _ in seq]
    wr = [(k, g, w_ * write_scale / 1024) for k, g, _, w_ in seq]
    _write(tmp_path / "f.csv", "FETCH_SIZE", cal_f + fe)
    _write(tmp_path / "w.csv", "WRITE_SIZE", cal_w + wr)
    return tmp_path / "f.csv", tmp_path / "w.csv"


def test_traffic_sums_one_level_with_calibrated_factors(tmp_path):
    # counters reporting half the reads and all the writes (as measured on the MI355X)
    level = [("k_giant_ks<4, 16>", 1000.0, 100.0), ("k_ntt_inv_b", 200.0, 200.0),
             ("k_moddown_ks_b<4, 8, true>", 3000.0, 600.0), ("k_mac_diag3<32>", 14000.0, 400.0)]
    f, w = _runs(tmp_path, 0.5, 1.0, level)
    txt = rs.traffic(str(f), str(w))
    vals = dict(line.split(": ") for line in txt.splitlines() if line.startswith("level_"))
    assert int(vals["level_read_bytes"]) == 18200
    assert int(vals["level_write_bytes"]) == 1300
    assert int(vals["level_traffic_bytes"]) == 19500
    assert "read factor 2.0000" in txt and "write factor 1.0000" in txt
    assert f"sources_sha256: {rs.sources_sha256()}" in txt


def test_traffic_refuses_runs_without_calibration(tmp_path):
    _write(tmp_path / "f.csv", "FETCH_SIZE", [("k_mac_diag3<32>", 64, 1.0), ("k_mac_diag3<32>", 64, 1.0)])
    _write(tmp_path / "w.csv", "WRITE_SIZE", [("k_mac_diag3<32>", 64, 1.0), ("k_mac_diag3<32>", 64, 1.0)])
    with pytest.raises(SystemExit):
        rs.traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"))


def test_trace_lists_the_level_span(tmp_path):
    rows = [("k_warm", 64, 0.0), ("k_mac_diag3<32>", 64, 0.0), ("k_ntt_inv_b", 64, 0.0), ("k_giant_ks<4, 16>", 64, 0.0),
            ("k_mac_diag3<32>", 64, 0.0)]
    _write(tmp_path / "t.csv", "none", rows)
    txt = rs.trace(str(tmp_path / "t.csv"))
    assert "| k_ntt_inv_b | 1 |" in txt and "| k_giant_ks | 1 |" in txt and "| k_mac_diag3 | 1 |" in txt
    assert "k_warm" not in txt


def test_waves_normalises_by_wave_cycles_over_the_level(tmp_path):
    # two counters per dispatch, as rocprofv3 writes them: one row per counter
    path = tmp_path / "sq.csv"
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(HEAD)
        disp = [("k_mac_diag3<32>", 8.0, 100.0), ("k_giant_ks<4, 16>", 30.0, 100.0), ("k_mac_diag3<32>", 40.0, 100.0)]
        for i, (name, wait, cyc) in enumerate(disp):
            for c, v in (("SQ_WAIT_ANY", wait), ("SQ_WAVE_CYCLES", cyc)):
                w.writerow([i + 1, i + 1, 64, name, c, v, 1000 * i, 1000 * i + 500])
    txt = rs.waves(str(path))
    assert "| k_giant_ks | 0.30 |" in txt and "| k_mac_diag3 | 0.40 |" in txt
