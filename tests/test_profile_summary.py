"""Host logic of the rocprofv3 summariser: the step window and the
calibrated counter combination, on small hand-written traces."""
import csv
import json

import pytest

from paper_2605_07243_amd import profile_summary as ps


def _trace(path, names, dur_us=1.0):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, ["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        t = 0
        for n in names:
            w.writerow({"Kernel_Name": n, "Start_Timestamp": t,
                        "End_Timestamp": t + int(dur_us * 1000)})
            t += 10_000


def test_window_keeps_last_complete_unprofiled_steps():
    # warmup, two timed steps, two profiled steps (with the row copy), tail
    m = "block1_reset_kernel"
    names = ["prefill", m, "a", m, "b", "b", m, "c", m, "d", "copy_int_kernel",
             m, "e", "copy_int_kernel", m, "tail"]
    win = ps.step_window(names, 2, m, "copy_int_kernel")
    assert [names[i] for i in win] == [m, "b", "b", m, "c"]
    # without skipping: the last two complete steps are the profiled ones
    win = ps.step_window(names, 2, m, "")
    assert [names[i] for i in win] == [m, "d", "copy_int_kernel",
                                       m, "e", "copy_int_kernel"]
    with pytest.raises(SystemExit):
        ps.step_window(names, 4, m, "copy_int_kernel")


def test_trace_summary_counts_dispatches_per_step(tmp_path):
    m = "void sb::block1_reset_kernel(int*)"
    names = [m, "void sb::gemm_tile_kernel<2, 1, 2, false, 0>(float*)",
             "void sb::gemm_tile_kernel<2, 1, 2, false, 0>(float*)"] * 3 + [m]
    p = tmp_path / "t.csv"
    _trace(p, names, dur_us=2.0)
    agg, busy, n = ps.summarise(str(p), 3, "block1_reset_kernel")
    assert n == 9
    assert agg["gemm_tile_kernel<2, 1, 2, false, 0>"] == [6, pytest.approx(12.0)]
    assert busy == pytest.approx(18.0)


def test_combine_scales_each_counter_by_its_calibration(tmp_path):
    fam = "gemm_tile_kernel<2, 1, 2, false, 0>"
    fetch = {"factor": {"FETCH_SIZE": 0.5}, "per_dispatch_kib": {
        fam: {"dispatches_per_step": 4.0, "FETCH_SIZE": 100.0},
        "residual_kernel<unsigned short>": {"dispatches_per_step": 9.0,
                                            "FETCH_SIZE": 7.0}}}
    write = {"factor": {"WRITE_SIZE": 1.0}, "per_dispatch_kib": {
        fam: {"dispatches_per_step": 4.0, "WRITE_SIZE": 10.0}}}
    fj, wj, oj = (tmp_path / n for n in ("f.json", "w.json", "o.json"))
    fj.write_text(json.dumps(fetch))
    wj.write_text(json.dumps(write))
    ps.combine(str(fj), str(wj), str(oj))
    out = json.loads(oj.read_text())
    assert out["fetch"]["bytes_per_dispatch"] == pytest.approx(100 * 1024 / 0.5)
    assert out["write"]["bytes_per_dispatch"] == pytest.approx(10 * 1024)
    assert out["bytes_per_dispatch"] == pytest.approx(200 * 1024 + 10 * 1024)
    assert out["sources_sha256"] == ps.gemm_sources_sha256()
