"""The rocprofv3 summary helpers, on small synthetic output directories."""
import csv
import json
import os

import pytest

from paper_2508_09001_amd import profiling

NAME = "void retro::(anonymous namespace)::attend_kernel<retro::bf16_t, 128, 1>(retro::AttendArgs)"
COPY = "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda(at::TensorIteratorBase&)::{lambda()#1}, std::array<char*, 2ul> >(int, float)"


def _write(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def _counters(d, counter, rows):
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    _write(os.path.join(d, "run_counter_collection.csv"), hdr,
           [[i, name, counter, v] for i, (name, v) in enumerate(rows)])


def test_short_names():
    assert profiling._short(NAME) == "attend_kernel<bf16_t, 128, 1>"
    assert profiling._short("void retro::(anonymous namespace)::topk_mask_kernel<256, 12>"
                            "(retro::TopkArgs, int const*)") == "topk_mask_kernel<256, 12>"
    assert profiling._short("__amd_rocclr_copyBuffer") == "__amd_rocclr_copyBuffer"


def test_stats_table(tmp_path):
    hdr = ["Kernel_Name", "Start_Timestamp", "End_Timestamp"]
    _write(str(tmp_path / "s" / "run_kernel_trace.csv"), hdr,
           [[NAME, 1000, 11000], [NAME, 20000, 32000], [COPY, 0, 500]])
    table = profiling.stats_table(str(tmp_path / "s"))
    lines = table.splitlines()
    assert lines[2].startswith("| attend_kernel<bf16_t, 128, 1> | 2 | 11.00 | 10.00 | 12.00 | 22.0 |")
    assert "| 1 | 0.50 |" in lines[3]


def test_last_dispatches_average(tmp_path):
    hdr = ["Kernel_Name", "Start_Timestamp", "End_Timestamp"]
    _write(str(tmp_path / "s" / "run_kernel_trace.csv"), hdr,
           [[NAME, 50000, 54000], [NAME, 1000, 11000], [COPY, 0, 500], [NAME, 60000, 62000]])
    n, avg = profiling.last_dispatches_avg(str(tmp_path / "s"), "attend_kernel", 2)
    assert n == 2 and avg == pytest.approx(3.0)   # the two latest: 4 us and 2 us
    n, avg = profiling.last_dispatches_avg(str(tmp_path / "s"), "attend_kernel", 10)
    assert n == 3 and avg == pytest.approx(16.0 / 3)


def test_traffic_scaling(tmp_path):
    # the kernel's counters are per dispatch, summed over counter instances; the
    # calibration copy of N bytes reports N/2 KiB for FETCH_SIZE, N KiB for WRITE_SIZE
    n = 512 << 20
    _counters(str(tmp_path / "f"), "FETCH_SIZE", [(NAME, 1000.0), (NAME, 3000.0), (COPY, 7.0)])
    _counters(str(tmp_path / "w"), "WRITE_SIZE", [(NAME, 500.0), (NAME, 500.0)])
    _counters(str(tmp_path / "cf"), "FETCH_SIZE", [(COPY, n / 1024 / 2)])
    _counters(str(tmp_path / "cw"), "WRITE_SIZE", [(COPY, n / 1024)])
    src = tmp_path / "k.hip"
    src.write_text("// kernel\n")
    out = tmp_path / "t.json"
    profiling.main(["traffic", "--kernel", "attend_kernel", "--fetch", str(tmp_path / "f"),
                    "--write", str(tmp_path / "w"), "--calib-fetch", str(tmp_path / "cf"),
                    "--calib-write", str(tmp_path / "cw"), "--calib-kernel", "neg_kernel",
                    "--calib-bytes", str(n), "--sources", str(src), "--out", str(out)])
    d = json.loads(out.read_text())
    assert d["dispatches"] == {"fetch": 2, "write": 2}
    assert d["fetch_scale"] == pytest.approx(2.0) and d["write_scale"] == pytest.approx(1.0)
    assert d["hbm_fetch_bytes_per_launch"] == 2000 * 1024 * 2
    assert d["hbm_write_bytes_per_launch"] == 500 * 1024
    assert d["hbm_bytes_per_launch"] == d["hbm_fetch_bytes_per_launch"] + d["hbm_write_bytes_per_launch"]
    assert d["source_sha256"] == profiling.sources_sha256([str(src)])
