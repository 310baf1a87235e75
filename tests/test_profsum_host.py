"""The profile summariser on a synthetic rocprofv3 output folder: which
dispatches it selects, the kernel-trace mean, the HBM traffic scaled by the
copy calibration and the traffic line it writes (the line bench.py reads)."""
import csv
import json
import os
import re

import pytest

from paper_1909_10616_amd import profsum

KERNEL = "void gt::gemm_kernel_dl<16, 8, 4, 4>(gt::KArgs)"
GRID_X, WAVES, LDS = 256, 8, 163840


def _csv(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)


def _counter_rows(kernel, name, values, grid=GRID_X * 64 * WAVES, lds=0):
    return [{"Dispatch_Id": i, "Kernel_Name": kernel, "Grid_Size": grid, "LDS_Block_Size": lds,
             "Counter_Name": name, "Counter_Value": v} for i, v in enumerate(values)]


@pytest.fixture
def out(tmp_path):
    d = tmp_path / "prof"
    bench = {"metric": "m", "value": 1234.5, "config": {
        "workload": "gemm4096_bf16", "M": 4096, "N": 4096, "K": 4096,
        "kernel_name": "gt::gemm_kernel_dl<16, 8, 4, 4>",
        "kernel": {"grid_x": GRID_X, "grid_y": 1, "waves": WAVES, "lds_bytes": LDS,
                   "BM": 256, "BN": 256, "BK": 32},
        "best_config": "m[16, 2, 8, 16]k[128, 1, 1, 32]n[16, 4, 2, 32]mfma16",
        "configs_timed": 1000, "space_size": 188392750, "fraction_of_space_pct": 0.00053,
        "search_wall_s": 7.3, "best_ms": 0.1114,
        "launch_signature": "gemm4096_bf16 gt::gemm_kernel_dl<16,8,4,4> grid=256x1 waves=8 "
                            "lds=163840 dl=1/5",
        "kernel_source": "0123456789abcdef"},
        "roofline": {"peak": 2516.6, "frac": 0.4905, "algorithmic_bytes": 134217728}}
    os.makedirs(d)
    with open(d / "bench_traced.json", "w") as f:
        f.write("[bench] progress line\n" + json.dumps(bench) + "\n")
    rows, t = [], 0
    # 250 dispatches of the kernel, durations 100.000 … 100.249 µs, between
    # them dispatches of another grid and another kernel that must not count
    for i in range(250):
        for name, grid, dur in ((KERNEL, GRID_X * 64 * WAVES, 100000 + i),
                                (KERNEL, 64 * 64 * WAVES, 5000),
                                ("copy_kernel", 1 << 20, 7000)):
            rows.append({"Kernel_Name": name, "Start_Timestamp": t, "End_Timestamp": t + dur,
                         "Grid_Size_X": grid, "Grid_Size_Y": 1, "Workgroup_Size_X": 512,
                         "LDS_Block_Size": 0, "VGPR_Count": 112, "Accum_VGPR_Count": 0,
                         "SGPR_Count": 112, "Scratch_Size": 0})
            t += dur + 10
    _csv(str(d / "trace" / "bench_kernel_trace.csv"), rows)
    _csv(str(d / "fetch" / "k_counter_collection.csv"),
         _counter_rows(KERNEL, "FETCH_SIZE", [98000, 99000]) +
         _counter_rows(KERNEL, "FETCH_SIZE", [1.0], grid=4096))
    _csv(str(d / "write" / "k_counter_collection.csv"), _counter_rows(KERNEL, "WRITE_SIZE", [65536]))
    _csv(str(d / "cfetch" / "c_counter_collection.csv"),
         _counter_rows("copy_kernel", "FETCH_SIZE", [524288, 524288], grid=1 << 28))
    _csv(str(d / "cwrite" / "c_counter_collection.csv"),
         _counter_rows("copy_kernel", "WRITE_SIZE", [1048576], grid=1 << 28))
    _csv(str(d / "util" / "u_counter_collection.csv"),
         _counter_rows(KERNEL, "SQ_WAIT_ANY", [10, 30]) + _counter_rows(KERNEL, "GRBM_GUI_ACTIVE", [7]))
    return str(d)


def test_traffic_scaled_by_the_copy(out):
    t = profsum.traffic(*(os.path.join(out, x) for x in ("fetch", "write", "cfetch", "cwrite")),
                        1 << 30, "gemm_kernel_dl<16, 8, 4, 4>", GRID_X * 64 * WAVES, LDS)
    # the copy of 1 GiB reads 512 MiB as FETCH_SIZE (factor 2) and 1 GiB as WRITE_SIZE (factor 1)
    assert t["fetch_factor"] == 2.0 and t["write_factor"] == 1.0
    assert t["fetch_kib"] == 98500.0 and t["write_kib"] == 65536.0
    assert t["traffic_bytes"] == 98500 * 1024 * 2 + 65536 * 1024


def test_report_selects_the_last_200_dispatches_of_the_tuned_launch(out):
    md = profsum.report(out, extra="--workload gemm4096_bf16 --no-enumeration")
    # last 200 of 250: durations 100.050 … 100.249 µs
    mean = sum(100000 + i for i in range(50, 250)) / 200 / 1e3
    assert f"| kernel trace, last 200 dispatches of CFG | 200 | {mean:.2f} |" in md
    assert "bench.py --no-cpu-baseline --workload gemm4096_bf16 --no-enumeration" in md
    assert 'report OUT --args "--workload gemm4096_bf16 --no-enumeration"' in md
    assert "- SQ_WAIT_ANY: 20" in md and "- GRBM_GUI_ACTIVE: 7" in md
    line = md.rstrip().splitlines()[-1].strip()
    assert line == ("gemm4096_bf16 gt::gemm_kernel_dl<16,8,4,4> grid=256x1 waves=8 lds=163840 "
                    f"dl=1/5 | source=0123456789abcdef traffic_bytes={98500 * 2048 + 65536 * 1024}")
    ratio = float(re.search(r"bytes \(A and B read once, C written once\): ([0-9.]+)x", md).group(1))
    assert ratio == round((98500 * 2048 + 65536 * 1024) / 134217728, 2)


def test_best_configuration_for_replay(out):
    assert profsum.best_cfg(os.path.join(out, "bench_traced.json")) == \
        [[16, 2, 8, 16], [128, 1, 1, 32], [16, 4, 2, 32], 16]
