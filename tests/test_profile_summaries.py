"""Host logic of the rocprofv3 summaries: dispatches are attributed to the
segment their marker opened, the calibration copy scales the byte counters,
and bench.py takes the traffic figure back only for the same conv source.

Synthetic CSVs in rocprofv3's column layout stand in for real runs."""
import contextlib
import csv
import io
import json
import os

import pytest

CONV = "void dstack::conv_igemm_kernel<64, 64, 2, 2, 4, 3, false, false>(dstack::ConvArgs)"
CONV1 = "void dstack::conv_igemm_1x1s_kernel<1>(dstack::ConvArgs)"
PROBE = "dstack::probe_kernel(unsigned int*)"
COPY = "void at::native::elementwise_kernel<copy>"
OTHER = "dstack::maxpool_kernel(...)"


def dispatches():
    """(name, grid threads, duration ns, fetch KiB, write KiB) in dispatch order."""
    return [
        (CONV, 4096, 9000, 99.0, 99.0),       # before any marker: ignored
        (PROBE, 1100 * 64, 1000, 0, 0),       # model 0
        (CONV, 4096, 10000, 100.0, 40.0),
        (OTHER, 4096, 3000, 7.0, 7.0),        # not a conv: ignored
        (CONV1, 4096, 6000, 50.0, 20.0),
        (PROBE, 999 * 64, 1000, 0, 0),
        (CONV, 4096, 50000, 999.0, 999.0),    # between segments: ignored
        (PROBE, 1103 * 64, 1000, 0, 0),       # model 3
        (CONV, 4096, 20000, 200.0, 80.0),
        (PROBE, 999 * 64, 1000, 0, 0),
        (PROBE, 1199 * 64, 1000, 0, 0),       # calibration: 256 MiB copy read at half, written at full count
        (COPY, 1 << 20, 40000, 131072.0, 262144.0),
        (PROBE, 999 * 64, 1000, 0, 0),
    ]


def write_trace(d):
    os.makedirs(d)
    with open(os.path.join(d, "x_kernel_trace.csv"), "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X", "Grid_Size_Y",
                    "Grid_Size_Z"])
        t = 1000
        for i, (name, grid, dur, _, _) in enumerate(dispatches()):
            w.writerow([i + 1, name, t, t + dur, grid, 1, 1])
            t += dur + 100
    with open(os.path.join(d, "x_kernel_stats.csv"), "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs", "StdDev"])
        w.writerow([CONV, 4, 89000, 22250.0, 50.0, 9000, 50000, 1.0])


def write_counters(d, counter, col):
    os.makedirs(d)
    with open(os.path.join(d, "x_counter_collection.csv"), "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
                    "End_Timestamp"])
        for i, row in enumerate(dispatches()):
            w.writerow([i + 1, row[1], row[0], counter, row[col], 0, 1])


def bench_log(path):
    line = dict(metric="m", config=dict(capacity_k=1.5, overprov_slots=0, batch=[8, 16, 4, 16],
                                        deployed_slots=[10, 6, 12, 4], home_offset=[0, 10, 16, 28]),
                roofline=dict(launches=3, avg_launch_us=11.0, flops_per_launch=1e9, algorithmic_bytes_per_launch=1e5))
    with open(path, "w") as f:
        f.write("progress text\n" + json.dumps(line) + "\n")


@pytest.fixture()
def runs(tmp_path):
    write_trace(str(tmp_path / "kt"))
    write_counters(str(tmp_path / "fetch"), "FETCH_SIZE", 3)
    write_counters(str(tmp_path / "write"), "WRITE_SIZE", 4)
    bench_log(str(tmp_path / "bench.log"))
    return tmp_path


def captured(fn, *a):
    buf = io.StringIO()
    with contextlib.redirect_stdout(buf):
        fn(*a)
    return buf.getvalue()


def test_bench_kernels_attributes_marked_conv_dispatches(runs):
    from paper_2304_13541_amd import layer_profile as lp
    out = captured(lp.bench_kernels, str(runs / "kt"), str(runs / "bench.log"))
    assert "| resnet50 conv dispatches / mean us (rocprofv3) | 2 / 8.00 |" in out
    assert "| lstm2 conv dispatches / mean us (rocprofv3) | 1 / 20.00 |" in out
    assert "| all conv dispatches of the roofline forwards / mean us (rocprofv3) | 3 / 12.00 |" in out
    assert "mobilenetv2 conv" not in out and "vgg19 conv" not in out
    # 1e9 FLOP / 12 us = 83.3 TFLOP/s
    assert "| 83.3 |" in out


def test_bench_traffic_calibrates_and_records_source(runs, monkeypatch):
    from paper_2304_13541_amd import layer_profile as lp
    out = captured(lp.bench_traffic, str(runs / "fetch"), str(runs / "write"), str(runs / "bench.log"))
    assert "| conv dispatches counted | 3 | 3 |" in out
    assert "| calibration factor | 2.0000 | 1.0000 |" in out
    # fetch (100 + 50 + 200) KiB x 2, write (40 + 20 + 80) KiB x 1, over 3 launches
    expect = ((100 + 50 + 200) * 2 + (40 + 20 + 80)) * 1024 / 3
    vals = dict(l.split(":", 1) for l in out.splitlines() if l.split(":")[0] in ("traffic_bytes_per_launch", "plan",
                                                                                  "source_sha256"))
    assert float(vals["traffic_bytes_per_launch"]) == pytest.approx(expect, rel=1e-5)
    assert json.loads(vals["plan"]) == dict(batch=[8, 16, 4, 16], deployed_slots=[10, 6, 12, 4],
                                            home_offset=[0, 10, 16, 28])

    # bench.py reads it back while the conv source is the one hashed, not after it changed
    import bench
    f = runs / "traffic.md"
    f.write_text("# summary\n" + out)
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    t, plan = bench.measured_traffic()
    assert t == pytest.approx(expect, rel=1e-5) and plan["batch"] == [8, 16, 4, 16]
    src = runs / "conv.hip"
    src.write_text("changed")
    monkeypatch.setattr(bench, "CONV_SRC", str(src))
    assert bench.measured_traffic() == (None, None)


def test_summarize_cases_and_wave_states(tmp_path, monkeypatch):
    """--cases labels the segments; the SQ counters become shares of the
    wave-cycles."""
    from paper_2304_13541_amd import layer_profile as lp
    d = tmp_path / "p1"
    os.makedirs(d)
    counters = {"SQ_WAVES": 8, "SQ_WAVE_CYCLES": 1000, "SQ_WAIT_ANY": 600, "SQ_WAIT_INST_ANY": 70,
                "SQ_ACTIVE_INST_ANY": 300, "SQ_ACTIVE_INST_VMEM": 50, "SQ_ACTIVE_INST_LDS": 40,
                "SQ_ACTIVE_INST_VALU": 100, "SQ_ACTIVE_INST_SCA": 30, "SQ_VALU_MFMA_BUSY_CYCLES": 2400,
                "GRBM_GUI_ACTIVE": 100}
    rows = [(PROBE, 1000 * 64, {}), (CONV, 4096, counters), (PROBE, 999 * 64, {}),
            (PROBE, 1001 * 64, {}), (OTHER, 4096, {"SQ_WAVES": 4}), (PROBE, 999 * 64, {}),
            (PROBE, 1002 * 64, {}), (COPY, 1 << 20, {"FETCH_SIZE": 131072.0}), (PROBE, 999 * 64, {})]
    with open(d / "x_counter_collection.csv", "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
                    "End_Timestamp"])
        for i, (name, grid, cs) in enumerate(rows):
            for cn, v in (cs or {"SQ_WAVES": 1}).items():
                w.writerow([i + 1, grid, name, cn, v, 0, 2000])
    monkeypatch.setattr(lp, "CASES", [("resnet50", 16, 3), ("lstm2", 32, 16)])
    out = captured(lp.summarize, [str(d)])
    assert "| 24 | resnet50 b16 | conv | 1 |" in out
    assert "| 128 | lstm2 b32 | pool | 1 |" in out
    # waiting 0.60, to issue 0.07, issuing 0.30 (VMEM 0.05, LDS 0.04, VALU
    # 0.10, scalar 0.03); MFMA busy 2400 / (100 x 24 CUs) = 1.000
    assert "| 24 | resnet50 b16 | conv | 8 | 0.60 | 0.07 | 0.30 | 0.05 | 0.04 | 0.10 | 0.03 | 1.000 |" in out


def test_summarize_lds_port(tmp_path, monkeypatch):
    """LDS reads and buffer-to-LDS fills per CU-cycle of the kernel time at
    the 2.4 GHz clock, per MFMA-busy cycle, and the MFMA share a 128-byte
    port allows at that ratio."""
    from paper_2304_13541_amd import layer_profile as lp
    d = tmp_path / "p1"
    os.makedirs(d)
    # 2 us on 24 CUs = 2 x 2400 x 24 = 115200 CU-cycles
    counters = {"SQ_INSTS_LDS_LOAD_BANDWIDTH": 115200, "TA_BUFFER_READ_LDS_WAVEFRONTS_sum": 3600,
                "SQ_VALU_MFMA_BUSY_CYCLES": 115200, "SQ_LDS_BANK_CONFLICT": 0, "SQ_LDS_DATA_FIFO_FULL": 1152,
                "GRBM_GUI_ACTIVE": 1}
    rows = [(PROBE, 1000 * 64, {}), (CONV, 4096, counters), (PROBE, 999 * 64, {}),
            (PROBE, 1001 * 64, {}), (COPY, 1 << 20, {"FETCH_SIZE": 131072.0}), (PROBE, 999 * 64, {})]
    with open(d / "x_counter_collection.csv", "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
                    "End_Timestamp"])
        for i, (name, grid, cs) in enumerate(rows):
            for cn, v in (cs or {"SQ_WAVES": 1}).items():
                w.writerow([i + 1, grid, name, cn, v, 0, 2000])
    monkeypatch.setattr(lp, "CASES", [("resnet50", 16, 3)])
    out = captured(lp.summarize, [str(d)])
    # reads 64 B/clk/CU, fills 3600 KB / 115200 = 32, total 96; MFMA busy
    # 115200 / (4 x 115200) = 0.25, so 384 LDS bytes per busy cycle and a
    # 128-byte port allows 0.33 of the MFMA rate
    assert "| 24 | resnet50 b16 | conv | 2.0 | 64.0 | 32.0 | 96.0 | 0.250 | 384 | 0.33 | 0.000 | 0.010 |" in out
