"""The rocprofv3 summarizer: counter aggregation, copy calibration, the
source stamp that tells bench.py whether recorded HBM bytes are current."""
import csv
import json
import os

import pytest

from paper_2511_13198_amd import profiling as pf

K = "void pdy::bwd_dkdv_kernel<128>(pdy::BwdArgs)"
COPY = "__amd_rocclr_copyBuffer"


def _write(d, name, header, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, name), "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def _counters(d, rows):
    _write(d, "run_counter_collection.csv", ["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                              "Counter_Value"], rows)


def _timed_counters(d, rows):
    """rows: (dispatch, kernel, counter, value, start_ns, end_ns)"""
    _write(d, "run_counter_collection.csv", ["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                              "Counter_Value", "Start_Timestamp",
                                              "End_Timestamp"], rows)


def test_summary_from_fake_rocprof_output(tmp_path):
    t = str(tmp_path)
    _write(t + "/trace", "run_kernel_stats.csv",
           ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs",
            "StdDev"], [[K, 2, 6e7, 3e7, 100, 2.9e7, 3.1e7, 1]])
    # 1000 active cycles per XCD over a 1 us dispatch: a 1 GHz clock
    ts = [5000, 6000]
    _timed_counters(t + "/pmc", [[1, K, "GRBM_GUI_ACTIVE", 8 * 1000, *ts],
                                 [1, K, "SQ_WAVE_CYCLES", 500, *ts],
                                 [1, K, "SQ_VALU_MFMA_BUSY_CYCLES", 512 * 1000, *ts],
                                 [1, K, "SQ_WAIT_ANY", 100, *ts],
                                 [1, K, "SQ_ACTIVE_INST_ANY", 250, *ts]])
    # two dispatches: 100 and 300 KiB fetched; the copy moved 1 MiB and read 512 KiB
    _counters(t + "/fetch", [[1, K, "FETCH_SIZE", 100], [2, K, "FETCH_SIZE", 300]])
    _counters(t + "/write", [[1, K, "WRITE_SIZE", 50], [2, K, "WRITE_SIZE", 50]])
    _counters(t + "/cf", [[9, COPY, "FETCH_SIZE", 512]])
    _counters(t + "/cw", [[9, COPY, "WRITE_SIZE", 1024]])
    args = pf.argparse.Namespace(trace=t + "/trace", pmc=t + "/pmc", fetch=t + "/fetch",
                                 write=t + "/write", copy_fetch=t + "/cf", copy_write=t + "/cw",
                                 copy_mib=1, workload="w")
    rec = pf.summarize(args)
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    e = rec["kernels"]["bwd_dkdv_kernel"]
    assert e["avg_ms"] == pytest.approx(30.0)
    assert e["fetch_bytes"] == pytest.approx(200 * 1024 * 2.0)
    assert e["write_bytes"] == pytest.approx(50 * 1024)
    assert e["mfma_busy_pct"] == pytest.approx(50.0)  # 512000 / (1000 * 1024)
    assert e["sq_wait_any_pct_of_wave"] == pytest.approx(20.0)
    assert e["clock_ghz"] == pytest.approx(1.0)
    md = pf.markdown(rec, ["cmd one"])
    assert "`cmd one`" in md and "bwd_dkdv_kernel" in md


def test_source_hash_is_stable_and_names_kernels():
    assert pf.source_hash() == pf.source_hash()
    assert len(pf.source_hash()) == 64
    assert pf.short_name("void pdy::fwd_kernel<128, 8>(pdy::FwdArgs)") == "fwd_kernel"
    assert pf.short_name("__amd_rocclr_copyBuffer") == ""


def test_committed_traffic_record_matches_its_summary():
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    rec = json.load(open(os.path.join(root, "profiles", "single131072_h4_d128_traffic.json")))
    md = open(os.path.join(root, "profiles", "single131072_h4_d128_kernels.md")).read()
    assert rec["source_sha256"] in md
    for k in ("fwd_kernel", "bwd_dkdv_kernel", "bwd_dq_kernel"):
        assert rec["kernels"][k]["fetch_bytes"] > 0 and rec["kernels"][k]["write_bytes"] > 0


def test_code_text_ignores_comments_and_layout_only():
    a = "int f(int x) {  // doubles\n  return 2 * x; /* done */\n}\n"
    b = "int f(int x) {\n    return 2 * x;\n}"
    c = "int f(int x) { return 3 * x; }"
    assert pf.code_text(a) == pf.code_text(b)
    assert pf.code_text(a) != pf.code_text(c)
