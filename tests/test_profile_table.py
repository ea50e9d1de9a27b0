"""The per-length profile table: its length sweep, per-batch columns, buffer
accounting and CSV round trip on the host; one small measured table on the
GPU whose times, rates and allocator peaks are checked for consistency."""
import math

import pytest

from paper_2511_13198_amd import accounting as acc
from paper_2511_13198_amd import profile_table as pt
from paper_2511_13198_amd import workloads as wl


def test_sweep_lengths():
    L = pt.sweep_lengths()
    assert L == sorted(set(L))
    assert [s for s in L if s & (s - 1) == 0] == [1 << e for e in range(6, 20)]
    # 624K and the single-sequence batches of the lognormal stream
    for s in (638976, 313313, 366775, 427570, 433630):
        assert s in L
    assert len(L) == 14 + 5
    assert pt.sweep_lengths(4096) == [64, 128, 256, 512, 1024, 2048, 4096]


def test_row_columns_for_a_packed_batch():
    lengths = [3, 0, 5, 64]
    r = pt._row_base("g", "stream_batch", "b", lengths, 32, 8, 128, True)
    assert r["n_seqs"] == 4 and r["tokens"] == 72 and r["max_s"] == 64
    assert r["sum_s2"] == 9 + 25 + 4096
    assert r["pairs_per_head"] == 6 + 15 + 64 * 65 // 2
    assert r["counted_flops"] == 14 * 128 * 32 * r["pairs_per_head"]
    # rates: counted FLOPs over the measured milliseconds
    r = pt._finish(r, lengths, 32, 128, True, 2.0, 5.0)
    f = acc.fwd_flops(lengths, 32, 128)
    assert math.isclose(r["fwd_tflops"], f / 2e-3 / 1e12)
    assert math.isclose(r["bwd_tflops"], 2.5 * f / 5e-3 / 1e12)
    assert math.isclose(r["fwdbwd_tflops"], 3.5 * f / 7e-3 / 1e12)
    assert math.isclose(r["pct_peak"], 100 * r["fwdbwd_tflops"] / 2516.6)


def test_buffer_bytes_by_hand():
    # T=10 tokens in 2 segments, 4 query heads over 2 KV heads, d=8
    b = pt.buffer_bytes(10, 2, 4, 2, 8, 100, 1000)
    q, kv, cu, o, lse = 10 * 4 * 8 * 2, 2 * 10 * 2 * 8 * 2, 3 * 4, 10 * 4 * 8 * 2, 4 * 10 * 4
    assert b["fwd"] == q + kv + cu + o + lse + 100
    do, dq, dkdv = 10 * 4 * 8 * 2, 10 * 4 * 8 * 4, 2 * 10 * 2 * 8 * 4
    assert b["step"] == b["fwd"] + do + dq + dkdv + 1000


def test_stream_total_aggregates():
    rows = []
    for i, (lengths, fm, bm) in enumerate([([100, 200], 1.0, 3.0), ([300000], 50.0, 120.0)]):
        r = pt._row_base("h32kv8_d128", "stream_batch", f"batch{i}", lengths, 32, 8, 128, True)
        r = pt._finish(r, lengths, 32, 128, True, fm, bm)
        r.update({"fwd_peak_bytes": 10 * (i + 1), "step_peak_bytes": 20 * (i + 1),
                  "step_buffer_bytes": 19 * (i + 1), "workspace_bytes": i, "reps": 1})
        rows.append(r)
    t = pt.stream_total(rows)
    allf = acc.fwd_bwd_flops([100, 200, 300000], 32, 128)
    assert math.isclose(t["fwdbwd_tflops"], allf / (174.0e-3) / 1e12, rel_tol=1e-12)
    assert t["n_seqs"] == 3 and t["max_s"] == 300000 and t["step_peak_bytes"] == 40


def test_csv_round_trip(tmp_path):
    r = pt._row_base("h4_d128", "single", "s=64", [64], 4, 4, 128, True)
    r = pt._finish(r, [64], 4, 128, True, 0.01, 0.03)
    r.update({"fwd_peak_bytes": 1, "step_peak_bytes": 2, "step_buffer_bytes": 2,
              "workspace_bytes": 0, "reps": 10})
    p = tmp_path / "t.csv"
    pt.write_csv([r], str(p), "python -m x")
    assert p.read_text().startswith("# command: python -m x\n")
    back = pt.read_csv(str(p))
    assert list(back[0]) == pt.COLUMNS
    assert int(back[0]["tokens"]) == 64 and float(back[0]["bwd_ms"]) == 0.03


def test_stream_batches_fit_the_packing_rule():
    for b in wl.stream_config5():
        assert len(b.lengths) == 1 or b.total_tokens == wl.PACKED_BATCH_TOKENS


@pytest.mark.gpu
def test_measured_table_small():
    """A few short lengths and a ragged packed batch, measured for real."""
    import torch
    rows = pt.run_sweep("h8_d64", [64, 1000])
    rows.append(pt.measure([5, 300, 1, 700], 4, 2, 128, True, warmup=1, reps=3,
                           group="gqa", kind="stream_batch", label="ragged"))
    for r in rows:
        assert r["fwd_ms"] > 0 and r["bwd_ms"] > 0
        assert math.isclose(r["fwdbwd_ms"], r["fwd_ms"] + r["bwd_ms"])
        # the library allocates nothing: the allocator's peak is the 13
        # buffers, each rounded up (to 512 bytes, or by less than 1 MiB when
        # a large buffer takes a whole cached block)
        assert 0 <= r["step_peak_bytes"] - r["step_buffer_bytes"] <= 13 * (1 << 20), r
        assert r["fwd_peak_bytes"] < r["step_peak_bytes"]
        assert r["pct_peak"] > 0
    torch.cuda.synchronize()


def _committed(name):
    import os
    return pt.read_csv(os.path.join(os.path.dirname(os.path.dirname(__file__)), "profiles", name))


@pytest.mark.parametrize("name,hq,hkv", [("length_profile_h4_d128.csv", 4, 4),
                                          ("length_profile_h32kv8_d128.csv", 32, 8)])
def test_committed_sweep_table_is_consistent(name, hq, hkv):
    rows = _committed(name)
    assert [int(r["tokens"]) for r in rows] == pt.sweep_lengths()
    for r in rows:
        s = int(r["tokens"])
        assert int(r["n_seqs"]) == 1 and int(r["max_s"]) == s and int(r["sum_s2"]) == s * s
        assert (int(r["heads_q"]), int(r["heads_kv"])) == (hq, hkv)
        f = acc.fwd_bwd_flops([s], hq, 128)
        assert float(r["counted_flops"]) == pytest.approx(f, rel=1e-5)
        assert float(r["fwdbwd_tflops"]) == pytest.approx(
            f / (float(r["fwdbwd_ms"]) * 1e-3) / 1e12, rel=1e-4)
        assert 0 <= int(r["step_peak_bytes"]) - int(r["step_buffer_bytes"]) <= 13 << 20


def test_committed_stream_table_matches_the_recipe():
    rows = _committed("length_profile_stream_h32kv8_d128.csv")
    batches = wl.stream_config5()
    assert len(rows) == len(batches) + 1 and rows[-1]["kind"] == "stream_total"
    for r, b in zip(rows, batches):
        assert r["kind"] == "stream_batch"
        assert int(r["n_seqs"]) == b.num_seqs and int(r["tokens"]) == b.total_tokens
        assert int(r["max_s"]) == b.max_seqlen
        assert int(r["sum_s2"]) == sum(s * s for s in b.lengths)
    tot = rows[-1]
    assert float(tot["fwdbwd_ms"]) == pytest.approx(sum(float(r["fwdbwd_ms"]) for r in rows[:-1]),
                                                    rel=1e-4)
    assert int(tot["step_peak_bytes"]) == max(int(r["step_peak_bytes"]) for r in rows[:-1])
