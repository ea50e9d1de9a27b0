"""Per-length time and peak-memory profile of the attention layer.

The paper's hybrid cost models (Section 4.3, Eq. 7) take the sequence length
s as their only input and are fitted, per configuration group, to the
measured wall-clock time and the peak device memory that PyTorch's allocator
reports while training on sequences of that length (Section 4.5, cost model
implementations).  This module measures that table for the fused causal
attention forward and backward of this library:

* part "sweep": one sequence of each length s in {64, 128, ..., 2^19},
  638,976 (the paper's "624K") and the single-sequence batches of the
  lognormal stream, for one configuration group;
* part "stream": one row per mini-batch of the lognormal stream (32 query
  heads over 8 KV heads, d = 128), plus one aggregate row.

Times are HIP events around each `attn_fwd` / `attn_bwd` call on the current
stream (median over the repetitions).  Memory is the allocator's peak over
the call's own buffers, which this library never adds to (it allocates
nothing): `fwd_peak_bytes` covers Q, K, V, O, LSE and the forward workspace;
`step_peak_bytes` adds dO, dQ, dK, dV and the backward workspace.
`step_buffer_bytes` is the same sum computed from the shapes (the allocator
rounds each buffer up to a multiple of 512 bytes, and a large buffer that
takes a whole cached block by less than 1 MiB).

Usage:
  python -m paper_2511_13198_amd.profile_table --part sweep --group h4_d128 --out t.csv
  python -m paper_2511_13198_amd.profile_table --part stream --out s.csv
"""
from __future__ import annotations

import argparse
import csv
import statistics
import sys
from typing import Dict, List, Optional, Sequence

from . import accounting as acc
from . import workloads as wl

# (query heads, KV heads, head_dim): one GPU's head share of a 32-head layer
# (4 of 32 heads), and the GQA heads of the lognormal stream
GROUPS: Dict[str, tuple] = {
    "h4_d128": (4, 4, 128),
    "h32kv8_d128": (32, 8, 128),
    "h8_d64": (8, 8, 64),
}

COLUMNS = [
    "group", "kind", "label", "heads_q", "heads_kv", "head_dim", "causal", "dtype",
    "n_seqs", "tokens", "max_s", "sum_s2", "pairs_per_head", "counted_flops",
    "fwd_ms", "bwd_ms", "fwdbwd_ms", "fwd_tflops", "bwd_tflops", "fwdbwd_tflops", "pct_peak",
    "fwd_peak_bytes", "step_peak_bytes", "step_buffer_bytes", "workspace_bytes", "reps",
]

# rough sustained rate used only to choose repetition counts
_PLAN_TFLOPS = 600.0


def sweep_lengths(max_len: int = wl.MAX_TOKENS_624K) -> List[int]:
    """Powers of two from 64 to 2^19, 638,976 and the lengths of the
    single-sequence batches of the lognormal stream, ascending, <= max_len."""
    out = {1 << e for e in range(6, 20)}
    out.add(wl.MAX_TOKENS_624K)
    for b in wl.lognormal_stream():
        if len(b) == 1:
            out.add(b[0])
    return sorted(s for s in out if s <= max_len)


def buffer_bytes(total_tokens: int, num_seqs: int, heads_q: int, heads_kv: int, head_dim: int,
                 fwd_ws: int, bwd_ws: int) -> Dict[str, int]:
    """Bytes of every buffer one forward and one forward+backward step use:
    Q, K, V, cu_seqlens, O, LSE, forward workspace; then dO, dQ, dK, dV and
    the backward workspace."""
    T, d = total_tokens, head_dim
    fwd = (2 * T * d * (2 * heads_q + 2 * heads_kv) + 4 * (num_seqs + 1) + 4 * heads_q * T
           + fwd_ws)
    step = fwd + 2 * T * heads_q * d + 4 * T * d * (heads_q + 2 * heads_kv) + bwd_ws
    return {"fwd": fwd, "step": step}


def reps_for(counted_flops: float) -> tuple:
    """(warmup, timed repetitions): 3 + 10 for calls under ~0.5 s, 1 + 3 above."""
    est = counted_flops / (_PLAN_TFLOPS * 1e12)
    return (3, 10) if est < 0.5 else (1, 3)


def _row_base(group: str, kind: str, label: str, lengths: Sequence[int], hq: int, hkv: int,
              d: int, causal: bool) -> dict:
    return {
        "group": group, "kind": kind, "label": label, "heads_q": hq, "heads_kv": hkv,
        "head_dim": d, "causal": int(causal), "dtype": "bf16",
        "n_seqs": len(lengths), "tokens": int(sum(lengths)),
        "max_s": int(max(lengths)) if lengths else 0,
        "sum_s2": int(sum(int(s) * int(s) for s in lengths)),
        "pairs_per_head": acc.pairs_per_head(lengths, causal),
        "counted_flops": acc.fwd_bwd_flops(lengths, hq, d, causal),
    }


def _finish(row: dict, lengths, hq, d, causal, fwd_ms, bwd_ms) -> dict:
    ff = acc.fwd_flops(lengths, hq, d, causal)
    fb = acc.bwd_flops(lengths, hq, d, causal)
    tot = fwd_ms + bwd_ms
    row.update({
        "fwd_ms": fwd_ms, "bwd_ms": bwd_ms, "fwdbwd_ms": tot,
        "fwd_tflops": ff / (fwd_ms * 1e-3) / 1e12 if fwd_ms > 0 else 0.0,
        "bwd_tflops": fb / (bwd_ms * 1e-3) / 1e12 if bwd_ms > 0 else 0.0,
        "fwdbwd_tflops": (ff + fb) / (tot * 1e-3) / 1e12 if tot > 0 else 0.0,
    })
    row["pct_peak"] = 100.0 * row["fwdbwd_tflops"] / acc.PEAK_BF16_TFLOPS
    return row


def measure(lengths: Sequence[int], heads_q: int, heads_kv: int, head_dim: int,
            causal: bool = True, warmup: Optional[int] = None, reps: Optional[int] = None,
            group: str = "", kind: str = "single", label: str = "") -> dict:
    """Time one packed batch (forward and backward separately) and record the
    allocator's peak over its buffers.  Inputs are the seeded device recipe."""
    import torch

    from . import pdyattn

    lengths = [int(s) for s in lengths]
    hq, hkv, d = heads_q, heads_kv, head_dim
    row = _row_base(group, kind, label, lengths, hq, hkv, d, causal)
    if warmup is None or reps is None:
        w0, r0 = reps_for(row["counted_flops"])
        warmup = w0 if warmup is None else warmup
        reps = r0 if reps is None else reps
    T, n, maxlen = row["tokens"], row["n_seqs"], row["max_s"]
    dev = torch.device("cuda")
    scale = 1.0 / (d ** 0.5)

    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    a0 = torch.cuda.memory_allocated()
    inp = wl.device_inputs(T, hq, hkv, d, device="cuda")
    q, k, v, do = inp["q"], inp["k"], inp["v"], inp["do"]
    cu = torch.from_numpy(wl.cu_from_lengths(lengths)).to(dev)
    torch.cuda.synchronize()
    # peak := what is allocated now; the float32 draws above are not counted
    torch.cuda.reset_peak_memory_stats()

    wsf_n = pdyattn.fwd_workspace_size(T, n, maxlen, hq, hkv, d)
    wsb_n = pdyattn.bwd_workspace_size(T, n, maxlen, hq, hkv, d)
    o = torch.empty_like(q)
    lse = torch.empty((hq, T), dtype=torch.float32, device=dev)
    wsf = torch.empty(wsf_n, dtype=torch.uint8, device=dev)

    def fwd():
        pdyattn.attn_fwd(q, k, v, cu, maxlen, causal, scale, out=o, lse=lse, workspace=wsf)

    for _ in range(max(1, warmup)):  # at least once: O and LSE for the backward
        fwd()
    torch.cuda.synchronize()
    fwd_peak = torch.cuda.max_memory_allocated() - a0 - do.numel() * do.element_size()

    dq = torch.empty((T, hq, d), dtype=torch.float32, device=dev)
    dk = torch.empty((T, hkv, d), dtype=torch.float32, device=dev)
    dv = torch.empty((T, hkv, d), dtype=torch.float32, device=dev)
    wsb = torch.empty(wsb_n, dtype=torch.uint8, device=dev)

    def bwd():
        pdyattn.attn_bwd(q, k, v, o, lse, do, cu, maxlen, causal, scale, dq=dq, dk=dk, dv=dv,
                         workspace=wsb)

    for _ in range(warmup):
        bwd()

    tf, tb = [], []
    for _ in range(reps):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record()
        fwd()
        e[1].record()
        bwd()
        e[2].record()
        e[2].synchronize()
        tf.append(e[0].elapsed_time(e[1]))
        tb.append(e[1].elapsed_time(e[2]))
    torch.cuda.synchronize()
    step_peak = torch.cuda.max_memory_allocated() - a0
    bb = buffer_bytes(T, n, hq, hkv, d, wsf_n, wsb_n)
    row.update({
        "fwd_peak_bytes": int(fwd_peak), "step_peak_bytes": int(step_peak),
        "step_buffer_bytes": bb["step"], "workspace_bytes": wsf_n + wsb_n, "reps": reps,
    })
    del q, k, v, do, o, lse, dq, dk, dv, wsf, wsb, inp
    torch.cuda.empty_cache()
    return _finish(row, lengths, hq, d, causal, statistics.median(tf), statistics.median(tb))


def stream_total(rows: List[dict]) -> dict:
    """Aggregate of the per-batch rows: summed FLOPs over summed time, the
    largest peak."""
    tot = {c: "" for c in COLUMNS}
    r0 = rows[0]
    tot.update({k: r0[k] for k in ("group", "heads_q", "heads_kv", "head_dim", "causal", "dtype")})
    tot.update({"kind": "stream_total", "label": f"{len(rows)} batches"})
    for c in ("n_seqs", "tokens", "sum_s2", "pairs_per_head", "counted_flops", "fwd_ms", "bwd_ms",
              "fwdbwd_ms"):
        tot[c] = sum(r[c] for r in rows)
    tot["max_s"] = max(r["max_s"] for r in rows)
    ff = sum(r["fwd_tflops"] * r["fwd_ms"] for r in rows)  # TFLOP/s * ms = GFLOP
    fb = sum(r["bwd_tflops"] * r["bwd_ms"] for r in rows)
    tot["fwd_tflops"] = ff / tot["fwd_ms"]
    tot["bwd_tflops"] = fb / tot["bwd_ms"]
    tot["fwdbwd_tflops"] = (ff + fb) / tot["fwdbwd_ms"]
    tot["pct_peak"] = 100.0 * tot["fwdbwd_tflops"] / acc.PEAK_BF16_TFLOPS
    for c in ("fwd_peak_bytes", "step_peak_bytes", "step_buffer_bytes", "workspace_bytes"):
        tot[c] = max(r[c] for r in rows)
    tot["reps"] = min(r["reps"] for r in rows)
    return tot


def _fmt(v):
    return f"{v:.6g}" if isinstance(v, float) else v


def write_csv(rows: List[dict], path: str, command: str = "") -> None:
    with open(path, "w", newline="") as f:
        if command:
            f.write(f"# command: {command}\n")
        w = csv.DictWriter(f, fieldnames=COLUMNS)
        w.writeheader()
        for r in rows:
            w.writerow({c: _fmt(r.get(c, "")) for c in COLUMNS})


def read_csv(path: str) -> List[dict]:
    with open(path) as f:
        return list(csv.DictReader(line for line in f if not line.startswith("#")))


def _log(row: dict) -> None:
    print(f"[profile] {row['group']} {row['kind']} {row['label']}: T={row['tokens']} "
          f"n={row['n_seqs']} fwd {row['fwd_ms']:.3f} ms, bwd {row['bwd_ms']:.3f} ms, "
          f"{row['fwdbwd_tflops']:.1f} TFLOP/s, peak {row['step_peak_bytes'] / 2**30:.3f} GiB",
          file=sys.stderr, flush=True)


def run_sweep(group: str, lengths: Sequence[int], causal: bool = True) -> List[dict]:
    hq, hkv, d = GROUPS[group]
    rows = []
    for s in lengths:
        r = measure([s], hq, hkv, d, causal, group=group, kind="single", label=f"s={s}")
        _log(r)
        rows.append(r)
    return rows


def run_stream(n_batches: int = 64) -> List[dict]:
    batches = wl.stream_config5(n_batches)
    hq, hkv, d = batches[0].heads_q, batches[0].heads_kv, batches[0].head_dim
    group = next(g for g, v in GROUPS.items() if v == (hq, hkv, d))
    longest = max(batches, key=lambda b: acc.pairs_per_head(b.lengths))
    # one warmup call on the longest batch, then each batch once
    measure(longest.lengths, hq, hkv, d, True, warmup=1, reps=1, group=group)
    rows = []
    for i, b in enumerate(batches):
        r = measure(b.lengths, hq, hkv, d, True, warmup=0, reps=1, group=group,
                    kind="stream_batch", label=f"batch{i:02d}")
        _log(r)
        rows.append(r)
    rows.append(stream_total(rows))
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--part", choices=("sweep", "stream"), required=True)
    ap.add_argument("--group", choices=sorted(GROUPS), default="h4_d128")
    ap.add_argument("--max-len", type=int, default=wl.MAX_TOKENS_624K)
    ap.add_argument("--lengths", type=str, default="",
                    help="comma-separated lengths instead of the default sweep")
    ap.add_argument("--batches", type=int, default=64)
    ap.add_argument("--out", required=True)
    a = ap.parse_args(argv)

    import torch
    if not torch.cuda.is_available():
        sys.exit("the profile table needs a GPU")
    from . import pdyattn
    pdyattn.lib()  # fail loudly if the HIP library is missing

    if a.part == "sweep":
        lengths = ([int(x) for x in a.lengths.split(",")] if a.lengths
                   else sweep_lengths(a.max_len))
        rows = run_sweep(a.group, lengths)
    else:
        rows = run_stream(a.batches)
    cmd = "python -m paper_2511_13198_amd.profile_table " + " ".join(sys.argv[1:] if argv is None
                                                                     else argv)
    write_csv(rows, a.out, cmd)
    print(f"[profile] wrote {len(rows)} rows to {a.out}", file=sys.stderr, flush=True)


if __name__ == "__main__":
    main()
