"""Context-parallel (sequence-sharded) attention: the ring steps of each
device, run one device after another on a single GPU.

With p devices every device owns some query positions of the sequence and
the keys/values of the same positions (section 2.2: the context-parallel
strategies shard the sequence and exchange K/V between the shards).  Two
layouts:

* contiguous: device r owns chunk r of p near-equal chunks;
* zigzag: the sequence is cut into 2p chunks and device r owns chunks r and
  2p-1-r, which evens out the causal work (an early chunk sees few keys, its
  partner near the end sees many).

Key/value shards travel around the ring, so at step t device r holds the
shard of device (r - t) mod p.  For every (own query range, visiting key
range) pair with at least one visible key the device calls attn_fwd_chunk
and folds the partial result into that range's running (O, LSE) with
attn_merge.  The backward, given the final O and LSE, calls attn_bwd_chunk
per pair, accumulating dQ of its own ranges and dK/dV of the visiting shard,
which travel on with it.  At step 0 a device's diagonal pairs run first and
overwrite, so each of its dQ and dK/dV buffers is written before anything
is added to it; every later call adds.

ring_forward / ring_backward run the devices' steps one after another on one
GPU (the exchanges become no-ops): a single-GPU check of the chunked path
against plain attention.  `python -m paper_2511_13198_amd.context_parallel`
times each device's share of a ring (its forward and backward calls) at a
full sequence length.  Every step runs in the library's kernels; this module
only orders the calls.
"""
from __future__ import annotations

import argparse
import json
import sys
import time
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

from . import pdyattn

Range = Tuple[int, int]


def chunk_bounds(total_tokens: int, n: int) -> List[Range]:
    """n contiguous chunks of near-equal length (the first T mod n one longer)."""
    if n < 1:
        raise ValueError("the number of chunks must be >= 1")
    base, extra = divmod(total_tokens, n)
    out, a = [], 0
    for r in range(n):
        b = a + base + (1 if r < extra else 0)
        out.append((a, b))
        a = b
    return out


def device_ranges(total_tokens: int, p: int, layout: str = "contiguous") -> List[List[Range]]:
    """Position ranges owned by each of the p devices, in position order."""
    if layout == "contiguous":
        return [[c] for c in chunk_bounds(total_tokens, p)]
    if layout == "zigzag":
        c = chunk_bounds(total_tokens, 2 * p)
        return [[c[r], c[2 * p - 1 - r]] for r in range(p)]
    raise ValueError(f"unknown layout {layout!r}")


def ring_order(r: int, p: int) -> List[int]:
    """Device whose key/value shard device r holds at steps 0 .. p-1."""
    return [(r - t) % p for t in range(p)]


def visible(q: Range, k: Range, causal: bool) -> bool:
    """Whether any key of range k is visible to a query of range q."""
    (qa, qb), (ka, kb) = q, k
    return qb > qa and kb > ka and (not causal or ka <= qb - 1)


def pair_count(q: Range, k: Range, causal: bool) -> int:
    """Number of (query, key) pairs of the two ranges that attend (per head)."""
    (qa, qb), (ka, kb) = q, k
    if qb <= qa or kb <= ka:
        return 0
    if not causal:
        return (qb - qa) * (kb - ka)

    def upto(n: int) -> int:
        # sum over query positions i < n of min(max(i - ka + 1, 0), kb - ka)
        if n <= ka:
            return 0
        ramp_end = min(n, kb)                   # i in [ka, ramp_end): i - ka + 1 keys
        m = ramp_end - ka
        return m * (m + 1) // 2 + max(0, n - kb) * (kb - ka)

    return upto(qb) - upto(qa)


def device_steps(r: int, ranges: Sequence[Sequence[Range]], causal: bool
                 ) -> List[Tuple[Range, Range, bool]]:
    """Chunk pairs of device r in call order: (query range, key range,
    accumulate).  Step 0 (its own shard) puts the diagonal pairs first; they
    are called even when empty so that every output buffer gets written."""
    p = len(ranges)
    own = ranges[r]
    out: List[Tuple[Range, Range, bool]] = [(rg, rg, False) for rg in own]
    for q in own:
        for k in own:
            if q != k and visible(q, k, causal):
                out.append((q, k, True))
    for src in ring_order(r, p)[1:]:
        for k in ranges[src]:
            for q in own:
                if visible(q, k, causal):
                    out.append((q, k, True))
    return out


def device_pairs(r: int, ranges: Sequence[Sequence[Range]], causal: bool) -> int:
    return sum(pair_count(q, k, causal) for q, k, _ in device_steps(r, ranges, causal))


def concurrent_groups(calls: Sequence[Tuple[Range, Range, bool]]
                      ) -> List[List[Tuple[Range, Range, bool]]]:
    """Split an ordered list of (query range, key range, accumulate) calls
    into consecutive groups of at most two calls that touch different query
    ranges and different key ranges: the calls of a group write disjoint
    dQ and dK/dV rows and may run at the same time, while a call still runs
    after every earlier call that writes the same rows."""
    groups: List[List[Tuple[Range, Range, bool]]] = []
    cur: List[Tuple[Range, Range, bool]] = []
    for c in calls:
        if len(cur) < 2 and all(c[0] != o[0] and c[1] != o[1] for o in cur):
            cur.append(c)
        else:
            groups.append(cur)
            cur = [c]
    if cur:
        groups.append(cur)
    return groups


_STREAMS: Dict[object, list] = {}


def _side_streams(device) -> list:
    """Two streams (default priority) for a device's independent calls: a
    zig-zag device's chunk pairs are separate launches of a few hundred
    workgroups each, and running two at once fills the tail of each."""
    import torch
    key = str(device)
    if key not in _STREAMS:
        _STREAMS[key] = [torch.cuda.Stream(device=device) for _ in range(2)]
    return _STREAMS[key]


def forward_chains(steps: Sequence[Tuple[Range, Range, bool]], causal: bool
                   ) -> List[Tuple[Range, List[Range]]]:
    """A device's forward calls as independent chains (query range, key
    ranges in call order): every query range's calls are split in two halves
    of near-equal work (pairs), each half folded into its own partial result,
    so that two streams can run them; the first chain of a range starts with
    its own (diagonal) pair."""
    by_q: Dict[Range, List[Range]] = {}
    for q, k, _ in steps:
        by_q.setdefault(q, []).append(k)
    chains: List[Tuple[Range, List[Range]]] = []
    for q, ks in by_q.items():
        if len(ks) < 2:
            chains.append((q, ks))
            continue
        work = [pair_count(q, k, causal) for k in ks]
        total, run, cut = sum(work), 0, 1
        for i, wk in enumerate(work):
            run += wk
            if run * 2 >= total:
                cut = max(1, min(len(ks) - 1, i + 1))
                break
        chains.append((q, ks[:cut]))
        chains.append((q, ks[cut:]))
    return chains


def ring_forward(q, k, v, p: int, causal: bool = True, scale: Optional[float] = None,
                 layout: str = "contiguous", devices: Optional[Iterable[int]] = None,
                 out=None):
    """O [T, Hq, d] and {query range: LSE [Hq, len]} of the sequence, computed
    range pair by range pair in each device's ring order.  `devices` limits
    the work to those devices' query ranges (the rest of O is left as is).
    A device's calls run as independent chains on two streams (a chain folds
    its pairs into its own partial result with attn_merge; the partials of a
    query range are merged at the end)."""
    import torch
    T, hq = q.shape[0], q.shape[1]
    ranges = device_ranges(T, p, layout)
    o = torch.empty_like(q) if out is None else out
    lses: Dict[Range, object] = {}
    main = torch.cuda.current_stream(q.device)
    side = _side_streams(q.device)
    for r in (range(p) if devices is None else devices):
        chains = forward_chains(device_steps(r, ranges, causal), causal)
        # outputs and partial results live on the caller's stream
        parts = []
        for c, (qr, _) in enumerate(chains):
            n = qr[1] - qr[0]
            if qr not in lses:
                lses[qr] = torch.empty((hq, n), dtype=torch.float32, device=q.device)
                parts.append((o[qr[0]:qr[1]], lses[qr]))
            else:
                parts.append((torch.empty((n,) + tuple(q.shape[1:]), dtype=q.dtype,
                                          device=q.device),
                              torch.empty((hq, n), dtype=torch.float32, device=q.device)))
        # longest chains first, each on the less loaded stream
        load = [0, 0]
        order = sorted(range(len(chains)),
                       key=lambda c: -sum(pair_count(chains[c][0], kr, causal)
                                          for kr in chains[c][1]))
        for st in side:
            st.wait_stream(main)
        for c in order:
            (qa, qb), krs = chains[c]
            si = 0 if load[0] <= load[1] else 1
            load[si] += sum(pair_count((qa, qb), kr, causal) for kr in krs) + 1
            po, pl = parts[c]
            with torch.cuda.stream(side[si]):
                for j, (ka, kb) in enumerate(krs):
                    if j == 0:
                        pdyattn.attn_fwd_chunk(q[qa:qb], k[ka:kb], v[ka:kb], qa, ka, causal,
                                               scale, out=po, lse=pl)
                    else:
                        part = pdyattn.attn_fwd_chunk(q[qa:qb], k[ka:kb], v[ka:kb], qa, ka,
                                                      causal, scale)
                        pdyattn.attn_merge(po, pl, part[0], part[1], out=po, lse=pl)
        for st in side:
            main.wait_stream(st)
        for c, (qr, _) in enumerate(chains):  # fold second halves into the outputs
            po, pl = parts[c]
            if po.data_ptr() != o[qr[0]:qr[1]].data_ptr() or qr[0] == qr[1]:
                if qr[0] < qr[1]:
                    pdyattn.attn_merge(o[qr[0]:qr[1]], lses[qr], po, pl, out=o[qr[0]:qr[1]],
                                       lse=lses[qr])
    return o, lses


def ring_backward(q, k, v, o, lses: Dict[Range, object], dout, p: int, causal: bool = True,
                  scale: Optional[float] = None, layout: str = "contiguous",
                  devices: Optional[Iterable[int]] = None, grads=None):
    """dQ [T, Hq, d], dK and dV [T, Hkv, d] (fp32) accumulated in the kernels
    over the range pairs, ring step by ring step.  With `devices` only those
    devices' calls run; a visiting shard's dK/dV then has to arrive in
    `grads` already holding the earlier devices' sums (zero for a timing).
    Calls that write disjoint rows run two at a time on two streams."""
    import torch
    T, hq, d = q.shape
    hkv = k.shape[1]
    ranges = device_ranges(T, p, layout)
    if grads is None:
        grads = (torch.empty((T, hq, d), dtype=torch.float32, device=q.device),
                 torch.empty((T, hkv, d), dtype=torch.float32, device=q.device),
                 torch.empty((T, hkv, d), dtype=torch.float32, device=q.device))
    dq, dk, dv = grads
    devs = list(range(p) if devices is None else devices)
    steps = {r: device_steps(r, ranges, causal) for r in devs}
    main = torch.cuda.current_stream(q.device)
    side = _side_streams(q.device)
    # step 0 of every device before any later step: each shard's own device
    # overwrites its dK/dV before other devices add to it
    n_own = {r: sum(1 for _, _, acc in steps[r] if not acc) for r in devs}
    for phase in (0, 1):
        for r in devs:
            calls = steps[r][:n_own[r]] if phase == 0 else steps[r][n_own[r]:]
            for group in concurrent_groups(calls):
                for i, ((qa, qb), (ka, kb), accumulate) in enumerate(group):
                    st = side[i]
                    st.wait_stream(main)
                    with torch.cuda.stream(st):
                        pdyattn.attn_bwd_chunk(q[qa:qb], k[ka:kb], v[ka:kb], o[qa:qb],
                                               lses[(qa, qb)], dout[qa:qb], qa, ka, causal, scale,
                                               dq=dq[qa:qb], dk=dk[ka:kb], dv=dv[ka:kb],
                                               accumulate=accumulate)
                for i in range(len(group)):
                    main.wait_stream(side[i])
    return dq, dk, dv


# ---------------------------------------------------------------------------
# Timing of one device's share
# ---------------------------------------------------------------------------
def time_device(inputs: dict, r: int, p: int, layout: str, causal: bool, reps: int,
                warmup: int, o, lses_all, grads) -> Tuple[float, float]:
    """Mean (forward ms, backward ms) of device r's calls over `reps` runs."""
    import torch
    q, k, v, do = inputs["q"], inputs["k"], inputs["v"], inputs["do"]
    fwd, bwd = [], []
    for it in range(warmup + reps):
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record()
        _, lses = ring_forward(q, k, v, p, causal, layout=layout, devices=[r], out=o)
        e1.record()
        lses_all.update(lses)
        ring_backward(q, k, v, o, lses_all, do, p, causal, layout=layout, devices=[r],
                      grads=grads)
        e2.record()
        torch.cuda.synchronize()
        if it >= warmup:
            fwd.append(e0.elapsed_time(e1))
            bwd.append(e1.elapsed_time(e2))
    return sum(fwd) / len(fwd), sum(bwd) / len(bwd)


def measure(tokens: int, p: int, hq: int, hkv: int, d: int, layouts: Sequence[str],
            causal: bool, reps: int, warmup: int, seed: int = 42) -> dict:
    """Per-device times of each layout plus the unsharded kernels' time, all at
    the same sequence.  Dk/dV/dQ buffers are zeroed outside the timed region
    (a visiting shard's partial sums arrive with it)."""
    import torch
    from . import accounting as acc
    from .workloads import device_inputs
    inputs = device_inputs(tokens, hq, hkv, d, seed=seed)
    q = inputs["q"]
    o = torch.empty_like(q)
    grads = (torch.zeros((tokens, hq, d), dtype=torch.float32, device=q.device),
             torch.zeros((tokens, hkv, d), dtype=torch.float32, device=q.device),
             torch.zeros((tokens, hkv, d), dtype=torch.float32, device=q.device))
    rec = {"tokens": tokens, "p": p, "heads_q": hq, "heads_kv": hkv, "head_dim": d,
           "causal": causal, "reps": reps, "warmup": warmup,
           "flops_per_pair": 14.0 * d * hq, "layouts": {}}
    # the unsharded step at the same length, for reference
    cu = torch.tensor([0, tokens], dtype=torch.int32, device=q.device)
    times = []
    for it in range(warmup + reps):
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record()
        out, lse = pdyattn.attn_fwd(q, inputs["k"], inputs["v"], cu, tokens, causal)
        e1.record()
        pdyattn.attn_bwd(q, inputs["k"], inputs["v"], out, lse, inputs["do"], cu, tokens, causal)
        e2.record()
        torch.cuda.synchronize()
        if it >= warmup:
            times.append((e0.elapsed_time(e1), e1.elapsed_time(e2)))
    del out, lse
    f, b = (sum(x) / len(x) for x in zip(*times))
    full_pairs = acc.pairs_per_head([tokens], causal)
    rec["unsharded"] = {"fwd_ms": f, "bwd_ms": b, "pairs_per_head": full_pairs,
                        "tflops": rec["flops_per_pair"] * full_pairs / ((f + b) * 1e9)}
    print(f"unsharded T={tokens}: fwd {f:.2f} ms bwd {b:.2f} ms "
          f"{rec['unsharded']['tflops']:.1f} TFLOP/s", flush=True)
    for layout in layouts:
        ranges = device_ranges(tokens, p, layout)
        devs = []
        lses_all: Dict[Range, object] = {}
        for r in range(p):
            f, b = time_device(inputs, r, p, layout, causal, reps, warmup, o, lses_all, grads)
            pairs = device_pairs(r, ranges, causal)
            n_calls = len(device_steps(r, ranges, causal))
            devs.append({"device": r, "ranges": ranges[r], "calls": n_calls,
                         "pairs_per_head": pairs, "fwd_ms": f, "bwd_ms": b,
                         "tflops": rec["flops_per_pair"] * pairs / ((f + b) * 1e9)})
            print(f"{layout} device {r}: {n_calls} pair calls, fwd {f:.2f} ms bwd {b:.2f} ms "
                  f"{devs[-1]['tflops']:.1f} TFLOP/s", flush=True)
        slowest = max(x["fwd_ms"] + x["bwd_ms"] for x in devs)
        rec["layouts"][layout] = {
            "devices": devs, "step_ms": slowest,
            "imbalance": slowest / (sum(x["fwd_ms"] + x["bwd_ms"] for x in devs) / p),
            "speedup_vs_unsharded": (rec["unsharded"]["fwd_ms"] + rec["unsharded"]["bwd_ms"])
            / slowest}
    return rec


def markdown(rec: dict, command: str) -> str:
    u = rec["unsharded"]
    lines = [f"# Context-parallel ring, one device's share: T={rec['tokens']}, p={rec['p']}, "
             f"Hq={rec['heads_q']}, Hkv={rec['heads_kv']}, d={rec['head_dim']}, "
             f"causal={rec['causal']}, MI355X", "",
             f"Command: `{command}`", "",
             "Each device's forward (chunk calls + merges) and backward (chunk calls with "
             "accumulation) timed with events, mean of "
             f"{rec['reps']} runs after {rec['warmup']} warm-up runs; exchanges are not "
             "modelled (a shard is already resident when its step starts).  TFLOP/s counts "
             "14 d Hq FLOPs per attending (query, key) pair.", "",
             f"Unsharded attn_fwd + attn_bwd at the same length: {u['fwd_ms']:.1f} + "
             f"{u['bwd_ms']:.1f} ms, {u['tflops']:.1f} TFLOP/s.", ""]
    for layout, L in rec["layouts"].items():
        lines += [f"## Layout {layout}: slowest device {L['step_ms']:.1f} ms, imbalance "
                  f"(slowest / mean) {L['imbalance']:.3f}, {L['speedup_vs_unsharded']:.2f}x the "
                  "unsharded step", "",
                  "| device | ranges | pair calls | pairs per head | fwd ms | bwd ms | TFLOP/s |",
                  "|---|---|---|---|---|---|---|"]
        for x in L["devices"]:
            rg = ", ".join(f"[{a}, {b})" for a, b in x["ranges"])
            lines.append(f"| {x['device']} | {rg} | {x['calls']} | {x['pairs_per_head']} | "
                         f"{x['fwd_ms']:.2f} | {x['bwd_ms']:.2f} | {x['tflops']:.1f} |")
        lines.append("")
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser(description="time each device's share of a context-parallel ring")
    ap.add_argument("--tokens", type=int, default=638976)
    ap.add_argument("--p", type=int, default=8)
    ap.add_argument("--heads-q", type=int, default=4)
    ap.add_argument("--heads-kv", type=int, default=4)
    ap.add_argument("--head-dim", type=int, default=128)
    ap.add_argument("--layouts", default="contiguous,zigzag")
    ap.add_argument("--non-causal", action="store_true")
    ap.add_argument("--reps", type=int, default=2)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--md")
    ap.add_argument("--json")
    a = ap.parse_args(argv)
    t0 = time.time()
    rec = measure(a.tokens, a.p, a.heads_q, a.heads_kv, a.head_dim, a.layouts.split(","),
                  not a.non_causal, a.reps, a.warmup)
    cmd = "python -m paper_2511_13198_amd.context_parallel " + " ".join(
        argv if argv is not None else sys.argv[1:])
    md = markdown(rec, cmd)
    if a.md:
        open(a.md, "w").write(md + "\n")
    else:
        print(md)
    if a.json:
        with open(a.json, "w") as fh:
            json.dump(rec, fh, indent=1)
    print(f"done in {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    main()
