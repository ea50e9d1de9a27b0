"""HIP path vs the fp64 oracle on every element of the full-size workloads
where the oracle can afford it, through the C-ABI:

* the packed 65,536-token batch (log-uniform lengths in [128, 8192], 32
  heads, d = 128): O, LSE, dQ, dK and dV, every element of every head;
* the 131,072-token sequence (4 heads, d = 128): O, LSE and dQ for every row
  of query head 0, and dK, dV of its kv head for the first 2,048 ("sink")
  keys, 2,048 keys in the middle and the last 2,048 keys, from the oracle's
  own row statistics (LSE and D of every row).

The oracle's pieces (heads, row ranges, key windows) run side by side on the
host's cores; each piece is the plain definition.  Tolerance per tensor, over
all compared elements: max |err| <= 2e-2 and relative L2 <= 5e-3; the margins
to both are printed."""
import math
import time

import numpy as np
import pytest

from oracle import attention as ora
from paper_2511_13198_amd import workloads as wl
from tests import parity_util as pu

pytestmark = pytest.mark.gpu


@pytest.mark.timeout(900)
def test_packed_65536_every_element():
    import torch
    w = wl.config(2)
    T, hq, hkv, d = w.total_tokens, w.heads_q, w.heads_kv, w.head_dim
    scale = w.softmax_scale
    pu.log(f"  workload {w.name}: T={T} N={w.num_seqs} Hq={hq} Hkv={hkv} d={d}")
    bits = wl.host_inputs(T, hq, hkv, d)
    dev = {n: pu.to_device_bf16(b) for n, b in bits.items()}
    cu = w.cu_seqlens()
    cu_d = torch.from_numpy(cu).cuda()
    o, lse, dq, dk, dv = pu.run_gpu(dev["q"], dev["k"], dev["v"], dev["do"], cu_d,
                                    w.max_seqlen, w.causal, scale)
    got = {"O": o.cpu().double().numpy(), "LSE": lse.cpu().double().numpy(),
           "dQ": dq.cpu().numpy(), "dK": dk.cpu().numpy(), "dV": dv.cpu().numpy()}
    del o, lse, dq, dk, dv, dev
    assert hq == hkv, "one query head per kv head: each head is its own oracle piece"

    def one_head(h):
        f = {n: wl.bf16_bits_to_f64(b[:, h:h + 1]) for n, b in bits.items()}
        return ora.backward(f["q"], f["k"], f["v"], f["do"], cu, w.causal, scale)

    t0 = time.perf_counter()
    refs = pu.run_pieces(one_head, list(range(hq)))
    pu.log(f"  oracle: {hq} heads in {time.perf_counter() - t0:.1f} s on "
           f"{pu.host_workers()} threads")
    acc = {n: pu.ErrAcc(n) for n in ("O", "LSE", "dQ", "dK", "dV")}
    for h, (ro, rl, rdq, rdk, rdv) in enumerate(refs):
        acc["O"].add(got["O"][:, h], ro[:, 0])
        acc["LSE"].add(got["LSE"][h], rl[0])
        acc["dQ"].add(got["dQ"][:, h], rdq[:, 0])
        acc["dK"].add(got["dK"][:, h], rdk[:, 0])
        acc["dV"].add(got["dV"][:, h], rdv[:, 0])
    for a in acc.values():
        a.check()


SINK_WINDOW = 2048


@pytest.mark.timeout(900)
def test_single_131072_every_row_of_a_head_and_sink_keys():
    import torch
    w = wl.config(3)
    T, hq, hkv, d = w.total_tokens, w.heads_q, w.heads_kv, w.head_dim
    scale = w.softmax_scale
    h, hk = 0, 0
    g = hq // hkv
    pu.log(f"  workload {w.name}: query head {h}, kv head {hk}")
    dev = wl.device_inputs(T, hq, hkv, d)
    cu = w.cu_seqlens()
    cu_d = torch.from_numpy(cu).cuda()
    o, lse, dq, dk, dv = pu.run_gpu(dev["q"], dev["k"], dev["v"], dev["do"], cu_d,
                                    w.max_seqlen, w.causal, scale)
    # the kv head's whole group of query heads, widened exactly to fp64
    qs = dev["q"][:, hk * g:(hk + 1) * g].contiguous().cpu().double().numpy()
    dos = dev["do"][:, hk * g:(hk + 1) * g].contiguous().cpu().double().numpy()
    ks = dev["k"][:, hk:hk + 1].contiguous().cpu().double().numpy()
    vs = dev["v"][:, hk:hk + 1].contiguous().cpu().double().numpy()
    got_o = o[:, h].cpu().double().numpy()
    got_l = lse[h].cpu().double().numpy()
    got_q = dq[:, h].cpu().numpy()
    got_k = dk[:, hk].cpu().numpy()
    got_v = dv[:, hk].cpu().numpy()
    del o, lse, dq, dk, dv, dev

    # every row of the group's query heads: O, LSE, D, dQ (row ranges side by side)
    step = 2048
    pieces = [(hh, r0, min(T, r0 + step)) for hh in range(g) for r0 in range(0, T, step)]
    t0 = time.perf_counter()
    rows = pu.run_pieces(lambda p: ora.head_rows(qs, ks, vs, dos, cu, w.causal, scale, p[0],
                                                 p[1], p[2]), pieces)
    pu.log(f"  oracle rows: {len(pieces)} pieces in {time.perf_counter() - t0:.1f} s")
    lse_all = np.zeros((g, T))
    dd_all = np.zeros((g, T))
    acc = {n: pu.ErrAcc(n) for n in ("O", "LSE", "dQ")}
    for (hh, r0, r1), (ro, rl, rd, rq) in zip(pieces, rows):
        lse_all[hh, r0:r1] = rl
        dd_all[hh, r0:r1] = rd
        if hh == h - hk * g:
            acc["O"].add(got_o[r0:r1], ro)
            acc["LSE"].add(got_l[r0:r1], rl)
            acc["dQ"].add(got_q[r0:r1], rq)
    for a in acc.values():
        a.check()

    # dK, dV of the kv head on three key windows, from the row statistics
    windows = [(0, SINK_WINDOW), (T // 2 - SINK_WINDOW // 2, T // 2 + SINK_WINDOW // 2),
               (T - SINK_WINDOW, T)]
    sub = 256
    kpieces = [(c, c + sub) for lo, hi in windows for c in range(lo, hi, sub)]
    t0 = time.perf_counter()
    cols = pu.run_pieces(lambda p: ora.key_window_backward(qs, ks, vs, dos, lse_all, dd_all, cu,
                                                           w.causal, scale, 0, p[0], p[1]),
                         kpieces)
    pu.log(f"  oracle key windows: {len(kpieces)} pieces in {time.perf_counter() - t0:.1f} s")
    for (lo, hi) in windows:
        acc = {n: pu.ErrAcc(f"{n}") for n in ("dK", "dV")}
        for (c0, c1), (rk, rv) in zip(kpieces, cols):
            if lo <= c0 < hi:
                acc["dK"].add(got_k[c0:c1], rk)
                acc["dV"].add(got_v[c0:c1], rv)
        pu.log(f"   keys [{lo}, {hi}): |dK| up to {float(np.max(np.abs(got_k[lo:hi]))):.3g}")
        for a in acc.values():
            a.check()
