"""Helpers shared by the GPU parity tests (HIP path vs the fp64 oracle)."""
from __future__ import annotations

import math
import sys
from typing import Dict, List, Optional, Sequence

import numpy as np

from paper_2511_13198_amd import workloads as wl

# tolerance for bf16 inputs with fp32 accumulation, applied per tensor
MAX_ABS = 2e-2
REL_L2 = 5e-3


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def check_close(name: str, got, ref, max_abs: float = MAX_ABS, rel_l2: float = REL_L2):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{name}: shape {got.shape} vs {ref.shape}"
    assert np.all(np.isfinite(got)), f"{name}: non-finite values in device output"
    diff = got - ref
    mx = float(np.max(np.abs(diff))) if diff.size else 0.0
    nref = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(diff)) / nref if nref > 0 else float(np.linalg.norm(diff))
    log(f"    {name:5s} max|err| {mx:.3e}  relL2 {rel:.3e}  (n={diff.size})")
    assert mx <= max_abs, f"{name}: max abs error {mx:.3e} > {max_abs}"
    assert rel <= rel_l2, f"{name}: relative L2 error {rel:.3e} > {rel_l2}"
    return mx, rel


class HeadView:
    """[T, H, d] bf16 tensor (host or device) handed to the oracle one head at
    a time, widened exactly to float64 on the host."""

    def __init__(self, t_bf16):
        self.t = t_bf16
        self.num_heads = int(t_bf16.shape[1])
        self._cache = {}

    def head(self, h: int) -> np.ndarray:
        if h not in self._cache:
            if len(self._cache) >= 2:
                self._cache.pop(next(iter(self._cache)))
            self._cache[h] = self.t[:, h].contiguous().cpu().double().numpy()
        return self._cache[h]


def to_device_bf16(bits: np.ndarray, device="cuda"):
    import torch
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(device)


def bf16_to_f64(t_bf16) -> np.ndarray:
    return t_bf16.detach().cpu().double().numpy()


def run_gpu(q, k, v, do, cu, max_seqlen, causal, scale, poison=True):
    """Forward + backward through the C-ABI; outputs poisoned with NaN first so
    an element the kernels never write is caught."""
    import torch
    from paper_2511_13198_amd import pdyattn
    T, hq, d = q.shape
    hkv = k.shape[1]
    o = torch.empty_like(q)
    lse = torch.empty((hq, T), dtype=torch.float32, device=q.device)
    dq = torch.empty((T, hq, d), dtype=torch.float32, device=q.device)
    dk = torch.empty((T, hkv, d), dtype=torch.float32, device=q.device)
    dv = torch.empty((T, hkv, d), dtype=torch.float32, device=q.device)
    if poison:
        for t in (o, lse, dq, dk, dv):
            t.fill_(float("nan"))
    pdyattn.attn_fwd(q, k, v, cu, max_seqlen, causal, scale, out=o, lse=lse)
    pdyattn.attn_bwd(q, k, v, o, lse, do, cu, max_seqlen, causal, scale, dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


def sample_rows(lengths: Sequence[int], per_seg_random: int, seed: int = 0,
                max_rows: Optional[int] = None) -> List[int]:
    """Stratified query rows: segment edges, tile edges near start/middle/end,
    and seeded random rows."""
    rng = np.random.default_rng(seed)
    rows = set()
    a = 0
    for s in lengths:
        if s == 0:
            continue
        b = a + s
        picks = [0, 1, 2, 3, s - 4, s - 3, s - 2, s - 1]
        for edge in (64, 128, 256):
            for c in (edge, s // 2 - s // 2 % edge, s - s % edge):
                picks += [c - 1, c, c + 1]
        picks += list(rng.integers(0, s, size=per_seg_random))
        rows.update(a + int(p) for p in picks if 0 <= p < s)
        a = b
    out = sorted(rows)
    if max_rows is not None and len(out) > max_rows:
        keep = rng.choice(len(out), size=max_rows, replace=False)
        out = sorted(out[i] for i in keep)
    return out


def gpu_invariants(o, lse, dq, dk, dv, q, k, v, do, cu_list, scale, causal=True):
    """Identities of the exact gradient, checked over every element in fp64 on
    the device (O(T d) work): per segment and key/value head,
      sum_j dK_j = 0,  sum_j dV_j = sum_i dO_i (over the group),
      sum_j <V_j, dV_j> = sum_i <dO_i, O_i>,  sum_i <Q_i, dQ_i> = sum_j <K_j, dK_j>.
    Residuals are relative to the norms of the summed terms."""
    import torch
    hq, hkv = q.shape[1], k.shape[1]
    g = hq // hkv
    worst = {}
    for si in range(len(cu_list) - 1):
        a, b = cu_list[si], cu_list[si + 1]
        if b - a < 2:
            continue
        for hk in range(hkv):
            hs = slice(hk * g, hk * g + g)
            dks = dk[a:b, hk].double()
            dvs = dv[a:b, hk].double()
            r1 = (dks.sum(0).norm() / (dks.norm() + 1e-30)).item()
            dos = do[a:b, hs].double()
            r2 = ((dvs.sum(0) - dos.sum((0, 1))).norm() / (dvs.norm() + 1e-30)).item()
            lhs = (v[a:b, hk].double() * dvs).sum()
            rhs = (dos * o[a:b, hs].double()).sum()
            r3 = (abs(lhs - rhs) / ((v[a:b, hk].double().norm() * dvs.norm()) + 1e-30)).item()
            lq = (q[a:b, hs].double() * dq[a:b, hs].double()).sum()
            rk = (k[a:b, hk].double() * dks).sum()
            r4 = (abs(lq - rk) / ((k[a:b, hk].double().norm() * dks.norm()) + 1e-30)).item()
            for name, r in (("sum_dK", r1), ("sum_dV", r2), ("V.dV", r3), ("Q.dQ", r4)):
                worst[name] = max(worst.get(name, 0.0), r)
    log("    invariants (relative residuals): " +
        ", ".join(f"{k_}={v_:.2e}" for k_, v_ in worst.items()))
    for name, r in worst.items():
        assert r < 5e-3, f"invariant {name} residual {r:.3e}"
    return worst


class ErrAcc:
    """Running max |err|, ||err||^2 and ||ref||^2 of one tensor compared in
    pieces (per head, per row range), checked against the same per-tensor
    tolerance as check_close once every piece is in."""

    def __init__(self, name: str):
        self.name = name
        self.max_abs = 0.0
        self.sq_err = 0.0
        self.sq_ref = 0.0
        self.n = 0

    def add(self, got, ref):
        got = np.asarray(got, dtype=np.float64)
        ref = np.asarray(ref, dtype=np.float64)
        assert got.shape == ref.shape, f"{self.name}: shape {got.shape} vs {ref.shape}"
        assert np.all(np.isfinite(got)), f"{self.name}: non-finite values in device output"
        diff = got - ref
        if diff.size:
            self.max_abs = max(self.max_abs, float(np.max(np.abs(diff))))
        self.sq_err += float(np.sum(diff * diff))
        self.sq_ref += float(np.sum(ref * ref))
        self.n += diff.size

    def check(self, max_abs: float = MAX_ABS, rel_l2: float = REL_L2):
        rel = math.sqrt(self.sq_err / self.sq_ref) if self.sq_ref > 0 else math.sqrt(self.sq_err)
        log(f"    {self.name:5s} max|err| {self.max_abs:.3e}  relL2 {rel:.3e}  (n={self.n})"
            f"  margins {max_abs / max(self.max_abs, 1e-30):.1f}x / {rel_l2 / max(rel, 1e-30):.1f}x")
        assert self.max_abs <= max_abs, f"{self.name}: max abs error {self.max_abs:.3e} > {max_abs}"
        assert rel <= rel_l2, f"{self.name}: relative L2 error {rel:.3e} > {rel_l2}"
        return self.max_abs, rel


def host_workers() -> int:
    """Threads for running independent oracle pieces side by side (the
    oracle's elementwise numpy work is single-threaded per call): the
    process's CPUs, at most 16."""
    import os
    return max(1, min(16, len(os.sched_getaffinity(0))))


def run_pieces(fn, pieces):
    """fn(piece) for every piece on host_workers() threads, each call with a
    single-threaded BLAS (numpy releases the GIL inside its array work).
    Returns the results in the order of `pieces`."""
    from concurrent.futures import ThreadPoolExecutor

    from threadpoolctl import threadpool_limits
    with threadpool_limits(1):
        with ThreadPoolExecutor(max_workers=host_workers()) as ex:
            return list(ex.map(fn, pieces))


def head_rows_and_key_windows(dev, outs, cu, causal, scale, h, windows, step=2048, sub=256):
    """Every row of query head h (O, LSE, dQ) and dK, dV of its kv head on the
    key windows [(lo, hi), ...] of a single segment cu = [0, T], against the
    oracle's row statistics pass (head_rows) and key-window gradients
    (key_window_backward), both run in pieces side by side on the host.
    dev: device bf16 inputs q, k, v, do; outs: device outputs (o, lse, dq, dk,
    dv)."""
    import time

    from oracle import attention as ora
    o, lse, dq, dk, dv = outs
    T, hq = dev["q"].shape[0], dev["q"].shape[1]
    hkv = dev["k"].shape[1]
    g = hq // hkv
    hk = h // g
    qs = dev["q"][:, hk * g:(hk + 1) * g].contiguous().cpu().double().numpy()
    dos = dev["do"][:, hk * g:(hk + 1) * g].contiguous().cpu().double().numpy()
    ks = dev["k"][:, hk:hk + 1].contiguous().cpu().double().numpy()
    vs = dev["v"][:, hk:hk + 1].contiguous().cpu().double().numpy()
    got_o = o[:, h].double().cpu().numpy()
    got_l = lse[h].double().cpu().numpy()
    got_q = dq[:, h].double().cpu().numpy()
    got_k = dk[:, hk].double().cpu().numpy()
    got_v = dv[:, hk].double().cpu().numpy()
    pieces = [(hh, r0, min(T, r0 + step)) for hh in range(g) for r0 in range(0, T, step)]
    t0 = time.perf_counter()
    rows = run_pieces(lambda p: ora.head_rows(qs, ks, vs, dos, cu, causal, scale, p[0], p[1],
                                              p[2]), pieces)
    log(f"  oracle rows of {g} head(s): {len(pieces)} pieces in {time.perf_counter() - t0:.1f} s")
    lse_all = np.zeros((g, T))
    dd_all = np.zeros((g, T))
    acc = {n: ErrAcc(n) for n in ("O", "LSE", "dQ")}
    for (hh, r0, r1), (ro, rl, rd, rq) in zip(pieces, rows):
        lse_all[hh, r0:r1] = rl
        dd_all[hh, r0:r1] = rd
        if hh == h - hk * g:
            acc["O"].add(got_o[r0:r1], ro)
            acc["LSE"].add(got_l[r0:r1], rl)
            acc["dQ"].add(got_q[r0:r1], rq)
    for a in acc.values():
        a.check()
    kpieces = [(c, min(hi, c + sub)) for lo, hi in windows for c in range(lo, hi, sub)]
    t0 = time.perf_counter()
    cols = run_pieces(lambda p: ora.key_window_backward(qs, ks, vs, dos, lse_all, dd_all, cu,
                                                        causal, scale, 0, p[0], p[1]), kpieces)
    log(f"  oracle key windows: {len(kpieces)} pieces in {time.perf_counter() - t0:.1f} s")
    for lo, hi in windows:
        acc = {n: ErrAcc(n) for n in ("dK", "dV")}
        for (c0, c1), (rk, rv) in zip(kpieces, cols):
            if lo <= c0 < hi:
                acc["dK"].add(got_k[c0:c1], rk)
                acc["dV"].add(got_v[c0:c1], rv)
        log(f"   keys [{lo}, {hi}) of kv head {hk}: |dK| up to "
            f"{float(np.max(np.abs(got_k[lo:hi]))):.3g}")
        for a in acc.values():
            a.check()
