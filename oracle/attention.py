"""fp64 CPU oracle for packed variable-length softmax attention and its gradient.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import or call this
module: only the tests, the smoke check and the benchmark's CPU-baseline leg
use it.  It shares no code with the HIP library.

What it computes is the plain definition of scaled dot-product attention,
Eq. (2) of the problem formulation (section 3):  A = Softmax(Q K^T / sqrt(d)) V,
applied per head to every packed segment, plus the exact calculus gradient of
that expression.  The paper leaves several points open; the readings taken
here are:
  * d is the head dimension h/n (Table 1 has no d; Table 4 gives h and n), and
    the softmax scale is passed in explicitly (1/sqrt(d) by default).
  * causal: key j is visible to query i iff j <= i, both inside the same
    segment; non-causal: every key of the segment is visible.
  * segments never attend to each other (packed batch = block-diagonal mask);
    the paper's b x s layout is the special case of equal lengths.
  * grouped heads (more query heads than key/value heads) use contiguous
    groups: query head h reads key/value head h // (Hq / Hkv); dK and dV sum
    over the group.
  * LSE is the natural-log log-sum-exp of the scaled logits of each row,
    laid out [Hq, T].  No dropout, no bias, no gradient flows into LSE.

Everything is float64.  Inputs are expected as float64 arrays holding the
bf16 values exactly (bf16 -> fp64 widening is exact), so any difference to a
device result is the device's own rounding.

Rows are processed in blocks of `row_block` query rows: each block is the
full definition for those rows (all visible keys at once, two-pass softmax),
so blocking changes nothing but memory use.
"""
from __future__ import annotations

from typing import Iterable, List, Sequence, Tuple

import numpy as np


def segments(cu_seqlens: Sequence[int]) -> List[Tuple[int, int]]:
    cu = [int(x) for x in cu_seqlens]
    return [(cu[i], cu[i + 1]) for i in range(len(cu) - 1)]


def _visible_keys(a: int, b: int, r0: int, r1: int, causal: bool) -> int:
    """Number of keys (from segment start a) any row in [r0, r1) may see."""
    return (r1 - a) if causal else (b - a)


def _logits(qr: np.ndarray, kk: np.ndarray, a: int, r0: int, causal: bool,
            scale: float) -> np.ndarray:
    """S[i, j] = scale * <q_i, k_j>, with -inf where key j is not visible.
    qr: [R, d] rows r0..r0+R-1; kk: [n, d] keys a..a+n-1."""
    s = scale * (qr @ kk.T)
    if causal:
        rows = np.arange(r0, r0 + qr.shape[0])[:, None]
        cols = np.arange(a, a + kk.shape[0])[None, :]
        s = np.where(cols <= rows, s, -np.inf)
    return s


def _softmax_stats(s: np.ndarray):
    """Two-pass log-sum-exp per row; returns (lse, P)."""
    m = np.max(s, axis=1)
    lse = m + np.log(np.sum(np.exp(s - m[:, None]), axis=1))
    p = np.exp(s - lse[:, None])
    return lse, p


def forward(q, k, v, cu_seqlens, causal: bool, scale: float, row_block: int = 256):
    """O [T, Hq, d] and LSE [Hq, T] (natural log) per Eq. (2)."""
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    g = Hq // Hkv
    o = np.zeros((T, Hq, v.shape[2]), dtype=np.float64)
    lse = np.zeros((Hq, T), dtype=np.float64)
    for a, b in segments(cu_seqlens):
        for h in range(Hq):
            hk = h // g
            for r0 in range(a, b, row_block):
                r1 = min(b, r0 + row_block)
                n = _visible_keys(a, b, r0, r1, causal)
                kk = k[a:a + n, hk]
                vv = v[a:a + n, hk]
                s = _logits(q[r0:r1, h], kk, a, r0, causal, scale)
                l, p = _softmax_stats(s)
                lse[h, r0:r1] = l
                o[r0:r1, h] = p @ vv
    return o, lse


def backward(q, k, v, do, cu_seqlens, causal: bool, scale: float, row_block: int = 256):
    """Gradient of L = sum(dO * O) with O from Eq. (2).

    Returns (O, LSE, dQ, dK, dV), all float64.  With P = softmax(S) and
    S = scale * Q K^T:
        dV = P^T dO
        dP = dO V^T
        dS = P * (dP - D),  D_i = <dO_i, O_i>   (softmax Jacobian)
        dQ = scale * dS K,  dK = scale * dS^T Q
    dK and dV of a key/value head sum the contributions of its query heads.
    """
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    g = Hq // Hkv
    o, lse = forward(q, k, v, cu_seqlens, causal, scale, row_block)
    dq = np.zeros_like(q, dtype=np.float64)
    dk = np.zeros_like(k, dtype=np.float64)
    dv = np.zeros_like(v, dtype=np.float64)
    for a, b in segments(cu_seqlens):
        for h in range(Hq):
            hk = h // g
            for r0 in range(a, b, row_block):
                r1 = min(b, r0 + row_block)
                n = _visible_keys(a, b, r0, r1, causal)
                kk = k[a:a + n, hk]
                vv = v[a:a + n, hk]
                s = _logits(q[r0:r1, h], kk, a, r0, causal, scale)
                p = np.exp(s - lse[h, r0:r1, None])
                dor = do[r0:r1, h]
                D = np.sum(dor * o[r0:r1, h], axis=1)
                dp = dor @ vv.T
                ds = p * (dp - D[:, None])
                dq[r0:r1, h] = scale * (ds @ kk)
                dk[a:a + n, hk] += scale * (ds.T @ q[r0:r1, h])
                dv[a:a + n, hk] += p.T @ dor
    return o, lse, dq, dk, dv


# ---------------------------------------------------------------------------
# Sampled mode: exact values for chosen rows / key columns at any size.
# Every function below evaluates the same definition as forward()/backward()
# for a subset of outputs; row results only need that row's visible keys,
# column results need the statistics (LSE, D) of every row that sees the key.
# ---------------------------------------------------------------------------
def _segment_of(cu: np.ndarray, idx: np.ndarray) -> np.ndarray:
    return np.searchsorted(cu, idx, side="right") - 1


def rows_forward_backward(q, k, v, do, cu_seqlens, causal: bool, scale: float,
                          heads: Iterable[int], rows: Sequence[int]):
    """For each query head in `heads` and each token index in `rows`:
    O_i [len(rows), d], LSE_i, dQ_i.  Inputs are [T, H, d] arrays, or objects
    with `num_heads` and a `head(h)` method returning the [T, d] float64 slice
    of head h (so large inputs can be widened one head at a time).

    Returns dict head -> (o, lse, dq) with arrays over `rows` (sorted order of
    the given list is preserved)."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    rows = np.asarray(rows, dtype=np.int64)
    seg = _segment_of(cu, rows)
    Hq = _nheads(q)
    Hkv = _nheads(k)
    g = Hq // Hkv
    out = {}
    for h in heads:
        hk = h // g
        qh, kh, vh, doh = _head(q, h), _head(k, hk), _head(v, hk), _head(do, h)
        o = np.zeros((len(rows), vh.shape[1]))
        lse = np.zeros(len(rows))
        dq = np.zeros((len(rows), qh.shape[1]))
        for si in np.unique(seg):
            a, b = int(cu[si]), int(cu[si + 1])
            sel = np.nonzero(seg == si)[0]
            r = rows[sel]
            n = (int(r.max()) + 1 - a) if causal else (b - a)
            kk, vv = kh[a:a + n], vh[a:a + n]
            s = scale * (qh[r] @ kk.T)
            if causal:
                s = np.where(np.arange(a, a + n)[None, :] <= r[:, None], s, -np.inf)
            l, p = _softmax_stats(s)
            orow = p @ vv
            D = np.sum(doh[r] * orow, axis=1)
            ds = p * (doh[r] @ vv.T - D[:, None])
            o[sel], lse[sel], dq[sel] = orow, l, scale * (ds @ kk)
        out[h] = (o, lse, dq)
    return out


def cols_backward(q, k, v, do, cu_seqlens, causal: bool, scale: float,
                  kv_heads: Iterable[int], seg_index: int, col_lo: int,
                  row_block: int = 512):
    """dK_j, dV_j for key columns j in [col_lo, b) of segment `seg_index`
    (b = segment end), summed over the query heads of each key/value head.
    Every row that sees one of these keys contributes; with causal masking
    these are rows i >= col_lo only, so a tail window is cheap at any length.
    Returns dict kv_head -> (dk [b-col_lo, d], dv [b-col_lo, d])."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    a, b = int(cu[seg_index]), int(cu[seg_index + 1])
    Hq, Hkv = _nheads(q), _nheads(k)
    g = Hq // Hkv
    out = {}
    for hk in kv_heads:
        kh, vh = _head(k, hk), _head(v, hk)
        dk = np.zeros((b - col_lo, kh.shape[1]))
        dv = np.zeros((b - col_lo, vh.shape[1]))
        r_start = col_lo if causal else a
        for h in range(hk * g, (hk + 1) * g):
            qh, doh = _head(q, h), _head(do, h)
            for r0 in range(r_start, b, row_block):
                r1 = min(b, r0 + row_block)
                n = (r1 - a) if causal else (b - a)
                kk, vv = kh[a:a + n], vh[a:a + n]
                s = _logits(qh[r0:r1], kk, a, r0, causal, scale)
                l, p = _softmax_stats(s)
                orow = p @ vv
                dor = doh[r0:r1]
                D = np.sum(dor * orow, axis=1)
                ds = p * (dor @ vv.T - D[:, None])
                c0 = col_lo - a
                dk[: n - c0] += scale * (ds[:, c0:n].T @ qh[r0:r1])
                dv[: n - c0] += p[:, c0:n].T @ dor
        out[hk] = (dk, dv)
    return out


def head_rows(q, k, v, do, cu_seqlens, causal: bool, scale: float, h: int, r_lo: int,
              r_hi: int, row_block: int = 256):
    """O_i, LSE_i, D_i = <dO_i, O_i> and dQ_i of query head h for every row
    r_lo <= i < r_hi (any range; rows take the keys of their own segment).
    Each block of rows is the full definition over all the keys it sees, as
    in backward(), so a range covering a whole segment is that segment's
    complete forward plus the dQ part of its gradient.  Inputs as for
    rows_forward_backward.  Returns (o [n, d], lse [n], dd [n], dq [n, d])."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    Hq, Hkv = _nheads(q), _nheads(k)
    hk = h // (Hq // Hkv)
    qh, kh, vh, doh = _head(q, h), _head(k, hk), _head(v, hk), _head(do, h)
    n = r_hi - r_lo
    o = np.zeros((n, vh.shape[1]))
    lse = np.zeros(n)
    dd = np.zeros(n)
    dq = np.zeros((n, qh.shape[1]))
    for si in range(len(cu) - 1):
        a, b = int(cu[si]), int(cu[si + 1])
        for r0 in range(max(a, r_lo), min(b, r_hi), row_block):
            r1 = min(b, r_hi, r0 + row_block)
            nk = _visible_keys(a, b, r0, r1, causal)
            kk, vv = kh[a:a + nk], vh[a:a + nk]
            s = _logits(qh[r0:r1], kk, a, r0, causal, scale)
            l, p = _softmax_stats(s)
            orow = p @ vv
            dor = doh[r0:r1]
            D = np.sum(dor * orow, axis=1)
            ds = p * (dor @ vv.T - D[:, None])
            sl = slice(r0 - r_lo, r1 - r_lo)
            o[sl], lse[sl], dd[sl], dq[sl] = orow, l, D, scale * (ds @ kk)
    return o, lse, dd, dq


def key_window_backward(q, k, v, do, lse, dd, cu_seqlens, causal: bool, scale: float,
                        kv_head: int, c_lo: int, c_hi: int, row_block: int = 512):
    """dK_j and dV_j of key/value head `kv_head` for the keys c_lo <= j < c_hi
    of one segment, summed over the query heads of its group, from the row
    statistics LSE [Hq, T] (natural log) and D [Hq, T] of the rows that see
    them (e.g. from head_rows over those rows; other entries are not read).
    With P_ij = exp(S_ij - LSE_i) and dS_ij = P_ij (<dO_i, V_j> - D_i):
    dK_j = scale sum_i dS_ij Q_i, dV_j = sum_i P_ij dO_i over the rows i that
    see key j (i >= j within the segment when causal, every row otherwise).
    Returns (dk [c_hi - c_lo, d], dv [c_hi - c_lo, d])."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    si = int(_segment_of(cu, np.array([c_lo]))[0])
    a, b = int(cu[si]), int(cu[si + 1])
    assert a <= c_lo < c_hi <= b, "the key window must lie inside one segment"
    Hq, Hkv = _nheads(q), _nheads(k)
    g = Hq // Hkv
    kw = _head(k, kv_head)[c_lo:c_hi]
    vw = _head(v, kv_head)[c_lo:c_hi]
    dk = np.zeros_like(kw)
    dv = np.zeros_like(vw)
    cols = np.arange(c_lo, c_hi)[None, :]
    for h in range(kv_head * g, (kv_head + 1) * g):
        qh, doh = _head(q, h), _head(do, h)
        for r0 in range(c_lo if causal else a, b, row_block):
            r1 = min(b, r0 + row_block)
            s = scale * (qh[r0:r1] @ kw.T)
            if causal:
                s = np.where(cols <= np.arange(r0, r1)[:, None], s, -np.inf)
            p = np.exp(s - lse[h, r0:r1, None])
            dor = doh[r0:r1]
            ds = p * (dor @ vw.T - dd[h, r0:r1, None])
            dk += scale * (ds.T @ qh[r0:r1])
            dv += p.T @ dor
    return dk, dv


def _nheads(x) -> int:
    if hasattr(x, "num_heads"):
        return x.num_heads
    return x.shape[1]


def _head(x, h):
    """[T, d] float64 view of head h; `x` is an array [T, H, d] or an object
    with a `head(h)` method returning that slice."""
    if hasattr(x, "head"):
        return x.head(h)
    return np.asarray(x[:, h], dtype=np.float64)


# ---------------------------------------------------------------------------
# Chunked (context-parallel) attention of one long sequence.
#
# Sequence sharding (the context-parallel strategies of section 2.2) gives a
# device the queries at absolute positions q_offset .. q_offset+Tq-1 and,
# one chunk at a time, the keys/values at k_offset .. k_offset+Tk-1.  Eq. (2)
# restricted to one key chunk yields a partial output and its log-sum-exp;
# the full result is their log-sum-exp weighted combination.  Readings: the
# causal rule compares absolute positions (key visible iff its position <=
# the query's); a row that sees no key of a chunk gets O = 0 and LSE = -inf
# (the neutral element of the combination).
# ---------------------------------------------------------------------------
def _chunk_logits(qh, kh, q_offset: int, k_offset: int, causal: bool, scale: float):
    s = scale * (qh @ kh.T)
    if causal:
        qpos = q_offset + np.arange(qh.shape[0])[:, None]
        kpos = k_offset + np.arange(kh.shape[0])[None, :]
        s = np.where(kpos <= qpos, s, -np.inf)
    return s


def partial_forward(q, k, v, q_offset: int, k_offset: int, causal: bool, scale: float):
    """O_c [Tq, Hq, d] and LSE_c [Hq, Tq] of a query chunk over one key/value
    chunk of the same sequence."""
    Tq, Hq, _ = q.shape
    Hkv = k.shape[1]
    g = Hq // Hkv
    o = np.zeros((Tq, Hq, v.shape[2]))
    lse = np.full((Hq, Tq), -np.inf)
    for h in range(Hq):
        hk = h // g
        s = _chunk_logits(q[:, h], k[:, hk], q_offset, k_offset, causal, scale)
        seen = np.isfinite(s).any(axis=1)
        if not seen.any():
            continue
        l, p = _softmax_stats(s[seen])
        lse[h, seen] = l
        o[seen, h] = p @ v[:, hk]
    return o, lse


def merge(parts):
    """Combine partial (O_c, LSE_c) pairs of the same query rows:
    LSE = log sum_c exp(LSE_c),  O = sum_c exp(LSE_c - LSE) O_c."""
    lses = np.stack([l for _, l in parts])           # [C, Hq, Tq]
    top = np.max(lses, axis=0)
    safe = np.where(np.isfinite(top), top, 0.0)
    w = np.exp(lses - safe[None])                    # exp(-inf) = 0
    tot = np.sum(w, axis=0)
    lse = np.where(tot > 0, safe + np.log(np.where(tot > 0, tot, 1.0)), -np.inf)
    o = np.zeros_like(parts[0][0])
    for (oc, _), wc in zip(parts, w):
        coef = np.where(tot > 0, wc / np.where(tot > 0, tot, 1.0), 0.0)  # [Hq, Tq]
        o += oc * coef.T[:, :, None]
    return o, lse


def partial_backward(q, k, v, o, lse, do, q_offset: int, k_offset: int, causal: bool,
                     scale: float):
    """Contribution of one (query chunk, key chunk) pair to the gradient of
    L = sum(dO * O), given the final O and LSE of the query rows (over all
    key chunks).  Returns (dQ_c [Tq, Hq, d], dK_c, dV_c [Tk, Hkv, d]); dQ of the
    query chunk is the sum over key chunks, dK/dV of a key chunk the sum over
    query chunks."""
    Tq, Hq, _ = q.shape
    Hkv = k.shape[1]
    g = Hq // Hkv
    dq = np.zeros_like(q, dtype=np.float64)
    dk = np.zeros_like(k, dtype=np.float64)
    dv = np.zeros_like(v, dtype=np.float64)
    for h in range(Hq):
        hk = h // g
        s = _chunk_logits(q[:, h], k[:, hk], q_offset, k_offset, causal, scale)
        l = lse[h][:, None]
        p = np.where(np.isfinite(l), np.exp(s - np.where(np.isfinite(l), l, 0.0)), 0.0)
        D = np.sum(do[:, h] * o[:, h], axis=1)
        ds = p * (do[:, h] @ v[:, hk].T - D[:, None])
        dq[:, h] = scale * (ds @ k[:, hk])
        dk[:, hk] += scale * (ds.T @ q[:, h])
        dv[:, hk] += p.T @ do[:, h]
    return dq, dk, dv
