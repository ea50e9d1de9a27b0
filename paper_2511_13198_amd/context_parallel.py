"""Context-parallel (sequence-sharded) attention: one device's ring steps,
and the whole ring run on one GPU.

With p devices, device r holds chunk r of the sequence (queries, keys and
values of positions chunk_bounds[r]).  Key/value chunks travel around the
ring, so at step t device r holds chunk (r - t) mod p (section 2.2: the
context-parallel strategies exchange K/V between sequence chunks).  Per step
the device calls attn_fwd_chunk and folds the partial result into its
running (O, LSE) with attn_merge.  The backward, given the final O and LSE,
calls attn_bwd_chunk per step, accumulating dQ of its own chunk and the dK/dV
of the visiting chunk, which travel on with it.  Under a causal mask a chunk
after the device's own contributes nothing and is skipped.

ring_forward / ring_backward run all devices' steps one after another on a
single GPU (the exchanges become no-ops): a single-GPU check of the chunked
path against plain attention, and a measure of its throughput.  Every step
runs in the library's kernels; this module only orders the calls.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

from . import pdyattn


def chunk_bounds(total_tokens: int, p: int) -> List[Tuple[int, int]]:
    """p contiguous chunks of near-equal length (the first T mod p one longer)."""
    if p < 1:
        raise ValueError("p must be >= 1")
    base, extra = divmod(total_tokens, p)
    out, a = [], 0
    for r in range(p):
        b = a + base + (1 if r < extra else 0)
        out.append((a, b))
        a = b
    return out


def _visible(qa: int, qb: int, ka: int, kb: int, causal: bool) -> bool:
    """Whether any key of [ka, kb) is visible to a query of [qa, qb)."""
    return qb > qa and kb > ka and (not causal or ka <= qb - 1)


def ring_order(r: int, p: int) -> List[int]:
    """Key/value chunk held by device r at steps 0 .. p-1."""
    return [(r - t) % p for t in range(p)]


def ring_forward(q, k, v, p: int, causal: bool = True, scale: Optional[float] = None):
    """O [T, Hq, d] and the per-chunk LSE list ([Hq, len_r] each) of the
    sequence, computed chunk by chunk in ring order."""
    import torch
    T = q.shape[0]
    bounds = chunk_bounds(T, p)
    o = torch.empty_like(q)
    lses = []
    for r, (qa, qb) in enumerate(bounds):
        acc = None
        for src in ring_order(r, p):
            ka, kb = bounds[src]
            if not _visible(qa, qb, ka, kb, causal):
                continue
            if acc is None:
                acc = pdyattn.attn_fwd_chunk(q[qa:qb], k[ka:kb], v[ka:kb], qa, ka, causal, scale,
                                             out=o[qa:qb])
            else:
                part = pdyattn.attn_fwd_chunk(q[qa:qb], k[ka:kb], v[ka:kb], qa, ka, causal,
                                              scale)
                acc = pdyattn.attn_merge(acc[0], acc[1], part[0], part[1], out=acc[0],
                                         lse=acc[1])
        if acc is None:  # an empty chunk
            acc = pdyattn.attn_fwd_chunk(q[qa:qb], k[qa:qa], v[qa:qa], qa, qa, causal, scale,
                                         out=o[qa:qb])
        lses.append(acc[1])
    return o, lses


def ring_backward(q, k, v, o, lses: Sequence, dout, p: int, causal: bool = True,
                  scale: Optional[float] = None):
    """dQ [T, Hq, d], dK and dV [T, Hkv, d] (fp32) from the chunk pairs in
    ring order, accumulated in the kernels."""
    import torch
    T, hq, d = q.shape
    hkv = k.shape[1]
    bounds = chunk_bounds(T, p)
    dq = torch.empty((T, hq, d), dtype=torch.float32, device=q.device)
    dk = torch.empty((T, hkv, d), dtype=torch.float32, device=q.device)
    dv = torch.empty((T, hkv, d), dtype=torch.float32, device=q.device)
    kv_started = [False] * p
    # every chunk's own (diagonal) pair comes first at step 0, so each dK/dV
    # chunk is written before anything is added to it
    for t in range(p):
        for r, (qa, qb) in enumerate(bounds):
            src = ring_order(r, p)[t]
            ka, kb = bounds[src]
            if t > 0 and not _visible(qa, qb, ka, kb, causal):
                continue
            pdyattn.attn_bwd_chunk(q[qa:qb], k[ka:kb], v[ka:kb], o[qa:qb], lses[r], dout[qa:qb],
                                   qa, ka, causal, scale, dq=dq[qa:qb], dk=dk[ka:kb],
                                   dv=dv[ka:kb], accumulate=(t > 0 or kv_started[src]))
            kv_started[src] = True
    return dq, dk, dv
