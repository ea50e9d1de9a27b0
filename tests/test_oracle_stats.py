"""Pins of the oracle's row-statistics pass (head_rows) and of the key-window
gradient computed from those statistics (key_window_backward), against an
independent library: torch's fp64 scaled_dot_product_attention with autograd
(per segment, key/value heads repeated for grouped heads) and torch's
logsumexp of the explicitly masked logits.  These are the functions the
full-length GPU parity tests use to check every row of a head and the
gradients of the first ("sink") keys of a long sequence.  CPU only."""
import math

import numpy as np
import pytest

from oracle import attention as ora
from paper_2511_13198_amd import workloads as wl


def _case(lengths, hq, hkv, d, seed):
    rng = np.random.default_rng(seed)
    T = sum(lengths)

    def draw(h):
        x = rng.standard_normal((T, h, d)).astype(np.float32)
        return wl.bf16_bits_to_f64(wl.f32_to_bf16_bits(x))
    return draw(hq), draw(hkv), draw(hkv), draw(hq), wl.cu_from_lengths(lengths)


def _torch_reference(q, k, v, do, cu, causal, scale):
    """O, LSE, dQ, dK, dV from torch fp64 (SDPA + autograd; LSE by logsumexp)."""
    import torch
    import torch.nn.functional as F
    Hq, Hkv = q.shape[1], k.shape[1]
    g = Hq // Hkv
    tq = torch.tensor(q, requires_grad=True)
    tk = torch.tensor(k, requires_grad=True)
    tv = torch.tensor(v, requires_grad=True)
    outs, lses = [], []
    for s in range(len(cu) - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        qs = tq[a:b].transpose(0, 1)
        ks = tk[a:b].repeat_interleave(g, dim=1).transpose(0, 1)
        vs = tv[a:b].repeat_interleave(g, dim=1).transpose(0, 1)
        outs.append(F.scaled_dot_product_attention(qs, ks, vs, is_causal=causal,
                                                   scale=scale).transpose(0, 1))
        with torch.no_grad():
            logits = scale * (qs @ ks.transpose(1, 2))
            if causal:
                n = b - a
                mask = torch.ones(n, n, dtype=torch.bool).tril()
                logits = logits.masked_fill(~mask, float("-inf"))
            lses.append(torch.logsumexp(logits, dim=-1))
    o = torch.cat(outs, 0)
    (o * torch.tensor(do)).sum().backward()
    lse = torch.cat(lses, 1)
    return (o.detach().numpy(), lse.numpy(), tq.grad.numpy(), tk.grad.numpy(),
            tv.grad.numpy())


CASES = [
    ([300], 2, 2, 32, True),
    ([40, 17, 171, 1], 4, 2, 16, True),   # packed, grouped heads, a 1-token segment
    ([90, 64], 2, 1, 16, False),          # non-causal
]


@pytest.mark.parametrize("lengths,hq,hkv,d,causal", CASES)
def test_head_rows_match_torch(lengths, hq, hkv, d, causal):
    q, k, v, do, cu = _case(lengths, hq, hkv, d, seed=21)
    scale = 1 / math.sqrt(d)
    to, tl, tdq, _, _ = _torch_reference(q, k, v, do, cu, causal, scale)
    T = sum(lengths)
    for h in range(hq):
        # the whole batch in one call and split at an arbitrary row, with a
        # row block that does not divide the segments
        for lo, hi in ((0, T), (0, 37), (37, T)):
            o, lse, dd, dq = ora.head_rows(q, k, v, do, cu, causal, scale, h, lo, hi,
                                           row_block=23)
            np.testing.assert_allclose(o, to[lo:hi, h], rtol=0, atol=1e-11)
            np.testing.assert_allclose(lse, tl[h, lo:hi], rtol=0, atol=1e-11)
            np.testing.assert_allclose(dd, np.sum(do[lo:hi, h] * to[lo:hi, h], axis=1),
                                       rtol=0, atol=1e-11)
            np.testing.assert_allclose(dq, tdq[lo:hi, h], rtol=0, atol=1e-11)


@pytest.mark.parametrize("lengths,hq,hkv,d,causal", CASES)
def test_key_windows_from_row_stats_match_torch(lengths, hq, hkv, d, causal):
    q, k, v, do, cu = _case(lengths, hq, hkv, d, seed=22)
    scale = 1 / math.sqrt(d)
    _, _, _, tdk, tdv = _torch_reference(q, k, v, do, cu, causal, scale)
    T = sum(lengths)
    lse = np.zeros((hq, T))
    dd = np.zeros((hq, T))
    for h in range(hq):
        _, lse[h], dd[h], _ = ora.head_rows(q, k, v, do, cu, causal, scale, h, 0, T)
    for si in range(len(lengths)):
        a, b = int(cu[si]), int(cu[si + 1])
        if b == a:
            continue
        mid = (a + b) // 2
        # sink keys, a window in the middle, the tail, the whole segment
        for lo, hi in {(a, min(b, a + 8)), (mid, min(b, mid + 5)), (max(a, b - 7), b), (a, b)}:
            for hk in range(hkv):
                dk, dv = ora.key_window_backward(q, k, v, do, lse, dd, cu, causal, scale, hk,
                                                 lo, hi, row_block=19)
                np.testing.assert_allclose(dk, tdk[lo:hi, hk], rtol=0, atol=1e-11)
                np.testing.assert_allclose(dv, tdv[lo:hi, hk], rtol=0, atol=1e-11)


def test_key_window_rows_that_do_not_see_it_are_not_read():
    """Causal: the rows before a window never see it, so their statistics
    may hold anything (here NaN) without changing the window's gradient."""
    q, k, v, do, cu = _case([200], 2, 1, 16, seed=23)
    scale = 0.25
    lse = np.zeros((2, 200))
    dd = np.zeros((2, 200))
    for h in range(2):
        _, lse[h], dd[h], _ = ora.head_rows(q, k, v, do, cu, True, scale, h, 0, 200)
    ref = ora.key_window_backward(q, k, v, do, lse, dd, cu, True, scale, 0, 120, 150)
    lse[:, :120] = np.nan
    dd[:, :120] = np.nan
    got = ora.key_window_backward(q, k, v, do, lse, dd, cu, True, scale, 0, 120, 150)
    np.testing.assert_array_equal(got[0], ref[0])
    np.testing.assert_array_equal(got[1], ref[1])
