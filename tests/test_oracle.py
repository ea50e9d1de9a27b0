"""Pins for the fp64 oracle: every check here compares it with something
other than itself -- a brute-force evaluation, a closed form, finite
differences, an independent library routine, or an invariant the mathematics
of Eq. (2) (section 3) fixes.  CPU only."""
import math

import numpy as np
import pytest

from oracle import attention as ora
from paper_2511_13198_amd import workloads as wl


def _case(lengths, hq, hkv, d, seed, bf16=True):
    rng = np.random.default_rng(seed)
    T = sum(lengths)
    def draw(h):
        x = rng.standard_normal((T, h, d)).astype(np.float32)
        return wl.bf16_bits_to_f64(wl.f32_to_bf16_bits(x)) if bf16 else x.astype(np.float64)
    q, k, v, do = draw(hq), draw(hkv), draw(hkv), draw(hq)
    return q, k, v, do, wl.cu_from_lengths(lengths)


# ---------------------------------------------------------------------------
# 1. brute force: explicit loops, no max shift, no blocking
# ---------------------------------------------------------------------------
def _brute_forward(q, k, v, cu, causal, scale):
    T, Hq, d = q.shape
    g = Hq // k.shape[1]
    o = np.zeros_like(q)
    lse = np.zeros((Hq, T))
    for s in range(len(cu) - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        for h in range(Hq):
            for i in range(a, b):
                js = range(a, i + 1) if causal else range(a, b)
                w = {j: math.exp(scale * sum(q[i, h, t] * k[j, h // g, t] for t in range(d)))
                     for j in js}
                z = sum(w.values())
                lse[h, i] = math.log(z)
                for t in range(d):
                    o[i, h, t] = sum(w[j] / z * v[j, h // g, t] for j in js)
    return o, lse


@pytest.mark.parametrize("lengths,hq,hkv,d,causal", [
    ([7], 1, 1, 4, True),
    ([5, 1, 9], 2, 1, 8, True),
    ([6, 3], 2, 2, 4, False),
    ([16], 4, 2, 8, True),
])
def test_forward_matches_brute_force(lengths, hq, hkv, d, causal):
    q, k, v, _, cu = _case(lengths, hq, hkv, d, seed=1)
    scale = 1 / math.sqrt(d)
    o, lse = ora.forward(q, k, v, cu, causal, scale, row_block=3)
    ob, lb = _brute_forward(q, k, v, cu, causal, scale)
    np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lb, rtol=0, atol=1e-12)


def test_rows_sum_to_one_v_ones():
    q, k, _, _, cu = _case([33, 64, 5], 4, 2, 16, seed=2)
    v = np.ones_like(k)
    for causal in (True, False):
        o, _ = ora.forward(q, k, v, cu, causal, 0.3, row_block=16)
        np.testing.assert_allclose(o, 1.0, rtol=0, atol=1e-14)


# ---------------------------------------------------------------------------
# 2. an independent library routine: torch's fp64 SDPA + autograd, per segment
# ---------------------------------------------------------------------------
def _torch_sdpa_grads(q, k, v, do, cu, causal, scale):
    import torch
    import torch.nn.functional as F
    Hq, Hkv = q.shape[1], k.shape[1]
    g = Hq // Hkv
    tq = torch.tensor(q, requires_grad=True)
    tk = torch.tensor(k, requires_grad=True)
    tv = torch.tensor(v, requires_grad=True)
    outs = []
    for s in range(len(cu) - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        qs = tq[a:b].transpose(0, 1)
        ks = tk[a:b].repeat_interleave(g, dim=1).transpose(0, 1)
        vs = tv[a:b].repeat_interleave(g, dim=1).transpose(0, 1)
        outs.append(F.scaled_dot_product_attention(qs, ks, vs, is_causal=causal,
                                                   scale=scale).transpose(0, 1))
    o = torch.cat(outs, 0)
    (o * torch.tensor(do)).sum().backward()
    return (o.detach().numpy(), tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy())


@pytest.mark.parametrize("lengths,hq,hkv,d,causal", [
    ([40, 17, 71], 4, 4, 32, True),
    ([40, 17, 71], 4, 2, 32, True),
    ([64, 3], 8, 2, 16, False),
    ([1, 130], 2, 1, 64, True),
])
def test_matches_torch_fp64_sdpa_and_autograd(lengths, hq, hkv, d, causal):
    q, k, v, do, cu = _case(lengths, hq, hkv, d, seed=3)
    scale = 1 / math.sqrt(d)
    o, lse, dq, dk, dv = ora.backward(q, k, v, do, cu, causal, scale, row_block=32)
    to, tdq, tdk, tdv = _torch_sdpa_grads(q, k, v, do, cu, causal, scale)
    np.testing.assert_allclose(o, to, rtol=0, atol=1e-10)
    np.testing.assert_allclose(dq, tdq, rtol=0, atol=1e-10)
    np.testing.assert_allclose(dk, tdk, rtol=0, atol=1e-10)
    np.testing.assert_allclose(dv, tdv, rtol=0, atol=1e-10)


# ---------------------------------------------------------------------------
# 3. closed forms
# ---------------------------------------------------------------------------
def test_single_token_segment():
    q, k, v, do, cu = _case([1, 1, 1], 2, 1, 8, seed=4)
    o, lse, dq, dk, dv = ora.backward(q, k, v, do, cu, True, 0.7)
    for h in range(2):
        np.testing.assert_array_equal(o[:, h], v[:, 0])
        np.testing.assert_allclose(lse[h], 0.7 * np.sum(q[:, h] * k[:, 0], axis=1), atol=1e-14)
    np.testing.assert_allclose(dq, 0, atol=1e-15)
    np.testing.assert_allclose(dk, 0, atol=1e-15)
    np.testing.assert_allclose(dv[:, 0], do[:, 0] + do[:, 1], atol=1e-15)


def test_zero_queries_give_prefix_means():
    _, k, v, _, cu = _case([37, 12], 2, 2, 8, seed=5)
    q = np.zeros((49, 2, 8))
    o, lse = ora.forward(q, k, v, cu, True, 0.5, row_block=8)
    for s in range(2):
        a, b = int(cu[s]), int(cu[s + 1])
        for i in range(a, b):
            np.testing.assert_allclose(o[i], v[a:i + 1].mean(axis=0), atol=1e-14)
            np.testing.assert_allclose(lse[:, i], math.log(i - a + 1), atol=1e-14)


def test_identical_keys_uniform_weights():
    q, k, v, _, cu = _case([20], 1, 1, 8, seed=6)
    k[:] = k[0:1]
    o, _ = ora.forward(q, k, v, cu, False, 1.0)
    np.testing.assert_allclose(o[:, 0], np.broadcast_to(v[:, 0].mean(0), (20, 8)), atol=1e-13)


def test_constant_values_zero_qk_grads():
    q, k, _, do, cu = _case([30, 9], 4, 2, 16, seed=7)
    v = np.broadcast_to(np.arange(16.0) - 3.0, k.shape).copy()
    o, _, dq, dk, dv = ora.backward(q, k, v, do, cu, True, 0.25, row_block=8)
    np.testing.assert_allclose(o, v[:, [0, 0, 1, 1]], atol=1e-13)
    np.testing.assert_allclose(dq, 0, atol=1e-12)
    np.testing.assert_allclose(dk, 0, atol=1e-12)


def test_dominant_key():
    q, k, v, _, cu = _case([10], 1, 1, 4, seed=8)
    q[:] = 1.0
    k[:] = 0.0
    k[3] = 100.0  # logit 400 * scale dominates every row that sees key 3
    o, _ = ora.forward(q, k, v, cu, True, 1.0)
    for i in range(3, 10):
        np.testing.assert_allclose(o[i, 0], v[3, 0], atol=1e-12)


# ---------------------------------------------------------------------------
# 4. finite differences of L = sum(dO * O)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("causal", [True, False])
def test_gradient_finite_differences(causal):
    q, k, v, do, cu = _case([5, 3], 2, 1, 4, seed=9, bf16=False)
    scale = 0.6
    _, _, dq, dk, dv = ora.backward(q, k, v, do, cu, causal, scale, row_block=2)

    def loss(q_, k_, v_):
        o, _ = ora.forward(q_, k_, v_, cu, causal, scale, row_block=2)
        return float(np.sum(do * o))

    h = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        for idx in np.ndindex(*x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            args_p = {"q": q, "k": k, "v": v}
            args_m = dict(args_p)
            args_p[name], args_m[name] = xp, xm
            num[idx] = (loss(args_p["q"], args_p["k"], args_p["v"])
                        - loss(args_m["q"], args_m["k"], args_m["v"])) / (2 * h)
        np.testing.assert_allclose(g, num, rtol=1e-6, atol=1e-8, err_msg=name)


# ---------------------------------------------------------------------------
# 5. causality and segment isolation (exact)
# ---------------------------------------------------------------------------
def test_causality_exact():
    q, k, v, do, cu = _case([50], 2, 2, 8, seed=10)
    o, lse, dq, dk, dv = ora.backward(q, k, v, do, cu, True, 0.35, row_block=16)
    i = 23
    q2, k2, v2, do2 = q.copy(), k.copy(), v.copy(), do.copy()
    q2[i + 1:] += 1.5
    k2[i + 1:] -= 2.0
    v2[i + 1:] *= 3.0
    o2, lse2, dq2, _, _ = ora.backward(q2, k2, v2, do, cu, True, 0.35, row_block=16)
    np.testing.assert_array_equal(o2[:i + 1], o[:i + 1])
    np.testing.assert_array_equal(lse2[:, :i + 1], lse[:, :i + 1])
    np.testing.assert_array_equal(dq2[:i + 1], dq[:i + 1])
    # upstream gradient of earlier rows does not reach later keys
    j = 30
    do2[:j] += 5.0
    _, _, _, dk3, dv3 = ora.backward(q, k, v, do2, cu, True, 0.35, row_block=16)
    np.testing.assert_array_equal(dk3[j:], dk[j:])
    np.testing.assert_array_equal(dv3[j:], dv[j:])


def test_segment_isolation_exact():
    lengths = [19, 40, 7]
    q, k, v, do, cu = _case(lengths, 2, 1, 8, seed=11)
    packed = ora.backward(q, k, v, do, cu, True, 0.4, row_block=8)
    for s in range(3):
        a, b = int(cu[s]), int(cu[s + 1])
        alone = ora.backward(q[a:b], k[a:b], v[a:b], do[a:b], [0, b - a], True, 0.4, row_block=8)
        np.testing.assert_array_equal(alone[0], packed[0][a:b])
        np.testing.assert_array_equal(alone[1], packed[1][:, a:b])
        for t in (2, 3, 4):
            np.testing.assert_array_equal(alone[t], packed[t][a:b])


# ---------------------------------------------------------------------------
# 6. grouped heads == repeated key/value heads
# ---------------------------------------------------------------------------
def test_gqa_equals_repeated_mha():
    q, k, v, do, cu = _case([33, 20], 8, 2, 16, seed=12)
    g = 4
    ga = ora.backward(q, k, v, do, cu, True, 0.25, row_block=16)
    kr, vr = np.repeat(k, g, axis=1), np.repeat(v, g, axis=1)
    ma = ora.backward(q, kr, vr, do, cu, True, 0.25, row_block=16)
    np.testing.assert_allclose(ga[0], ma[0], atol=1e-14)
    np.testing.assert_allclose(ga[2], ma[2], atol=1e-13)
    for t in (3, 4):
        summed = ma[t].reshape(ma[t].shape[0], 2, g, -1).sum(axis=2)
        np.testing.assert_allclose(ga[t], summed, atol=1e-12)


# ---------------------------------------------------------------------------
# 7. global invariants
# ---------------------------------------------------------------------------
def test_global_invariants():
    q, k, v, do, cu = _case([70, 129, 1, 31], 4, 2, 16, seed=13)
    scale = 0.25
    o, lse, dq, dk, dv = ora.backward(q, k, v, do, cu, True, scale, row_block=32)
    g = 2
    for s in range(4):
        a, b = int(cu[s]), int(cu[s + 1])
        for hk in range(2):
            hs = list(range(hk * g, hk * g + g))
            # softmax shift invariance: rows of dS sum to zero
            np.testing.assert_allclose(dk[a:b, hk].sum(0), 0, atol=1e-11)
            # rows of P sum to one
            np.testing.assert_allclose(dv[a:b, hk].sum(0), do[a:b, hs].sum((0, 1)), atol=1e-11)
            # O is linear in V
            np.testing.assert_allclose(np.sum(v[a:b, hk] * dv[a:b, hk]),
                                       np.sum(do[a:b, hs] * o[a:b, hs]), rtol=1e-12, atol=1e-10)
            # S is bilinear in Q and K
            np.testing.assert_allclose(np.sum(q[a:b, hs] * dq[a:b, hs]),
                                       np.sum(k[a:b, hk] * dk[a:b, hk]), rtol=1e-12, atol=1e-10)
        for h in range(4):
            for i in range(a, b):
                vis = v[a:i + 1, h // g]
                assert np.all(o[i, h] >= vis.min(0) - 1e-13)
                assert np.all(o[i, h] <= vis.max(0) + 1e-13)
                smax = np.max(scale * k[a:i + 1, h // g] @ q[i, h])
                assert smax - 1e-13 <= lse[h, i] <= smax + math.log(i - a + 1) + 1e-13


# ---------------------------------------------------------------------------
# 8. sampled mode agrees with the full oracle
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("causal", [True, False])
def test_sampled_rows_and_cols_match_full(causal):
    lengths = [90, 200, 13]
    q, k, v, do, cu = _case(lengths, 4, 2, 16, seed=14)
    full = ora.backward(q, k, v, do, cu, causal, 0.25, row_block=64)
    rows = [0, 1, 89, 90, 91, 150, 289, 290, 302]
    res = ora.rows_forward_backward(q, k, v, do, cu, causal, 0.25, heads=[0, 3], rows=rows)
    for h, (o, lse, dq) in res.items():
        np.testing.assert_allclose(o, full[0][rows, h], atol=1e-13)
        np.testing.assert_allclose(lse, full[1][h, rows], atol=1e-13)
        np.testing.assert_allclose(dq, full[2][rows, h], atol=1e-12)
    cols = ora.cols_backward(q, k, v, do, cu, causal, 0.25, kv_heads=[0, 1], seg_index=1,
                             col_lo=230, row_block=37)
    for hk, (dk, dv) in cols.items():
        np.testing.assert_allclose(dk, full[3][230:290, hk], atol=1e-12)
        np.testing.assert_allclose(dv, full[4][230:290, hk], atol=1e-12)
