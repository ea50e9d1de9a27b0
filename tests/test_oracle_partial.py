"""Pins of the chunked (context-parallel) oracle functions: chunks combined
with merge() reproduce the full-sequence oracle (itself pinned by brute
force, closed forms, finite differences and a library reference), the
chunk-pair gradients sum to the full gradient, and the neutral element of
the combination behaves as such."""
import numpy as np
import pytest

from oracle import attention as ora


def _inputs(T, Hq, Hkv, d, seed):
    rng = np.random.default_rng(seed)
    f = lambda h: rng.standard_normal((T, h, d))
    return f(Hq), f(Hkv), f(Hkv), f(Hq)


CASES = [
    (50, 2, 1, 8, [0, 13, 30, 50], True),
    (64, 4, 2, 16, [0, 32, 64], True),
    (37, 2, 2, 8, [0, 1, 20, 36, 37], True),
    (40, 2, 1, 8, [0, 17, 40], False),
]


@pytest.mark.parametrize("T,Hq,Hkv,d,cuts,causal", CASES)
def test_chunks_merge_to_the_full_forward(T, Hq, Hkv, d, cuts, causal):
    q, k, v, _ = _inputs(T, Hq, Hkv, d, 1)
    O, L = ora.forward(q, k, v, np.array([0, T]), causal, 0.3)
    spans = list(zip(cuts[:-1], cuts[1:]))
    for qa, qb in spans:
        parts = [ora.partial_forward(q[qa:qb], k[ka:kb], v[ka:kb], qa, ka, causal, 0.3)
                 for ka, kb in spans]
        o, lse = ora.merge(parts)
        assert np.allclose(o, O[qa:qb], atol=1e-12)
        assert np.allclose(lse, L[:, qa:qb], atol=1e-12)
        # merging in another order gives the same result
        o2, l2 = ora.merge(parts[::-1])
        assert np.allclose(o2, o, atol=1e-13) and np.allclose(l2, lse, atol=1e-13)


@pytest.mark.parametrize("T,Hq,Hkv,d,cuts,causal", CASES)
def test_chunk_pair_gradients_sum_to_the_full_gradient(T, Hq, Hkv, d, cuts, causal):
    q, k, v, do = _inputs(T, Hq, Hkv, d, 2)
    O, L, dQ, dK, dV = ora.backward(q, k, v, do, np.array([0, T]), causal, 0.3)
    spans = list(zip(cuts[:-1], cuts[1:]))
    dq = np.zeros_like(dQ)
    dk = np.zeros_like(dK)
    dv = np.zeros_like(dV)
    for qa, qb in spans:
        for ka, kb in spans:
            gq, gk, gv = ora.partial_backward(q[qa:qb], k[ka:kb], v[ka:kb], O[qa:qb],
                                              L[:, qa:qb], do[qa:qb], qa, ka, causal, 0.3)
            dq[qa:qb] += gq
            dk[ka:kb] += gk
            dv[ka:kb] += gv
    assert np.allclose(dq, dQ, atol=1e-11)
    assert np.allclose(dk, dK, atol=1e-11)
    assert np.allclose(dv, dV, atol=1e-11)


def test_rows_that_see_nothing_are_neutral():
    q, k, v, _ = _inputs(10, 1, 1, 4, 3)
    # keys at positions 20..29, queries at 0..9: nothing visible (causal)
    o, lse = ora.partial_forward(q, k, v, 0, 20, True, 1.0)
    assert np.all(o == 0) and np.all(np.isneginf(lse))
    # partially visible: queries 0..9 at positions 5..14, keys at 10..19
    o, lse = ora.partial_forward(q, k, v, 5, 10, True, 1.0)
    assert np.all(np.isneginf(lse[:, :5])) and np.all(np.isfinite(lse[:, 5:]))
    # merging with a neutral part changes nothing
    full = ora.partial_forward(q, k, v, 10, 0, True, 1.0)
    m = ora.merge([full, (np.zeros_like(full[0]), np.full_like(full[1], -np.inf))])
    assert np.array_equal(m[0], full[0]) and np.array_equal(m[1], full[1])
    # the first visible key of a row is the only one: O = its value row
    o, lse = ora.partial_forward(q, k, v, 10, 10, True, 0.5)
    assert np.allclose(o[0, 0], v[0, 0]) and np.isclose(lse[0, 0], 0.5 * q[0, 0] @ k[0, 0])


def test_brute_force_partial_on_a_tiny_chunk():
    q, k, v, _ = _inputs(3, 1, 1, 2, 4)
    o, lse = ora.partial_forward(q, k, v, 7, 6, True, 1.0)
    for i in range(3):
        w = [np.exp(q[i, 0] @ k[j, 0]) if 6 + j <= 7 + i else 0.0 for j in range(3)]
        z = sum(w)
        assert np.isclose(lse[0, i], np.log(z))
        assert np.allclose(o[i, 0], sum(wj * v[j, 0] for j, wj in enumerate(w)) / z)
