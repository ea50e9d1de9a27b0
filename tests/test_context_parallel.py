"""Host-side bookkeeping of the context-parallel ring: layouts, pair counts
and the call order, checked by brute force on small sequences."""
import itertools

import pytest

from paper_2511_13198_amd import accounting as acc
from paper_2511_13198_amd import context_parallel as cp


def brute_pairs(q, k, causal):
    return sum(1 for i in range(*q) for j in range(*k) if (not causal or j <= i))


@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
@pytest.mark.parametrize("T,p", [(10, 3), (2, 4), (64, 8), (37, 5), (0, 2)])
def test_layout_partitions_the_sequence(layout, T, p):
    ranges = cp.device_ranges(T, p, layout)
    assert len(ranges) == p
    covered = sorted(x for rs in ranges for a, b in rs for x in range(a, b))
    assert covered == list(range(T))
    for rs in ranges:
        assert all(a <= b for a, b in rs)
        assert list(rs) == sorted(rs)


def test_chunk_bounds_and_ring_order():
    assert cp.chunk_bounds(10, 3) == [(0, 4), (4, 7), (7, 10)]
    assert cp.chunk_bounds(2, 4) == [(0, 1), (1, 2), (2, 2), (2, 2)]
    assert cp.device_ranges(8, 2, "zigzag") == [[(0, 2), (6, 8)], [(2, 4), (4, 6)]]
    assert cp.ring_order(1, 4) == [1, 0, 3, 2]
    with pytest.raises(ValueError):
        cp.chunk_bounds(5, 0)
    with pytest.raises(ValueError):
        cp.device_ranges(5, 2, "striped")


@pytest.mark.parametrize("causal", [True, False])
def test_pair_count_by_brute_force(causal):
    for qa, qb, ka, kb in itertools.product(range(0, 9, 2), range(0, 10, 3), range(0, 9, 3),
                                            range(0, 10, 2)):
        q, k = (qa, qb), (ka, kb)
        assert cp.pair_count(q, k, causal) == brute_pairs(q, k, causal), (q, k)
        assert cp.visible(q, k, causal) == (brute_pairs(q, k, causal) > 0), (q, k)


@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("T,p", [(50, 4), (3, 5), (97, 3), (16, 1)])
def test_every_visible_pair_is_called_once(layout, causal, T, p):
    """Over all devices, the calls cover each attending (query, key) pair
    exactly once, and the first call on every query range and every key
    range overwrites (accumulate False) while all others add."""
    ranges = cp.device_ranges(T, p, layout)
    seen = {}
    written_q, written_k = set(), set()
    steps = [cp.device_steps(r, ranges, causal) for r in range(p)]
    n_own = [sum(1 for _, _, a in st if not a) for st in steps]
    for st, n in zip(steps, n_own):
        assert all(not a for _, _, a in st[:n]) and all(a for _, _, a in st[n:])
    # every device's step 0 runs before any later step
    order = [st[:n] for st, n in zip(steps, n_own)] + [st[n:] for st, n in zip(steps, n_own)]
    for calls in order:
        for q, k, accumulate in calls:
            if accumulate:
                assert q in written_q or q[0] == q[1]
                assert k in written_k or k[0] == k[1]
            written_q.add(q)
            written_k.add(k)
            for i in range(*q):
                for j in range(*k):
                    if not causal or j <= i:
                        assert (i, j) not in seen
                        seen[(i, j)] = True
    assert len(seen) == acc.pairs_per_head([T], causal) if T else len(seen) == 0


@pytest.mark.parametrize("T,p", [(638976, 8), (131072, 4)])
def test_zigzag_balances_causal_work(T, p):
    """Device shares sum to the whole, and zig-zag brings the busiest device
    to within 1% of the mean where the contiguous layout is ~(2p-1)/p times it."""
    total = acc.pairs_per_head([T], True)
    for layout in ("contiguous", "zigzag"):
        ranges = cp.device_ranges(T, p, layout)
        shares = [cp.device_pairs(r, ranges, True) for r in range(p)]
        assert sum(shares) == total
        ratio = max(shares) / (total / p)
        if layout == "zigzag":
            assert ratio < 1.01
        else:
            assert abs(ratio - (2 * p - 1) / p) < 0.01


@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("T,p", [(50, 4), (3, 5), (638976, 8)])
def test_forward_chains_partition_the_calls(layout, causal, T, p):
    """The forward's chains cover every call of a device exactly once, each
    chain is non-empty, and a range is split into at most two chains."""
    ranges = cp.device_ranges(T, p, layout)
    for r in range(p):
        steps = cp.device_steps(r, ranges, causal)
        chains = cp.forward_chains(steps, causal)
        got = sorted((qr, kr) for qr, krs in chains for kr in krs)
        assert got == sorted((qr, kr) for qr, kr, _ in steps)
        assert all(krs for _, krs in chains)
        per_q = {}
        for qr, _ in chains:
            per_q[qr] = per_q.get(qr, 0) + 1
        assert max(per_q.values()) <= 2


def test_concurrent_groups_keep_buffers_apart():
    calls = [((0, 4), (0, 4), False), ((4, 8), (4, 8), False), ((4, 8), (0, 4), True),
             ((0, 4), (8, 12), True), ((4, 8), (8, 12), True), ((0, 4), (12, 16), True)]
    groups = cp.concurrent_groups(calls)
    assert [c for g in groups for c in g] == calls
    for g in groups:
        assert len(g) <= 2
        if len(g) == 2:
            assert g[0][0] != g[1][0] and g[0][1] != g[1][1]
