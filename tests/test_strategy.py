"""Algorithm 1 (layer-wise strategy selection): pruning, early termination,
the candidate family against brute force on tiny layer counts, the
least-memory fallback, the (b, s) cache and smoothing."""
import itertools

import numpy as np
import pytest

from paper_2511_13198_amd.strategy import Strategy, StrategySelector, prune


def const(name, t, m):
    return Strategy(name, lambda b, s, t=t: t, lambda b, s, m=m: m)


def brute_force(sel, b, s):
    names = [st.name for st in sel.strategies]
    best = None
    for combo in itertools.product(names, repeat=sel.L):
        if sel.fits(combo, b, s):
            t = sel.list_time(combo, b, s)
            if best is None or t < best[0] - 1e-12:
                best = (t, combo)
    return best


def test_prune_drops_dominated_and_sorts_by_time():
    ss = [const("slow_big", 5, 9), const("fast", 1, 8), const("lean", 4, 1), const("mid", 2, 5),
          const("dominated", 3, 6)]
    assert [x.name for x in prune(ss, 1, 1)] == ["fast", "mid", "lean"]


def test_early_termination_when_the_fastest_fits():
    sel = StrategySelector([const("a", 1, 3), const("b", 2, 1)], n_layers=4, memory_limit=12)
    assert sel.select(1, 1) == ("a",) * 4


def test_mixes_when_the_fastest_does_not_fit():
    # a: fast, 3 per layer; b: slower, 1 per layer; budget 8 over 4 layers
    sel = StrategySelector([const("a", 1, 3), const("b", 2, 1)], n_layers=4, memory_limit=8)
    got = sel.select(1, 1)
    assert sel.fits(got, 1, 1)
    assert sorted(got) == ["a", "a", "b", "b"]        # 2*3 + 2*1 = 8, time 6
    assert sel.list_time(got, 1, 1) == brute_force(sel, 1, 1)[0]


def test_fallback_to_the_least_memory_strategy():
    sel = StrategySelector([const("a", 1, 3), const("b", 2, 2)], n_layers=3, memory_limit=1)
    assert sel.select(1, 1) == ("b",) * 3


def family_optimum(sel, b, s):
    """Least time over the lists the selection can consider, built by
    counting: every strategy on every layer, and every split of the layers
    between two neighbours in the pruned time order (layer costs add up, so
    the order of layers inside a list does not matter)."""
    order = [st.name for st in prune(sel.strategies, b, s)]
    cands = [(n,) * sel.L for n in order]
    for j in range(len(order) - 1):
        for a in range(sel.L + 1):
            cands.append((order[j],) * a + (order[j + 1],) * (sel.L - a))
    feas = [c for c in cands if sel.fits(c, b, s)]
    return min(sel.list_time(c, b, s) for c in feas) if feas else None


@pytest.mark.parametrize("seed", range(40))
def test_tradeoff_frontiers_match_the_counted_family(seed):
    """Strategies trading memory for time: the selection returns the best
    list of its candidate family (checked by counting), which is never
    better than the brute-force optimum over all assignments."""
    rng = np.random.default_rng(seed)
    k = int(rng.integers(2, 5))
    mem = np.sort(rng.uniform(1, 10, k))[::-1]            # memory descending
    c = rng.uniform(5, 20)
    strategies = [const(f"s{i}", c / mem[i], mem[i]) for i in range(k)]  # time ascending
    L = int(rng.integers(1, 5))
    limit = rng.uniform(mem[-1] * L, mem[0] * L)
    sel = StrategySelector(strategies, L, limit)
    got = sel.select(1, 1)
    assert sel.fits(got, 1, 1)
    assert sel.list_time(got, 1, 1) == pytest.approx(family_optimum(sel, 1, 1), rel=1e-12)
    assert sel.list_time(got, 1, 1) >= brute_force(sel, 1, 1)[0] - 1e-9


@pytest.mark.parametrize("seed", range(40))
def test_arbitrary_instances_are_feasible_and_never_beat_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    k = int(rng.integers(1, 5))
    strategies = [const(f"s{i}", rng.uniform(1, 10), rng.uniform(1, 10)) for i in range(k)]
    L = int(rng.integers(1, 5))
    fixed = rng.uniform(0, 5)
    limit = rng.uniform(fixed, fixed + 10 * L)
    sel = StrategySelector(strategies, L, limit, fixed_memory=fixed)
    got = sel.select(1, 1)
    assert len(got) == L
    bf = brute_force(sel, 1, 1)
    if bf is None:
        lean = min(strategies, key=lambda s: s.memory(1, 1))
        assert got == (lean.name,) * L
    elif sel.fits(got, 1, 1):
        assert sel.list_time(got, 1, 1) >= bf[0] - 1e-9


def test_cache_answers_repeated_inputs_without_recomputing():
    calls = {"n": 0}

    def t(b, s):
        calls["n"] += 1
        return s * 1.0

    sel = StrategySelector([Strategy("x", t, lambda b, s: 1.0)], n_layers=2, memory_limit=10)
    first = sel.select(2, 100)
    n = calls["n"]
    assert sel.select(2, 100) == first and calls["n"] == n
    sel.select(2, 200)
    assert calls["n"] > n


def test_smoothing_keeps_a_nearly_optimal_previous_choice():
    # at s=1 the fast strategy "a" fits; at s=2 "a" needs more memory and a
    # mix is optimal, but all-"b" is within 5% of it and was chosen before
    a = Strategy("a", lambda b, s: 1.0, lambda b, s: 3.0 * s)
    bb = Strategy("b", lambda b, s: 1.02, lambda b, s: 1.0)
    sel = StrategySelector([a, bb], n_layers=2, memory_limit=7.5, gamma=0.05)
    sel.previous = ("b", "b")
    got = sel.select(1, 2)   # optimum: one layer each (time 2.02); all-b costs 2.04
    assert got == ("b", "b")
    assert sel.optimum(1, 2) != ("b", "b")
    sel0 = StrategySelector([a, bb], n_layers=2, memory_limit=7.5, gamma=0.0)
    sel0.previous = ("b", "b")
    assert sel0.select(1, 2) != ("b", "b")


def test_strategies_from_fitted_cost_models():
    import os

    from paper_2511_13198_amd import cost_model as cm
    from paper_2511_13198_amd import profile_table as pt
    from paper_2511_13198_amd.strategy import from_cost_model
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    rows = pt.read_csv(os.path.join(root, "profiles", "length_profile_h4_d128.csv"))
    model = cm.GroupCostModel.from_rows(rows)
    st = from_cost_model("heads", model)
    assert st.time(2, 131072) == pytest.approx(2 * float(model.time_ms(131072)[0]))
    sel = StrategySelector([st], n_layers=4, memory_limit=288 * 2 ** 30)
    assert sel.select(1, 131072) == ("heads",) * 4
