"""Layer-wise parallel strategy selection (Algorithm 1, Section 4.4).

Given candidate strategies with per-layer time and memory cost models (for
example the hybrid models of cost_model.py, one per strategy) and a device
memory budget, choose one strategy per layer for an input of batch size b
and sequence length s:

1. drop strategies that another strategy beats in both time and memory, and
   order the rest by per-layer time (then memory);
2. answer repeated (b, s) from a cache;
3. take the fastest strategy for every layer if that fits in memory;
4. otherwise collect memory-feasible candidates: each strategy used for every
   layer, and, for each strategy whose uniform use does not fit, the lists
   obtained by handing the layers one at a time, oldest first, to each later
   strategy in turn;
5. pick the candidate with the least total time, or the least-memory
   strategy on every layer when no candidate fits;
6. smoothing (Section 4.4, Optimizations; gamma = 5%, Section 5.3): keep the
   previously chosen list if it still fits and its time is within gamma of
   the new choice.

A list's time and memory are the sums over layers of the chosen strategies'
per-layer costs, plus a fixed memory term (weights, optimizer state, ...)
that does not depend on the assignment.

Readings: smoothing is described in the text but not in the printed
listing; it is applied to what select() returns while the cache keeps the
unsmoothed optimum, so that cached answers do not depend on history.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence, Tuple

CostFn = Callable[[int, int], float]  # (b, s) -> per-layer cost


@dataclass(frozen=True)
class Strategy:
    name: str
    time: CostFn    # per-layer time cost
    memory: CostFn  # per-layer memory cost


def prune(strategies: Sequence[Strategy], b: int, s: int) -> List[Strategy]:
    """Strategies not dominated in (time, memory), sorted by time then memory."""
    cost = [(st.time(b, s), st.memory(b, s), st) for st in strategies]
    keep = []
    for t, m, st in cost:
        dominated = any((t2 <= t and m2 <= m) and (t2 < t or m2 < m) for t2, m2, _ in cost)
        if not dominated:
            keep.append((t, m, st))
    keep.sort(key=lambda x: (x[0], x[1]))
    return [st for _, _, st in keep]


class StrategySelector:
    def __init__(self, strategies: Sequence[Strategy], n_layers: int, memory_limit: float,
                 fixed_memory: float = 0.0, gamma: float = 0.05):
        if n_layers < 1:
            raise ValueError("n_layers must be >= 1")
        if not strategies:
            raise ValueError("no strategies")
        self.strategies = list(strategies)
        self.L = n_layers
        self.limit = memory_limit
        self.fixed = fixed_memory
        self.gamma = gamma
        self.cache: Dict[Tuple[int, int], Tuple[str, ...]] = {}
        self.previous: Optional[Tuple[str, ...]] = None
        self.by_name = {st.name: st for st in self.strategies}

    # -- costs of a layer-wise list -------------------------------------
    def list_time(self, names: Sequence[str], b: int, s: int) -> float:
        return sum(self.by_name[n].time(b, s) for n in names)

    def list_memory(self, names: Sequence[str], b: int, s: int) -> float:
        return self.fixed + sum(self.by_name[n].memory(b, s) for n in names)

    def fits(self, names: Sequence[str], b: int, s: int) -> bool:
        """Memory check that stops as soon as the running sum exceeds the budget."""
        total = self.fixed
        for n in names:
            total += self.by_name[n].memory(b, s)
            if total > self.limit:
                return False
        return True

    # -- candidate lists ---------------------------------------------------
    def candidates(self, b: int, s: int) -> Tuple[List[Tuple[str, ...]], Optional[Tuple[str, ...]]]:
        """(feasible candidate lists, early choice or None)."""
        order = prune(self.strategies, b, s)
        feasible: List[Tuple[str, ...]] = []
        for i, st in enumerate(order):
            layers = [st.name] * self.L
            ok = self.fits(layers, b, s)
            if i == 0 and ok:
                return feasible, tuple(layers)
            if ok:
                feasible.append(tuple(layers))
                continue
            # hand the layers, oldest first, to each later strategy in turn
            for later in order[i + 1:]:
                for _ in range(self.L):
                    layers.pop(0)
                    layers.append(later.name)
                    if self.fits(layers, b, s):
                        feasible.append(tuple(layers))
        return feasible, None

    def optimum(self, b: int, s: int) -> Tuple[str, ...]:
        key = (b, s)
        if key in self.cache:
            return self.cache[key]
        feasible, early = self.candidates(b, s)
        if early is not None:
            best = early
        elif feasible:
            best = min(feasible, key=lambda c: self.list_time(c, b, s))
        else:
            lean = min(self.strategies, key=lambda st: st.memory(b, s))
            best = tuple([lean.name] * self.L)
        self.cache[key] = best
        return best

    def select(self, b: int, s: int) -> Tuple[str, ...]:
        best = self.optimum(b, s)
        prev = self.previous
        if (prev is not None and prev != best and self.fits(prev, b, s)
                and self.list_time(prev, b, s) <= (1.0 + self.gamma) * self.list_time(best, b, s)):
            best = prev
        self.previous = best
        return best


def from_cost_model(name: str, model) -> Strategy:
    """A strategy whose per-layer costs for b sequences of length s are b
    times the per-sequence predictions of a cost_model.GroupCostModel
    (packed segments are independent)."""
    def t(b: int, s: int) -> float:
        return b * float(model.time_ms(s)[0])

    def m(b: int, s: int) -> float:
        return b * float(model.memory_bytes(s)[0])

    return Strategy(name, t, m)
