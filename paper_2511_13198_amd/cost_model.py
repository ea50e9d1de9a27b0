"""Sequence-aware hybrid cost model (Section 4.3, Eq. 7) on the profile table.

For one configuration group the model predicts the time cost T(s) and the
memory cost M(s) of a step from the sequence length s alone:

* inside the profiled range (s <= the largest profiled length) a random
  forest regressor, the mean over its trees, interpolates;
* beyond it a polynomial of degree 1, 2 or 3 extrapolates; the degree is
  the one with the lowest Akaike information criterion on the profile
  points (Section 4.5: numpy polyfit, degree chosen by AIC);
* OOM risk: a length whose predicted memory exceeds the group's threshold
  (the device memory, or the largest memory the group may use) is flagged.

The forest uses the sizes Section 4.5 gives (50 trees, depth at most 10) and
seed 42, the paper's seed.  The profile rows come from profile_table.py
(single-sequence sweep; s = tokens).

Usage:
  python -m paper_2511_13198_amd.cost_model profiles/length_profile_h4_d128.csv \
      [--holdout 524288] [--predict 786432,1048576]
"""
from __future__ import annotations

import argparse
import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

RF_TREES = 50
RF_MAX_DEPTH = 10
SEED = 42
DEFAULT_OOM_BYTES = 288 * 2 ** 30  # HBM3E of one MI355X


def aic(y: np.ndarray, yhat: np.ndarray, n_params: int) -> float:
    """Akaike information criterion of a least-squares fit with Gaussian
    residuals: n ln(RSS / n) + 2 k."""
    n = len(y)
    rss = float(np.sum((np.asarray(y) - np.asarray(yhat)) ** 2))
    rss = max(rss, 1e-300 * n)  # an exact fit would give -inf
    return n * math.log(rss / n) + 2 * n_params


@dataclass
class PolyFit:
    """Least-squares polynomial in s with the degree (1..3) of lowest AIC."""
    coef: np.ndarray
    degree: int
    aics: Dict[int, float]

    @classmethod
    def fit(cls, s: Sequence[float], y: Sequence[float], degrees=(1, 2, 3)) -> "PolyFit":
        x = np.asarray(s, dtype=np.float64)
        y = np.asarray(y, dtype=np.float64)
        best, aics = None, {}
        for d in degrees:
            if len(x) <= d:  # not enough points to fit (and score) this degree
                continue
            c = np.polyfit(x, y, d)
            aics[d] = aic(y, np.polyval(c, x), d + 1)
            if best is None or aics[d] < aics[best[0]]:
                best = (d, c)
        if best is None:
            raise ValueError("need at least two profile points")
        return cls(coef=best[1], degree=best[0], aics=aics)

    def __call__(self, s) -> np.ndarray:
        return np.polyval(self.coef, np.asarray(s, dtype=np.float64))


@dataclass
class HybridModel:
    """Eq. (7) for one quantity: forest inside the profiled range, polynomial
    beyond it."""
    s_max: float
    forest: object
    poly: PolyFit

    @classmethod
    def fit(cls, s: Sequence[float], y: Sequence[float], seed: int = SEED) -> "HybridModel":
        from sklearn.ensemble import RandomForestRegressor
        x = np.asarray(s, dtype=np.float64).reshape(-1, 1)
        rf = RandomForestRegressor(n_estimators=RF_TREES, max_depth=RF_MAX_DEPTH,
                                   random_state=seed)
        rf.fit(x, np.asarray(y, dtype=np.float64))
        return cls(s_max=float(np.max(x)), forest=rf, poly=PolyFit.fit(s, y))

    def __call__(self, s) -> np.ndarray:
        s = np.atleast_1d(np.asarray(s, dtype=np.float64))
        out = np.empty_like(s)
        inside = s <= self.s_max
        if inside.any():
            out[inside] = self.forest.predict(s[inside].reshape(-1, 1))
        if (~inside).any():
            out[~inside] = self.poly(s[~inside])
        return out

    def regime(self, s: float) -> str:
        return "RF" if s <= self.s_max else f"PR{self.poly.degree}"


@dataclass
class GroupCostModel:
    """Time and memory models of one configuration group, with its OOM
    threshold."""
    group: str
    time_ms: HybridModel
    memory_bytes: HybridModel
    oom_bytes: float = DEFAULT_OOM_BYTES
    meta: dict = field(default_factory=dict)

    @classmethod
    def from_rows(cls, rows: List[dict], oom_bytes: float = DEFAULT_OOM_BYTES,
                  time_col: str = "fwdbwd_ms", mem_col: str = "step_peak_bytes",
                  max_s: Optional[int] = None) -> "GroupCostModel":
        rows = [r for r in rows if r.get("kind", "single") == "single"]
        if max_s is not None:
            rows = [r for r in rows if int(r["tokens"]) <= max_s]
        if not rows:
            raise ValueError("no single-sequence profile rows")
        groups = {r["group"] for r in rows}
        if len(groups) != 1:
            raise ValueError(f"rows of several configuration groups: {sorted(groups)}")
        s = [int(r["tokens"]) for r in rows]
        t = [float(r[time_col]) for r in rows]
        m = [float(r[mem_col]) for r in rows]
        return cls(group=groups.pop(), time_ms=HybridModel.fit(s, t),
                   memory_bytes=HybridModel.fit(s, m), oom_bytes=oom_bytes,
                   meta={"profiled_lengths": s})

    def predict(self, s) -> dict:
        t = self.time_ms(s)
        m = self.memory_bytes(s)
        return {"time_ms": t, "memory_bytes": m, "oom": m > self.oom_bytes}


def main(argv=None):
    from .profile_table import read_csv
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("csv")
    ap.add_argument("--holdout", type=int, default=0,
                    help="fit on lengths below this and report the error on the rest")
    ap.add_argument("--predict", type=str, default="", help="comma-separated lengths")
    ap.add_argument("--oom-gib", type=float, default=288.0)
    a = ap.parse_args(argv)
    rows = read_csv(a.csv)
    oom = a.oom_gib * 2 ** 30
    model = GroupCostModel.from_rows(rows, oom, max_s=(a.holdout - 1) if a.holdout else None)
    print(f"group {model.group}: fitted on {len(model.meta['profiled_lengths'])} lengths "
          f"<= {int(model.time_ms.s_max)}; time PR degree {model.time_ms.poly.degree}, "
          f"memory PR degree {model.memory_bytes.poly.degree}")
    if a.holdout:
        for r in rows:
            s = int(r["tokens"])
            if r.get("kind", "single") != "single" or s < a.holdout:
                continue
            p = model.predict(s)
            t, mem = float(p["time_ms"][0]), float(p["memory_bytes"][0])
            print(f"  s={s}: time {t:.1f} ms vs measured {float(r['fwdbwd_ms']):.1f} "
                  f"({100 * (t / float(r['fwdbwd_ms']) - 1):+.1f}%), memory "
                  f"{mem / 2**30:.3f} GiB vs {int(r['step_peak_bytes']) / 2**30:.3f} GiB "
                  f"({100 * (mem / int(r['step_peak_bytes']) - 1):+.2f}%) [{model.time_ms.regime(s)}]")
    for s in [int(x) for x in a.predict.split(",") if x]:
        p = model.predict(s)
        print(f"  s={s}: time {float(p['time_ms'][0]):.1f} ms, memory "
              f"{float(p['memory_bytes'][0]) / 2**30:.3f} GiB, OOM {bool(p['oom'][0])} "
              f"[{model.time_ms.regime(s)}]")


if __name__ == "__main__":
    main()
