"""The hybrid cost model of Eq. (7): polynomial extrapolation with AIC
degree choice, forest interpolation inside the profiled range, the switch
between them, OOM flags, and its accuracy on the measured profile table."""
import math
import os

import numpy as np
import pytest

from paper_2511_13198_amd import cost_model as cm
from paper_2511_13198_amd import profile_table as pt

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_aic_by_hand():
    y = np.array([1.0, 2.0, 4.0])
    yhat = np.array([1.5, 2.0, 3.0])  # RSS = 0.25 + 0 + 1 = 1.25
    assert cm.aic(y, yhat, 2) == pytest.approx(3 * math.log(1.25 / 3) + 4)


def test_polyfit_recovers_planted_cubic():
    s = np.linspace(1.0, 40.0, 15)
    true = np.array([0.002, -0.3, 5.0, 7.0])   # 0.002 s^3 - 0.3 s^2 + 5 s + 7
    f = cm.PolyFit.fit(s, np.polyval(true, s))
    assert f.degree == 3
    assert np.allclose(f.coef, true, rtol=1e-6, atol=1e-8)
    # extrapolation of an exact cubic stays exact
    assert f(100.0) == pytest.approx(np.polyval(true, 100.0), rel=1e-6)


def test_aic_prefers_the_simple_model_for_noisy_linear_data():
    rng = np.random.default_rng(42)
    s = np.linspace(64, 65536, 20)
    y = 3.0 * s + 100.0 + rng.normal(0, 50.0, s.size)
    f = cm.PolyFit.fit(s, y)
    assert f.degree == 1
    assert f.coef[0] == pytest.approx(3.0, rel=1e-3)


def test_polyfit_needs_points():
    with pytest.raises(ValueError):
        cm.PolyFit.fit([1.0], [2.0])
    # two points: only the linear fit is possible
    assert cm.PolyFit.fit([1.0, 2.0], [2.0, 4.0]).degree == 1


def test_hybrid_switches_at_the_largest_profiled_length():
    s = np.array([2.0 ** e for e in range(6, 20)])
    y = 1e-8 * s ** 2 + 1e-3 * s                      # quadratic cost curve
    h = cm.HybridModel.fit(s, y)
    assert h.s_max == s.max()
    assert h.regime(s.max()) == "RF" and h.regime(s.max() + 1).startswith("PR")
    # forest inside the range: a prediction lies between the neighbouring
    # profiled values (a mean over trees of training targets)
    mid = np.sqrt(s[:-1] * s[1:])
    pm = h(mid)
    assert np.all(pm >= y[:-1] * 0.999) and np.all(pm <= y[1:] * 1.001)
    # polynomial beyond the range: the quadratic extrapolates exactly
    big = np.array([1.5e6, 4e6])
    assert np.allclose(h(big), 1e-8 * big ** 2 + 1e-3 * big, rtol=1e-6)
    assert h.poly.degree in (2, 3)


def test_oom_flag_and_group_rows():
    rows = []
    for e in range(6, 16):
        s = 2 ** e
        rows.append({"group": "g", "kind": "single", "tokens": s, "fwdbwd_ms": 1e-6 * s * s,
                     "step_peak_bytes": 1000 * s})
    m = cm.GroupCostModel.from_rows(rows, oom_bytes=1000 * 40000)
    p = m.predict([1024, 30000, 50000])
    assert list(p["oom"]) == [False, False, True]
    with pytest.raises(ValueError):
        cm.GroupCostModel.from_rows(rows + [dict(rows[0], group="other")])


def test_measured_table_extrapolates_within_a_few_percent():
    """Fit on lengths < 500,000 of the committed MI355X sweep and predict the
    two longest measured lengths (524,288 and 638,976)."""
    rows = pt.read_csv(os.path.join(ROOT, "profiles", "length_profile_h4_d128.csv"))
    m = cm.GroupCostModel.from_rows(rows, max_s=499_999)
    for r in rows:
        s = int(r["tokens"])
        if s < 500_000:
            continue
        p = m.predict(s)
        assert float(p["time_ms"][0]) == pytest.approx(float(r["fwdbwd_ms"]), rel=0.05)
        assert float(p["memory_bytes"][0]) == pytest.approx(int(r["step_peak_bytes"]), rel=0.02)
        assert not p["oom"][0]


def test_forest_interpolates_a_densely_profiled_curve():
    s = np.linspace(1000, 100000, 200)
    y = 2e-6 * s ** 2 + 0.01 * s
    train, held = s[::2], s[1::2]
    h = cm.HybridModel.fit(train, 2e-6 * train ** 2 + 0.01 * train)
    assert h.regime(held[-2]) == "RF" and h.regime(held[-1]).startswith("PR")
    pred = h(held[:-1])  # the last held-out length lies beyond the range
    want = 2e-6 * held[:-1] ** 2 + 0.01 * held[:-1]
    # piecewise-constant trees: small relative error in the bulk, and an
    # absolute error far below the spread of the curve everywhere
    assert np.median(np.abs(pred / want - 1)) < 0.02
    assert np.max(np.abs(pred - want)) < 0.01 * want.max()
