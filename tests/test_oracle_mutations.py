"""Planted mistakes in a copy of the oracle must each trip at least one pin.

Each mutation edits the oracle's source text (on the CPU, in memory), loads
the edited copy as a throwaway module, and re-runs the pin tests of
test_oracle.py against it.  A mutation that no pin detects fails this test."""
import importlib.util
import os
import types

import pytest

import tests.test_oracle as pins
import tests.test_oracle_stats as stat_pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "attention.py")

MUTATIONS = {
    "mask_strict": ("cols <= rows", "cols < rows"),
    "mask_open": ("np.where(cols <= rows, s, -np.inf)", "s"),
    "scale_dropped": ("s = scale * (qr @ kk.T)", "s = (qr @ kk.T)"),
    "lse_log2": ("lse = m + np.log(np.sum", "lse = m + np.log2(np.sum"),
    "ds_sign": ("ds = p * (dp - D[:, None])", "ds = p * (D[:, None] - dp)"),
    "d_dropped": ("ds = p * (dp - D[:, None])", "ds = p * dp"),
    "dq_no_scale": ("dq[r0:r1, h] = scale * (ds @ kk)", "dq[r0:r1, h] = (ds @ kk)"),
    "dk_uses_p": ("dk[a:a + n, hk] += scale * (ds.T @ q[r0:r1, h])",
                  "dk[a:a + n, hk] += scale * (p.T @ q[r0:r1, h])"),
    "dv_uses_ds": ("dv[a:a + n, hk] += p.T @ dor", "dv[a:a + n, hk] += ds.T @ dor"),
    "gqa_modulo": ("hk = h // g\n            for r0 in range(a, b, row_block):\n                r1 = min(b, r0 + row_block)\n                n = _visible_keys(a, b, r0, r1, causal)\n                kk = k[a:a + n, hk]\n                vv = v[a:a + n, hk]\n                s = _logits(q[r0:r1, h], kk, a, r0, causal, scale)\n                l, p",
                   "hk = h % Hkv\n            for r0 in range(a, b, row_block):\n                r1 = min(b, r0 + row_block)\n                n = _visible_keys(a, b, r0, r1, causal)\n                kk = k[a:a + n, hk]\n                vv = v[a:a + n, hk]\n                s = _logits(q[r0:r1, h], kk, a, r0, causal, scale)\n                l, p"),
    "segment_leak": ("kk = k[a:a + n, hk]\n                vv = v[a:a + n, hk]\n                s = _logits(q[r0:r1, h], kk, a, r0, causal, scale)\n                l, p",
                     "kk = k[max(0, a - 1):max(0, a - 1) + n, hk]\n                vv = v[max(0, a - 1):max(0, a - 1) + n, hk]\n                s = _logits(q[r0:r1, h], kk, a, r0, causal, scale)\n                l, p"),
    "visible_short": ("return (r1 - a) if causal else (b - a)", "return (r1 - a - 1) if causal else (b - a)"),
    # the row-statistics pass and the key-window gradient
    "rows_dq_no_scale": ("dd[sl], dq[sl] = orow, l, D, scale * (ds @ kk)",
                         "dd[sl], dq[sl] = orow, l, D, (ds @ kk)"),
    "rows_d_from_dq": ("D = np.sum(dor * orow, axis=1)\n            ds = p * (dor @ vv.T - D[:, None])\n            sl",
                       "D = np.sum(dor * dor, axis=1)\n            ds = p * (dor @ vv.T - D[:, None])\n            sl"),
    "rows_block_overrun": ("r1 = min(b, r_hi, r0 + row_block)", "r1 = min(b, r0 + row_block)"),
    "window_mask_strict": ("s = np.where(cols <= np.arange(r0, r1)[:, None], s, -np.inf)",
                           "s = np.where(cols < np.arange(r0, r1)[:, None], s, -np.inf)"),
    "window_skips_diagonal_row": ("for r0 in range(c_lo if causal else a, b, row_block):",
                                  "for r0 in range(c_lo + 1 if causal else a, b, row_block):"),
    "window_no_d": ("ds = p * (dor @ vw.T - dd[h, r0:r1, None])", "ds = p * (dor @ vw.T)"),
    "window_lse_log2": ("p = np.exp(s - lse[h, r0:r1, None])",
                        "p = np.exp2(s - lse[h, r0:r1, None])"),
    "window_one_head": ("for h in range(kv_head * g, (kv_head + 1) * g):",
                        "for h in range(kv_head * g, kv_head * g + 1):"),
}

PIN_TESTS = [
    ("test_forward_matches_brute_force", [([7], 1, 1, 4, True), ([5, 1, 9], 2, 1, 8, True),
                                           ([6, 3], 2, 2, 4, False), ([16], 4, 2, 8, True)]),
    ("test_rows_sum_to_one_v_ones", [()]),
    ("test_matches_torch_fp64_sdpa_and_autograd", [([40, 17, 71], 4, 2, 32, True),
                                                   ([64, 3], 8, 2, 16, False)]),
    ("test_single_token_segment", [()]),
    ("test_zero_queries_give_prefix_means", [()]),
    ("test_gradient_finite_differences", [(True,), (False,)]),
    ("test_gqa_equals_repeated_mha", [()]),
    ("test_global_invariants", [()]),
]

# pins of the row-statistics pass and the key-window gradient
STAT_PIN_TESTS = [
    ("test_head_rows_match_torch", list(stat_pins.CASES)),
    ("test_key_windows_from_row_stats_match_torch", list(stat_pins.CASES)),
]


def _mutant(name):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert old in src, f"mutation {name} no longer applies"
    mod = types.ModuleType(f"oracle_mutant_{name}")
    exec(compile(src.replace(old, new, 1), SRC, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    mutant = _mutant(name)
    monkeypatch.setattr(pins, "ora", mutant)
    monkeypatch.setattr(stat_pins, "ora", mutant)
    for module, tests in ((pins, PIN_TESTS), (stat_pins, STAT_PIN_TESTS)):
        for test_name, cases in tests:
            fn = getattr(module, test_name)
            for args in cases:
                try:
                    fn(*args)
                except Exception:
                    return  # detected
    pytest.fail(f"planted mistake '{name}' passed every pin")
