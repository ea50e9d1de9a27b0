"""Write the golden fixtures of this directory from the fp64 oracle.

Each fixture is a small packed batch: its bf16 inputs (raw bits, drawn once
from numpy's seeded generator and stored, so the fixture does not depend on
the generator staying the same) and the oracle's outputs O, LSE, dQ, dK, dV
of Eq. (2) (section 3) and its gradient, as decimal strings that round-trip
float64 exactly.  Only the oracle and the input helpers are called.

Usage: python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import attention as ora  # noqa: E402
from paper_2511_13198_amd import workloads as wl  # noqa: E402

CASES = {
    # a ragged packed batch with a one-token segment and grouped heads
    "packed_5_1_9_h2kv1_d64_causal": dict(lengths=[5, 1, 9], hq=2, hkv=1, d=64, causal=True,
                                          scale=0.125, seed=2024),
    # the same segments without the causal mask
    "packed_5_1_9_h2kv1_d64_full": dict(lengths=[5, 1, 9], hq=2, hkv=1, d=64, causal=False,
                                        scale=0.125, seed=2024),
}


def make(case):
    T = sum(case["lengths"])
    rng = np.random.default_rng(case["seed"])
    bits = {}
    for name, h in (("q", case["hq"]), ("k", case["hkv"]), ("v", case["hkv"]), ("do", case["hq"])):
        x = rng.standard_normal((T, h, case["d"])).astype(np.float32)
        bits[name] = wl.f32_to_bf16_bits(x)
    f = {n: wl.bf16_bits_to_f64(b) for n, b in bits.items()}
    cu = wl.cu_from_lengths(case["lengths"])
    o, lse, dq, dk, dv = ora.backward(f["q"], f["k"], f["v"], f["do"], cu, case["causal"],
                                      case["scale"])
    enc = lambda a: [repr(float(x)) for x in np.asarray(a).ravel()]  # noqa: E731
    return {
        "case": case,
        "inputs_bf16_bits": {n: [int(x) for x in b.ravel()] for n, b in bits.items()},
        "outputs": {"O": enc(o), "LSE": enc(lse), "dQ": enc(dq), "dK": enc(dk), "dV": enc(dv)},
        "shapes": {"O": list(o.shape), "LSE": list(lse.shape), "dQ": list(dq.shape),
                   "dK": list(dk.shape), "dV": list(dv.shape)},
    }


def main():
    for name, case in CASES.items():
        path = os.path.join(HERE, f"{name}.json")
        with open(path, "w") as fh:
            json.dump(make(case), fh, indent=0)
        print("wrote", path)


if __name__ == "__main__":
    main()
