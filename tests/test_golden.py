"""The golden fixtures of tests/golden (small packed batches: stored bf16
inputs and the fp64 oracle's outputs, written by tests/golden/make_golden.py
from the oracle alone).  On the CPU the oracle must still produce the stored
values (any change to its arithmetic shows here and has to be justified by
the paper); on the GPU the HIP path must match them within the parity
tolerance."""
import glob
import json
import os

import numpy as np
import pytest

from oracle import attention as ora
from paper_2511_13198_amd import workloads as wl

HERE = os.path.dirname(os.path.abspath(__file__))
FIXTURES = sorted(glob.glob(os.path.join(HERE, "golden", "*.json")))
NAMES = ("O", "LSE", "dQ", "dK", "dV")


def _load(path):
    rec = json.load(open(path))
    c = rec["case"]
    T = sum(c["lengths"])
    shapes = {"q": (T, c["hq"], c["d"]), "k": (T, c["hkv"], c["d"]), "v": (T, c["hkv"], c["d"]),
              "do": (T, c["hq"], c["d"])}
    bits = {n: np.array(v, dtype=np.uint16).reshape(shapes[n])
            for n, v in rec["inputs_bf16_bits"].items()}
    want = {n: np.array([float(x) for x in rec["outputs"][n]]).reshape(rec["shapes"][n])
            for n in NAMES}
    return c, bits, want


def test_fixtures_present():
    assert len(FIXTURES) >= 2


@pytest.mark.parametrize("path", FIXTURES, ids=[os.path.basename(p) for p in FIXTURES])
def test_oracle_reproduces_golden(path):
    c, bits, want = _load(path)
    f = {n: wl.bf16_bits_to_f64(b) for n, b in bits.items()}
    got = ora.backward(f["q"], f["k"], f["v"], f["do"], wl.cu_from_lengths(c["lengths"]),
                       c["causal"], c["scale"])
    for name, g in zip(NAMES, got):
        np.testing.assert_allclose(g, want[name], rtol=0, atol=1e-13, err_msg=name)


@pytest.mark.gpu
@pytest.mark.parametrize("path", FIXTURES, ids=[os.path.basename(p) for p in FIXTURES])
def test_hip_path_matches_golden(path):
    import torch

    from tests import parity_util as pu
    c, bits, want = _load(path)
    dev = {n: pu.to_device_bf16(b) for n, b in bits.items()}
    cu = torch.from_numpy(wl.cu_from_lengths(c["lengths"])).cuda()
    outs = pu.run_gpu(dev["q"], dev["k"], dev["v"], dev["do"], cu, max(c["lengths"]),
                      c["causal"], c["scale"])
    for name, g in zip(NAMES, outs):
        pu.check_close(name, g.double().cpu().numpy(), want[name])
