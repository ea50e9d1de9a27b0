"""Seeded workload generators: determinism, recipe shape, bf16 rounding."""
import math

import numpy as np
import pytest

from paper_2511_13198_amd import workloads as wl


def test_bf16_rounding_matches_torch():
    import torch
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 3.0e38, 1e-40],
                                 dtype=np.float32)])
    ours = wl.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = wl.bf16_bits_to_f64(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(x).to(torch.bfloat16).double().numpy())


def test_cu_seqlens():
    cu = wl.cu_from_lengths([3, 0, 5])
    assert cu.dtype == np.int32 and cu.tolist() == [0, 3, 3, 8]


def test_loguniform_recipe():
    L = wl.loguniform_lengths()
    assert sum(L) == 65536
    assert L == wl.loguniform_lengths()  # deterministic
    assert all(128 <= s <= 8192 for s in L[:-1])
    assert 1 <= L[-1] <= 8192
    assert len(L) == 25 and min(L) == 167 and max(L) == 7402


def test_lognormal_stream_recipe():
    B = wl.lognormal_stream()
    assert len(B) == 64
    singles = sorted(b[0] for b in B if len(b) == 1)
    assert singles == [313313, 366775, 427570, 433630, 638976]
    for b in B:
        if len(b) > 1:
            assert sum(b) == 262144
            assert all(1 <= s < 262144 for s in b)
        else:
            assert 262144 <= b[0] <= 638976
    # long tail: a small share of draws at >= 128K (Table 3 puts 1.1-1.9% there)
    flat = [s for b in B for s in b]
    assert 0.0 < sum(s >= 131072 for s in flat) / len(flat) < 0.05


def test_configs():
    c1 = wl.config(1)
    assert (c1.total_tokens, c1.heads_q, c1.head_dim, c1.softmax_scale) == (512, 8, 64, 0.125)
    c4 = wl.config(4)
    assert c4.total_tokens == 638976 and c4.heads_q == 4
    s5 = wl.stream_config5(3)
    assert all(w.heads_q == 32 and w.heads_kv == 8 for w in s5)
    assert math.isclose(wl.config(3).softmax_scale, 1 / math.sqrt(128))


def test_host_inputs_deterministic():
    a = wl.host_inputs(100, 4, 2, 16, seed=5)
    b = wl.host_inputs(100, 4, 2, 16, seed=5)
    for n in "q k v do".split():
        np.testing.assert_array_equal(a[n], b[n])
    assert a["q"].shape == (100, 4, 16) and a["k"].shape == (100, 2, 16)
    x = wl.bf16_bits_to_f64(a["q"])
    assert abs(x.mean()) < 0.1 and abs(x.std() - 1) < 0.1


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: asked for more it exits with status 2 and a
    message, before touching a GPU."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""
