"""GPU parity of the context-parallel chunk entry points (attn_fwd_chunk,
attn_merge, attn_bwd_chunk) against the fp64 chunked oracle, and end to end:
chunked-and-merged forward and summed chunk gradients against the
full-sequence oracle."""
import numpy as np
import pytest

from oracle import attention as ora
from paper_2511_13198_amd import workloads as wl
from tests.parity_util import check_close, log, to_device_bf16

pytestmark = pytest.mark.gpu


def _host(T, hq, hkv, d, seed):
    bits = wl.host_inputs(T, hq, hkv, d, seed=seed)
    f64 = {n: wl.bf16_bits_to_f64(b) for n, b in bits.items()}
    return bits, f64


def _dev(bits, name, lo, hi):
    return to_device_bf16(np.ascontiguousarray(bits[name][lo:hi]))


def _check_partial(name_o, name_l, o_gpu, l_gpu, o_ref, l_ref):
    """-inf rows must match exactly (with O = 0); the rest within tolerance."""
    l_gpu = np.asarray(l_gpu, dtype=np.float64)
    dead_ref = np.isneginf(l_ref)
    assert np.array_equal(np.isneginf(l_gpu), dead_ref), f"{name_l}: rows without keys differ"
    assert np.all(np.isfinite(l_gpu[~dead_ref]))
    if (~dead_ref).any():
        check_close(name_l, l_gpu[~dead_ref], l_ref[~dead_ref])
    o_gpu = np.asarray(o_gpu, dtype=np.float64)
    dead_rows = dead_ref.T  # [Tq, Hq]
    assert np.all(o_gpu[dead_rows] == 0), f"{name_o}: rows without keys are not zero"
    check_close(name_o, o_gpu, o_ref)


PAIRS = [
    # (T, hq, hkv, d, causal, (qa, qb), (ka, kb))
    (700, 4, 2, 128, True, (300, 700), (0, 300)),     # every key visible
    (700, 4, 2, 128, True, (300, 700), (300, 700)),   # diagonal chunk
    (700, 4, 2, 128, True, (0, 300), (300, 700)),     # nothing visible
    (700, 4, 2, 128, True, (200, 500), (350, 650)),   # first 150 rows see nothing
    (700, 2, 2, 64, True, (129, 700), (1, 257)),
    (600, 2, 1, 128, False, (0, 333), (100, 600)),
    (300, 2, 2, 128, True, (0, 300), (0, 0)),         # empty key chunk
    # query chunks over 2,048 rows: the 8-wave kernels
    (5000, 2, 1, 128, True, (2100, 5000), (1000, 3500)),
    (4500, 2, 2, 64, False, (0, 2300), (2000, 4500)),
]


@pytest.mark.parametrize("T,hq,hkv,d,causal,qs,ks", PAIRS)
def test_partial_forward(T, hq, hkv, d, causal, qs, ks):
    import torch
    from paper_2511_13198_amd import pdyattn
    bits, f = _host(T, hq, hkv, d, 7)
    scale = 1.0 / np.sqrt(d)
    (qa, qb), (ka, kb) = qs, ks
    log(f"  chunk q[{qa},{qb}) k[{ka},{kb}) Hq={hq} Hkv={hkv} d={d} causal={causal}")
    o_ref, l_ref = ora.partial_forward(f["q"][qa:qb], f["k"][ka:kb], f["v"][ka:kb], qa, ka,
                                       causal, scale)
    q, k, v = _dev(bits, "q", qa, qb), _dev(bits, "k", ka, kb), _dev(bits, "v", ka, kb)
    o = torch.full_like(q, float("nan"))
    lse = torch.full((hq, qb - qa), float("nan"), dtype=torch.float32, device=q.device)
    pdyattn.attn_fwd_chunk(q, k, v, qa, ka, causal, scale, out=o, lse=lse)
    torch.cuda.synchronize()
    _check_partial("O", "LSE", o.double().cpu().numpy(), lse.cpu().numpy(), o_ref, l_ref)


def _split_forward_gpu(bits, cuts, hq, causal, scale):
    """Forward of every query chunk over every key chunk, merged on the GPU."""
    from paper_2511_13198_amd import pdyattn
    spans = list(zip(cuts[:-1], cuts[1:]))
    outs = []
    for qa, qb in spans:
        q = _dev(bits, "q", qa, qb)
        acc = None
        for ka, kb in spans:
            part = pdyattn.attn_fwd_chunk(q, _dev(bits, "k", ka, kb), _dev(bits, "v", ka, kb),
                                          qa, ka, causal, scale)
            acc = part if acc is None else pdyattn.attn_merge(acc[0], acc[1], part[0], part[1],
                                                              out=acc[0], lse=acc[1])
        outs.append(acc)
    return outs


@pytest.mark.parametrize("T,hq,hkv,d,causal,cuts", [
    (1500, 4, 2, 128, True, [0, 400, 1000, 1500]),
    (1024, 2, 2, 64, True, [0, 1, 512, 1024]),
    (900, 2, 1, 128, False, [0, 450, 900]),
])
def test_chunks_merge_to_full_attention(T, hq, hkv, d, causal, cuts):
    import torch
    bits, f = _host(T, hq, hkv, d, 11)
    scale = 1.0 / np.sqrt(d)
    log(f"  sequence T={T} cut at {cuts} Hq={hq} Hkv={hkv} d={d} causal={causal}")
    O, L = ora.forward(f["q"], f["k"], f["v"], np.array([0, T]), causal, scale)
    outs = _split_forward_gpu(bits, cuts, hq, causal, scale)
    torch.cuda.synchronize()
    o = np.concatenate([x[0].double().cpu().numpy() for x in outs], axis=0)
    lse = np.concatenate([x[1].cpu().numpy() for x in outs], axis=1)
    check_close("O", o, O)
    check_close("LSE", lse, L)


@pytest.mark.parametrize("T,hq,hkv,d,causal,cuts", [
    (1200, 4, 2, 128, True, [0, 300, 700, 1200]),
    (800, 2, 2, 64, True, [0, 257, 800]),
    (600, 2, 1, 128, False, [0, 200, 600]),
    (5000, 2, 1, 128, True, [0, 2200, 5000]),     # chunks over 2,048 rows: 8-wave kernels
])
def test_chunk_gradients(T, hq, hkv, d, causal, cuts):
    """Each pair against the oracle's pair contribution, and the sums against
    the full-sequence gradient.  O and LSE fed to the device are the oracle's
    (O rounded to bf16, LSE to fp32)."""
    import torch
    from paper_2511_13198_amd import pdyattn
    bits, f = _host(T, hq, hkv, d, 13)
    scale = 1.0 / np.sqrt(d)
    log(f"  sequence T={T} cut at {cuts} Hq={hq} Hkv={hkv} d={d} causal={causal}")
    O, L, dQ, dK, dV = ora.backward(f["q"], f["k"], f["v"], f["do"], np.array([0, T]), causal,
                                    scale)
    o_bits = wl.f32_to_bf16_bits(O.astype(np.float32))
    o_dev = to_device_bf16(o_bits)
    l_dev = torch.from_numpy(L.astype(np.float32)).cuda()
    spans = list(zip(cuts[:-1], cuts[1:]))
    dq = torch.zeros((T, hq, d), dtype=torch.float32, device="cuda")
    dk = torch.zeros((T, hkv, d), dtype=torch.float32, device="cuda")
    dv = torch.zeros((T, hkv, d), dtype=torch.float32, device="cuda")
    for qa, qb in spans:
        for ka, kb in spans:
            gq, gk, gv = pdyattn.attn_bwd_chunk(
                _dev(bits, "q", qa, qb), _dev(bits, "k", ka, kb), _dev(bits, "v", ka, kb),
                o_dev[qa:qb].contiguous(), l_dev[:, qa:qb].contiguous(),
                _dev(bits, "do", qa, qb), qa, ka, causal, scale)
            torch.cuda.synchronize()
            rq, rk, rv = ora.partial_backward(
                f["q"][qa:qb], f["k"][ka:kb], f["v"][ka:kb], wl.bf16_bits_to_f64(o_bits[qa:qb]),
                L[:, qa:qb].astype(np.float32).astype(np.float64), f["do"][qa:qb], qa, ka,
                causal, scale)
            log(f"   pair q[{qa},{qb}) k[{ka},{kb})")
            # a pair with no visible key gives exact zeros on both sides
            for nm, g, r in (("dQc", gq, rq), ("dKc", gk, rk), ("dVc", gv, rv)):
                gn = g.double().cpu().numpy()
                if not np.any(r):
                    assert not np.any(gn), f"{nm}: nonzero gradient for an invisible pair"
                else:
                    check_close(nm, gn, r)
            dq[qa:qb] += gq
            dk[ka:kb] += gk
            dv[ka:kb] += gv
    torch.cuda.synchronize()
    check_close("dQ", dq.double().cpu().numpy(), dQ)
    check_close("dK", dk.double().cpu().numpy(), dK)
    check_close("dV", dv.double().cpu().numpy(), dV)


def _random_pairs(n=20, seed=13198):
    """Seeded random (query chunk, key chunk) pairs of one sequence of 64-5,000
    tokens: chunks of 1-3,000 rows anywhere (before, across or after each
    other, empty key chunks included), 1-3 kv heads in groups of 1, 2 or 4,
    d in {64, 128}, either causal flag."""
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        T = int(rng.integers(64, 5001))
        qa = int(rng.integers(0, T))
        qb = int(rng.integers(qa + 1, min(T, qa + 3000) + 1))
        ka = int(rng.integers(0, T))
        kb = ka if rng.random() < 0.1 else int(rng.integers(ka + 1, min(T, ka + 3000) + 1))
        hkv = int(rng.choice([1, 2, 3]))
        hq = hkv * int(rng.choice([1, 2, 4]))
        cases.append((T, hq, hkv, int(rng.choice([64, 128])), bool(rng.integers(0, 2)),
                      (qa, qb), (ka, kb)))
    return cases


@pytest.mark.parametrize("T,hq,hkv,d,causal,qs,ks", _random_pairs())
def test_random_chunk_pairs(T, hq, hkv, d, causal, qs, ks):
    """Partial forward and the pair's gradient contribution of random chunk
    pairs against the oracle's (O and LSE fed to the backward are the
    oracle's final ones over the whole sequence, rounded as the device
    stores them)."""
    import torch
    from paper_2511_13198_amd import pdyattn
    bits, f = _host(T, hq, hkv, d, 17)
    scale = 1.0 / np.sqrt(d)
    (qa, qb), (ka, kb) = qs, ks
    log(f"  T={T} chunk q[{qa},{qb}) k[{ka},{kb}) Hq={hq} Hkv={hkv} d={d} causal={causal}")
    o_ref, l_ref = ora.partial_forward(f["q"][qa:qb], f["k"][ka:kb], f["v"][ka:kb], qa, ka,
                                       causal, scale)
    q, do = _dev(bits, "q", qa, qb), _dev(bits, "do", qa, qb)
    if kb > ka:
        k, v = _dev(bits, "k", ka, kb), _dev(bits, "v", ka, kb)
    else:  # an empty key chunk
        k = v = torch.empty((0, hkv, d), dtype=torch.bfloat16, device="cuda")
    o = torch.full_like(q, float("nan"))
    lse = torch.full((hq, qb - qa), float("nan"), dtype=torch.float32, device=q.device)
    pdyattn.attn_fwd_chunk(q, k, v, qa, ka, causal, scale, out=o, lse=lse)
    torch.cuda.synchronize()
    _check_partial("O", "LSE", o.double().cpu().numpy(), lse.cpu().numpy(), o_ref, l_ref)
    if kb == ka:
        return
    O, L = ora.forward(f["q"], f["k"], f["v"], np.array([0, T]), causal, scale)
    o_bits = wl.f32_to_bf16_bits(O[qa:qb].astype(np.float32))
    l32 = np.ascontiguousarray(L[:, qa:qb].astype(np.float32))
    gq, gk, gv = pdyattn.attn_bwd_chunk(q, k, v, to_device_bf16(o_bits),
                                        torch.from_numpy(l32).cuda(), do, qa, ka, causal, scale)
    torch.cuda.synchronize()
    rq, rk, rv = ora.partial_backward(f["q"][qa:qb], f["k"][ka:kb], f["v"][ka:kb],
                                      wl.bf16_bits_to_f64(o_bits), l32.astype(np.float64),
                                      f["do"][qa:qb], qa, ka, causal, scale)
    for nm, g, r in (("dQc", gq, rq), ("dKc", gk, rk), ("dVc", gv, rv)):
        gn = g.double().cpu().numpy()
        if not np.any(r):
            assert not np.any(gn), f"{nm}: nonzero gradient for an invisible pair"
        else:
            check_close(nm, gn, r)


def test_merge_against_the_oracle():
    import torch
    from paper_2511_13198_amd import pdyattn
    rng = np.random.default_rng(5)
    T, hq, d = 333, 3, 128
    parts = []
    for _ in range(2):
        o = wl.f32_to_bf16_bits(rng.standard_normal((T, hq, d)).astype(np.float32))
        l = rng.normal(0, 3, (hq, T)).astype(np.float32)
        l[0, :7] = -np.inf       # one side empty
        parts.append((o, l))
    parts[1][1][0, :3] = -np.inf  # both sides empty for three rows
    ref = ora.merge([(wl.bf16_bits_to_f64(o), l.astype(np.float64)) for o, l in parts])
    a = (to_device_bf16(parts[0][0]), torch.from_numpy(parts[0][1]).cuda())
    b = (to_device_bf16(parts[1][0]), torch.from_numpy(parts[1][1]).cuda())
    o, l = pdyattn.attn_merge(a[0], a[1], b[0], b[1])
    torch.cuda.synchronize()
    _check_partial("O", "LSE", o.double().cpu().numpy(), l.cpu().numpy(), ref[0], ref[1])
    # in place into the first operand gives the same bytes
    o2, l2 = pdyattn.attn_merge(a[0], a[1], b[0], b[1], out=a[0], lse=a[1])
    torch.cuda.synchronize()
    assert torch.equal(o2, o) and torch.equal(l2.isneginf(), l.isneginf())
