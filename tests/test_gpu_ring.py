"""The whole context-parallel ring run on one GPU (chunk forward + merges,
chunk backward with in-kernel accumulation) against the full-sequence fp64
oracle."""
import numpy as np
import pytest

from oracle import attention as ora
from paper_2511_13198_amd import context_parallel as cp
from paper_2511_13198_amd import workloads as wl
from tests.parity_util import check_close, log, to_device_bf16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
@pytest.mark.parametrize("T,hq,hkv,d,causal,p", [
    (1500, 4, 2, 128, True, 3),
    (1024, 2, 2, 64, True, 4),
    (1001, 2, 1, 128, True, 4),
    (700, 2, 2, 128, False, 2),
    (3, 1, 1, 128, True, 5),      # more devices than tokens: empty chunks
])
def test_ring_matches_full_attention(T, hq, hkv, d, causal, p, layout):
    import torch
    bits = wl.host_inputs(T, hq, hkv, d, seed=17)
    f = {n: wl.bf16_bits_to_f64(b) for n, b in bits.items()}
    scale = 1.0 / np.sqrt(d)
    log(f"  ring {layout} p={p} T={T} Hq={hq} Hkv={hkv} d={d} causal={causal}")
    O, L, dQ, dK, dV = ora.backward(f["q"], f["k"], f["v"], f["do"], np.array([0, T]), causal,
                                    scale)
    q, k, v, do = (to_device_bf16(bits[n]) for n in ("q", "k", "v", "do"))
    o, lses = cp.ring_forward(q, k, v, p, causal, scale, layout=layout)
    dq, dk, dv = cp.ring_backward(q, k, v, o, lses, do, p, causal, scale, layout=layout)
    torch.cuda.synchronize()
    lse = np.concatenate([lses[rg].cpu().numpy() for rg in sorted(lses)], axis=1)
    check_close("O", o.double().cpu().numpy(), O)
    check_close("LSE", lse, L)
    check_close("dQ", dq.double().cpu().numpy(), dQ)
    check_close("dK", dk.double().cpu().numpy(), dK)
    check_close("dV", dv.double().cpu().numpy(), dV)


def test_accumulate_adds_to_what_is_there():
    """attn_bwd_chunk with accumulate=True on buffers holding X gives X + the
    pair's part (checked against the same call with accumulate=False)."""
    import torch
    from paper_2511_13198_amd import pdyattn
    T, hq, hkv, d = 600, 2, 2, 128
    bits = wl.host_inputs(T, hq, hkv, d, seed=19)
    q, k, v, do = (to_device_bf16(bits[n]) for n in ("q", "k", "v", "do"))
    o, lse = pdyattn.attn_fwd_chunk(q[300:], k[:300], v[:300], 300, 0, True)
    fresh = pdyattn.attn_bwd_chunk(q[300:], k[:300], v[:300], o, lse, do[300:], 300, 0, True)
    base = [torch.randn_like(x) for x in fresh]
    acc = [b.clone() for b in base]
    pdyattn.attn_bwd_chunk(q[300:], k[:300], v[:300], o, lse, do[300:], 300, 0, True,
                           dq=acc[0], dk=acc[1], dv=acc[2], accumulate=True)
    torch.cuda.synchronize()
    for a, b, fr in zip(acc, base, fresh):
        assert torch.allclose(a, b + fr, rtol=0, atol=1e-5)
