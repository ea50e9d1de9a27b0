"""The whole context-parallel ring run on one GPU (chunk forward + merges,
chunk backward with in-kernel accumulation) against the full-sequence fp64
oracle."""
import numpy as np
import pytest

from oracle import attention as ora
from paper_2511_13198_amd import context_parallel as cp
from paper_2511_13198_amd import workloads as wl
from tests.parity_util import (HeadView, check_close, head_rows_and_key_windows, log, sample_rows,
                               to_device_bf16)

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


@pytest.mark.timeout(900)
def test_zigzag_ring_at_131072_tokens():
    """The p=8 zig-zag ring over one 131,072-token sequence (4 heads, d=128)
    against the oracle: every row of query head 3 (O, LSE, dQ) and dK, dV of
    kv head 3 on its first, middle and last 2,048 keys; sampled rows of head
    0 and the last 64 keys of kv heads 1 and 2; and every element against the
    unsharded library call within twice the tolerance (both carry their own
    rounding)."""
    import torch
    from paper_2511_13198_amd import pdyattn
    w = wl.config(3)
    T, hq, hkv, d = w.total_tokens, w.heads_q, w.heads_kv, w.head_dim
    scale = w.softmax_scale
    p = 8
    log(f"  zig-zag ring p={p} T={T} Hq={hq} d={d}")
    dev = wl.device_inputs(T, hq, hkv, d)
    q, k, v, do = dev["q"], dev["k"], dev["v"], dev["do"]
    o, lses = cp.ring_forward(q, k, v, p, True, scale, layout="zigzag")
    dq, dk, dv = cp.ring_backward(q, k, v, o, lses, do, p, True, scale, layout="zigzag")
    lse = torch.empty((hq, T), dtype=torch.float32, device=q.device)
    for (a, b), l in lses.items():
        lse[:, a:b] = l
    cu = torch.tensor([0, T], dtype=torch.int32, device=q.device)
    o_u, lse_u = pdyattn.attn_fwd(q, k, v, cu, T, True, scale)
    dq_u, dk_u, dv_u = pdyattn.attn_bwd(q, k, v, o_u, lse_u, do, cu, T, True, scale)
    torch.cuda.synchronize()
    for name, g, u in (("O", o, o_u), ("LSE", lse, lse_u), ("dQ", dq, dq_u), ("dK", dk, dk_u),
                       ("dV", dv, dv_u)):
        check_close(name + " vs unsharded", g.double().cpu().numpy(), u.double().cpu().numpy(),
                    max_abs=4e-2, rel_l2=1e-2)
    cu_h = np.array([0, T])
    del o_u, lse_u, dq_u, dk_u, dv_u
    w2 = 2048
    head_rows_and_key_windows(dev, (o, lse, dq, dk, dv), cu_h, True, scale, 3,
                              [(0, w2), (T // 2 - w2 // 2, T // 2 + w2 // 2), (T - w2, T)])
    host = {n: HeadView(t) for n, t in dev.items()}
    rows = sample_rows([T], 24, max_rows=48)
    res = ora.rows_forward_backward(host["q"], host["k"], host["v"], host["do"], cu_h, True,
                                    scale, heads=[0], rows=rows)
    ridx = torch.tensor(rows, dtype=torch.long, device=q.device)
    for h in (0,):
        check_close("O", o[ridx, h].double().cpu().numpy(), res[h][0])
        check_close("LSE", lse[h, ridx].double().cpu().numpy(), res[h][1])
        check_close("dQ", dq[ridx, h].double().cpu().numpy(), res[h][2])
    cols = ora.cols_backward(host["q"], host["k"], host["v"], host["do"], cu_h, True, scale,
                             kv_heads=[1, 2], seg_index=0, col_lo=T - 64)
    for hk in (1, 2):
        check_close("dK", dk[T - 64:, hk].double().cpu().numpy(), cols[hk][0])
        check_close("dV", dv[T - 64:, hk].double().cpu().numpy(), cols[hk][1])
