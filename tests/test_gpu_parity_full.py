"""HIP path vs the fp64 oracle on every element of the full-size workloads
where the oracle can afford it, through the C-ABI:

* the packed 65,536-token batch (log-uniform lengths in [128, 8192], 32
  heads, d = 128): O, LSE, dQ, dK and dV, every element of every head;
* the 131,072-token sequence (4 heads, d = 128): O, LSE and dQ for every row
  of query head 0, and dK, dV of its kv head for the first 2,048 ("sink")
  keys, 2,048 keys in the middle and the last 2,048 keys, from the oracle's
  own row statistics (LSE and D of every row);
* a 65,536-token sequence with 4 query heads on one kv head (grouped heads):
  every row of query head 2, and the kv head's dK, dV -- summed over the
  four query heads -- on the same three key windows.

The oracle's pieces (heads, row ranges, key windows) run side by side on the
host's cores; each piece is the plain definition.  Tolerance per tensor, over
all compared elements: max |err| <= 2e-2 and relative L2 <= 5e-3; the margins
to both are printed."""
import time

import pytest

from oracle import attention as ora
from paper_2511_13198_amd import workloads as wl
from tests import parity_util as pu

pytestmark = pytest.mark.gpu


@pytest.mark.timeout(900)
def test_packed_65536_every_element():
    import torch
    w = wl.config(2)
    T, hq, hkv, d = w.total_tokens, w.heads_q, w.heads_kv, w.head_dim
    scale = w.softmax_scale
    pu.log(f"  workload {w.name}: T={T} N={w.num_seqs} Hq={hq} Hkv={hkv} d={d}")
    bits = wl.host_inputs(T, hq, hkv, d)
    dev = {n: pu.to_device_bf16(b) for n, b in bits.items()}
    cu = w.cu_seqlens()
    cu_d = torch.from_numpy(cu).cuda()
    o, lse, dq, dk, dv = pu.run_gpu(dev["q"], dev["k"], dev["v"], dev["do"], cu_d,
                                    w.max_seqlen, w.causal, scale)
    got = {"O": o.cpu().double().numpy(), "LSE": lse.cpu().double().numpy(),
           "dQ": dq.cpu().numpy(), "dK": dk.cpu().numpy(), "dV": dv.cpu().numpy()}
    del o, lse, dq, dk, dv, dev
    assert hq == hkv, "one query head per kv head: each head is its own oracle piece"

    def one_head(h):
        f = {n: wl.bf16_bits_to_f64(b[:, h:h + 1]) for n, b in bits.items()}
        return ora.backward(f["q"], f["k"], f["v"], f["do"], cu, w.causal, scale)

    t0 = time.perf_counter()
    refs = pu.run_pieces(one_head, list(range(hq)))
    pu.log(f"  oracle: {hq} heads in {time.perf_counter() - t0:.1f} s on "
           f"{pu.host_workers()} threads")
    acc = {n: pu.ErrAcc(n) for n in ("O", "LSE", "dQ", "dK", "dV")}
    for h, (ro, rl, rdq, rdk, rdv) in enumerate(refs):
        acc["O"].add(got["O"][:, h], ro[:, 0])
        acc["LSE"].add(got["LSE"][h], rl[0])
        acc["dQ"].add(got["dQ"][:, h], rdq[:, 0])
        acc["dK"].add(got["dK"][:, h], rdk[:, 0])
        acc["dV"].add(got["dV"][:, h], rdv[:, 0])
    for a in acc.values():
        a.check()


SINK_WINDOW = 2048


def sink_middle_tail(T, w=SINK_WINDOW):
    """The first w ("sink") keys, w keys in the middle and the last w keys."""
    return [(0, w), (T // 2 - w // 2, T // 2 + w // 2), (T - w, T)]


@pytest.mark.timeout(900)
def test_single_131072_every_row_of_a_head_and_sink_keys():
    import torch
    w = wl.config(3)
    T, hq, hkv, d = w.total_tokens, w.heads_q, w.heads_kv, w.head_dim
    pu.log(f"  workload {w.name}: query head 0")
    dev = wl.device_inputs(T, hq, hkv, d)
    cu = w.cu_seqlens()
    cu_d = torch.from_numpy(cu).cuda()
    outs = pu.run_gpu(dev["q"], dev["k"], dev["v"], dev["do"], cu_d, w.max_seqlen, w.causal,
                      w.softmax_scale)
    pu.head_rows_and_key_windows(dev, outs, cu, w.causal, w.softmax_scale, 0,
                                 sink_middle_tail(T))


@pytest.mark.timeout(900)
def test_single_65536_grouped_heads_every_row_and_sink_keys():
    import torch
    w = wl.Workload("single65536_h4kv1", [65536], 4, 1, 128)
    T = w.total_tokens
    pu.log(f"  workload {w.name}: query head 2 of the group of 4 on kv head 0")
    dev = wl.device_inputs(T, w.heads_q, w.heads_kv, w.head_dim, seed=5)
    cu = w.cu_seqlens()
    cu_d = torch.from_numpy(cu).cuda()
    outs = pu.run_gpu(dev["q"], dev["k"], dev["v"], dev["do"], cu_d, w.max_seqlen, w.causal,
                      w.softmax_scale)
    pu.head_rows_and_key_windows(dev, outs, cu, w.causal, w.softmax_scale, 2,
                                 sink_middle_tail(T))
