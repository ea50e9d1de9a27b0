"""HIP path vs the fp64 oracle, through the C-ABI, on seeded inputs.

Small shapes are compared element by element in full; the full-size workloads
are compared on sampled rows (O, LSE, dQ) and tail key columns (dK, dV) that
the oracle evaluates one by one, plus identities of the exact gradient over
every element.  Tolerance per tensor: max |err| <= 2e-2 and relative L2 <= 5e-3."""
import math

import numpy as np
import pytest

from oracle import attention as ora
from paper_2511_13198_amd import workloads as wl
from tests import parity_util as pu

pytestmark = pytest.mark.gpu


def _host_case(lengths, hq, hkv, d, seed=wl.SEED):
    T = sum(lengths)
    bits = wl.host_inputs(T, hq, hkv, d, seed=seed)
    return bits, wl.cu_from_lengths(lengths)


def _full_parity(lengths, hq, hkv, d, causal, scale=None, seed=wl.SEED):
    import torch
    scale = scale if scale is not None else 1.0 / math.sqrt(d)
    pu.log(f"  case lengths={lengths[:8]}{'...' if len(lengths) > 8 else ''} T={sum(lengths)} "
           f"Hq={hq} Hkv={hkv} d={d} causal={causal}")
    bits, cu = _host_case(lengths, hq, hkv, d, seed)
    dev = {n: pu.to_device_bf16(b) for n, b in bits.items()}
    cu_d = torch.from_numpy(cu).cuda()
    o, lse, dq, dk, dv = pu.run_gpu(dev["q"], dev["k"], dev["v"], dev["do"], cu_d,
                                    max(lengths) if lengths else 0, causal, scale)
    f = {n: wl.bf16_bits_to_f64(b) for n, b in bits.items()}
    ro, rlse, rdq, rdk, rdv = ora.backward(f["q"], f["k"], f["v"], f["do"], cu, causal, scale)
    pu.check_close("O", pu.bf16_to_f64(o), ro)
    pu.check_close("LSE", lse.cpu().numpy(), rlse)
    pu.check_close("dQ", dq.cpu().numpy(), rdq)
    pu.check_close("dK", dk.cpu().numpy(), rdk)
    pu.check_close("dV", dv.cpu().numpy(), rdv)
    return (o, lse, dq, dk, dv), dev, cu_d


@pytest.mark.parametrize("lengths,hq,hkv,d,causal,scale", [
    ([512], 8, 8, 64, True, 0.125),                         # 512-token, 8-head, d=64 workload
    ([1, 127, 128, 129, 300, 64, 1000], 4, 2, 128, True, None),  # ragged tails + grouped heads
    ([0, 5, 0, 200, 0], 2, 1, 128, True, None),             # empty segments
    ([777], 2, 2, 64, False, None),                         # non-causal (BERT-like)
    ([300, 65, 1], 4, 4, 128, False, None),
    ([2048, 33], 8, 2, 128, True, None),
    ([1], 1, 1, 64, True, None),                            # single token
    ([128, 1, 100, 37, 128], 4, 2, 128, True, None),        # every segment <= 2048: 4-wave kernels
    ([96, 3, 128], 2, 2, 128, False, None),                 # same, non-causal
    ([700, 1300, 45], 6, 2, 128, True, None),               # three query heads per kv head
    ([900, 257], 3, 3, 64, False, None),                    # odd head count, non-causal
    ([2100, 300, 1], 4, 2, 128, True, None),                # a segment > 2048: 8-wave kernels
    ([2200], 2, 2, 64, False, None),                        # same, non-causal, d = 64
])
def test_full_parity_small(lengths, hq, hkv, d, causal, scale):
    _full_parity(lengths, hq, hkv, d, causal, scale)


def _random_shapes(n=40, seed=2511):
    """Seeded random small shapes: 1-4 segments of 0-3,000 tokens (some
    empty), query/kv head groups of 1-4, d in {64, 128}, either causal flag
    and scales around 1/sqrt(d): across the 4-/8-wave threshold, ragged
    tails and the split paths."""
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        nseg = int(rng.integers(1, 5))
        kind = rng.choice(3, size=nseg, p=[0.15, 0.25, 0.6])  # empty, short, longer
        lengths = [0 if k == 0 else int(rng.integers(1, 65)) if k == 1 else
                   int(rng.integers(65, 3001)) for k in kind]
        if sum(lengths) == 0:
            lengths[0] = 1
        hkv = int(rng.choice([1, 2, 3]))
        hq = hkv * int(rng.choice([1, 2, 4]))
        d = int(rng.choice([64, 128]))
        causal = bool(rng.integers(0, 2))
        scale = float(rng.uniform(0.6, 1.4) / math.sqrt(d))
        cases.append((lengths, hq, hkv, d, causal, scale))
    return cases


@pytest.mark.parametrize("lengths,hq,hkv,d,causal,scale", _random_shapes())
def test_random_shapes_full_parity(lengths, hq, hkv, d, causal, scale):
    _full_parity(lengths, hq, hkv, d, causal, scale)


@pytest.mark.parametrize("lengths,hq,hkv,d,causal", [
    ([3000], 2, 1, 128, True),        # 8-wave forward
    ([1500, 700], 2, 2, 64, True),    # 4-wave forward
    ([2600], 2, 2, 128, False),       # non-causal
    ([4096], 2, 2, 128, True),        # balanced split-K: every part sets its own offset
])
def test_forward_logits_rising_past_first_keys(lengths, hq, hkv, d, causal):
    """Keys 512-1023 of each segment scaled by 64 and keys from 1024 on by
    128 (exact in bf16): their logits rise 100-300 (natural units) above the
    first keys' maximum, so the forward must raise its exponent offset both
    where 2^(s c - m) overflows to inf and where it only grows large.  O and
    LSE against the oracle; V is halved (exact) because such peaked rows put
    O on single values of V, whose bf16 rounding alone would otherwise sit at
    the absolute tolerance.  (The gradients of such rows scale with the key
    norms, beyond the absolute tolerance, and take no part in this path.)"""
    import torch
    from paper_2511_13198_amd import pdyattn
    scale = 1.0 / math.sqrt(d)
    pu.log(f"  case lengths={lengths} Hq={hq} Hkv={hkv} d={d} causal={causal}")
    bits, cu = _host_case(lengths, hq, hkv, d)
    f = {n: wl.bf16_bits_to_f64(b) for n, b in bits.items()}
    k = f["k"].copy()
    for a, b in zip(cu[:-1], cu[1:]):
        k[a + 512:min(b, a + 1024)] *= 64.0
        k[a + 1024:b] *= 128.0
    vh = f["v"] * 0.5
    q = pu.to_device_bf16(bits["q"])
    kd = torch.from_numpy(k).to(torch.bfloat16).cuda()
    v = torch.from_numpy(vh).to(torch.bfloat16).cuda()
    assert np.array_equal(kd.double().cpu().numpy(), k), "scaling by powers of two stays exact"
    assert np.array_equal(v.double().cpu().numpy(), vh), "scaling by powers of two stays exact"
    cu_d = torch.from_numpy(cu).cuda()
    o = torch.full_like(q, float("nan"))
    lse = torch.full((hq, q.shape[0]), float("nan"), dtype=torch.float32, device="cuda")
    pdyattn.attn_fwd(q, kd, v, cu_d, max(lengths), causal, scale, out=o, lse=lse)
    torch.cuda.synchronize()
    ro, rlse = ora.forward(f["q"], k, vh, cu, causal, scale)
    assert np.max(rlse) > 100.0, "the inputs reach the large-logit regime"
    pu.check_close("O", pu.bf16_to_f64(o), ro)
    pu.check_close("LSE", lse.cpu().numpy(), rlse)


def _run_counted(dev, cu_d, max_seqlen, scale):
    """run_gpu, and whether any split-K combining kernel ran."""
    from paper_2511_13198_amd import pdyattn
    pdyattn.profile_start()
    out = pu.run_gpu(dev["q"], dev["k"], dev["v"], dev["do"], cu_d, max_seqlen, True, scale)
    prof = pdyattn.profile_stop()
    return out, any(k in prof for k in ("split_merge_kernel", "split_sum_kernel"))


def _same(a, b, exact, what):
    """Bitwise when both launches took the same path.  Otherwise (one of them
    split-K) within the parity tolerance: the forward's O may round to the
    neighbouring bf16 value, which moves D = rowsum(dO * O) and with it the
    gradients by about 1e-3 relative."""
    import torch
    if exact:
        assert torch.equal(a, b), f"{what} differs"
        return
    pu.check_close(what, a.double().cpu().numpy(), b.double().cpu().numpy())


@pytest.mark.parametrize("lengths,hq,hkv", [
    ([300, 129, 511], 4, 2),       # small: the lone segments run split-K
    ([4096, 6000, 4500], 64, 32),  # every launch fills the chip: bitwise throughout
])
def test_determinism_and_isolation(lengths, hq, hkv):
    """A second run gives the same bytes; a packed batch gives each segment
    what it gets alone (bitwise unless one of the two launches is split-K);
    future keys do not change earlier rows (bitwise, same launch)."""
    import torch
    d = 128
    T = sum(lengths)
    dev = wl.device_inputs(T, hq, hkv, d, seed=3)
    cu = wl.cu_from_lengths(lengths)
    cu_d = torch.from_numpy(cu).cuda()
    r1, split1 = _run_counted(dev, cu_d, max(lengths), 0.09)
    r2, _ = _run_counted(dev, cu_d, max(lengths), 0.09)
    for a, b in zip(r1, r2):
        assert torch.equal(a, b), "non-deterministic output"
    names = ("O", "LSE", "dQ", "dK", "dV")
    for si in range(len(lengths)):
        a, b = int(cu[si]), int(cu[si + 1])
        cu1 = torch.tensor([0, b - a], dtype=torch.int32, device="cuda")
        seg = {n: dev[n][a:b].contiguous() for n in ("q", "k", "v", "do")}
        alone, split_a = _run_counted(seg, cu1, b - a, 0.09)
        exact = not (split1 or split_a)
        if len(lengths) == 3 and lengths[0] == 4096:
            assert exact, "the large case is meant to run without split-K"
        _same(alone[0], r1[0][a:b], exact, f"segment {si}: O")
        _same(alone[1], r1[1][:, a:b], exact, f"segment {si}: LSE")
        for t in (2, 3, 4):
            _same(alone[t], r1[t][a:b], exact, f"segment {si}: {names[t]}")
    # causality: perturb everything after row i of the last segment
    a = int(cu[-2])
    i = a + 200
    q2, k2, v2 = (dev[n].clone() for n in ("q", "k", "v"))
    q2[i + 1:] = 3.0
    k2[i + 1:] = -2.0
    v2[i + 1:] = 7.0
    r3, _ = _run_counted({"q": q2, "k": k2, "v": v2, "do": dev["do"]}, cu_d, max(lengths), 0.09)
    assert torch.equal(r3[0][: i + 1], r1[0][: i + 1])
    assert torch.equal(r3[1][:, : i + 1], r1[1][:, : i + 1])
    assert torch.equal(r3[2][: i + 1], r1[2][: i + 1])


# ---------------------------------------------------------------------------
# Full-size workloads: sampled parity + invariants
# ---------------------------------------------------------------------------
def _sampled_parity(w: wl.Workload, device_gen: bool, heads, kv_heads, per_seg_random,
                    tail_cols, tail_segs=None, max_rows=None, expect_split=None,
                    invariants=True, max_plan_ms=None, max_seqlen=None):
    """expect_split: {"merge": n, "sum": m} -- the split-K combining kernels the
    forward + backward must launch; max_plan_ms: bound on the tile schedule's
    time per launch (both checked with the library's launch counters).
    invariants: the whole-tensor gradient identities (one pass per segment).
    max_seqlen: the bound passed to the library (default: the true maximum)."""
    import torch
    from paper_2511_13198_amd import pdyattn
    T, hq, hkv, d = w.total_tokens, w.heads_q, w.heads_kv, w.head_dim
    scale = w.softmax_scale
    pu.log(f"  workload {w.name}: T={T} N={w.num_seqs} Hq={hq} Hkv={hkv} d={d}")
    if device_gen:
        dev = wl.device_inputs(T, hq, hkv, d)
    else:
        bits = wl.host_inputs(T, hq, hkv, d)
        dev = {n: pu.to_device_bf16(b) for n, b in bits.items()}
    cu = w.cu_seqlens()
    cu_d = torch.from_numpy(cu).cuda()
    counted = expect_split is not None or max_plan_ms is not None
    if counted:
        pdyattn.profile_start()
    o, lse, dq, dk, dv = pu.run_gpu(dev["q"], dev["k"], dev["v"], dev["do"], cu_d,
                                    max_seqlen or w.max_seqlen, w.causal, scale)
    if counted:
        prof = pdyattn.profile_stop()
    if expect_split is not None:
        got = {"merge": prof.get("split_merge_kernel", (0, 0.0))[0],
               "sum": prof.get("split_sum_kernel", (0, 0.0))[0]}
        assert got == expect_split, f"split-K launches {got}, expected {expect_split}"
    if max_plan_ms is not None:
        launches, total_ms = prof["plan_kernel"]
        pu.log(f"  plan_kernel {total_ms / launches:.4f} ms per launch")
        assert total_ms / launches < max_plan_ms, f"plan {total_ms / launches:.3f} ms per launch"
    cu_list = [int(x) for x in cu]
    if invariants:
        pu.gpu_invariants(o, lse, dq, dk, dv, dev["q"], dev["k"], dev["v"], dev["do"], cu_list,
                          scale, w.causal)
    host = {n: pu.HeadView(t) for n, t in dev.items()}
    rows = pu.sample_rows(w.lengths, per_seg_random, max_rows=max_rows)
    res = ora.rows_forward_backward(host["q"], host["k"], host["v"], host["do"], cu, w.causal,
                                    scale, heads=heads, rows=rows)
    ridx = torch.tensor(rows, dtype=torch.long, device=o.device)
    got_o = np.concatenate([o[ridx, h].cpu().double().numpy() for h in heads])
    got_l = np.concatenate([lse[h, ridx].cpu().double().numpy() for h in heads])
    got_q = np.concatenate([dq[ridx, h].cpu().double().numpy() for h in heads])
    pu.check_close("O", got_o, np.concatenate([res[h][0] for h in heads]))
    pu.check_close("LSE", got_l, np.concatenate([res[h][1] for h in heads]))
    pu.check_close("dQ", got_q, np.concatenate([res[h][2] for h in heads]))
    segs = tail_segs if tail_segs is not None else [int(np.argmax(w.lengths))]
    gk, gv, rk, rv = [], [], [], []
    for si in segs:
        b = cu_list[si + 1]
        lo = max(cu_list[si], b - tail_cols)
        cols = ora.cols_backward(host["q"], host["k"], host["v"], host["do"], cu, w.causal, scale,
                                 kv_heads=kv_heads, seg_index=si, col_lo=lo)
        for hk in kv_heads:
            gk.append(dk[lo:b, hk].cpu().double().numpy())
            gv.append(dv[lo:b, hk].cpu().double().numpy())
            rk.append(cols[hk][0])
            rv.append(cols[hk][1])
    pu.check_close("dK", np.concatenate(gk), np.concatenate(rk))
    pu.check_close("dV", np.concatenate(gv), np.concatenate(rv))


def test_packed_65536_loguniform():
    w = wl.config(2)
    _sampled_parity(w, device_gen=False, heads=[0, 13, 31], kv_heads=[0, 31],
                    per_seg_random=8, tail_cols=256, tail_segs=[0, 7, 24])


def test_single_131072_h4():
    _sampled_parity(wl.config(3), device_gen=True, heads=[0, 3], kv_heads=[1, 2],
                    per_seg_random=96, tail_cols=128, expect_split={"merge": 0, "sum": 0})


# Launches too small to fill 256 CUs split each work item's inner loop into
# parts (split-K): forward and dQ by key tiles, dK/dV by query steps.  The
# expected combining launches follow from the sizes: one forward merge when
# the forward splits, one sum for whatever of dQ and dK/dV split.
@pytest.mark.parametrize("lengths,hq,hkv,d,expect", [
    ([8192], 4, 4, 128, {"merge": 1, "sum": 1}),        # forward, dQ and dK/dV in 4 parts
    ([16384], 8, 2, 128, {"merge": 0, "sum": 1}),       # only dK/dV (grouped heads) splits
    ([3000, 5000, 77], 2, 1, 64, {"merge": 1, "sum": 1}),  # packed, d = 64, 4 parts each
    ([16384], 8, 8, 64, {"merge": 0, "sum": 0}),        # fills the chip: no split
])
def test_split_k(lengths, hq, hkv, d, expect):
    w = wl.Workload(f"split_{len(lengths)}x{max(lengths)}_h{hq}kv{hkv}_d{d}", lengths, hq, hkv, d)
    _sampled_parity(w, device_gen=False, heads=[0, hq - 1], kv_heads=[0, hkv - 1],
                    per_seg_random=24, tail_cols=192, tail_segs=list(range(len(lengths))),
                    expect_split=expect)


# Causal single sequences too short to fill the chip take the balanced
# split when its workgroups fit one round on the chip: the heaviest items (the
# last query tiles, the first key tiles) are cut into more parts than light
# ones.  Every element against the oracle; the combining launches show that
# the split ran.
@pytest.mark.parametrize("lengths,hq,hkv,d,expect", [
    ([1024], 4, 4, 128, {"merge": 1, "sum": 1}),
    ([2048], 4, 4, 128, {"merge": 1, "sum": 1}),
    ([4096], 4, 4, 128, {"merge": 1, "sum": 1}),
    ([3000], 8, 2, 128, {"merge": 1, "sum": 1}),   # ragged tail, grouped heads (dK/dV balanced)
    ([1500], 2, 1, 64, {"merge": 1, "sum": 1}),    # d = 64
    ([2048], 32, 8, 128, {"merge": 0, "sum": 1}),  # dK/dV balanced, dQ uniform, forward whole
    ([2500], 6, 2, 128, {"merge": 1, "sum": 1}),   # three query heads per kv head
])
def test_balanced_split_full_parity(lengths, hq, hkv, d, expect):
    from paper_2511_13198_amd import pdyattn
    pdyattn.profile_start()
    _full_parity(lengths, hq, hkv, d, True)
    prof = pdyattn.profile_stop()
    got = {"merge": prof.get("split_merge_kernel", (0, 0.0))[0],
           "sum": prof.get("split_sum_kernel", (0, 0.0))[0]}
    assert got == expect, f"split-K launches {got}, expected {expect}"


@pytest.mark.parametrize("nseg,hi,hq,hkv,d", [
    (16384, 64, 2, 1, 64),    # every segment <= 2048 tokens: the 4-wave kernels
    (6000, 300, 4, 2, 128),   # same, d = 128
    (1000, 3000, 2, 1, 128),  # segments up to 3000 tokens: the 8-wave kernels
])
def test_many_segments(nseg, hi, hq, hkv, d):
    """Batches of a thousand or more segments (lengths uniform in 1..hi): the
    tile schedule is a counting sort, far below a millisecond per launch, and
    sampled rows and the tail key columns of three segments match the oracle."""
    rng = np.random.default_rng(7)
    lengths = [int(x) for x in rng.integers(1, hi + 1, size=nseg)]
    w = wl.Workload(f"many{nseg}x{hi}", lengths, hq, hkv, d)
    _sampled_parity(w, device_gen=True, heads=[0, hq - 1], kv_heads=[0, hkv - 1],
                    per_seg_random=0, tail_cols=hi, tail_segs=[0, nseg // 2, nseg - 1],
                    max_rows=512, invariants=False, max_plan_ms=0.5)


def test_single_65536_one_kv_head():
    """4 query heads on one kv head (one GPU's share of a 32/8-head model over
    8 GPUs): the dK/dV workgroups run in the XCD order for few kv heads.  Its
    256 key tiles of 256 keys (one per CU) split in two parts (one sum)."""
    w = wl.Workload("single65536_h4kv1", [65536], 4, 1, 128)
    _sampled_parity(w, device_gen=True, heads=[0, 3], kv_heads=[0], per_seg_random=48,
                    tail_cols=256, expect_split={"merge": 0, "sum": 1})


def test_single_65536_head_dim_64():
    """The d = 64 kernels on a long sequence (8 heads, 256 query tiles per
    head: no split), sampled rows and tail keys against the oracle plus the
    identities over every element."""
    w = wl.Workload("single65536_h8_d64", [65536], 8, 8, 64)
    _sampled_parity(w, device_gen=True, heads=[0, 7], kv_heads=[3], per_seg_random=48,
                    tail_cols=256, expect_split={"merge": 0, "sum": 0})


def test_plan_with_a_loose_length_bound():
    """max_seqlen only bounds the segment lengths: 1000 segments (about 800K
    tokens, one head) passed with max_seqlen = T give more tile counts than
    the schedule bins in LDS, so it bins in the workspace instead."""
    rng = np.random.default_rng(11)
    lengths = [int(x) for x in rng.integers(1, 1601, size=1000)]
    w = wl.Workload("loose_bound", lengths, 1, 1, 64)
    assert w.total_tokens // 128 > 6144
    _sampled_parity(w, device_gen=True, heads=[0], kv_heads=[0], per_seg_random=0,
                    tail_cols=128, tail_segs=[0, 500, 999], max_rows=384, invariants=False,
                    max_plan_ms=0.5, max_seqlen=w.total_tokens)


def test_single_638976_h4():
    _sampled_parity(wl.config(4), device_gen=True, heads=[1, 2], kv_heads=[0, 3],
                    per_seg_random=48, tail_cols=96, max_rows=96)


def _stream_cases():
    """Batches of the lognormal GQA stream checked against the oracle: every
    single-sequence batch but the longest (which has a test of its own), the
    most- and least-segmented packed batches, the packed batches with the
    longest and the shortest longest segment, and two more spread over the
    stream."""
    stream = wl.stream_config5()
    idx = range(len(stream))
    singles = [i for i in idx if stream[i].num_seqs == 1]
    longest = max(singles, key=lambda i: stream[i].max_seqlen)
    packed = [i for i in idx if stream[i].num_seqs > 1]
    picks = {max(packed, key=lambda i: stream[i].num_seqs),
             min(packed, key=lambda i: stream[i].num_seqs),
             max(packed, key=lambda i: stream[i].max_seqlen),
             min(packed, key=lambda i: stream[i].max_seqlen),
             packed[0], packed[len(packed) // 3], packed[2 * len(packed) // 3]}
    return sorted(set(singles) - {longest}) + sorted(picks)


@pytest.mark.parametrize("batch", _stream_cases())
def test_stream_batches_gqa(batch):
    w = wl.stream_config5()[batch]
    _sampled_parity(w, device_gen=True, heads=[0, 17, 31], kv_heads=[0, 7],
                    per_seg_random=4 if w.num_seqs > 1 else 32, tail_cols=64,
                    tail_segs=sorted({0, int(np.argmax(w.lengths)), w.num_seqs - 1}),
                    max_rows=64)


def test_stream_longest_batch_gqa():
    """The 638,976-token batch with 32 query and 8 kv heads: element offsets
    of q, o and dq pass 2**31."""
    stream = wl.stream_config5()
    i = max(range(len(stream)), key=lambda j: stream[j].max_seqlen)
    w = stream[i]
    assert w.total_tokens * w.heads_q * w.head_dim > 2 ** 31
    _sampled_parity(w, device_gen=True, heads=[0, 30], kv_heads=[0, 7], per_seg_random=16,
                    tail_cols=64, max_rows=48)
