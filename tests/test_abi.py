"""The C-ABI library loads without a GPU, exports every function the header
declares, and rejects bad arguments before touching HIP."""
import ctypes
import os
import re

import pytest

from paper_2511_13198_amd import pdyattn as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pdyattn.h")

FAKE = 0x10000  # aligned, never dereferenced: every call below fails validation first


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", text)) - {"defined"})


def test_header_symbols_exported():
    names = header_functions()
    assert "attn_fwd" in names and "attn_bwd" in names
    L = P.lib()
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, f"missing exports: {missing}"
    assert sorted(P.SYMBOLS) == names


def _fwd(**kw):
    args = dict(q=FAKE, k=FAKE, v=FAKE, cu=FAKE, n=1, T=512, maxlen=512, hq=8, hkv=8, d=128,
                causal=1, scale=0.1, o=FAKE, lse=FAKE, ws=FAKE, wsb=1 << 20, stream=None)
    args.update(kw)
    return P.lib().attn_fwd(args["q"], args["k"], args["v"], args["cu"], args["n"], args["T"],
                            args["maxlen"], args["hq"], args["hkv"], args["d"], args["causal"],
                            args["scale"], args["o"], args["lse"], args["ws"], args["wsb"],
                            args["stream"])


def _bwd(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=FAKE, do=FAKE, cu=FAKE, n=1, T=512, maxlen=512,
             hq=8, hkv=8, d=128, causal=1, scale=0.1, dq=FAKE, dk=FAKE, dv=FAKE, ws=FAKE,
             wsb=1 << 30, stream=None)
    a.update(kw)
    return P.lib().attn_bwd(a["q"], a["k"], a["v"], a["o"], a["lse"], a["do"], a["cu"], a["n"],
                            a["T"], a["maxlen"], a["hq"], a["hkv"], a["d"], a["causal"],
                            a["scale"], a["dq"], a["dk"], a["dv"], a["ws"], a["wsb"],
                            a["stream"])


@pytest.mark.parametrize("kw,status,msg", [
    (dict(d=96), P.PDY_ERR_UNSUPPORTED, "head_dim"),
    (dict(hq=6, hkv=4), P.PDY_ERR_INVALID_ARG, "multiple"),
    (dict(hkv=0), P.PDY_ERR_INVALID_ARG, "head counts"),
    (dict(n=0), P.PDY_ERR_INVALID_ARG, "num_seqs"),
    (dict(T=-1), P.PDY_ERR_INVALID_ARG, "total_tokens"),
    (dict(maxlen=513), P.PDY_ERR_INVALID_ARG, "max_seqlen"),
    (dict(maxlen=0), P.PDY_ERR_INVALID_ARG, "max_seqlen"),
    # one segment is [0, T): a smaller bound would leave rows unwritten
    (dict(maxlen=500), P.PDY_ERR_INVALID_ARG, "num_seqs = 1"),
    (dict(causal=2), P.PDY_ERR_INVALID_ARG, "causal"),
    (dict(scale=0.0), P.PDY_ERR_INVALID_ARG, "scale"),
    (dict(scale=float("nan")), P.PDY_ERR_INVALID_ARG, "scale"),
    (dict(q=0), P.PDY_ERR_INVALID_ARG, "q is NULL"),
    (dict(o=FAKE + 8), P.PDY_ERR_INVALID_ARG, "aligned"),
    (dict(cu=0), P.PDY_ERR_INVALID_ARG, "cu_seqlens"),
    (dict(cu=FAKE + 2), P.PDY_ERR_INVALID_ARG, "cu_seqlens"),
    (dict(wsb=16), P.PDY_ERR_WORKSPACE, "workspace"),
])
def test_fwd_argument_errors(kw, status, msg):
    st = _fwd(**kw)
    assert st == status, (st, P.last_error())
    assert msg in P.last_error()


@pytest.mark.parametrize("kw,status,msg", [
    (dict(d=32), P.PDY_ERR_UNSUPPORTED, "head_dim"),
    (dict(dk=0), P.PDY_ERR_INVALID_ARG, "dk is NULL"),
    (dict(do=FAKE + 4), P.PDY_ERR_INVALID_ARG, "aligned"),
    (dict(wsb=1024), P.PDY_ERR_WORKSPACE, "workspace"),
    (dict(hq=32, hkv=5), P.PDY_ERR_INVALID_ARG, "multiple"),
    (dict(maxlen=1), P.PDY_ERR_INVALID_ARG, "num_seqs = 1"),
])
def test_bwd_argument_errors(kw, status, msg):
    st = _bwd(**kw)
    assert st == status, (st, P.last_error())
    assert msg in P.last_error()


def test_empty_batch_is_noop():
    # T = 0 returns before any pointer check or launch
    assert _fwd(T=0, maxlen=0, q=0, k=0, v=0, o=0, lse=0, ws=0, wsb=0) == P.PDY_OK
    assert _bwd(T=0, maxlen=0, q=0) == P.PDY_OK


def test_workspace_sizes():
    f = P.fwd_workspace_size(65536, 25, 7402, 32, 32, 128)
    b = P.bwd_workspace_size(65536, 25, 7402, 32, 32, 128)
    assert 256 <= f < 1 << 20
    assert b >= 32 * 65536 * 4  # D = rowsum(dO*O), fp32 [Hq, T]
    assert P.fwd_workspace_size(512, 1, 512, 8, 8, 96) == 0
    assert P.bwd_workspace_size(512, 1, 513, 8, 8, 128) == 0


MiB = 1 << 20


def test_split_k_workspace():
    """Launches too small to fill the chip split their work (split-K) and need
    fp32 partial buffers; the size queries make the same decision as the
    calls.  8192 tokens x 4 heads: forward, dQ and dK/dV in 4 parts."""
    part_o = 4 * 8192 * 4 * 128 * 4
    assert P.fwd_workspace_size(8192, 1, 8192, 4, 4, 128) >= part_o + 4 * 4 * 8192 * 4
    assert P.bwd_workspace_size(8192, 1, 8192, 4, 4, 128) >= 2 * (4 * 8192 * 4 * 128 * 4) + part_o
    # grouped heads at 16K: only dK/dV (2 kv heads: 128 key tiles) splits, in
    # 4 parts per key tile (not causal) or a balanced split of at most 16
    # partial slices (causal; the size query covers both)
    b = P.bwd_workspace_size(16384, 1, 16384, 8, 2, 128)
    slice_kv = 2 * 16384 * 2 * 128 * 4
    assert 4 * slice_kv <= b < 16 * slice_kv + 2 * MiB
    # launches that fill the chip need no partial buffers
    assert P.fwd_workspace_size(131072, 1, 131072, 4, 4, 128) < MiB
    assert P.bwd_workspace_size(16384, 1, 16384, 8, 8, 64) < 2 * MiB
    # segments of at most 128 tokens leave nothing to split
    assert P.fwd_workspace_size(1024, 8, 128, 1, 1, 64) < MiB
    # context-parallel pair calls never split
    assert P.fwd_chunk_workspace_size(8192, 8192, 4, 4, 128) < MiB


def test_status_strings_and_kernel_names():
    L = P.lib()
    assert L.pdy_status_string(0) == b"ok"
    assert L.pdy_status_string(-3) == b"workspace too small"
    names = [L.pdy_kernel_name(i).decode() for i in range(L.pdy_kernel_count())]
    assert {"fwd_kernel", "bwd_dkdv_kernel", "bwd_dq_kernel", "split_merge_kernel",
            "split_sum_kernel"} <= set(names)
    # profiling with nothing launched reports nothing
    P.profile_start()
    assert P.profile_stop() == {}


def _fwd_chunk(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, tq=256, tk=256, qo=0, ko=0, hq=4, hkv=2, d=128, causal=1,
             scale=0.1, o=FAKE, lse=FAKE, ws=FAKE, wsb=1 << 20, stream=None)
    a.update(kw)
    return P.lib().attn_fwd_chunk(a["q"], a["k"], a["v"], a["tq"], a["tk"], a["qo"], a["ko"],
                                  a["hq"], a["hkv"], a["d"], a["causal"], a["scale"], a["o"],
                                  a["lse"], a["ws"], a["wsb"], a["stream"])


def _bwd_chunk(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=FAKE, do=FAKE, tq=256, tk=256, qo=0, ko=0, hq=4,
             hkv=2, d=128, causal=1, scale=0.1, dq=FAKE, dk=FAKE, dv=FAKE, acc=0, ws=FAKE,
             wsb=1 << 30, stream=None)
    a.update(kw)
    return P.lib().attn_bwd_chunk(a["q"], a["k"], a["v"], a["o"], a["lse"], a["do"], a["tq"],
                                  a["tk"], a["qo"], a["ko"], a["hq"], a["hkv"], a["d"],
                                  a["causal"], a["scale"], a["dq"], a["dk"], a["dv"], a["acc"],
                                  a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status,msg", [
    (dict(tq=-1), P.PDY_ERR_INVALID_ARG, "chunk lengths"),
    (dict(ko=-5), P.PDY_ERR_INVALID_ARG, "offsets"),
    (dict(d=96), P.PDY_ERR_UNSUPPORTED, "head_dim"),
    (dict(hq=6, hkv=4), P.PDY_ERR_INVALID_ARG, "multiple"),
    (dict(scale=-1.0), P.PDY_ERR_INVALID_ARG, "scale"),
    (dict(o=0), P.PDY_ERR_INVALID_ARG, "o is NULL"),
    (dict(k=0), P.PDY_ERR_INVALID_ARG, "k is NULL"),
    (dict(wsb=8), P.PDY_ERR_WORKSPACE, "attn_fwd_chunk"),
])
def test_fwd_chunk_argument_errors(kw, status, msg):
    st = _fwd_chunk(**kw)
    assert st == status, (st, P.last_error())
    assert msg in P.last_error()


@pytest.mark.parametrize("kw,status,msg", [
    (dict(tk=-1), P.PDY_ERR_INVALID_ARG, "chunk lengths"),
    (dict(qo=-1), P.PDY_ERR_INVALID_ARG, "offsets"),
    (dict(dv=0), P.PDY_ERR_INVALID_ARG, "dv is NULL"),
    (dict(lse=FAKE + 4), P.PDY_ERR_INVALID_ARG, "aligned"),
    (dict(wsb=64), P.PDY_ERR_WORKSPACE, "attn_bwd_chunk"),
    (dict(acc=2), P.PDY_ERR_INVALID_ARG, "accumulate"),
])
def test_bwd_chunk_argument_errors(kw, status, msg):
    st = _bwd_chunk(**kw)
    assert st == status, (st, P.last_error())
    assert msg in P.last_error()


def test_workspace_bounds_over_a_size_sweep():
    """The header's bounds on the split-K workspaces (forward under 129 MiB,
    backward under 384 MiB) over single sequences and packed batches of the
    sizes that split (the largest: two parts of a 130,816-token sequence)."""
    worst_f = worst_b = 0
    for d in (64, 128):
        for hq, hkv in ((1, 1), (2, 1), (4, 4), (6, 2), (8, 2), (32, 8)):
            for T in list(range(64, 8192, 448)) + list(range(8192, 131073, 4096)) + [130816]:
                for n in (1, 3):
                    maxlen = T if n == 1 else (T + n - 1) // n
                    worst_f = max(worst_f, P.fwd_workspace_size(T, n, maxlen, hq, hkv, d))
                    worst_b = max(worst_b, P.bwd_workspace_size(T, n, maxlen, hq, hkv, d))
    assert 128 * MiB < worst_f < 129 * MiB
    assert 383 * MiB < worst_b < 384 * MiB


def test_chunk_noops_and_workspace_sizes():
    # no query rows: nothing to do (k and v may be absent)
    assert _fwd_chunk(tq=0, q=0, k=0, v=0, o=0, lse=0, ws=0, wsb=0) == P.PDY_OK
    assert _bwd_chunk(tq=0, tk=0, q=0, k=0, v=0, o=0, lse=0, do=0, dq=0, dk=0, dv=0, ws=0,
                      wsb=0) == P.PDY_OK
    # a pair that fills the chip needs only the schedule (and D for the backward)
    f = P.fwd_chunk_workspace_size(32768, 65536, 32, 8, 128)
    b = P.bwd_chunk_workspace_size(32768, 65536, 32, 8, 128)
    assert 256 <= f < 1 << 20 and 32 * 32768 * 4 <= b < 32 * 32768 * 4 + (1 << 20)
    assert P.fwd_chunk_workspace_size(-1, 5, 4, 4, 128) == 0
    L = P.lib()
    assert L.attn_merge(FAKE, FAKE, FAKE, FAKE, 10, 4, 96, FAKE, FAKE, None) == P.PDY_ERR_UNSUPPORTED
    assert L.attn_merge(FAKE, FAKE, FAKE, FAKE, 0, 4, 128, 0, 0, None) == P.PDY_OK
    assert L.attn_merge(FAKE, 0, FAKE, FAKE, 10, 4, 128, FAKE, FAKE, None) == P.PDY_ERR_INVALID_ARG


def _bwd_noalloc(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=FAKE, do=FAKE, cu=FAKE, n=1, T=512, maxlen=512,
             hq=8, hkv=8, d=128, causal=1, scale=0.1, dq=FAKE, dk=FAKE, dv=FAKE, stream=None)
    a.update(kw)
    return P.lib().attn_bwd_noalloc(a["q"], a["k"], a["v"], a["o"], a["lse"], a["do"], a["cu"],
                                    a["n"], a["T"], a["maxlen"], a["hq"], a["hkv"], a["d"],
                                    a["causal"], a["scale"], a["dq"], a["dk"], a["dv"],
                                    a["stream"])


@pytest.mark.parametrize("kw,status,msg", [
    (dict(dq=0), P.PDY_ERR_INVALID_ARG, "dq is NULL"),
    (dict(maxlen=511), P.PDY_ERR_INVALID_ARG, "num_seqs = 1"),
    (dict(d=80), P.PDY_ERR_UNSUPPORTED, "head_dim"),
    # D alone (fp32 [Hq, T]) is 64 MiB here: beyond the static scratch
    (dict(T=1 << 20, maxlen=1 << 20, hq=16, hkv=4), P.PDY_ERR_WORKSPACE, "static scratch"),
])
def test_bwd_noalloc_argument_errors(kw, status, msg):
    st = _bwd_noalloc(**kw)
    assert st == status, (st, P.last_error())
    assert msg in P.last_error()


def test_bwd_noalloc_empty_batch_is_noop():
    assert _bwd_noalloc(T=0, maxlen=0, q=0, dq=0) == P.PDY_OK
