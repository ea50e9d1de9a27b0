"""Forward + backward captured in a HIP graph (torch.cuda.CUDAGraph) through
the C-ABI: every replay gives exactly the eager results.  The library records
no memset or allocation into the graph (its scratch is the caller's
workspace, or the static array of attn_bwd_noalloc), so replays are plain
kernel launches.  Each replay starts from outputs poisoned with NaN by eager
work outside the graph, with other eager attention calls and synchronisations
in between, as a serving loop would have them."""
import math

import pytest

from paper_2511_13198_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("lengths,hq,hkv,d,noalloc", [
    ([300, 1000, 2048, 77], 4, 2, 128, False),  # packed: tile schedules in the workspace
    ([8192], 4, 4, 128, False),                 # split-K partials and their sums
    ([3000, 5000, 77], 2, 1, 64, True),         # the allocation-free backward
])
def test_graph_replays_match_eager(lengths, hq, hkv, d, noalloc):
    import torch
    from paper_2511_13198_amd import pdyattn
    T, n, ml = sum(lengths), len(lengths), max(lengths)
    scale = 1.0 / math.sqrt(d)
    dev = wl.device_inputs(T, hq, hkv, d, seed=9)
    other = wl.device_inputs(T, hq, hkv, d, seed=10)
    cu = torch.from_numpy(wl.cu_from_lengths(lengths)).cuda()
    q, k, v, do = dev["q"], dev["k"], dev["v"], dev["do"]
    wsf = torch.empty(max(256, pdyattn.fwd_workspace_size(T, n, ml, hq, hkv, d)),
                      dtype=torch.uint8, device="cuda")
    wsb = torch.empty(max(256, pdyattn.bwd_workspace_size(T, n, ml, hq, hkv, d)),
                      dtype=torch.uint8, device="cuda")
    o = torch.empty_like(q)
    lse = torch.empty((hq, T), dtype=torch.float32, device="cuda")
    dq = torch.empty((T, hq, d), dtype=torch.float32, device="cuda")
    dk = torch.empty((T, hkv, d), dtype=torch.float32, device="cuda")
    dv = torch.empty_like(dk)

    def step():
        pdyattn.attn_fwd(q, k, v, cu, ml, True, scale, out=o, lse=lse, workspace=wsf)
        if noalloc:
            pdyattn.attn_bwd_noalloc(q, k, v, o, lse, do, cu, ml, True, scale, dq=dq, dk=dk,
                                     dv=dv)
        else:
            pdyattn.attn_bwd(q, k, v, o, lse, do, cu, ml, True, scale, dq=dq, dk=dk, dv=dv,
                             workspace=wsb)

    # eager reference (also the first call of every entry point, outside capture)
    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (o, lse, dq, dk, dv)]

    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()  # warm the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for rep in range(4):
        for t in (o, lse, dq, dk, dv):
            t.fill_(float("nan"))
        # unrelated eager attention calls between the replays
        pdyattn.attn_fwd(other["q"], other["k"], other["v"], cu, ml, True, scale)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, got, want in zip(("O", "LSE", "dQ", "dK", "dV"), (o, lse, dq, dk, dv), ref):
            assert torch.equal(got, want), f"replay {rep}: {name} differs from the eager result"
