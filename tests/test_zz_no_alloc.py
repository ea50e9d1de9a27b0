"""attn_bwd_noalloc (scratch in a static device array, no workspace) against
attn_bwd through the C-ABI, on three calls in a row with shrinking inputs:
bit for bit where both take the same path, within the parity tolerance where
the static scratch holds fewer split-K parts than attn_bwd's workspace."""
import math

import pytest

from paper_2511_13198_amd import workloads as wl
from tests import parity_util as pu

pytestmark = pytest.mark.gpu

CASES = [
    # (lengths, Hq, Hkv, d, same_path): the first splits its work into parts
    # whose partial gradients exceed the 64 MiB scratch, so it runs with fewer
    ([3000, 5000, 77], 4, 2, 128, False),
    # a causal single sequence: a balanced split whose partials exceed the
    # scratch, so its parts are halved (larger units per part)
    ([4096], 4, 4, 128, False),
    ([16384], 8, 8, 64, True),          # fills the chip: no split
    ([700, 1, 129], 2, 1, 64, True),    # split parts that fit
]


def test_noalloc_matches_attn_bwd_on_consecutive_calls():
    import torch
    from paper_2511_13198_amd import pdyattn
    for lengths, hq, hkv, d, same in CASES:
        T = sum(lengths)
        pu.log(f"  case lengths={lengths} Hq={hq} Hkv={hkv} d={d}")
        need = pdyattn.bwd_workspace_size(T, len(lengths), max(lengths), hq, hkv, d)
        assert (need <= 64 << 20) == same, f"workspace {need} bytes"
        dev = wl.device_inputs(T, hq, hkv, d, seed=5)
        cu = torch.from_numpy(wl.cu_from_lengths(lengths)).cuda()
        scale = 1.0 / math.sqrt(d)
        o, lse = pdyattn.attn_fwd(dev["q"], dev["k"], dev["v"], cu, max(lengths), True, scale)
        ref = pdyattn.attn_bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["do"], cu, max(lengths),
                               True, scale)
        outs = tuple(torch.full_like(t, float("nan")) for t in ref)
        got = pdyattn.attn_bwd_noalloc(dev["q"], dev["k"], dev["v"], o, lse, dev["do"], cu,
                                       max(lengths), True, scale, dq=outs[0], dk=outs[1],
                                       dv=outs[2])
        torch.cuda.synchronize()
        for name, g, r in zip(("dQ", "dK", "dV"), got, ref):
            pu.check_close(name, g.double().cpu().numpy(), r.double().cpu().numpy())
            if same:
                assert torch.equal(g, r), f"{name} differs from attn_bwd"
