"""Seeded synthetic workloads for packed variable-length causal attention.

This module only *draws* inputs: segment lengths, the packed-offset array and
N(0,1) activations rounded to bf16.  It holds none of the attention arithmetic,
so both the fp64 oracle (test infrastructure) and the HIP path can consume the
very same bytes.

Shapes follow the paper's workloads:
  * head shapes from the LLM configuration table (Table 4, section 5.1):
    BERT h=1024/n=16 -> d=64, LLaMA 8192/64 -> d=128, GPT 12288/96 -> d=128;
  * length distributions shaped after the dataset table (Table 3, section 5.1):
    long-tailed, with maxima of 309K (GitHubCode) and 624K (GRCh38) tokens;
  * the activation layout b x s/p x h of the tensor-layout specification
    (Table 2, section 4.2) packed as [T, H, d] with int32 segment offsets.
The datasets themselves are not used: token values do not change attention
cost, so N(0,1) activations stand in for them.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

SEED = 42                 # the only seed the paper states (section 5.1)
MAX_TOKENS_624K = 624 * 1024  # "624K" read as 624 * 1024 = 638,976 tokens
PACKED_BATCH_TOKENS = 256 * 1024


# ---------------------------------------------------------------------------
# bf16 helpers (pure bit manipulation, round-to-nearest-even)
# ---------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (RNE) and return the raw uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bits to float64."""
    u = np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32)


# ---------------------------------------------------------------------------
# Segment-length recipes
# ---------------------------------------------------------------------------
def cu_from_lengths(lengths: Sequence[int]) -> np.ndarray:
    """Packed offsets: cu[0] = 0, cu[i+1] = cu[i] + lengths[i] (int32)."""
    cu = np.zeros(len(lengths) + 1, dtype=np.int64)
    cu[1:] = np.cumsum(np.asarray(lengths, dtype=np.int64))
    if cu[-1] >= 2 ** 31:
        raise ValueError("total tokens exceed int32")
    return cu.astype(np.int32)


def loguniform_lengths(total: int = 65536, lo: int = 128, hi: int = 8192,
                       seed: int = SEED) -> List[int]:
    """Lengths s = round(exp(U(ln lo, ln hi))) drawn until the running total
    would exceed `total`; the last one is truncated to the remainder."""
    rng = np.random.default_rng(seed)
    out: List[int] = []
    used = 0
    while used < total:
        s = int(round(math.exp(rng.uniform(math.log(lo), math.log(hi)))))
        s = min(s, total - used)
        out.append(s)
        used += s
    return out


def lognormal_stream(n_batches: int = 64, median: int = 4096, sigma: float = 1.6,
                     lo: int = 64, hi: int = MAX_TOKENS_624K,
                     batch_tokens: int = PACKED_BATCH_TOKENS,
                     seed: int = SEED) -> List[List[int]]:
    """Dynamic stream of mini-batches with long-tailed lengths.

    Draws s = clip(round(exp(N(ln median, sigma))), lo, hi) one at a time.  A
    draw of at least `batch_tokens` becomes a batch of its own.  Shorter draws
    are packed greedily; the draw that overflows `batch_tokens` is truncated
    to fit and closes the batch.  sigma = 1.6 puts about 1.5% of draws at
    >= 128K, between the two datasets' long-tail fractions (Table 3).
    """
    rng = np.random.default_rng(seed)
    batches: List[List[int]] = []
    cur: List[int] = []
    used = 0
    while len(batches) < n_batches:
        s = int(round(math.exp(rng.normal(math.log(median), sigma))))
        s = max(lo, min(hi, s))
        if s >= batch_tokens:
            batches.append([s])
            continue
        if used + s >= batch_tokens:
            cur.append(batch_tokens - used)
            batches.append(cur)
            cur, used = [], 0
        else:
            cur.append(s)
            used += s
    return batches[:n_batches]


# ---------------------------------------------------------------------------
# Workload configurations
# ---------------------------------------------------------------------------
@dataclass
class Workload:
    name: str
    lengths: List[int]
    heads_q: int
    heads_kv: int
    head_dim: int
    causal: bool = True
    scale: Optional[float] = None
    extra: dict = field(default_factory=dict)

    @property
    def total_tokens(self) -> int:
        return int(sum(self.lengths))

    @property
    def num_seqs(self) -> int:
        return len(self.lengths)

    @property
    def max_seqlen(self) -> int:
        return int(max(self.lengths)) if self.lengths else 0

    @property
    def softmax_scale(self) -> float:
        return self.scale if self.scale is not None else 1.0 / math.sqrt(self.head_dim)

    def cu_seqlens(self) -> np.ndarray:
        return cu_from_lengths(self.lengths)


def config(n: int) -> Workload:
    """The five synthetic workloads (index 1..5)."""
    if n == 1:
        return Workload("single512_h8_d64", [512], 8, 8, 64, True, 1.0 / 8.0)
    if n == 2:
        return Workload("packed65536_loguniform128-8192_h32_d128",
                        loguniform_lengths(), 32, 32, 128, True)
    if n == 3:
        return Workload("single131072_h4_d128", [131072], 4, 4, 128, True)
    if n == 4:
        return Workload("single638976_h4_d128", [MAX_TOKENS_624K], 4, 4, 128, True)
    if n == 5:
        raise ValueError("config 5 is a stream; use stream_config5()")
    raise ValueError(f"unknown config {n}")


def stream_config5(n_batches: int = 64) -> List[Workload]:
    return [Workload(f"stream5_batch{i:02d}", b, 32, 8, 128, True)
            for i, b in enumerate(lognormal_stream(n_batches))]


# ---------------------------------------------------------------------------
# Activations
# ---------------------------------------------------------------------------
def host_inputs(total_tokens: int, heads_q: int, heads_kv: int, head_dim: int,
                seed: int = SEED, with_grad: bool = True) -> dict:
    """N(0,1) float32 from default_rng(seed) in the order q, k, v, dO, each
    rounded to bf16 (RNE).  Returns uint16 bit arrays of shape [T, H, d]."""
    rng = np.random.default_rng(seed)
    shapes = [("q", heads_q), ("k", heads_kv), ("v", heads_kv)]
    if with_grad:
        shapes.append(("do", heads_q))
    out = {}
    for name, h in shapes:
        x = rng.standard_normal((total_tokens, h, head_dim), dtype=np.float32)
        out[name] = f32_to_bf16_bits(x)
    return out


def device_inputs(total_tokens: int, heads_q: int, heads_kv: int, head_dim: int,
                  seed: int = SEED, device: str = "cuda", with_grad: bool = True) -> dict:
    """Same recipe on the device (torch's Philox generator seeded with
    `seed`), for workloads too large to draw quickly on the host.  Values are
    N(0,1) drawn in float32 and rounded to bf16.  Returns torch bf16 tensors."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    shapes = [("q", heads_q), ("k", heads_kv), ("v", heads_kv)]
    if with_grad:
        shapes.append(("do", heads_q))
    out = {}
    for name, h in shapes:
        x = torch.empty((total_tokens, h, head_dim), dtype=torch.bfloat16, device=device)
        # draw in float32 chunks to bound the transient footprint
        step = max(1, (1 << 26) // max(1, h * head_dim))
        for t0 in range(0, total_tokens, step):
            t1 = min(total_tokens, t0 + step)
            x[t0:t1] = torch.randn((t1 - t0, h, head_dim), generator=g,
                                   dtype=torch.float32, device=device).to(torch.bfloat16)
        out[name] = x
    return out
