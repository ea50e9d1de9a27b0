"""Work accounting for packed attention: pair counts, counted FLOPs and
compulsory HBM bytes.

Counted FLOPs follow the usual convention for fused attention kernels: per
visible (query, key) pair and query head, 2*d multiply-adds per matrix
product.  The forward has two products (Q K^T and P V): 4*d per pair.  The
backward has five (S recomputed, dV, dP, dK, dQ): 10*d per pair, i.e. 2.5x
the forward; fwd+bwd = 3.5x forward = 14*d per pair.  Masked-out halves of
diagonal tiles and any extra recomputation are not counted.

Peak figures are AMD's published dense MI355X numbers.
"""
from __future__ import annotations

from typing import Sequence

PEAK_BF16_TFLOPS = 2516.6      # dense bf16 MFMA, 256 CUs x 2.4 GHz x 4096 FLOP/clk
PEAK_HBM_GBPS = 8000.0         # HBM3E


def pairs_per_head(lengths: Sequence[int], causal: bool = True) -> int:
    if causal:
        return int(sum(s * (s + 1) // 2 for s in lengths))
    return int(sum(s * s for s in lengths))


def fwd_flops(lengths, heads_q, head_dim, causal=True) -> float:
    return 4.0 * head_dim * heads_q * pairs_per_head(lengths, causal)


def bwd_flops(lengths, heads_q, head_dim, causal=True) -> float:
    return 2.5 * fwd_flops(lengths, heads_q, head_dim, causal)


def fwd_bwd_flops(lengths, heads_q, head_dim, causal=True) -> float:
    return 3.5 * fwd_flops(lengths, heads_q, head_dim, causal)


# Algorithmic FLOPs of each kernel of the library (matrix products it is
# required to perform per visible pair, 2*d each):
#   fwd_kernel      S, PV                -> 2 products
#   bwd_dkdv_kernel S, dP, dV, dK        -> 4 products
#   bwd_dq_kernel   S, dP, dQ            -> 3 products (S and dP recomputed)
KERNEL_PRODUCTS = {"fwd_kernel": 2, "bwd_dkdv_kernel": 4, "bwd_dq_kernel": 3}


def kernel_flops(kernel: str, lengths, heads_q, head_dim, causal=True) -> float:
    return KERNEL_PRODUCTS[kernel] * 2.0 * head_dim * heads_q * pairs_per_head(lengths, causal)


def fwd_bytes(total_tokens, heads_q, heads_kv, head_dim) -> float:
    """Compulsory HBM traffic of the forward: read Q, K, V; write O (bf16) and LSE."""
    return 2.0 * total_tokens * head_dim * (2 * heads_q + 2 * heads_kv) + 4.0 * total_tokens * heads_q


def bwd_bytes(total_tokens, heads_q, heads_kv, head_dim) -> float:
    """Compulsory HBM traffic of the backward: read Q, K, V, O, dO (bf16), LSE;
    write dQ, dK, dV (fp32) and D (fp32, written and read once)."""
    T, d = total_tokens, head_dim
    return (2.0 * T * d * (3 * heads_q + 2 * heads_kv) + 4.0 * T * d * (heads_q + 2 * heads_kv)
            + 12.0 * T * heads_q)
