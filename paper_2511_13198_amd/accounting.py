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


# Algorithmic FLOPs of each kernel: the matrix products of the method it
# accounts for, 2*d per visible pair each.  The dQ kernel's share of the
# gradient is the single product dQ = scale * dS K; it also recomputes S and
# dP (which the dK/dV kernel already formed), and those are issued work, not
# algorithmic work:
#   fwd_kernel      S, PV                -> 2 products (issued 2)
#   bwd_dkdv_kernel S, dP, dV, dK        -> 4 products (issued 4)
#   bwd_dq_kernel   dQ                   -> 1 product  (issued 3: S, dP, dQ)
KERNEL_PRODUCTS = {"fwd_kernel": 2, "bwd_dkdv_kernel": 4, "bwd_dq_kernel": 1}
ISSUED_PRODUCTS = {"fwd_kernel": 2, "bwd_dkdv_kernel": 4, "bwd_dq_kernel": 3}


def kernel_flops(kernel: str, lengths, heads_q, head_dim, causal=True) -> float:
    """Algorithmic FLOPs of one launch of `kernel` (visible pairs only)."""
    return KERNEL_PRODUCTS[kernel] * 2.0 * head_dim * heads_q * pairs_per_head(lengths, causal)


def kernel_issued_flops(kernel: str, lengths, heads_q, head_dim, causal=True) -> float:
    """Matrix-product FLOPs the kernel issues on visible pairs, recomputation
    included (masked halves of diagonal tiles still not counted)."""
    return ISSUED_PRODUCTS[kernel] * 2.0 * head_dim * heads_q * pairs_per_head(lengths, causal)


def fwd_bytes(total_tokens, heads_q, heads_kv, head_dim) -> float:
    """Compulsory HBM traffic of the forward: read Q, K, V; write O (bf16) and LSE."""
    return 2.0 * total_tokens * head_dim * (2 * heads_q + 2 * heads_kv) + 4.0 * total_tokens * heads_q


def bwd_bytes(total_tokens, heads_q, heads_kv, head_dim) -> float:
    """Compulsory HBM traffic of the backward: read Q, K, V, O, dO (bf16), LSE;
    write dQ, dK, dV (fp32) and D (fp32, written and read once)."""
    T, d = total_tokens, head_dim
    return (2.0 * T * d * (3 * heads_q + 2 * heads_kv) + 4.0 * T * d * (heads_q + 2 * heads_kv)
            + 12.0 * T * heads_q)
