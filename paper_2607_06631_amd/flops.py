"""Algorithmic FLOP and byte accounting for the pruned block stack.

The paper never defines "FLOPs" (it reports per-step FLOP removal in the
abstract and Sec. 5.4 and per-step retention in Sec. 6).  Convention used
here: 2 flops per multiply-accumulate over every GEMM plus the QK^T and PV
products of both attentions; softmax, norms, elementwise work and the
patch-embed / output head are not counted.  Kept counts are exact (not
padded to tiles).
"""
from __future__ import annotations


def gemm_flops(M: int, N: int, K: int) -> int:
    return 2 * M * N * K


def block_terms(L: int, Lc: int, D: int, dh: int, h: int, hc: int, f: int, B: int = 1) -> dict:
    """FLOPs of each contraction in one block, for B samples."""
    a, ac = h * dh, hc * dh
    t = {
        "qkv": 2 * L * D * 3 * a,
        "self_attn": 4 * L * L * dh * h,
        "self_out": 2 * L * a * D,
        "cross_q": 2 * L * D * ac,
        "cross_kv": 4 * Lc * D * ac,
        "cross_attn": 4 * L * Lc * dh * hc,
        "cross_out": 2 * L * ac * D,
        "ffn": 4 * L * D * f,
    }
    return {k: B * v for k, v in t.items()}


def block_flops(L, Lc, D, dh, h, hc, f, B: int = 1) -> int:
    return sum(block_terms(L, Lc, D, dh, h, hc, f, B).values())


def structure_flops(L, Lc, D, dh, heads, cross_heads, ffn, block_keep=None, B: int = 1) -> int:
    """FLOPs of one step structure: per-layer kept counts (sequences)."""
    n = len(heads)
    keep = [1] * n if block_keep is None else block_keep
    return sum(block_flops(L, Lc, D, dh, heads[l], cross_heads[l], ffn[l], B)
               for l in range(n) if keep[l])


def self_attn_flops(L: int, dh: int, h: int, B: int = 1) -> int:
    return B * 4 * L * L * dh * h


def exp_count(L: int, Lk: int, h: int, B: int = 1) -> int:
    """Softmax exponentials of one attention call."""
    return B * L * Lk * h
