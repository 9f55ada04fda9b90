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


# --------------------------------------------------------------------------
# executed (tile-padded) work of the kernels as launched
# --------------------------------------------------------------------------

def _tiles(n: int, t: int) -> int:
    return -(-n // t) * t


def gemm_executed(M: int, N: int, K: int, store_small: bool = False, nseg: int = 1) -> int:
    """MFMA flops a GEMM launch executes: M and N rounded up to the workgroup
    tile (256 x 256; 128 x 128 for store-epilogue problems with fewer than
    128 of the big tiles), K as given (already padded by the plan)."""
    big = -(-M // 256) * -(-N // 256) * nseg
    t = 128 if (store_small and big < 128) else 256
    return 2 * _tiles(M, t) * _tiles(N, t) * nseg * K


def attention_executed(Lq: int, Lk: int, dh: int, h: int, B: int = 1, waves: int = 8) -> int:
    """MFMA flops of one attention launch: queries in blocks of 32 * waves,
    keys in tiles of 64 (masked keys are computed, then discarded)."""
    return B * 4 * dh * h * _tiles(Lq, 32 * waves) * _tiles(Lk, 64)


def block_executed_terms(L: int, Lc: int, D: int, dh: int, h: int, hc: int, f_pad: int,
                         B: int = 1) -> dict:
    """Executed MFMA flops of one block (compact plan, bf16): the contractions
    of block_terms with the FFN at its padded width f_pad and every launch
    rounded to its tiles."""
    a, ac = h * dh, hc * dh
    M, Mc = B * L, B * Lc
    long_keys = L >= 4096
    return {
        "qkv": gemm_executed(M, 3 * a, D, store_small=True) if a else 0,
        "self_attn": attention_executed(L, L, dh, h, B, 8 if long_keys else 4),
        "self_out": gemm_executed(M, D, a),
        "cross_q": gemm_executed(M, ac, D, store_small=True) if ac else 0,
        "cross_kv": gemm_executed(Mc, 2 * ac, D, store_small=True) if ac else 0,
        "cross_attn": attention_executed(L, Lc, dh, hc, B, 4),
        "cross_out": gemm_executed(M, D, ac),
        "ffn": (gemm_executed(M, f_pad, D) + gemm_executed(M, D, f_pad)) if f_pad else 0,
    }
