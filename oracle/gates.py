"""Oracle: hard gates from continuous masks, and the FFN channel reorder.

TEST INFRASTRUCTURE (see the package header).

Sec. 4.1 ("Unifying Step Reduction and Dynamic Sparsification") maps the
continuous masks m of one step to binary gates g per granularity:
  * block:  g = 1 if m > 0
  * head:   a head of D_head features is kept if the mean of its D_head
            mask values is > 0
  * FFN:    the hidden channels form consecutive chunks of C; one scalar mask
            per chunk, g = 1(m > 0) repeated C times.
The comparison is strict (m = 0 prunes).

App. A ("FFN Reordering and Chunking") sorts the FFN hidden channels by the
L2 norm of their weights before chunking.  Reading taken here: a channel's
weights are its W1 row, its b1 entry and its W2 column, sorted by
decreasing norm, ties kept in index order.  Permuting W1 rows, b1 and W2
columns together leaves the block's output unchanged.
"""
from __future__ import annotations

import numpy as np


def hard_gates(m_block, m_self, m_cross, m_ffn, n_heads: int, head_dim: int, chunk: int):
    """One step's continuous masks -> keep masks.

    m_block [N]; m_self, m_cross [N, n_heads * head_dim]; m_ffn [N, F / chunk].
    Returns uint8 arrays block_keep [N], self_head_keep [N, H],
    cross_head_keep [N, H], ffn_keep [N, F].
    """
    m_block = np.asarray(m_block, dtype=np.float64)
    N = m_block.shape[0]
    out = {"block_keep": np.zeros(N, np.uint8)}
    for l in range(N):
        out["block_keep"][l] = 1 if m_block[l] > 0 else 0
    for key, m in (("self_head_keep", m_self), ("cross_head_keep", m_cross)):
        m = np.asarray(m, dtype=np.float64)
        keep = np.zeros((N, n_heads), np.uint8)
        for l in range(N):
            for h in range(n_heads):
                mean = sum(m[l, h * head_dim + d] for d in range(head_dim)) / head_dim
                keep[l, h] = 1 if mean > 0 else 0
        out[key] = keep
    m_ffn = np.asarray(m_ffn, dtype=np.float64)
    n_chunks = m_ffn.shape[1]
    keep = np.zeros((N, n_chunks * chunk), np.uint8)
    for l in range(N):
        for c in range(n_chunks):
            if m_ffn[l, c] > 0:
                keep[l, c * chunk:(c + 1) * chunk] = 1
    out["ffn_keep"] = keep
    return out


def ffn_channel_norms(wl: dict) -> np.ndarray:
    """L2 norm of each hidden channel's weights: W1 row, b1 entry, W2 column."""
    w1 = np.asarray(wl["ffn_w1"], dtype=np.float64)
    b1 = np.asarray(wl["ffn_b1"], dtype=np.float64)
    w2 = np.asarray(wl["ffn_w2"], dtype=np.float64)
    return np.sqrt((w1 * w1).sum(axis=1) + b1 * b1 + (w2 * w2).sum(axis=0))


def ffn_reorder(wl: dict):
    """(permutation, reordered copy of the layer): channel i of the result is
    channel perm[i] of the input, by decreasing norm."""
    norms = ffn_channel_norms(wl)
    perm = np.argsort(-norms, kind="stable")
    out = dict(wl)
    out["ffn_w1"] = np.asarray(wl["ffn_w1"])[perm]
    out["ffn_b1"] = np.asarray(wl["ffn_b1"])[perm]
    out["ffn_w2"] = np.asarray(wl["ffn_w2"])[:, perm]
    return perm, out
