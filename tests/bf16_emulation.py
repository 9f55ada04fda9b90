"""The oracle's block with the bfloat16 rounding points of the GPU path.

Test infrastructure (never used by the product path).  The HIP path stores
every activation between kernels in bfloat16 and computes in float32; the
oracle computes in float64 on the same bf16-rounded weights and inputs.
The difference between the two is therefore set by where the GPU rounds to
bf16, not by its arithmetic.  This module re-runs the oracle's block (built
from the oracle's own primitives, in float64) rounding to bf16 exactly where
the GPU path stores:

  the LayerNorm outputs; q, k, v after their projection; q and k after
  QK-RMSNorm and RoPE, with q already multiplied by log2(e)/sqrt(dh) (the
  attention kernel takes base-2 exponents); the probabilities fed to the PV
  product (the row sums use the unrounded ones); the attention output; the
  residual stream after each of its three updates; the GELU output.

Its distance to the oracle is the error floor that bf16 storage alone
imposes on a block: tolerances above 2e-2 are justified by it, and the
power of a check is measured against it.
"""
from __future__ import annotations

import math

import numpy as np

import oracle as O
from workloads.synth import bf16_round

LOG2E = 1.4426950408889634


def r(a):
    """Round to bfloat16 (ties to even), back in float64."""
    return bf16_round(np.asarray(a, dtype=np.float32)).astype(np.float64)


def attention_base2(qs, k, v, n_heads, dh, chunk=512):
    """softmax over base-2 scores s = qs . k with the probabilities rounded to
    bf16 for the PV product and the row sums taken unrounded."""
    Lq = qs.shape[0]
    out = np.empty((Lq, n_heads * dh))
    for h in range(n_heads):
        cs = slice(h * dh, (h + 1) * dh)
        kt = np.ascontiguousarray(k[:, cs].T)
        vh = np.ascontiguousarray(v[:, cs])
        for r0 in range(0, Lq, chunk):
            s = qs[r0:r0 + chunk, cs] @ kt
            p = np.exp2(s - s.max(axis=1, keepdims=True))
            out[r0:r0 + chunk, cs] = (r(p) @ vh) / p.sum(axis=1, keepdims=True)
    return out


def block(x, ctx, e0, wz, keep_block, n_heads, dh, grid, theta=10000.0, eps=1e-6,
          rows=None):
    """Same arguments and result as oracle.block (float64 only), with the
    GPU path's bf16 storage points; `rows` selects query rows as there."""
    x = np.asarray(x, dtype=np.float64)
    ctx = np.asarray(ctx, dtype=np.float64)
    rows = np.arange(x.shape[0]) if rows is None else np.asarray(rows)
    if not keep_block:
        return x[rows].copy()
    w = {k: np.asarray(v, dtype=np.float64) for k, v in wz.items()}
    sh1, sc1, g1, sh2, sc2, g2 = w["mod"] + np.asarray(e0, dtype=np.float64)
    phi = O.rope_angles(grid, dh, theta)
    scale = LOG2E / math.sqrt(dh)

    a = r(O.layer_norm(x, eps) * (1.0 + sc1) + sh1)
    qs = r(O.apply_rope(O.rms_norm(r(a[rows] @ w["self_wq"].T + w["self_bq"]), w["self_gq"], eps),
                        phi[rows], n_heads, dh) * scale)
    k = r(O.apply_rope(O.rms_norm(r(a @ w["self_wk"].T + w["self_bk"]), w["self_gk"], eps),
                       phi, n_heads, dh))
    v = r(a @ w["self_wv"].T + w["self_bv"])
    o = r(attention_base2(qs, k, v, n_heads, dh))
    y = r(x[rows] + g1 * (o @ w["self_wo"].T + w["self_bo"]))

    a = r(O.layer_norm(y, eps) * w["norm3_w"] + w["norm3_b"])
    qs = r(O.rms_norm(r(a @ w["cross_wq"].T + w["cross_bq"]), w["cross_gq"], eps) * scale)
    k = r(O.rms_norm(r(ctx @ w["cross_wk"].T + w["cross_bk"]), w["cross_gk"], eps))
    v = r(ctx @ w["cross_wv"].T + w["cross_bv"])
    o = r(attention_base2(qs, k, v, n_heads, dh))
    y = r(y + (o @ w["cross_wo"].T + w["cross_bo"]))

    a = r(O.layer_norm(y, eps) * (1.0 + sc2) + sh2)
    u = r(O.gelu_tanh(a @ w["ffn_w1"].T + w["ffn_b1"]))
    return r(y + g2 * (u @ w["ffn_w2"].T + w["ffn_b2"]))
