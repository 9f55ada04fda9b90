"""Plain numpy oracle of one denoising step of a step-pruned video DiT.

TEST INFRASTRUCTURE (see oracle/__init__.py): never used by the product path.

What the paper fixes, and where:
  * the few-step sampler visits T = 4 discrete timesteps t_1 (most noise)
    .. t_T (Sec. 3.1, "Modified Distribution Matching Distillation");
  * each step t_i has its own binary gates for blocks, attention heads and
    FFN hidden channels, shapes [T, N_block], [T, N_head], [T, N_channel]
    (Sec. 3.2, "Step-Aware Tri-level Structural Pruning");
  * a gate multiplies the output of the component it controls, broadcast
    (Sec. 3.2, equation "gating"); once trained the gated network is
    exported to a dense one per step (same paragraph) and the inference
    engine gathers each step's active parameters from the union of all
    steps' parameters through per-step index tables (Sec. 4.3);
  * FFN gates act on chunks of C hidden channels (Sec. 4.1; C = 8, App. A).

The paper is silent on the block internals (it names a DiT, Wan2.1; Sec.
3.2 and Sec. 5.1).  The readings taken here, identical on the GPU side:
  R1  Wan2.1-style block: AdaLN-modulated self-attention with per-head 3D
      RoPE and full-width QK-RMSNorm, LayerNorm-affine cross-attention to
      the text tokens with QK-RMSNorm, AdaLN-modulated GELU(tanh) FFN.
  R2  A head gate zeroes that head's q, k and v projections (rows of Wq,
      Wk, Wv and their biases) and its Wo columns; an FFN gate zeroes the
      channel's W1 row, b1 entry and W2 column.  A block gate of 0 makes
      the block the identity.
  R3  QK-RMSNorm spans the full model width D: pruned channels enter the
      mean square as zeros and the divisor stays D.
  R4  LayerNorm / RMSNorm eps = 1e-6, biased variance; the self-attention
      and FFN LayerNorms have no affine, the cross-attention one does.
  R5  Timestep features: 256 sinusoids [cos, sin], omega_j = 10000^(-j/128);
      two SiLU MLPs give e [D] and e0 [6, D]; rows of (block modulation +
      e0) are (shift1, scale1, gate1, shift2, scale2, gate2); the output
      head uses (shift, scale) = head modulation + e.
  R6  Attention scale 1/sqrt(dh), bidirectional, no padding mask.
  R7  Inter-step update: Euler in sigma = t / 1000 with sigma after the last
      step = 0, timesteps (999, 750, 500, 250).
  R8  3D RoPE: head_dim split (dh - 4*(dh//6), 2*(dh//6), 2*(dh//6)) over
      (frame, row, column); consecutive pairs rotate by pos * theta^(-2j/d).
"""
from __future__ import annotations

import numpy as np

EPS = 1e-6


# --------------------------------------------------------------------------
# elementwise pieces
# --------------------------------------------------------------------------

def sinusoid(t: float, dim: int = 256, dtype=np.float64) -> np.ndarray:
    """Timestep features [cos(t w_j), sin(t w_j)], w_j = 10000^(-j/(dim/2)) (R5)."""
    half = dim // 2
    j = np.arange(half, dtype=np.float64)
    arg = float(t) * np.power(10000.0, -j / half)
    return np.concatenate([np.cos(arg), np.sin(arg)]).astype(dtype)


def silu(x):
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x):
    """GELU, tanh form (R1)."""
    c = np.sqrt(2.0 / np.pi)
    return 0.5 * x * (1.0 + np.tanh(c * (x + 0.044715 * x ** 3)))


def layer_norm(x, eps: float = EPS):
    """Per-row (x - mean) / sqrt(biased var + eps), no affine (R4)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def rms_norm(x, gain, eps: float = EPS):
    """x / sqrt(mean(x^2) + eps) * gain over the last axis (R3 when the
    last axis is the full width D with pruned channels at zero)."""
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * gain


# --------------------------------------------------------------------------
# 3D rotary position embedding (R8)
# --------------------------------------------------------------------------

def rope_split(dh: int):
    d_hw = 2 * (dh // 6)
    return dh - 2 * d_hw, d_hw, d_hw


def rope_angles(grid, dh: int, theta: float = 10000.0) -> np.ndarray:
    """Rotation angle of every (token, pair) for one head: [L, dh/2], fp64.

    Token n = (f * rows + r) * cols + w; the first d_t/2 pairs follow f,
    the next d_h/2 follow r, the last d_w/2 follow w.
    """
    gf, gh, gw = grid
    f_idx, r_idx, w_idx = np.meshgrid(np.arange(gf), np.arange(gh), np.arange(gw),
                                      indexing="ij")
    pos = [f_idx.reshape(-1), r_idx.reshape(-1), w_idx.reshape(-1)]
    cols = []
    for axis, d in enumerate(rope_split(dh)):
        j = np.arange(d // 2, dtype=np.float64)
        omega = np.power(float(theta), -2.0 * j / d)
        cols.append(np.outer(pos[axis].astype(np.float64), omega))
    return np.concatenate(cols, axis=1)


def apply_rope(x, phi, n_heads: int, dh: int):
    """Rotate each head's consecutive pairs (x0, x1) by the token's angle."""
    L = x.shape[0]
    xr = x.reshape(L, n_heads, dh // 2, 2)
    c = np.cos(phi)[:, None, :].astype(x.dtype)
    s = np.sin(phi)[:, None, :].astype(x.dtype)
    x0, x1 = xr[..., 0], xr[..., 1]
    out = np.stack([x0 * c - x1 * s, x0 * s + x1 * c], axis=-1)
    return out.reshape(L, n_heads * dh)


# --------------------------------------------------------------------------
# attention (R6)
# --------------------------------------------------------------------------

def softmax_rows(s):
    """Two-pass softmax along the last axis: subtract the row max, exp, divide."""
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def attention(q, k, v, n_heads: int, dh: int, chunk: int = 512):
    """softmax(q_h k_h^T / sqrt(dh)) v_h for every head; q [Lq, H*dh],
    k, v [Lk, H*dh].  Query rows go in chunks so Lq x Lk is never held."""
    Lq = q.shape[0]
    out = np.empty((Lq, n_heads * dh), dtype=q.dtype)
    scale = 1.0 / np.sqrt(dh)
    for h in range(n_heads):
        cs = slice(h * dh, (h + 1) * dh)
        kt = np.ascontiguousarray(k[:, cs].T)
        vh = np.ascontiguousarray(v[:, cs])
        for r0 in range(0, Lq, chunk):
            p = softmax_rows((q[r0:r0 + chunk, cs] @ kt) * scale)
            out[r0:r0 + chunk, cs] = p @ vh
    return out


# --------------------------------------------------------------------------
# keep masks -> zeroed dense weights (Sec. 3.2 gating equation; R2)
# --------------------------------------------------------------------------

def apply_keep(wl: dict, self_keep, cross_keep, ffn_keep, dh: int, dtype=np.float64) -> dict:
    """Copy of one layer's weights with pruned heads / channels zeroed.

    A head gate g_h multiplies that head's features; zeroing the head's rows
    of Wq, Wk, Wv (and biases) makes its q, k, v exactly zero, and zeroing
    its Wo columns removes its contribution to the output.  An FFN channel
    gate zeroes the channel's W1 row, b1 entry and W2 column.
    """
    w = {k: np.asarray(v, dtype=dtype) for k, v in wl.items()}
    ms = np.repeat(np.asarray(self_keep, dtype=dtype), dh)
    mc = np.repeat(np.asarray(cross_keep, dtype=dtype), dh)
    mf = np.asarray(ffn_keep, dtype=dtype)
    for pre, m in (("self", ms), ("cross", mc)):
        for p in ("q", "k", "v"):
            w[f"{pre}_w{p}"] = w[f"{pre}_w{p}"] * m[:, None]
            w[f"{pre}_b{p}"] = w[f"{pre}_b{p}"] * m
        w[f"{pre}_wo"] = w[f"{pre}_wo"] * m[None, :]
    w["ffn_w1"] = w["ffn_w1"] * mf[:, None]
    w["ffn_b1"] = w["ffn_b1"] * mf
    w["ffn_w2"] = w["ffn_w2"] * mf[None, :]
    return w


# --------------------------------------------------------------------------
# timestep embedding and modulation (R5)
# --------------------------------------------------------------------------

def time_embedding(w: dict, t: float, dtype=np.float64):
    """e [D] and e0 [6, D] for timestep t."""
    g = lambda k: np.asarray(w[k], dtype=dtype)
    emb = sinusoid(t, g("t_w1").shape[1], dtype)
    e = g("t_w2") @ silu(g("t_w1") @ emb + g("t_b1")) + g("t_b2")
    e0 = (g("t_w3") @ silu(e) + g("t_b3")).reshape(6, -1)
    return e, e0


# --------------------------------------------------------------------------
# one block (R1-R4, R6, R8)
# --------------------------------------------------------------------------

def block(x, ctx, e0, wz: dict, keep_block: bool, n_heads: int, dh: int, grid,
          theta: float = 10000.0, eps: float = EPS, rows=None, dtype=np.float64):
    """One DiT block on one sample with already-zeroed weights `wz`.

    x [L, D] residual stream, ctx [Lc, D] text tokens, e0 [6, D].
    `rows` (optional index array) selects the query rows whose outputs are
    returned; keys and values of self-attention always span all L tokens.
    """
    x = np.asarray(x, dtype=dtype)
    ctx = np.asarray(ctx, dtype=dtype)
    rows = np.arange(x.shape[0]) if rows is None else np.asarray(rows)
    if not keep_block:
        return x[rows].copy()
    w = {k: np.asarray(v, dtype=dtype) for k, v in wz.items()}
    sh1, sc1, g1, sh2, sc2, g2 = w["mod"] + np.asarray(e0, dtype=dtype)
    phi = rope_angles(grid, dh, theta)

    # self-attention
    a = layer_norm(x, eps) * (1.0 + sc1) + sh1
    q = rms_norm(a[rows] @ w["self_wq"].T + w["self_bq"], w["self_gq"], eps)
    k = rms_norm(a @ w["self_wk"].T + w["self_bk"], w["self_gk"], eps)
    v = a @ w["self_wv"].T + w["self_bv"]
    q = apply_rope(q, phi[rows], n_heads, dh)
    k = apply_rope(k, phi, n_heads, dh)
    o = attention(q, k, v, n_heads, dh)
    y = x[rows] + g1 * (o @ w["self_wo"].T + w["self_bo"])

    # cross-attention to the text tokens
    a = layer_norm(y, eps) * w["norm3_w"] + w["norm3_b"]
    q = rms_norm(a @ w["cross_wq"].T + w["cross_bq"], w["cross_gq"], eps)
    k = rms_norm(ctx @ w["cross_wk"].T + w["cross_bk"], w["cross_gk"], eps)
    v = ctx @ w["cross_wv"].T + w["cross_bv"]
    o = attention(q, k, v, n_heads, dh)
    y = y + (o @ w["cross_wo"].T + w["cross_bo"])

    # FFN
    a = layer_norm(y, eps) * (1.0 + sc2) + sh2
    u = gelu_tanh(a @ w["ffn_w1"].T + w["ffn_b1"])
    y = y + g2 * (u @ w["ffn_w2"].T + w["ffn_b2"])
    return y


# --------------------------------------------------------------------------
# one step and the 4-step denoise (Sec. 3.1 sampler; R7)
# --------------------------------------------------------------------------

def step(z, t: float, ctx, w: dict, masks: dict, cfg, dtype=np.float64):
    """Model prediction v for latents z [B, L, Cp] at timestep t under the
    step structure `masks`."""
    z = np.asarray(z, dtype=dtype)
    ctx = np.asarray(ctx, dtype=dtype)
    e, e0 = time_embedding(w, t, dtype)
    g = lambda k: np.asarray(w[k], dtype=dtype)
    dh = cfg.head_dim
    zeroed = [apply_keep(w["layers"][l], masks["self_head_keep"][l],
                         masks["cross_head_keep"][l], masks["ffn_keep"][l], dh, dtype)
              for l in range(cfg.n_layers)]
    out = np.empty(z.shape, dtype=dtype)
    sh, sc = g("head_mod") + e
    for b in range(z.shape[0]):
        x = z[b] @ g("patch_w").T + g("patch_b")
        for l in range(cfg.n_layers):
            x = block(x, ctx[b], e0, zeroed[l], bool(masks["block_keep"][l]),
                      cfg.n_heads, dh, cfg.grid, cfg.rope_theta, cfg.eps, dtype=dtype)
        out[b] = (layer_norm(x, cfg.eps) * (1.0 + sc) + sh) @ g("head_w").T + g("head_b")
    return out


def sigmas(timesteps):
    """sigma_s = t_s / 1000, followed by sigma = 0 after the last step (R7)."""
    return [t / 1000.0 for t in timesteps] + [0.0]


def euler(z, v, sigma_from: float, sigma_to: float):
    return z + (sigma_to - sigma_from) * v


def predict_clean(z, v, sigma: float):
    """Clean-data estimate from the model prediction at noise level sigma
    (the single-step prediction of Sec. 4.2).  With z = (1 - sigma) x +
    sigma eps and v = eps - x (R7) this is x."""
    return z - sigma * v


def renoise(x_hat, sigma_to: float, eps):
    """Re-noise a clean estimate to level sigma_to with noise eps (the
    re-noising of Sec. 3.1, written in sigma = 1 - tau)."""
    return (1.0 - sigma_to) * x_hat + sigma_to * eps


def rollout(z, ctx, w: dict, masks_per_step, cfg, eps_per_step=None, start: int = 0,
            sampler: str = "renoise", dtype=np.float64):
    """Sequential denoise from step `start` to the last step (the output
    rollout of Sec. 4.2 / Fig. 2(b)).  sampler "euler": z += dsigma v;
    "renoise": x_hat = z - sigma_s v, then z = (1 - sigma_{s+1}) x_hat +
    sigma_{s+1} eps_s; the last step returns x_hat (sigma after it is 0)."""
    z = np.asarray(z, dtype=dtype)
    sig = sigmas(cfg.timesteps)
    T = len(cfg.timesteps)
    for s in range(start, T):
        v = step(z, cfg.timesteps[s], ctx, w, masks_per_step[s], cfg, dtype)
        if sampler == "euler":
            z = euler(z, v, sig[s], sig[s + 1])
        else:
            x_hat = predict_clean(z, v, sig[s])
            z = x_hat if s + 1 == T else renoise(x_hat, sig[s + 1], np.asarray(eps_per_step[s], dtype))
    return z


def denoise(z, ctx, w: dict, masks_per_step, cfg, dtype=np.float64):
    """Run the T-step sampler; step s uses its own structure masks_per_step[s]."""
    z = np.asarray(z, dtype=dtype)
    sig = sigmas(cfg.timesteps)
    for s, t in enumerate(cfg.timesteps):
        v = step(z, t, ctx, w, masks_per_step[s], cfg, dtype)
        z = euler(z, v, sig[s], sig[s + 1])
    return z
