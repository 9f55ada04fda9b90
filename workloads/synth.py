"""Seeded synthetic inputs: weights, latents, text context and keep masks.

Every value the oracle tests and the HIP path consume is drawn here, from
named seed streams (weights=0, inputs=1, masks=2), so the two sides see the
same numbers.  Nothing here computes any part of the block forward.

Distributions (the paper ships no weights, Sec. 5.1 initialises from a
pre-trained Wan2.1 checkpoint that is not available):
  * every matrix and bias ~ N(0, 0.02)
  * RMSNorm / LayerNorm gains 1 + N(0, 0.02); LayerNorm bias N(0, 0.02)
  * per-layer modulation table and head modulation ~ N(0, 0.02)
  * latents z ~ N(0, 1) [B, L, Cp]; text context ~ N(0, 1) [B, Lc, D]

For "bf16" configurations the matrices and the text context are rounded to
bfloat16 (round to nearest even) here, so the oracle's fp32/fp64 arithmetic
runs on exactly the values the GPU stores.
"""
from __future__ import annotations

import zlib
from typing import Dict, List, Optional

import numpy as np

from .configs import Config, get_config

SEED_WEIGHTS, SEED_INPUTS, SEED_MASKS = 0, 1, 2

MATRIX_KEYS_GLOBAL = ("patch_w", "t_w1", "t_w2", "t_w3", "head_w")
MATRIX_KEYS_LAYER = ("self_wq", "self_wk", "self_wv", "self_wo",
                     "cross_wq", "cross_wk", "cross_wv", "cross_wo",
                     "ffn_w1", "ffn_w2")


def rng(stream: int, *tags) -> np.random.Generator:
    """Generator for a named stream; `tags` (ints/strings) split it further."""
    words = [stream]
    for t in tags:
        words.append(zlib.crc32(t.encode()) if isinstance(t, str) else int(t))
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(words)))


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def _store(cfg: Config, a: np.ndarray) -> np.ndarray:
    return bf16_round(a) if cfg.dtype == "bf16" else a.astype(np.float32)


def _normal(g, shape, std):
    return (g.standard_normal(shape, dtype=np.float32) * np.float32(std))


def make_global_weights(cfg: Config, seed: int = 0) -> Dict[str, np.ndarray]:
    D, Cp, Fq, s = cfg.dim, cfg.patch_dim, cfg.freq_dim, cfg.std
    g = rng(SEED_WEIGHTS, seed, cfg.name, "global")
    w = {
        "patch_w": _normal(g, (D, Cp), s), "patch_b": _normal(g, (D,), s),
        "t_w1": _normal(g, (D, Fq), s), "t_b1": _normal(g, (D,), s),
        "t_w2": _normal(g, (D, D), s), "t_b2": _normal(g, (D,), s),
        "t_w3": _normal(g, (6 * D, D), s), "t_b3": _normal(g, (6 * D,), s),
        "head_mod": _normal(g, (2, D), s),
        "head_w": _normal(g, (Cp, D), s), "head_b": _normal(g, (Cp,), s),
    }
    for k in MATRIX_KEYS_GLOBAL:
        w[k] = _store(cfg, w[k])
    return w


def make_layer_weights(cfg: Config, layer: int, seed: int = 0,
                       qk_gain: Optional[float] = None) -> Dict[str, np.ndarray]:
    """One block's weights in nn.Linear layout ([out, in], row-major)."""
    D, F, s = cfg.dim, cfg.ffn_dim, cfg.std
    g = rng(SEED_WEIGHTS, seed, cfg.name, "layer", layer)
    w = {"mod": _normal(g, (6, D), s)}
    for pre in ("self", "cross"):
        for m in ("q", "k", "v", "o"):
            w[f"{pre}_w{m}"] = _normal(g, (D, D), s)
            w[f"{pre}_b{m}"] = _normal(g, (D,), s)
        for m in ("q", "k"):
            w[f"{pre}_g{m}"] = 1.0 + _normal(g, (D,), s)
        if pre == "self":
            w["norm3_w"] = 1.0 + _normal(g, (D,), s)
            w["norm3_b"] = _normal(g, (D,), s)
    w["ffn_w1"] = _normal(g, (F, D), s)
    w["ffn_b1"] = _normal(g, (F,), s)
    w["ffn_w2"] = _normal(g, (D, F), s)
    w["ffn_b2"] = _normal(g, (D,), s)
    if qk_gain is not None:   # stress variant: sharper attention
        for pre in ("self", "cross"):
            w[f"{pre}_gq"] = w[f"{pre}_gq"] * np.float32(qk_gain)
            w[f"{pre}_gk"] = w[f"{pre}_gk"] * np.float32(qk_gain)
    for k in MATRIX_KEYS_LAYER:
        w[k] = _store(cfg, w[k])
    for k in list(w):
        w[k] = np.ascontiguousarray(w[k], dtype=np.float32)
    return w


def make_weights(cfg: Config, seed: int = 0, qk_gain: Optional[float] = None,
                 layers: Optional[List[int]] = None) -> Dict:
    """Full model weights: global tensors plus a list of per-layer dicts."""
    w = make_global_weights(cfg, seed)
    idx = range(cfg.n_layers) if layers is None else layers
    w["layers"] = [make_layer_weights(cfg, l, seed, qk_gain) for l in idx]
    return w


def make_latents(cfg: Config, seed: int = 0) -> np.ndarray:
    g = rng(SEED_INPUTS, seed, cfg.name, "z")
    return g.standard_normal((cfg.batch, cfg.seq_len, cfg.patch_dim), dtype=np.float32)


def make_renoise_eps(cfg: Config, seed: int = 0) -> List[np.ndarray]:
    """Noise drawn for the re-noise sampler, one latent-shaped array per step
    transition (the method's random draws, passed in as inputs)."""
    return [rng(SEED_INPUTS, seed, cfg.name, "eps", s).standard_normal(
        (cfg.batch, cfg.seq_len, cfg.patch_dim), dtype=np.float32)
        for s in range(len(cfg.timesteps) - 1)]


def make_context(cfg: Config, seed: int = 0, text_len: Optional[int] = None) -> np.ndarray:
    Lc = cfg.text_len if text_len is None else text_len
    g = rng(SEED_INPUTS, seed, cfg.name, "ctx")
    return _store(cfg, g.standard_normal((cfg.batch, Lc, cfg.dim), dtype=np.float32))


def make_block_input(cfg: Config, seed: int = 0, scale: float = 1.0) -> np.ndarray:
    """Synthetic residual-stream input x [B, L, D] for single-block tests."""
    g = rng(SEED_INPUTS, seed, cfg.name, "x")
    x = g.standard_normal((cfg.batch, cfg.seq_len, cfg.dim), dtype=np.float32)
    return _store(cfg, x * np.float32(scale))


def make_attention_inputs(L: int, n_heads: int, dh: int, q_std: float, k_std: float,
                          seed: int = 0, heads=None, bf16: bool = True):
    """q, k, v [L, len(heads) * dh] for attention operator tests, float32:
    q ~ N(0, q_std^2), k ~ N(0, k_std^2), v ~ N(0, 1), rounded to bfloat16
    when `bf16`.  Scores q.k / sqrt(dh) then have standard deviation
    q_std * k_std.  Every head has its own stream, so any subset of heads
    (default: all n_heads) is drawn identically on its own."""
    hs = list(range(n_heads)) if heads is None else list(heads)
    out = [np.empty((L, len(hs) * dh), dtype=np.float32) for _ in range(3)]
    for i, h in enumerate(hs):
        g = rng(SEED_INPUTS, seed, "attention", L, n_heads, dh, h)
        cs = slice(i * dh, (i + 1) * dh)
        out[0][:, cs] = _normal(g, (L, dh), q_std)
        out[1][:, cs] = _normal(g, (L, dh), k_std)
        out[2][:, cs] = _normal(g, (L, dh), 1.0)
    return tuple(bf16_round(a) if bf16 else a for a in out)


def make_e0(cfg: Config, seed: int = 0, std: float = 0.1) -> np.ndarray:
    """Synthetic per-step modulation e0 [6, D] for single-block tests."""
    g = rng(SEED_INPUTS, seed, cfg.name, "e0")
    return _normal(g, (6, cfg.dim), std)


# --------------------------------------------------------------------------
# keep masks
# --------------------------------------------------------------------------

def _subset(g, n: int, k: int) -> np.ndarray:
    keep = np.zeros(n, dtype=np.uint8)
    if k > 0:
        keep[np.sort(g.choice(n, size=k, replace=False))] = 1
    return keep


def _ffn_subset(g, F: int, k: int, chunk: int) -> np.ndarray:
    """k kept channels; whole chunks of `chunk` when both divide."""
    if chunk > 1 and F % chunk == 0 and k % chunk == 0:
        ck = _subset(g, F // chunk, k // chunk)
        return np.repeat(ck, chunk).astype(np.uint8)
    return _subset(g, F, k)


def masks_from_counts(cfg: Config, heads, cross_heads, ffn, seed: int = 0,
                      step: int = 0, block_keep=None) -> Dict[str, np.ndarray]:
    """Seeded masks with the given per-layer kept counts (lists of length N)."""
    N, H, F = cfg.n_layers, cfg.n_heads, cfg.ffn_dim
    out = {
        "block_keep": np.ones(N, np.uint8) if block_keep is None
        else np.asarray(block_keep, np.uint8).copy(),
        "self_head_keep": np.zeros((N, H), np.uint8),
        "cross_head_keep": np.zeros((N, H), np.uint8),
        "ffn_keep": np.zeros((N, F), np.uint8),
    }
    for l in range(N):
        out["self_head_keep"][l] = _subset(rng(SEED_MASKS, seed, cfg.name, step, l, "self"), H, heads[l])
        out["cross_head_keep"][l] = _subset(rng(SEED_MASKS, seed, cfg.name, step, l, "cross"), H, cross_heads[l])
        out["ffn_keep"][l] = _ffn_subset(rng(SEED_MASKS, seed, cfg.name, step, l, "ffn"), F, ffn[l], cfg.ffn_chunk)
    return out


# FLOP retention targets for the depth-tilted recipe: the paper's Wan-1.3B
# per-step retention (88.4 / 78.5 / 77.1 / 89.1 %, Sec. 6 "U-Shaped
# Computational Allocation") rescaled so the mean removal is the 24 % the
# paper reports for Wan-14B (abstract; Sec. 5.4 "Speedup on Wan-14B").
RECIPE_RHO = (0.834, 0.691, 0.671, 0.844)
# depth tilt of attention retention, larger at t2/t3 (Sec. 6 "Semantic
# Freezing in Deep Layers")
RECIPE_DELTA = (0.10, 0.30, 0.30, 0.10)
RECIPE_TOL = 0.0025


def layer_flops(cfg: Config, h: int, hc: int, f: int, L: Optional[int] = None,
                Lc: Optional[int] = None) -> float:
    """Per-block FLOP count used only to balance the synthetic recipe."""
    L = cfg.seq_len if L is None else L
    Lc = cfg.text_len if Lc is None else Lc
    D, dh = cfg.dim, cfg.head_dim
    a, ac = h * dh, hc * dh
    return float(2 * L * D * 3 * a + 4 * L * L * dh * h + 2 * L * a * D
                 + 2 * L * D * ac + 4 * Lc * D * ac + 4 * L * Lc * dh * hc
                 + 2 * L * ac * D + 4 * L * D * f)


def recipe_counts(cfg: Config, step: int, seed: int = 0):
    """Per-layer kept (heads, cross heads, FFN channels) for one step."""
    N, H, F = cfg.n_layers, cfg.n_heads, cfg.ffn_dim
    rho, delta = RECIPE_RHO[step], RECIPE_DELTA[step]
    g = rng(SEED_MASKS, seed, cfg.name, "recipe", step)
    heads, cheads, ffn = [], [], []
    for l in range(N):
        tilt = delta * ((l / max(N - 1, 1)) - 0.5)
        ra = np.clip(rho - 0.05 - tilt + g.uniform(-0.03, 0.03), 0.3, 1.0)
        rc = np.clip(rho - 0.05 - tilt + g.uniform(-0.03, 0.03), 0.3, 1.0)
        rf = np.clip(rho + 0.05 + g.uniform(-0.03, 0.03), 0.3, 1.0)
        heads.append(int(round(ra * H)))
        cheads.append(int(round(rc * H)))
        ffn.append(int(round(rf * F / 8)) * 8)
    dense = N * layer_flops(cfg, H, H, F)

    def frac():
        return sum(layer_flops(cfg, heads[l], cheads[l], ffn[l]) for l in range(N)) / dense

    lo_h = max(1, int(np.ceil(0.3 * H)))
    for _ in range(100 * N):
        fr = frac()
        if abs(fr - rho) <= RECIPE_TOL:
            break
        l = int(g.integers(N))
        if fr > rho and heads[l] > lo_h:
            heads[l] -= 1
        elif fr < rho and heads[l] < H:
            heads[l] += 1
    return heads, cheads, ffn


def make_masks(cfg: Config, step: int, seed: int = 0) -> Dict[str, np.ndarray]:
    """Keep masks of one step structure.

    Configs with fixed per-step counts use them for every layer; the 40-layer
    stacks use the depth-tilted recipe (the 720p stack reuses the 480p
    structures).
    """
    if cfg.keep_heads is not None:
        N = cfg.n_layers
        return masks_from_counts(cfg, [cfg.keep_heads[step]] * N,
                                 [cfg.keep_heads[step]] * N,
                                 [cfg.keep_ffn[step]] * N, seed, step)
    base = get_config("wan14b_480p") if cfg.name == "wan14b_720p" else cfg
    h, hc, f = recipe_counts(base, step, seed)
    m = masks_from_counts(base, h, hc, f, seed, step)
    return m


def all_keep_masks(cfg: Config) -> Dict[str, np.ndarray]:
    N, H, F = cfg.n_layers, cfg.n_heads, cfg.ffn_dim
    return {"block_keep": np.ones(N, np.uint8),
            "self_head_keep": np.ones((N, H), np.uint8),
            "cross_head_keep": np.ones((N, H), np.uint8),
            "ffn_keep": np.ones((N, F), np.uint8)}


# --------------------------------------------------------------------------
# device-side generation for the 40-layer stacks (about 28 GB of weights)
# --------------------------------------------------------------------------

def make_weights_torch(cfg: Config, device, seed: int = 0):
    """Seeded random-init weights generated directly in device memory.

    Matrices are bfloat16 (the config dtype), everything else float32.
    Each tensor has its own seed so any layer can be regenerated alone.
    """
    import torch
    D, F, Cp, Fq, s = cfg.dim, cfg.ffn_dim, cfg.patch_dim, cfg.freq_dim, cfg.std
    mdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    gen = torch.Generator(device=device)
    counter = [0]

    def normal(shape, std=s, mean=0.0, dtype=torch.float32):
        gen.manual_seed(zlib.crc32(f"{seed}/{cfg.name}/{counter[0]}".encode()))
        counter[0] += 1
        t = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
        t.mul_(std).add_(mean)
        return t.to(dtype)

    w = {"patch_w": normal((D, Cp), dtype=mdt), "patch_b": normal((D,)),
         "t_w1": normal((D, Fq), dtype=mdt), "t_b1": normal((D,)),
         "t_w2": normal((D, D), dtype=mdt), "t_b2": normal((D,)),
         "t_w3": normal((6 * D, D), dtype=mdt), "t_b3": normal((6 * D,)),
         "head_mod": normal((2, D)), "head_w": normal((Cp, D), dtype=mdt),
         "head_b": normal((Cp,)), "layers": []}
    for _ in range(cfg.n_layers):
        lw = {"mod": normal((6, D))}
        for pre in ("self", "cross"):
            for m in ("q", "k", "v", "o"):
                lw[f"{pre}_w{m}"] = normal((D, D), dtype=mdt)
                lw[f"{pre}_b{m}"] = normal((D,))
            for m in ("q", "k"):
                lw[f"{pre}_g{m}"] = normal((D,), mean=1.0)
            if pre == "self":
                lw["norm3_w"] = normal((D,), mean=1.0)
                lw["norm3_b"] = normal((D,))
        lw["ffn_w1"] = normal((F, D), dtype=mdt)
        lw["ffn_b1"] = normal((F,))
        lw["ffn_w2"] = normal((D, F), dtype=mdt)
        lw["ffn_b2"] = normal((D,))
        w["layers"].append(lw)
    return w
