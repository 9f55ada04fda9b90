"""Pins of the oracle against things other than itself.

Each test fixes a part of oracle/dit.py against an independent fact:
library routines (torch CPU), textbook closed forms, invariants the paper's
gating equation implies (Sec. 3.2), brute force on tiny inputs, or a second
formulation (compacted weights, feature gating).  A plausible slip in the
oracle (a dropped term, a wrong sign or index, a transposed operand, a
wrong divisor) fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as O
from workloads import get_config
from workloads import synth

MICRO = get_config("tiny").with_(name="micro", dim=24, n_heads=2, head_dim=12, ffn_dim=32,
                                  n_layers=2, grid=(2, 2, 3), text_len=5, dtype="f32",
                                  keep_heads=(2, 1, 1, 1), keep_ffn=(32, 24, 16, 8))
TINY = get_config("tiny")


def _layer_inputs(cfg, seed=0, layer=0, qk_gain=None):
    wl = synth.make_layer_weights(cfg, layer, seed, qk_gain)
    x = synth.make_block_input(cfg, seed)[0].astype(np.float64)
    ctx = synth.make_context(cfg, seed)[0].astype(np.float64)
    e0 = synth.make_e0(cfg, seed).astype(np.float64)
    return wl, x, ctx, e0


def _run_block(cfg, wl, x, ctx, e0, ms, mc, mf, keep=True, rows=None):
    wz = O.apply_keep(wl, ms, mc, mf, cfg.head_dim)
    return O.block(x, ctx, e0, wz, keep, cfg.n_heads, cfg.head_dim, cfg.grid,
                   cfg.rope_theta, cfg.eps, rows=rows)


# --------------------------------------------------------------------------
# primitives against library routines and closed forms
# --------------------------------------------------------------------------

def test_layer_norm_matches_torch():
    x = np.random.default_rng(0).standard_normal((7, 33)) * 3 + 1.5
    ref = F.layer_norm(torch.from_numpy(x), (33,), eps=1e-6).numpy()
    np.testing.assert_allclose(O.layer_norm(x, 1e-6), ref, rtol=0, atol=1e-12)


def test_layer_norm_constant_row_is_zero():
    x = np.full((3, 16), 2.75)
    assert np.all(O.layer_norm(x) == 0.0)


def test_rms_norm_matches_torch():
    g = np.random.default_rng(1)
    x, w = g.standard_normal((5, 40)), 1 + 0.1 * g.standard_normal(40)
    ref = F.rms_norm(torch.from_numpy(x), (40,), weight=torch.from_numpy(w), eps=1e-6).numpy()
    np.testing.assert_allclose(O.rms_norm(x, w, 1e-6), ref, rtol=0, atol=1e-12)


def test_gelu_tanh_matches_torch_and_erf_form():
    x = np.linspace(-8, 8, 1001)
    ref = F.gelu(torch.from_numpy(x), approximate="tanh").numpy()
    np.testing.assert_allclose(O.gelu_tanh(x), ref, rtol=0, atol=1e-13)
    erf_form = np.array([0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in x])
    assert np.max(np.abs(O.gelu_tanh(x) - erf_form)) < 1e-3
    # odd part: gelu(x) - gelu(-x) == x ; gelu(0) == 0
    np.testing.assert_allclose(O.gelu_tanh(x) - O.gelu_tanh(-x), x, atol=1e-13)
    assert O.gelu_tanh(np.zeros(1))[0] == 0.0


def test_silu_matches_torch():
    x = np.linspace(-20, 20, 401)
    np.testing.assert_allclose(O.silu(x), F.silu(torch.from_numpy(x)).numpy(), atol=1e-14)


def test_sinusoid_closed_forms():
    s0 = O.sinusoid(0.0, 256)
    assert np.all(s0[:128] == 1.0) and np.all(s0[128:] == 0.0)
    t = 750.0
    s = O.sinusoid(t, 256)
    z = np.exp(1j * t * 10000.0 ** (-np.arange(128) / 128.0))
    np.testing.assert_allclose(s[:128], z.real, atol=1e-12)
    np.testing.assert_allclose(s[128:], z.imag, atol=1e-12)


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------

def _brute_attention(q, k, v, H, dh):
    """Triple loop over (head, query, key) in plain Python floats."""
    Lq, Lk = q.shape[0], k.shape[0]
    out = np.zeros((Lq, H * dh))
    for h in range(H):
        for i in range(Lq):
            s = []
            for j in range(Lk):
                acc = 0.0
                for d in range(dh):
                    acc += q[i, h * dh + d] * k[j, h * dh + d]
                s.append(acc / math.sqrt(dh))
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = sum(e)
            for d in range(dh):
                out[i, h * dh + d] = sum(e[j] * v[j, h * dh + d] for j in range(Lk)) / z
    return out


def test_attention_brute_force():
    g = np.random.default_rng(2)
    H, dh = 2, 6
    q, k, v = (g.standard_normal((n, H * dh)) for n in (5, 7, 7))
    q *= 2.0
    np.testing.assert_allclose(O.attention(q, k, v, H, dh), _brute_attention(q, k, v, H, dh),
                               rtol=0, atol=1e-12)


def test_attention_matches_torch_sdpa_and_chunking():
    g = np.random.default_rng(3)
    H, dh, Lq, Lk = 3, 16, 70, 53
    q, k, v = g.standard_normal((Lq, H * dh)), g.standard_normal((Lk, H * dh)), g.standard_normal((Lk, H * dh))
    tq = torch.from_numpy(q).reshape(Lq, H, dh).transpose(0, 1)
    tk = torch.from_numpy(k).reshape(Lk, H, dh).transpose(0, 1)
    tv = torch.from_numpy(v).reshape(Lk, H, dh).transpose(0, 1)
    ref = F.scaled_dot_product_attention(tq, tk, tv).transpose(0, 1).reshape(Lq, H * dh).numpy()
    for chunk in (512, 16, 7):
        np.testing.assert_allclose(O.attention(q, k, v, H, dh, chunk=chunk), ref, atol=1e-12)


def test_softmax_rows_sum_to_one():
    s = np.random.default_rng(4).standard_normal((9, 300)) * 30
    p = O.softmax_rows(s)
    np.testing.assert_allclose(p.sum(axis=-1), 1.0, atol=1e-12)
    assert np.all(p >= 0)


def test_attention_special_cases():
    g = np.random.default_rng(5)
    H, dh = 2, 4
    q = g.standard_normal((6, H * dh))
    v1 = g.standard_normal((1, H * dh))
    # one key: the output is that key's value
    out = O.attention(q, g.standard_normal((1, H * dh)), v1, H, dh)
    np.testing.assert_allclose(out, np.repeat(v1, 6, axis=0), atol=1e-15)
    # identical keys: the output is the mean of the values
    k = np.repeat(g.standard_normal((1, H * dh)), 9, axis=0)
    v = g.standard_normal((9, H * dh))
    out = O.attention(q, k, v, H, dh)
    np.testing.assert_allclose(out, np.repeat(v.mean(0, keepdims=True), 6, axis=0), atol=1e-14)


# --------------------------------------------------------------------------
# 3D RoPE
# --------------------------------------------------------------------------

def test_rope_split():
    assert O.rope_split(128) == (44, 42, 42)
    assert O.rope_split(64) == (24, 20, 20)
    assert O.rope_split(12) == (4, 4, 4)


def test_rope_complex_form_and_invariants():
    grid, H, dh = (3, 4, 5), 2, 12
    L = 60
    g = np.random.default_rng(6)
    x = g.standard_normal((L, H * dh))
    phi = O.rope_angles(grid, dh)
    out = O.apply_rope(x, phi, H, dh)
    # complex multiplication of each pair by exp(i phi)
    xc = x.reshape(L, H, dh // 2, 2)
    z = (xc[..., 0] + 1j * xc[..., 1]) * np.exp(1j * phi)[:, None, :]
    np.testing.assert_allclose(out.reshape(L, H, dh // 2, 2)[..., 0], z.real, atol=1e-13)
    np.testing.assert_allclose(out.reshape(L, H, dh // 2, 2)[..., 1], z.imag, atol=1e-13)
    # token 0 sits at the origin: identity
    np.testing.assert_allclose(out[0], x[0], atol=0)
    # pair norms are preserved
    np.testing.assert_allclose(np.linalg.norm(out.reshape(L, -1, 2), axis=-1),
                               np.linalg.norm(x.reshape(L, -1, 2), axis=-1), atol=1e-12)


def test_rope_axis_layout_and_relative_positions():
    grid, dh = (3, 4, 5), 12
    dt, dhh, dw = O.rope_split(dh)
    phi = O.rope_angles(grid, dh)
    tok = lambda f, r, w: (f * grid[1] + r) * grid[2] + w
    # moving along one axis changes only that axis's block of pairs
    d = phi[tok(0, 0, 3)] - phi[tok(0, 0, 0)]
    assert np.all(d[: (dt + dhh) // 2] == 0) and np.all(d[(dt + dhh) // 2:] != 0)
    d = phi[tok(2, 0, 0)] - phi[tok(0, 0, 0)]
    assert np.all(d[dt // 2:] == 0) and np.all(d[: dt // 2] != 0)
    # first-pair frequency of each axis is 1 (theta^0): angle == position
    assert phi[tok(2, 3, 4)][0] == 2.0
    assert phi[tok(2, 3, 4)][dt // 2] == 3.0
    assert phi[tok(2, 3, 4)][(dt + dhh) // 2] == 4.0
    # <R(p) q, R(p') k> depends only on p - p'
    g = np.random.default_rng(7)
    q, k = g.standard_normal((1, dh)), g.standard_normal((1, dh))

    def dot(p1, p2):
        a = O.apply_rope(q, phi[[tok(*p1)]], 1, dh)
        b = O.apply_rope(k, phi[[tok(*p2)]], 1, dh)
        return float((a * b).sum())
    assert dot((0, 1, 2), (1, 0, 0)) == pytest.approx(dot((1, 2, 4), (2, 1, 2)), abs=1e-12)


# --------------------------------------------------------------------------
# keep-mask semantics (Sec. 3.2 gating equation; R2, R3)
# --------------------------------------------------------------------------

def test_all_keep_equals_unpruned():
    cfg = TINY
    wl, x, ctx, e0 = _layer_inputs(cfg)
    ones_h, ones_f = np.ones(cfg.n_heads), np.ones(cfg.ffn_dim)
    masked = _run_block(cfg, wl, x, ctx, e0, ones_h, ones_h, ones_f)
    raw = O.block(x, ctx, e0, wl, True, cfg.n_heads, cfg.head_dim, cfg.grid)
    assert np.array_equal(masked, raw)


def _compact_block(cfg, wl, x, ctx, e0, ms, mc, mf):
    """Second formulation: gather the kept rows / columns (numpy fancy
    indexing), run narrow matmuls, divide the QK mean square by D."""
    D, dh, eps = cfg.dim, cfg.head_dim, cfg.eps
    w = {k: np.asarray(v, np.float64) for k, v in wl.items()}
    ks = np.flatnonzero(np.repeat(ms, dh))
    kc = np.flatnonzero(np.repeat(mc, dh))
    kf = np.flatnonzero(mf)
    sh1, sc1, g1, sh2, sc2, g2 = w["mod"] + e0
    phi = O.rope_angles(cfg.grid, dh)

    def rms_full_width(t, gain):
        return t / np.sqrt((t * t).sum(-1, keepdims=True) / D + eps) * gain

    a = O.layer_norm(x, eps) * (1 + sc1) + sh1
    y = x.copy()
    if ks.size:
        q = rms_full_width(a @ w["self_wq"][ks].T + w["self_bq"][ks], w["self_gq"][ks])
        k = rms_full_width(a @ w["self_wk"][ks].T + w["self_bk"][ks], w["self_gk"][ks])
        v = a @ w["self_wv"][ks].T + w["self_bv"][ks]
        hk = ks.size // dh
        q, k = O.apply_rope(q, phi, hk, dh), O.apply_rope(k, phi, hk, dh)
        o = O.attention(q, k, v, hk, dh)
        y = y + g1 * (o @ w["self_wo"][:, ks].T + w["self_bo"])
    else:
        y = y + g1 * w["self_bo"]
    a = O.layer_norm(y, eps) * w["norm3_w"] + w["norm3_b"]
    if kc.size:
        q = rms_full_width(a @ w["cross_wq"][kc].T + w["cross_bq"][kc], w["cross_gq"][kc])
        k = rms_full_width(ctx @ w["cross_wk"][kc].T + w["cross_bk"][kc], w["cross_gk"][kc])
        v = ctx @ w["cross_wv"][kc].T + w["cross_bv"][kc]
        o = O.attention(q, k, v, kc.size // dh, dh)
        y = y + o @ w["cross_wo"][:, kc].T + w["cross_bo"]
    else:
        y = y + w["cross_bo"]
    a = O.layer_norm(y, eps) * (1 + sc2) + sh2
    u = O.gelu_tanh(a @ w["ffn_w1"][kf].T + w["ffn_b1"][kf])
    return y + g2 * (u @ w["ffn_w2"][:, kf].T + w["ffn_b2"])


@pytest.mark.parametrize("counts", [(3, 2, 640), (1, 3, 8), (2, 0, 1000), (0, 4, 0), (4, 1, 1023)])
def test_masked_dense_equals_compacted(counts):
    cfg = TINY
    h, hc, f = counts
    wl, x, ctx, e0 = _layer_inputs(cfg, seed=1, qk_gain=4.0)
    m = synth.masks_from_counts(cfg.with_(n_layers=1, ffn_chunk=1), [h], [hc], [f], seed=5)
    ms, mc, mf = m["self_head_keep"][0], m["cross_head_keep"][0], m["ffn_keep"][0]
    dense = _run_block(cfg, wl, x, ctx, e0, ms, mc, mf)
    comp = _compact_block(cfg, wl, x, ctx, e0, ms, mc, mf)
    np.testing.assert_allclose(dense, comp, rtol=0, atol=1e-11 * np.abs(dense).max())


def test_gating_equation_equals_weight_zeroing():
    """x_out = g (.) F(x_in) on the heads' projection features and the FFN
    hidden features (Sec. 3.2) is what zeroing the dense weights computes."""
    cfg = TINY
    D, dh, H, eps = cfg.dim, cfg.head_dim, cfg.n_heads, cfg.eps
    wl, x, ctx, e0 = _layer_inputs(cfg, seed=2)
    m = synth.make_masks(cfg.with_(n_layers=1), step=3, seed=9)
    ms, mc, mf = m["self_head_keep"][0], m["cross_head_keep"][0], m["ffn_keep"][0]
    w = {k: np.asarray(v, np.float64) for k, v in wl.items()}
    gs, gc = np.repeat(ms, dh).astype(float), np.repeat(mc, dh).astype(float)
    sh1, sc1, g1, sh2, sc2, g2 = w["mod"] + e0
    phi = O.rope_angles(cfg.grid, dh)
    a = O.layer_norm(x, eps) * (1 + sc1) + sh1
    q = O.rms_norm(gs * (a @ w["self_wq"].T + w["self_bq"]), w["self_gq"], eps)
    k = O.rms_norm(gs * (a @ w["self_wk"].T + w["self_bk"]), w["self_gk"], eps)
    v = gs * (a @ w["self_wv"].T + w["self_bv"])
    o = O.attention(O.apply_rope(q, phi, H, dh), O.apply_rope(k, phi, H, dh), v, H, dh)
    y = x + g1 * (o @ w["self_wo"].T + w["self_bo"])
    a = O.layer_norm(y, eps) * w["norm3_w"] + w["norm3_b"]
    q = O.rms_norm(gc * (a @ w["cross_wq"].T + w["cross_bq"]), w["cross_gq"], eps)
    k = O.rms_norm(gc * (ctx @ w["cross_wk"].T + w["cross_bk"]), w["cross_gk"], eps)
    v = gc * (ctx @ w["cross_wv"].T + w["cross_bv"])
    y = y + O.attention(q, k, v, H, dh) @ w["cross_wo"].T + w["cross_bo"]
    a = O.layer_norm(y, eps) * (1 + sc2) + sh2
    u = mf * O.gelu_tanh(a @ w["ffn_w1"].T + w["ffn_b1"])
    gated = y + g2 * (u @ w["ffn_w2"].T + w["ffn_b2"])
    zeroed = _run_block(cfg, wl, x, ctx, e0, ms, mc, mf)
    np.testing.assert_allclose(zeroed, gated, rtol=0, atol=1e-12 * np.abs(gated).max())


def test_everything_pruned_closed_form():
    cfg = TINY
    wl, x, ctx, e0 = _layer_inputs(cfg, seed=3)
    z_h, z_f = np.zeros(cfg.n_heads), np.zeros(cfg.ffn_dim)
    out = _run_block(cfg, wl, x, ctx, e0, z_h, z_h, z_f)
    mod = wl["mod"] + e0
    expect = x + mod[2] * wl["self_bo"] + wl["cross_bo"] + mod[5] * wl["ffn_b2"]
    np.testing.assert_allclose(out, expect, rtol=0, atol=1e-14)


def test_block_gate_and_zero_gates_give_identity():
    cfg = TINY
    wl, x, ctx, e0 = _layer_inputs(cfg, seed=4)
    ones_h, ones_f = np.ones(cfg.n_heads), np.ones(cfg.ffn_dim)
    assert np.array_equal(_run_block(cfg, wl, x, ctx, e0, ones_h, ones_h, ones_f, keep=False), x)
    wl = dict(wl)
    wl["mod"] = wl["mod"].copy()
    wl["mod"][2] = -e0[2]
    wl["mod"][5] = -e0[5]
    wl["cross_bo"] = np.zeros_like(wl["cross_bo"])
    out = _run_block(cfg, wl, x, ctx, e0, ones_h, np.zeros(cfg.n_heads), ones_f)
    np.testing.assert_allclose(out, x, rtol=0, atol=1e-14)


def test_row_sampling_matches_full_block():
    cfg = TINY
    wl, x, ctx, e0 = _layer_inputs(cfg, seed=5)
    m = synth.make_masks(cfg.with_(n_layers=1), step=2)
    args = (m["self_head_keep"][0], m["cross_head_keep"][0], m["ffn_keep"][0])
    full = _run_block(cfg, wl, x, ctx, e0, *args)
    rows = np.array([0, 5, 77, 127])
    np.testing.assert_allclose(_run_block(cfg, wl, x, ctx, e0, *args, rows=rows), full[rows],
                               rtol=0, atol=1e-13)


def _permute_heads(wl, pre, perm, dh):
    chan = (perm[:, None] * dh + np.arange(dh)[None, :]).reshape(-1)
    w = dict(wl)
    for p in ("q", "k", "v"):
        w[f"{pre}_w{p}"] = wl[f"{pre}_w{p}"][chan]
        w[f"{pre}_b{p}"] = wl[f"{pre}_b{p}"][chan]
    for p in ("q", "k"):
        w[f"{pre}_g{p}"] = wl[f"{pre}_g{p}"][chan]
    w[f"{pre}_wo"] = wl[f"{pre}_wo"][:, chan]
    return w


def test_permutation_invariance():
    cfg = TINY
    wl, x, ctx, e0 = _layer_inputs(cfg, seed=6)
    m = synth.make_masks(cfg.with_(n_layers=1), step=1, seed=3)
    ms, mc, mf = m["self_head_keep"][0], m["cross_head_keep"][0], m["ffn_keep"][0]
    base = _run_block(cfg, wl, x, ctx, e0, ms, mc, mf)
    g = np.random.default_rng(8)
    ph, pc, pf = g.permutation(cfg.n_heads), g.permutation(cfg.n_heads), g.permutation(cfg.ffn_dim)
    w2 = _permute_heads(_permute_heads(wl, "self", ph, cfg.head_dim), "cross", pc, cfg.head_dim)
    w2["ffn_w1"], w2["ffn_b1"], w2["ffn_w2"] = wl["ffn_w1"][pf], wl["ffn_b1"][pf], wl["ffn_w2"][:, pf]
    out = _run_block(cfg, w2, x, ctx, e0, ms[ph], mc[pc], mf[pf])
    np.testing.assert_allclose(out, base, rtol=0, atol=1e-12 * np.abs(base).max())


# --------------------------------------------------------------------------
# step, sampler
# --------------------------------------------------------------------------

def test_step_with_all_blocks_gated_off_closed_form():
    cfg = MICRO
    w = synth.make_weights(cfg, seed=1)
    D = cfg.dim
    c = np.linspace(-0.5, 0.5, D).astype(np.float32)
    w["t_w2"] = np.zeros_like(w["t_w2"])
    w["t_b2"] = c
    z = synth.make_latents(cfg, seed=2)
    ctx = synth.make_context(cfg, seed=2)
    m = synth.make_masks(cfg, step=0)
    m["block_keep"][:] = 0
    v = O.step(z, 750, ctx, w, m, cfg)
    x = z[0].astype(np.float64) @ w["patch_w"].T.astype(np.float64) + w["patch_b"]
    hm = w["head_mod"].astype(np.float64)
    sh, sc = hm[0] + c, hm[1] + c
    expect = (O.layer_norm(x) * (1 + sc) + sh) @ w["head_w"].T.astype(np.float64) + w["head_b"]
    np.testing.assert_allclose(v[0], expect, rtol=0, atol=1e-12)


def test_time_embedding_reshape_order():
    cfg = MICRO
    w = synth.make_weights(cfg, seed=1)
    w["t_w3"] = np.zeros_like(w["t_w3"])
    e, e0 = O.time_embedding(w, 500.0)
    assert e0.shape == (6, cfg.dim)
    np.testing.assert_array_equal(e0[4], w["t_b3"][4 * cfg.dim:5 * cfg.dim])


def test_time_embedding_matches_torch_modules():
    """e = Linear2(SiLU(Linear1(emb))) and e0 = Linear3(SiLU(e)) reshaped to
    [6, D], built from torch.nn modules loaded with the same weights, every
    weight and bias non-zero: a dropped inner layer or SiLU, a transposed
    matrix, a missing bias or a wrong reshape order fails here."""
    cfg = MICRO
    w = synth.make_weights(cfg, seed=4)
    D, Fq = cfg.dim, cfg.freq_dim
    for k in ("t_w1", "t_w2", "t_w3", "t_b1", "t_b2", "t_b3"):
        assert np.all(w[k] != 0), k

    def lin(wk, bk):
        m = torch.nn.Linear(w[wk].shape[1], w[wk].shape[0], dtype=torch.float64)
        with torch.no_grad():
            m.weight.copy_(torch.from_numpy(w[wk].astype(np.float64)))
            m.bias.copy_(torch.from_numpy(w[bk].astype(np.float64)))
        return m

    mlp = torch.nn.Sequential(lin("t_w1", "t_b1"), torch.nn.SiLU(), lin("t_w2", "t_b2"))
    head = torch.nn.Sequential(torch.nn.SiLU(), lin("t_w3", "t_b3"), torch.nn.Unflatten(-1, (6, D)))
    for t in (999.0, 750.0, 250.0, 0.0):
        emb = torch.from_numpy(O.sinusoid(t, Fq))
        with torch.no_grad():
            e_ref = mlp(emb)
            e0_ref = head(e_ref)
        e, e0 = O.time_embedding(w, t)
        np.testing.assert_allclose(e, e_ref.numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(e0, e0_ref.numpy(), rtol=0, atol=1e-12)
    # the modulation rows differ between timesteps (t reaches every row)
    assert not np.allclose(O.time_embedding(w, 999.0)[1], O.time_embedding(w, 250.0)[1])


def test_euler_and_sigma_schedule():
    sig = O.sigmas((999, 750, 500, 250))
    assert sig == [0.999, 0.75, 0.5, 0.25, 0.0]
    assert sum(sig[s + 1] - sig[s] for s in range(4)) == pytest.approx(-0.999, abs=1e-15)
    z = np.arange(5.0)
    assert np.array_equal(O.euler(z, np.zeros(5), 0.999, 0.75), z)


def test_denoise_constant_prediction_closed_form():
    """With zero patch weights and constant time embedding the prediction is
    the same vector at every step, so four Euler steps move z by -sigma_1 v."""
    cfg = MICRO
    w = synth.make_weights(cfg, seed=3)
    w["patch_w"] = np.zeros_like(w["patch_w"])
    w["t_w2"] = np.zeros_like(w["t_w2"])
    masks = [synth.make_masks(cfg, s) for s in range(4)]
    for m in masks:
        m["block_keep"][:] = 0
    z = synth.make_latents(cfg, seed=4)
    ctx = synth.make_context(cfg, seed=4)
    v = O.step(z, 999, ctx, w, masks[0], cfg)
    out = O.denoise(z, ctx, w, masks, cfg)
    np.testing.assert_allclose(out, z - 0.999 * v, rtol=0, atol=1e-12)


def test_full_denoise_runs_and_is_finite():
    cfg = MICRO
    w = synth.make_weights(cfg, seed=0)
    masks = [synth.make_masks(cfg, s) for s in range(4)]
    z = synth.make_latents(cfg)
    ctx = synth.make_context(cfg)
    out = O.denoise(z, ctx, w, masks, cfg)
    assert out.shape == z.shape and np.all(np.isfinite(out))
    # float32 and float64 oracles agree to float32 rounding
    out32 = O.denoise(z, ctx, w, masks, cfg, dtype=np.float32)
    assert np.max(np.abs(out32 - out)) / np.max(np.abs(out)) < 1e-5


def test_renoise_sampler_on_the_exact_flow():
    """On the straight path z_sigma = (1 - sigma) x + sigma eps with the exact
    velocity v = eps - x (R7): the clean estimate is x at every level,
    re-noising with the same eps lands on the path, and it coincides with
    the Euler step; to sigma = 0 both give x."""
    g = np.random.default_rng(5)
    x, eps = g.standard_normal(64), g.standard_normal(64)
    v = eps - x
    for s_from, s_to in [(0.999, 0.75), (0.75, 0.5), (0.25, 0.0)]:
        z = (1 - s_from) * x + s_from * eps
        np.testing.assert_allclose(O.predict_clean(z, v, s_from), x, rtol=0, atol=1e-12)
        on_path = (1 - s_to) * x + s_to * eps
        np.testing.assert_allclose(O.renoise(O.predict_clean(z, v, s_from), s_to, eps), on_path,
                                   rtol=0, atol=1e-12)
        np.testing.assert_allclose(O.euler(z, v, s_from, s_to), on_path, rtol=0, atol=1e-12)
    # a different eps moves the re-noised point by sigma_to (eps' - eps) only
    eps2 = g.standard_normal(64)
    z = 0.25 * x + 0.75 * eps
    np.testing.assert_allclose(O.renoise(O.predict_clean(z, v, 0.75), 0.5, eps2) -
                               O.euler(z, v, 0.75, 0.5), 0.5 * (eps2 - eps), rtol=0, atol=1e-12)


def test_rollout_samplers_and_start_step():
    """Both samplers end with the clean estimate of the last step; the Euler
    rollout is the plain denoise; a rollout started at step s equals steps
    s.. of the full chain fed the same intermediate latent."""
    cfg = MICRO
    w = synth.make_weights(cfg, seed=2)
    masks = [synth.make_masks(cfg, s) for s in range(4)]
    z = synth.make_latents(cfg, seed=6)
    ctx = synth.make_context(cfg, seed=6)
    g = np.random.default_rng(7)
    eps = [g.standard_normal(z.shape) for _ in range(4)]
    np.testing.assert_array_equal(O.rollout(z, ctx, w, masks, cfg, sampler="euler"),
                                  O.denoise(z, ctx, w, masks, cfg))
    # one step by hand, then the rest through rollout(start=1)
    sig = O.sigmas(cfg.timesteps)
    v0 = O.step(z, cfg.timesteps[0], ctx, w, masks[0], cfg)
    z1 = O.renoise(O.predict_clean(z, v0, sig[0]), sig[1], eps[0])
    full = O.rollout(z, ctx, w, masks, cfg, eps, sampler="renoise")
    np.testing.assert_allclose(O.rollout(z1, ctx, w, masks, cfg, eps, start=1), full,
                               rtol=0, atol=1e-12)
    # the last step returns z - sigma_T v regardless of the sampler
    z3 = synth.make_latents(cfg, seed=8)
    v3 = O.step(z3, cfg.timesteps[3], ctx, w, masks[3], cfg)
    np.testing.assert_allclose(O.rollout(z3, ctx, w, masks, cfg, eps, start=3),
                               z3 - sig[3] * v3, rtol=0, atol=1e-12)
    np.testing.assert_allclose(O.rollout(z3, ctx, w, masks, cfg, start=3, sampler="euler"),
                               z3 - sig[3] * v3, rtol=0, atol=1e-12)
