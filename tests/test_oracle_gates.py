"""Pins of the oracle's hard-gate rules and FFN reorder (Sec. 4.1, App. A)."""
import numpy as np

import oracle as O
from workloads import get_config, synth

MICRO = get_config("tiny").with_(name="micro", n_layers=1, grid=(1, 4, 4), text_len=8)


def test_block_gate_is_strict_indicator():
    m = np.array([0.5, 0.0, -1e-9, 1e-30, -0.0], np.float32)
    g = O.hard_gates(m, np.zeros((5, 8)), np.zeros((5, 8)), np.zeros((5, 1)), 2, 4, 8)
    assert g["block_keep"].tolist() == [1, 0, 0, 1, 0]


def test_head_gate_uses_the_mean_of_its_mask_values():
    # two heads of 4 features per layer
    m_self = np.array([[3, -1, -1, -1,   1, -1, 1, -1],     # mean 0 -> pruned, mean 0 -> pruned
                       [3, -1, -1, -0.5, -1, -1, -1, 5]],   # mean 0.125 -> kept, 0.5 -> kept
                      np.float32)
    m_cross = -m_self
    g = O.hard_gates(np.ones(2), m_self, m_cross, np.zeros((2, 1)), 2, 4, 8)
    assert g["self_head_keep"].tolist() == [[0, 0], [1, 1]]
    assert g["cross_head_keep"].tolist() == [[0, 0], [0, 0]]
    # a head whose values are all positive but one large negative is pruned
    g = O.hard_gates(np.ones(1), np.array([[1, 1, 1, -3.5, 0, 0, 0, 1e-3]]),
                     np.zeros((1, 8)), np.zeros((1, 1)), 2, 4, 8)
    assert g["self_head_keep"].tolist() == [[0, 1]]


def test_ffn_gate_repeats_one_mask_per_chunk():
    m_ffn = np.array([[1.0, 0.0, -1.0, 2e-7]])
    g = O.hard_gates(np.ones(1), np.zeros((1, 8)), np.zeros((1, 8)), m_ffn, 2, 4, 8)
    assert g["ffn_keep"].tolist() == [[1] * 8 + [0] * 16 + [1] * 8]


def test_hard_gates_of_random_masks_are_valid_structures():
    g = np.random.default_rng(0)
    N, H, dh, F, C = 3, 4, 64, 1024, 8
    out = O.hard_gates(g.standard_normal(N), g.standard_normal((N, H * dh)),
                       g.standard_normal((N, H * dh)), g.standard_normal((N, F // C)), H, dh, C)
    f = out["ffn_keep"].reshape(N, F // C, C)
    assert np.all(f.min(axis=2) == f.max(axis=2))            # whole chunks
    for k in ("block_keep", "self_head_keep", "cross_head_keep", "ffn_keep"):
        assert out[k].dtype == np.uint8 and set(np.unique(out[k])) <= {0, 1}


def test_ffn_norms_and_reorder():
    cfg = MICRO
    wl = synth.make_layer_weights(cfg, 0, 3)
    norms = O.ffn_channel_norms(wl)
    j = 17   # brute force for one channel
    s = sum(float(v) ** 2 for v in wl["ffn_w1"][j]) + float(wl["ffn_b1"][j]) ** 2 + \
        sum(float(wl["ffn_w2"][d, j]) ** 2 for d in range(cfg.dim))
    assert abs(norms[j] - np.sqrt(s)) <= 1e-12 * np.sqrt(s)
    perm, wr = O.ffn_reorder(wl)
    assert sorted(perm.tolist()) == list(range(cfg.ffn_dim))
    assert np.all(np.diff(norms[perm]) <= 0)
    np.testing.assert_array_equal(wr["ffn_w2"][:, 5], wl["ffn_w2"][:, perm[5]])


def test_ffn_reorder_preserves_the_block():
    """Permuting the hidden channels (W1 rows, b1, W2 columns) together is
    function-preserving: the block output is unchanged."""
    cfg = MICRO
    wl = synth.make_layer_weights(cfg, 0, 4)
    _, wr = O.ffn_reorder(wl)
    x = synth.make_block_input(cfg, 4)[0]
    ctx = synth.make_context(cfg, 4)[0]
    e0 = synth.make_e0(cfg, 4, std=0.3)
    ones_h = np.ones(cfg.n_heads)
    ref = O.block(x, ctx, e0, O.apply_keep(wl, ones_h, ones_h, np.ones(cfg.ffn_dim), cfg.head_dim),
                  True, cfg.n_heads, cfg.head_dim, cfg.grid, cfg.rope_theta, cfg.eps)
    got = O.block(x, ctx, e0, O.apply_keep(wr, ones_h, ones_h, np.ones(cfg.ffn_dim), cfg.head_dim),
                  True, cfg.n_heads, cfg.head_dim, cfg.grid, cfg.rope_theta, cfg.eps)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * np.abs(ref).max())
