"""Seeded input generators, the FLOP counter and the paper's printed figures."""
import json
import os

import numpy as np
import pytest
import torch

from paper_2607_06631_amd import flops
from workloads import get_config, synth

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")))


def test_bf16_round_matches_torch():
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(10000).astype(np.float32) * 10,
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, 1e-40], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    assert np.array_equal(synth.bf16_round(x), ref)


@pytest.mark.parametrize("name", ["tiny", "wan1.3b_block", "wan14b_block"])
def test_fixed_count_masks(name):
    cfg = get_config(name)
    for s in range(len(cfg.keep_heads)):
        m = synth.make_masks(cfg, s)
        assert m["self_head_keep"].shape == (cfg.n_layers, cfg.n_heads)
        assert np.all(m["self_head_keep"].sum(1) == cfg.keep_heads[s])
        assert np.all(m["cross_head_keep"].sum(1) == cfg.keep_heads[s])
        assert np.all(m["ffn_keep"].sum(1) == cfg.keep_ffn[s])
        assert np.all(m["block_keep"] == 1)
        m2 = synth.make_masks(cfg, s)
        for k in m:
            assert np.array_equal(m[k], m2[k])


def test_masks_chunked_and_independent():
    cfg = get_config("tiny")
    m = synth.make_masks(cfg, 2)
    chunks = m["ffn_keep"].reshape(cfg.n_layers, -1, GOLDEN["ffn_chunk_size"]["value"])
    assert np.all((chunks.min(-1) == chunks.max(-1)))
    # self and cross subsets drawn independently (not all equal across layers/steps)
    diffs = sum(not np.array_equal(synth.make_masks(cfg, s)["self_head_keep"],
                                   synth.make_masks(cfg, s)["cross_head_keep"]) for s in range(1, 4))
    assert diffs >= 1


def _frac(cfg, m, L=None):
    N, dh = cfg.n_layers, cfg.head_dim
    L = cfg.seq_len if L is None else L
    kept = flops.structure_flops(L, cfg.text_len, cfg.dim, dh, m["self_head_keep"].sum(1),
                                 m["cross_head_keep"].sum(1), m["ffn_keep"].sum(1))
    dense = flops.structure_flops(L, cfg.text_len, cfg.dim, dh, [cfg.n_heads] * N,
                                  [cfg.n_heads] * N, [cfg.ffn_dim] * N)
    return kept / dense


def test_flop_fractions_closed_form():
    c3 = get_config("wan14b_block")
    got = [_frac(c3, synth.make_masks(c3, s)) for s in range(4)]
    np.testing.assert_allclose(got, [1.0, 0.8, 0.7, 0.6], atol=2e-5)
    c2 = get_config("wan1.3b_block")
    assert _frac(c2, synth.make_masks(c2, 0)) == pytest.approx(0.75, abs=1e-12)
    c1 = get_config("tiny")
    got = [_frac(c1, synth.make_masks(c1, s)) for s in range(4)]
    np.testing.assert_allclose(got, [1.0, 0.75, 0.685, 0.5], atol=2e-3)


def test_dense_block_flops_known_values():
    c3 = get_config("wan14b_block")
    t = flops.block_terms(c3.seq_len, c3.text_len, c3.dim, c3.head_dim, 40, 40, c3.ffn_dim)
    assert sum(t.values()) / 1e12 == pytest.approx(41.96, abs=0.01)
    assert t["self_attn"] / 1e12 == pytest.approx(21.98, abs=0.01)
    c5 = get_config("wan14b_720p")
    assert flops.block_flops(c5.seq_len, 512, 5120, 128, 40, 40, 13824) / 1e12 == pytest.approx(163.1, abs=0.1)


def test_recipe_matches_paper_figures():
    rho = np.array(synth.RECIPE_RHO)
    assert rho.mean() == pytest.approx(1 - GOLDEN["wan14b_per_step_flops_removed"]["value"], abs=1e-3)
    # same U shape as the paper's Wan-1.3B retention (ends high, middle low)
    paper = np.array(GOLDEN["wan13b_step_flops_retention"]["value"])
    assert np.array_equal(np.argsort(rho), np.argsort(paper))
    cfg = get_config("wan14b_480p")
    fr = []
    for s in range(4):
        m = synth.make_masks(cfg, s)
        fr.append(_frac(cfg, m))
        assert abs(fr[-1] - rho[s]) <= synth.RECIPE_TOL + 1e-12
        # deeper layers keep fewer attention heads at the middle steps
        h = m["self_head_keep"].sum(1)
        if s in (1, 2):
            assert h[:10].mean() > h[-10:].mean()
        assert np.all(m["ffn_keep"].sum(1) % 8 == 0)
    assert np.mean(fr) == pytest.approx(0.76, abs=0.005)
