"""The bf16 storage floor behind the block tolerances (CPU).

tests/bf16_emulation.py re-runs the oracle's block rounding to bfloat16
exactly where the GPU path stores activations.  Its distance to the oracle
is the error that bf16 storage alone causes; a GPU tolerance must sit above
it with margin, and a check only has power if a plausible kernel mistake
moves the result well past the tolerance.  These cases are the GPU tests'
own inputs; each prints its floor.
"""
import numpy as np

import oracle as O
from tests import bf16_emulation as E
from workloads import get_config, synth

TOL = 2e-2


def _floor(cfg, wl, masks, x, ctx, e0, rows=None):
    wz = O.apply_keep(wl, masks["self_head_keep"][0], masks["cross_head_keep"][0],
                      masks["ffn_keep"][0], cfg.head_dim)
    ref = O.block(x, ctx, e0, wz, True, cfg.n_heads, cfg.head_dim, cfg.grid, cfg.rope_theta,
                  cfg.eps, rows=rows)
    em = E.block(x, ctx, e0, wz, True, cfg.n_heads, cfg.head_dim, cfg.grid, cfg.rope_theta,
                 cfg.eps, rows=rows)
    xr = np.asarray(x, dtype=np.float64)[rows if rows is not None else slice(None)]
    err = np.abs(em - ref).max()
    return err / np.abs(ref).max(), err / np.abs(ref - xr).max()


def test_sharp_attention_block_floor():
    """test_gpu_block.py::test_wan13b_width_block_sharp_attention's inputs."""
    cfg = get_config("wan1.3b_block").with_(name="mid13", grid=(3, 10, 13), text_len=77, batch=1)
    w = synth.make_weights(cfg, seed=1, qk_gain=2.0)
    masks = synth.make_masks(cfg, 0)
    x = synth.make_block_input(cfg, 8, scale=0.5)[0]
    ctx = synth.make_context(cfg, 8)[0]
    e0 = synth.make_e0(cfg, 8, std=0.3)
    e0[5] = -w["layers"][0]["mod"][5]
    out, upd = _floor(cfg, w["layers"][0], masks, x, ctx, e0)
    print(f"sharp-attention block: bf16 storage floor {out:.3e} (update-relative {upd:.3e})")
    assert out < TOL / 1.5


def test_self_attention_dominated_floor_and_power():
    """test_gpu_fullsize.py::test_block_fullsize_self_attention_dominates's
    Wan-1.3B-width inputs at full length (QK gains x2, cross heads pruned,
    FFN gate 0, 9 of 12 heads; 96 of its rows): the floor on the update is
    below the tolerance, and a uniform self-attention is far above it."""
    cfg = get_config("wan1.3b_block")
    wl = synth.make_layer_weights(cfg, 0, 0, qk_gain=2.0)
    masks = synth.masks_from_counts(cfg, [9], [0], [cfg.keep_ffn[-1]])
    x = synth.make_block_input(cfg, 90, scale=0.5)[0]
    ctx = synth.make_context(cfg, 90)[0]
    e0 = synth.make_e0(cfg, 90, std=0.3)
    e0[5] = -wl["mod"][5]
    rows = np.random.default_rng(90).choice(cfg.seq_len, 96, replace=False)
    out, upd = _floor(cfg, wl, masks, x, ctx, e0, rows)
    print(f"self-attention-dominated block: floor {out:.3e} (update-relative {upd:.3e})")
    assert upd < TOL / 1.25
    # uniform attention: zero queries give every key the same score
    wz = O.apply_keep(wl, masks["self_head_keep"][0], masks["cross_head_keep"][0],
                      masks["ffn_keep"][0], cfg.head_dim)
    ref = O.block(x, ctx, e0, wz, True, cfg.n_heads, cfg.head_dim, cfg.grid, rows=rows)
    wu = dict(wz, self_wq=wz["self_wq"] * 0, self_bq=wz["self_bq"] * 0)
    uni = O.block(x, ctx, e0, wu, True, cfg.n_heads, cfg.head_dim, cfg.grid, rows=rows)
    power = np.abs(uni - ref).max() / np.abs(ref - x[rows]).max()
    print(f"  uniform self-attention moves the update by {power:.3e}")
    assert power > 3 * TOL
