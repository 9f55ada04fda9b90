"""dif_ffn_reorder: the App. A channel sort, checked against the oracle."""
import numpy as np
import pytest

import oracle as O
from paper_2607_06631_amd import binding as B
from tests.gpu_util import make_model, rel_err, say, to_dev, to_np
from workloads import get_config, synth

pytestmark = pytest.mark.gpu

TINY = get_config("tiny")
MID14 = get_config("wan14b_block").with_(name="mid14", grid=(1, 4, 6), text_len=32)


@pytest.mark.parametrize("cfg", [TINY, MID14], ids=["tiny_f32", "wan14b_width_bf16"])
def test_reorder_permutation_and_gathers(cfg):
    say(f"ffn reorder {cfg.name}")
    w = synth.make_weights(cfg.with_(n_layers=1), seed=5)
    model = make_model(cfg.with_(n_layers=1), w)
    perm, w1, b1, w2 = B.dif_ffn_reorder(model, 0)
    wl = w["layers"][0]
    F = cfg.ffn_dim
    assert sorted(perm.tolist()) == list(range(F))
    norms = O.ffn_channel_norms(wl)
    # non-increasing along the permutation (up to rounding of near-equal norms)
    assert np.all(np.diff(norms[perm]) <= 1e-9 * norms.max())
    assert np.array_equal(to_np(w1), wl["ffn_w1"][perm])
    assert np.array_equal(to_np(b1), wl["ffn_b1"][perm])
    assert np.array_equal(to_np(w2), wl["ffn_w2"][:, perm])


def test_reordered_model_computes_the_same_block():
    import torch
    cfg = TINY.with_(n_layers=1)
    say("ffn reorder is function-preserving through the GPU block")
    w = synth.make_weights(cfg, seed=6)
    model = make_model(cfg, w)
    perm, w1, b1, w2 = B.dif_ffn_reorder(model, 0)
    w_re = dict(w)
    w_re["layers"] = [dict(w["layers"][0], ffn_w1=to_np(w1), ffn_b1=to_np(b1), ffn_w2=to_np(w2))]
    model_re = make_model(cfg, w_re)
    masks = synth.all_keep_masks(cfg)
    x = synth.make_block_input(cfg, 6, scale=0.5)
    ctx = synth.make_context(cfg, 6)
    e0 = synth.make_e0(cfg, 6, std=0.3)
    outs = []
    for m in (model, model_re):
        plan = B.dif_plan_step(m, 0, cfg.timesteps[0], masks)
        xd = to_dev(x, cfg)
        ws = B.workspace(m, 1, cfg.seq_len, cfg.text_len)
        B.dif_block_forward(plan, 0, xd, to_dev(ctx, cfg), to_dev(e0, dtype=torch.float32), ws)
        torch.cuda.synchronize()
        outs.append(to_np(xd))
    assert rel_err(outs[1], outs[0]) <= 1e-5
