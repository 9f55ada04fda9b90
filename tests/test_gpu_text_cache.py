"""Cross-attention text cache through the C ABI.

The cached calls must give the same bits as the calls that take the context
(the cache holds exactly the projections those calls compute, and each step
takes its kept heads from it), and so the oracle's results at the usual
tolerances: 1e-4 for the float32 configuration, 2e-2 for bf16.
"""
import numpy as np
import pytest

import oracle as O
from paper_2607_06631_amd import binding as B
from tests.gpu_util import make_model, rel_err, say, to_dev, to_np
from workloads import get_config, synth

pytestmark = pytest.mark.gpu

TINY = get_config("tiny")
MID14 = get_config("wan14b_block").with_(name="mid14c", grid=(2, 5, 7), text_len=77, batch=2)


@pytest.fixture(scope="module")
def tiny():
    w = synth.make_weights(TINY, seed=0, qk_gain=2.0)
    return w, make_model(TINY, w)


def _step_pair(model, cfg, masks, kind, t, z0, ctx):
    import torch
    plan = B.dif_plan_step(model, 0, t, masks, kind=kind)
    cd = to_dev(ctx, cfg)
    ws = B.workspace(model, z0.shape[0], cfg.seq_len, ctx.shape[1])
    cache = B.dif_text_cache_build(model, cd)
    z = to_dev(z0, dtype=torch.float32)
    va, vb = torch.empty_like(z), torch.empty_like(z)
    B.dif_step_forward(plan, z, t, cd, va, ws)
    B.dif_step_forward_cached(plan, z, t, cache, vb, ws)
    torch.cuda.synchronize()
    return to_np(va), to_np(vb)


@pytest.mark.parametrize("kind", ["compact", "indexed"])
@pytest.mark.parametrize("step", [0, 2, 3])
def test_tiny_cached_step_equals_uncached(tiny, kind, step):
    w, model = tiny
    say(f"tiny cached step {step}, {kind} plan")
    masks = synth.make_masks(TINY, step)
    z0 = synth.make_latents(TINY, seed=70 + step)
    ctx = synth.make_context(TINY, seed=70 + step)
    va, vb = _step_pair(model, TINY, masks, kind, TINY.timesteps[step], z0, ctx)
    assert np.array_equal(va, vb)
    ref = O.step(z0, TINY.timesteps[step], ctx, w, masks, TINY)
    assert rel_err(vb, ref) <= 1e-4


@pytest.mark.parametrize("case", ["no_cross_heads", "one_cross_head", "block_off", "text_len_1",
                                  "ragged_text_batch_3"])
def test_tiny_cached_edge_cases(tiny, case):
    w, model = tiny
    say(f"tiny cached step, {case}")
    N, H = TINY.n_layers, TINY.n_heads
    cfg = TINY.with_(batch=3) if case == "ragged_text_batch_3" else TINY
    cross = {"no_cross_heads": 0, "one_cross_head": 1}.get(case, H - 1)
    masks = synth.masks_from_counts(TINY.with_(ffn_chunk=1), [H] * N, [cross] * N, [900] * N, seed=9,
                                    block_keep=[1, 0] if case == "block_off" else None)
    Lc = {"text_len_1": 1, "ragged_text_batch_3": 13}.get(case, TINY.text_len)
    z0 = synth.make_latents(cfg, seed=80)
    ctx = synth.make_context(cfg, seed=80, text_len=Lc)
    va, vb = _step_pair(model, TINY, masks, "compact", TINY.timesteps[1], z0, ctx)
    assert np.array_equal(va, vb)
    ref = np.stack([O.step(z0[b:b + 1], TINY.timesteps[1], ctx[b:b + 1], w, masks, TINY)[0]
                    for b in range(z0.shape[0])])
    assert rel_err(vb, ref) <= 1e-4


def test_tiny_cached_rollout_matches_oracle(tiny):
    """One cache shared by the four steps of a re-noise rollout."""
    import torch
    w, model = tiny
    say("tiny cached 4-step rollout")
    masks = [synth.make_masks(TINY, s) for s in range(4)]
    plans = [B.dif_plan_step(model, s, TINY.timesteps[s], masks[s], kind="indexed") for s in range(4)]
    z0 = synth.make_latents(TINY, seed=90)
    ctx = synth.make_context(TINY, seed=90)
    eps = synth.make_renoise_eps(TINY, seed=90)
    cd = to_dev(ctx, TINY)
    ws = B.workspace(model, 1, TINY.seq_len, TINY.text_len)
    ed = [to_dev(e, dtype=torch.float32) for e in eps]
    cache = B.dif_text_cache_build(model, cd)
    za = to_dev(z0, dtype=torch.float32)
    zb = to_dev(z0, dtype=torch.float32)
    v = torch.empty_like(za)
    B.dif_rollout(plans, TINY.timesteps, za, cd, v, ws, eps=ed, sampler="renoise")
    B.dif_rollout_cached(plans, TINY.timesteps, zb, cache, v, ws, eps=ed, sampler="renoise")
    torch.cuda.synchronize()
    assert np.array_equal(to_np(za), to_np(zb))
    ref = O.rollout(z0, ctx, w, masks, TINY, eps, sampler="renoise")
    assert rel_err(to_np(zb), ref) <= 1e-4


def test_cache_errors(tiny):
    import torch
    _, model = tiny
    say("text cache argument errors")
    masks = synth.make_masks(TINY, 1)
    plan = B.dif_plan_step(model, 1, 750.0, masks)
    cd = to_dev(synth.make_context(TINY, seed=1), TINY)
    cache = B.dif_text_cache_build(model, cd)
    z = torch.zeros(1, TINY.seq_len, TINY.patch_dim, device="cuda")
    v = torch.empty_like(z)
    ws = B.workspace(model, 1, TINY.seq_len, TINY.text_len)
    small = B.TextCache(cache.mem[: cache.mem.numel() - 256], 1, TINY.text_len)
    with pytest.raises(B.DifError):
        B.dif_step_forward_cached(plan, z, 750.0, small, v, ws)
    with pytest.raises(B.DifError):
        B.dif_text_cache_bytes(model, 1, TINY.text_len + 1)
    with pytest.raises(B.DifError):
        B.dif_text_cache_bytes(model, 0, 4)
    torch.cuda.synchronize()


@pytest.fixture(scope="module")
def mid14():
    w = synth.make_weights(MID14, seed=0)
    return w, make_model(MID14, w)


@pytest.mark.parametrize("kind", ["compact", "indexed"])
def test_wan14b_width_cached_block_batch_2(mid14, kind):
    """bf16, 40 heads of 128, two samples (the per-sample value stride), 77 text tokens."""
    import torch
    w, model = mid14
    say(f"wan14b-width cached block B=2, {kind} plan")
    masks = synth.make_masks(MID14, 2)
    x = synth.make_block_input(MID14, 5, scale=0.5)
    ctx = synth.make_context(MID14, 5)
    e0 = synth.make_e0(MID14, 5, std=0.3)
    plan = B.dif_plan_step(model, 0, MID14.timesteps[0], masks, kind=kind)
    cd, ed = to_dev(ctx, MID14), to_dev(e0, dtype=torch.float32)
    ws = B.workspace(model, MID14.batch, MID14.seq_len, MID14.text_len)
    cache = B.dif_text_cache_build(model, cd)
    xa, xb = to_dev(x, MID14), to_dev(x, MID14)
    B.dif_block_forward(plan, 0, xa, cd, ed, ws)
    B.dif_block_forward_cached(plan, 0, xb, cache, ed, ws)
    torch.cuda.synchronize()
    got = to_np(xb)
    assert np.array_equal(to_np(xa), got)
    wl = w["layers"][0]
    wz = O.apply_keep(wl, masks["self_head_keep"][0], masks["cross_head_keep"][0],
                      masks["ffn_keep"][0], MID14.head_dim, np.float64)
    ref = np.stack([O.block(x[b], ctx[b], e0, wz, True, MID14.n_heads, MID14.head_dim, MID14.grid,
                            MID14.rope_theta, MID14.eps) for b in range(MID14.batch)])
    err = rel_err(got, ref)
    say(f"  rel err {err:.3e}")
    assert err <= 2e-2
