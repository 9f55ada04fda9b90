"""Block and step parity of the HIP path (through the C ABI) with the oracle.

Tolerances (max |g - r| / max |r|): 1e-4 for float32 configurations, 2e-2
for bfloat16 ones.  bf16 cases feed both sides the same bf16-rounded
weights and inputs; the oracle computes in float64.
"""
import numpy as np
import pytest

import oracle as O
from paper_2607_06631_amd import binding as B
from tests.gpu_util import make_model, rel_err, say, to_dev, to_np
from workloads import get_config, synth

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}
TINY = get_config("tiny")
# Wan-1.3B / Wan-14B block widths on small ragged token grids
MID13 = get_config("wan1.3b_block").with_(name="mid13", grid=(3, 10, 13), text_len=77, batch=2)
MID14 = get_config("wan14b_block").with_(name="mid14", grid=(2, 7, 11), text_len=512)


def oracle_block(cfg, wl, masks, layer, x, ctx, e0, rows=None, dtype=np.float64):
    wz = O.apply_keep(wl, masks["self_head_keep"][layer], masks["cross_head_keep"][layer],
                      masks["ffn_keep"][layer], cfg.head_dim, dtype)
    return np.stack([O.block(x[b], ctx[b], e0, wz, bool(masks["block_keep"][layer]), cfg.n_heads,
                             cfg.head_dim, cfg.grid, cfg.rope_theta, cfg.eps, rows=rows, dtype=dtype)
                     for b in range(x.shape[0])])


def gpu_block(model, cfg, masks, step, layer, x, ctx, e0):
    import torch
    plan = B.dif_plan_step(model, step, cfg.timesteps[step], masks)
    xd, cd = to_dev(x, cfg), to_dev(ctx, cfg)
    ed = to_dev(e0, dtype=torch.float32)
    ws = B.workspace(model, x.shape[0], x.shape[1], ctx.shape[1])
    B.dif_block_forward(plan, layer, xd, cd, ed, ws)
    torch.cuda.synchronize()
    return to_np(xd), plan


def _inputs(cfg, seed, x_scale=0.5, e0_std=0.3):
    x = synth.make_block_input(cfg, seed, scale=x_scale)
    ctx = synth.make_context(cfg, seed)
    e0 = synth.make_e0(cfg, seed, std=e0_std)
    return x, ctx, e0


# --------------------------------------------------------------------------
# tiny float32 stack
# --------------------------------------------------------------------------

@pytest.fixture(scope="module")
def tiny_model():
    w = synth.make_weights(TINY, seed=0, qk_gain=2.0)
    return w, make_model(TINY, w)


@pytest.mark.parametrize("step", [0, 1, 2, 3])
@pytest.mark.parametrize("layer", [0, 1])
def test_tiny_block_each_structure(tiny_model, step, layer):
    w, model = tiny_model
    say(f"tiny block step={step} layer={layer}")
    masks = synth.make_masks(TINY, step)
    x, ctx, e0 = _inputs(TINY, 10 + step)
    got, plan = gpu_block(model, TINY, masks, step, layer, x, ctx, e0)
    info = plan.layer_info(layer)
    assert info.self_heads == TINY.keep_heads[step] and info.ffn_channels == TINY.keep_ffn[step]
    ref = oracle_block(TINY, w["layers"][layer], masks, layer, x, ctx, e0)
    assert rel_err(got, ref) <= TOL["f32"]


@pytest.mark.parametrize("case", ["all_pruned", "block_off", "one_head_one_channel",
                                  "no_self_heads", "no_cross_no_ffn"])
def test_tiny_block_edge_cases(tiny_model, case):
    w, model = tiny_model
    say(f"tiny edge case {case}")
    cfg = TINY
    H, F = cfg.n_heads, cfg.ffn_dim
    counts = {"all_pruned": (0, 0, 0), "block_off": (4, 4, 1024),
              "one_head_one_channel": (1, 1, 1), "no_self_heads": (0, 3, 640),
              "no_cross_no_ffn": (2, 0, 0)}[case]
    N = cfg.n_layers
    masks = synth.masks_from_counts(cfg.with_(ffn_chunk=1), [counts[0]] * N, [counts[1]] * N,
                                    [counts[2]] * N, seed=3,
                                    block_keep=[0] * N if case == "block_off" else None)
    x, ctx, e0 = _inputs(cfg, 21)
    got, _ = gpu_block(model, cfg, masks, 0, 1, x, ctx, e0)
    ref = oracle_block(cfg, w["layers"][1], masks, 1, x, ctx, e0)
    if case == "block_off":
        assert np.array_equal(got, x)
    assert rel_err(got, ref) <= TOL["f32"]


def test_tiny_block_batch_and_bit_stability(tiny_model):
    w, model = tiny_model
    say("tiny batch=3 twice")
    cfg = TINY.with_(batch=3)
    masks = synth.make_masks(TINY, 2)
    x, ctx, e0 = _inputs(cfg, 5)
    got1, _ = gpu_block(model, TINY, masks, 2, 0, x, ctx, e0)
    got2, _ = gpu_block(model, TINY, masks, 2, 0, x, ctx, e0)
    assert np.array_equal(got1, got2)
    ref = oracle_block(TINY, w["layers"][0], masks, 0, x, ctx, e0)
    assert rel_err(got1, ref) <= TOL["f32"]


def test_tiny_time_embedding(tiny_model):
    import torch
    w, model = tiny_model
    say("tiny time embedding")
    ws = B.workspace(model, 1, TINY.seq_len, TINY.text_len)
    for t in TINY.timesteps:
        e = torch.empty(TINY.dim, device="cuda")
        e0 = torch.empty(6 * TINY.dim, device="cuda")
        B.dif_time_embed(model, t, e, e0, ws)
        torch.cuda.synchronize()
        re, re0 = O.time_embedding(w, t)
        assert rel_err(to_np(e), re) <= TOL["f32"]
        assert rel_err(to_np(e0).reshape(6, -1), re0) <= TOL["f32"]


def test_tiny_full_denoise_matches_oracle(tiny_model):
    """All four step structures, both layers, Euler between steps."""
    import torch
    w, model = tiny_model
    cfg = TINY
    say("tiny 4-step denoise")
    masks = [synth.make_masks(cfg, s) for s in range(4)]
    plans = [B.dif_plan_step(model, s, cfg.timesteps[s], masks[s]) for s in range(4)]
    z0 = synth.make_latents(cfg, seed=1)
    ctx = synth.make_context(cfg, seed=1)
    z = to_dev(z0, dtype=torch.float32)
    cd = to_dev(ctx, cfg)
    v = torch.empty_like(z)
    ws = B.workspace(model, 1, cfg.seq_len, cfg.text_len)
    sig = O.sigmas(cfg.timesteps)
    vs = []
    for s, t in enumerate(cfg.timesteps):
        B.dif_step_forward(plans[s], z, t, cd, v, ws)
        vs.append(to_np(v))
        B.dif_euler(z, v, sig[s], sig[s + 1])
    torch.cuda.synchronize()
    ref_v0 = O.step(z0, cfg.timesteps[0], ctx, w, masks[0], cfg)
    assert rel_err(vs[0], ref_v0) <= TOL["f32"]
    ref = O.denoise(z0, ctx, w, masks, cfg)
    assert rel_err(to_np(z), ref) <= TOL["f32"]


# --------------------------------------------------------------------------
# bf16 blocks with Wan-1.3B / Wan-14B widths, small ragged grids
# --------------------------------------------------------------------------

@pytest.fixture(scope="module")
def mid13():
    w = synth.make_weights(MID13, seed=0)
    return w, make_model(MID13, w)


@pytest.mark.parametrize("variant", ["default", "attention_visible"])
def test_wan13b_width_block(mid13, variant):
    w, model = mid13
    cfg = MID13
    say(f"wan1.3b-width block {variant} L={cfg.seq_len} B={cfg.batch}")
    masks = synth.make_masks(cfg, 0)
    x, ctx, e0 = _inputs(cfg, 3)
    if variant == "attention_visible":   # FFN gate 0: the attention branches dominate the update
        e0[5] = -w["layers"][0]["mod"][5]
    got, _ = gpu_block(model, cfg, masks, 0, 0, x, ctx, e0)
    ref = oracle_block(cfg, w["layers"][0], masks, 0, x, ctx, e0)
    err = rel_err(got, ref)
    say(f"  rel err {err:.3e}")
    assert err <= TOL["bf16"]


def test_wan13b_width_step(mid13):
    import torch
    w, model = mid13
    cfg = MID13
    say("wan1.3b-width single-layer step forward")
    masks = synth.make_masks(cfg, 0)
    plan = B.dif_plan_step(model, 0, 750, masks)
    z0 = synth.make_latents(cfg, seed=2)
    ctx = synth.make_context(cfg, seed=2)
    z = to_dev(z0, dtype=torch.float32)
    v = torch.empty_like(z)
    ws = B.workspace(model, cfg.batch, cfg.seq_len, cfg.text_len)
    B.dif_step_forward(plan, z, 750, to_dev(ctx, cfg), v, ws)
    torch.cuda.synchronize()
    ref = O.step(z0, 750, ctx, w, masks, cfg)
    assert rel_err(to_np(v), ref) <= TOL["bf16"]


@pytest.fixture(scope="module")
def mid14():
    w = synth.make_weights(MID14, seed=0)
    return w, make_model(MID14, w)


@pytest.mark.parametrize("step", [0, 1, 2, 3])
def test_wan14b_width_block_each_structure(mid14, step):
    w, model = mid14
    cfg = MID14
    say(f"wan14b-width block step={step} L={cfg.seq_len}")
    masks = synth.make_masks(cfg, step)
    x, ctx, e0 = _inputs(cfg, 4 + step)
    got, plan = gpu_block(model, cfg, masks, step, 0, x, ctx, e0)
    assert plan.layer_info(0).ffn_padded == -(-cfg.keep_ffn[step] // 64) * 64
    ref = oracle_block(cfg, w["layers"][0], masks, 0, x, ctx, e0)
    err = rel_err(got, ref)
    say(f"  rel err {err:.3e}")
    assert err <= TOL["bf16"]


def test_wan13b_width_block_attention_key_split():
    """Self-attention whose last round of workgroups is split along the keys
    and merged: 4551 tokens (18 query blocks of 256, the last ragged), 9 kept
    heads, batch 2 -> 324 work items on 256 CUs, so the 68 items of the final
    round run as two key halves each; the second half ends in a 7-key tile."""
    cfg = get_config("wan1.3b_block").with_(name="split13", grid=(3, 37, 41), text_len=77, batch=2)
    masks = synth.make_masks(cfg, 0)
    heads = int(masks["self_head_keep"][0].sum())
    items = -(-cfg.seq_len // 256) * heads * cfg.batch
    assert 0 < items % 256 <= 128 and cfg.seq_len % 64 == 7
    say(f"wan1.3b-width block L={cfg.seq_len} B={cfg.batch} heads={heads}: {items} attention items")
    w = synth.make_weights(cfg, seed=3)
    model = make_model(cfg, w)
    x, ctx, e0 = _inputs(cfg, 9)
    e0[5] = -w["layers"][0]["mod"][5]   # FFN gate 0: the attention branches dominate the update
    got, _ = gpu_block(model, cfg, masks, 0, 0, x, ctx, e0)
    ref = oracle_block(cfg, w["layers"][0], masks, 0, x, ctx, e0, dtype=np.float32)
    err = rel_err(got, ref)
    say(f"  rel err {err:.3e}")
    assert err <= TOL["bf16"]


def test_wan13b_width_block_sharp_attention():
    """QK-RMSNorm gains x2 (score std about 4).  The bf16 storage floor of
    these inputs is 9.5e-3 (tests/test_bf16_floor.py, on CPU)."""
    cfg = MID13.with_(batch=1)
    say("wan1.3b-width block, sharp attention (QK gains x2)")
    w = synth.make_weights(cfg, seed=1, qk_gain=2.0)
    model = make_model(cfg, w)
    masks = synth.make_masks(cfg, 0)
    x, ctx, e0 = _inputs(cfg, 8)
    e0[5] = -w["layers"][0]["mod"][5]
    got, _ = gpu_block(model, cfg, masks, 0, 0, x, ctx, e0)
    ref = oracle_block(cfg, w["layers"][0], masks, 0, x, ctx, e0)
    err = rel_err(got, ref)
    say(f"  rel err {err:.3e}")
    assert err <= TOL["bf16"]


def test_wan14b_width_step_with_block_skips():
    """A 4-layer stack at Wan-14B widths whose step structure gates off two
    blocks and keeps a different head / channel subset in every other layer
    (block gates, Sec. 4.1; per-layer structures, Sec. 6), through
    dif_step_forward, for both plan kinds."""
    import torch
    cfg = MID14.with_(name="mid14x4", n_layers=4, grid=(1, 7, 11), text_len=64)
    say(f"wan14b-width 4-layer step with block skips L={cfg.seq_len}")
    w = synth.make_weights(cfg, seed=2)
    model = make_model(cfg, w)
    masks = synth.masks_from_counts(cfg.with_(ffn_chunk=8), [40, 24, 30, 36], [28, 40, 20, 32],
                                    [13824, 8296, 9680, 11056], seed=9, block_keep=[1, 0, 1, 0])
    z0 = synth.make_latents(cfg, seed=9)
    ctx = synth.make_context(cfg, seed=9)
    ref = O.step(z0, 500, ctx, w, masks, cfg)
    for kind in ("compact", "indexed"):
        plan = B.dif_plan_step(model, 2, 500, masks, kind=kind)
        assert [plan.layer_info(l).block_keep for l in range(4)] == [1, 0, 1, 0]
        z = to_dev(z0, dtype=torch.float32)
        v = torch.empty_like(z)
        ws = B.workspace(model, 1, cfg.seq_len, cfg.text_len)
        B.dif_step_forward(plan, z, 500, to_dev(ctx, cfg), v, ws)
        torch.cuda.synchronize()
        err = rel_err(to_np(v), ref)
        say(f"  {kind}: rel err {err:.3e}")
        assert err <= TOL["bf16"]


def test_step_rejects_a_timestep_other_than_the_plans(tiny_model):
    """A plan is bound to its step's timestep (Sec. 3.1: the structure of
    step i belongs to t_i); DIF_PLAN_ANY_T lifts the binding."""
    import torch
    w, model = tiny_model[0], tiny_model[1]
    cfg = TINY
    masks = synth.make_masks(cfg, 1)
    plan = B.dif_plan_step(model, 1, cfg.timesteps[1], masks)
    assert B.dif_plan_timestep(plan) == (float(cfg.timesteps[1]), 0)
    z = torch.zeros((1, cfg.seq_len, cfg.patch_dim), device="cuda")
    v = torch.empty_like(z)
    ctx = to_dev(synth.make_context(cfg, seed=1), cfg)
    ws = B.workspace(model, 1, cfg.seq_len, cfg.text_len)
    with pytest.raises(B.DifError) as ei:
        B.dif_step_forward(plan, z, cfg.timesteps[2], ctx, v, ws)
    assert ei.value.code == -1
    free = B.dif_plan_step(model, 1, float("nan"), masks, any_t=True)
    B.dif_step_forward(free, z, cfg.timesteps[2], ctx, v, ws)
    torch.cuda.synchronize()


def test_single_token_grid_step():
    """The degenerate grid 1 x 1 x 1: one video token (attention over one
    key returns its value) and one text token, through dif_step_forward, at
    float32 against the oracle's step."""
    import torch
    cfg = TINY.with_(name="one_token", grid=(1, 1, 1), text_len=1)
    say("single-token grid step")
    w = synth.make_weights(cfg, seed=5, qk_gain=2.0)
    model = make_model(cfg, w)
    masks = synth.make_masks(cfg, 2)
    plan = B.dif_plan_step(model, 2, cfg.timesteps[2], masks)
    z0 = synth.make_latents(cfg, seed=5)
    ctx = synth.make_context(cfg, seed=5)
    z = to_dev(z0, dtype=torch.float32)
    v = torch.empty_like(z)
    ws = B.workspace(model, 1, 1, 1)
    B.dif_step_forward(plan, z, cfg.timesteps[2], to_dev(ctx, cfg), v, ws)
    torch.cuda.synchronize()
    ref = O.step(z0, cfg.timesteps[2], ctx, w, masks, cfg)
    err = rel_err(to_np(v), ref)
    say(f"  rel err {err:.3e}")
    assert err <= TOL["f32"]


def test_widest_bf16_block():
    """dim 8192 (64 heads of 128), the widest model the library accepts in
    bfloat16, on a small ragged grid: a pruned block against the oracle."""
    cfg = get_config("wan14b_block").with_(name="wide8192", dim=8192, n_heads=64, ffn_dim=2048,
                                           grid=(1, 5, 7), text_len=9,
                                           keep_heads=(47,), keep_ffn=(1384,), ffn_chunk=1)
    say(f"dim-8192 block L={cfg.seq_len}")
    w = synth.make_weights(cfg, seed=6)
    model = make_model(cfg, w)
    masks = synth.make_masks(cfg, 0)
    x, ctx, e0 = _inputs(cfg, 6)
    got, plan = gpu_block(model, cfg, masks, 0, 0, x, ctx, e0)
    assert plan.layer_info(0).self_heads == 47
    ref = oracle_block(cfg, w["layers"][0], masks, 0, x, ctx, e0)
    err = rel_err(got, ref)
    say(f"  rel err {err:.3e}")
    assert err <= TOL["bf16"]
