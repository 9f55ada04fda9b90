"""Indexed plans: step t's active parameters read in place from the union
weights through the index tables I_t (Sec. 4.3), no compacted copy.

Against the oracle at the usual tolerances, and against the compact plan:
bit-identical whenever every FFN chunk of 16 bytes (8 bf16 / 4 float32
channels) is wholly kept or wholly dropped, because both plans then feed
the same operands to the same MFMA sequence; with per-channel FFN masks
the indexed plan also runs the zeroed channels of partly kept chunks, so
only the oracle tolerance applies.
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
MID14 = get_config("wan14b_block").with_(name="mid14", grid=(2, 7, 11), text_len=512)


def oracle_block(cfg, wl, masks, layer, x, ctx, e0):
    wz = O.apply_keep(wl, masks["self_head_keep"][layer], masks["cross_head_keep"][layer],
                      masks["ffn_keep"][layer], cfg.head_dim, np.float64)
    return np.stack([O.block(x[b], ctx[b], e0, wz, bool(masks["block_keep"][layer]), cfg.n_heads,
                             cfg.head_dim, cfg.grid, cfg.rope_theta, cfg.eps)
                     for b in range(x.shape[0])])


def run_block(model, cfg, masks, layer, x, ctx, e0, kind):
    import torch
    plan = B.dif_plan_step(model, 0, cfg.timesteps[0], masks, kind=kind)
    xd, cd = to_dev(x, cfg), to_dev(ctx, cfg)
    ed = to_dev(e0, dtype=torch.float32)
    ws = B.workspace(model, x.shape[0], x.shape[1], ctx.shape[1])
    B.dif_block_forward(plan, layer, xd, cd, ed, ws)
    torch.cuda.synchronize()
    return to_np(xd), plan


def inputs(cfg, seed):
    return (synth.make_block_input(cfg, seed, scale=0.5), synth.make_context(cfg, seed),
            synth.make_e0(cfg, seed, std=0.3))


def chunk_aligned(m, vec):
    f = m["ffn_keep"].reshape(m["ffn_keep"].shape[0], -1, vec)
    return bool(np.all((f.min(axis=2) == f.max(axis=2))))


@pytest.fixture(scope="module")
def tiny_model():
    w = synth.make_weights(TINY, seed=0, qk_gain=2.0)
    return w, make_model(TINY, w)


@pytest.mark.parametrize("step", [0, 1, 2, 3])
@pytest.mark.parametrize("layer", [0, 1])
def test_tiny_indexed_equals_compact(tiny_model, step, layer):
    w, model = tiny_model
    say(f"tiny indexed vs compact step={step} layer={layer}")
    masks = synth.make_masks(TINY, step)
    assert chunk_aligned(masks, 4)
    x, ctx, e0 = inputs(TINY, 30 + step)
    got, plan = run_block(model, TINY, masks, layer, x, ctx, e0, "indexed")
    ref_c, plan_c = run_block(model, TINY, masks, layer, x, ctx, e0, "compact")
    assert plan.layer_info(layer).ffn_padded == plan_c.layer_info(layer).ffn_padded
    assert np.array_equal(got, ref_c)
    ref = oracle_block(TINY, w["layers"][layer], masks, layer, x, ctx, e0)
    assert rel_err(got, ref) <= TOL["f32"]


@pytest.mark.parametrize("ffn", [1, 3, 517, 1023])
def test_tiny_indexed_per_channel_ffn(tiny_model, ffn):
    """FFN masks that split 4-channel chunks: dropped channels inside a kept
    chunk must contribute exactly nothing."""
    w, model = tiny_model
    say(f"tiny indexed per-channel ffn={ffn}")
    cfg1 = TINY.with_(ffn_chunk=1)
    N = TINY.n_layers
    masks = synth.masks_from_counts(cfg1, [3] * N, [2] * N, [ffn] * N, seed=7)
    x, ctx, e0 = inputs(TINY, 40)
    got, plan = run_block(model, TINY, masks, 1, x, ctx, e0, "indexed")
    info = plan.layer_info(1)
    chunks = int(np.any(masks["ffn_keep"][1].reshape(-1, 4), axis=1).sum())
    assert info.ffn_channels == ffn and info.ffn_padded == -(-4 * chunks // 64) * 64
    ref = oracle_block(TINY, w["layers"][1], masks, 1, x, ctx, e0)
    assert rel_err(got, ref) <= TOL["f32"]


@pytest.mark.parametrize("case", ["all_pruned", "block_off", "one_head_one_channel",
                                  "no_self_heads", "no_cross_no_ffn"])
def test_tiny_indexed_edge_cases(tiny_model, case):
    w, model = tiny_model
    say(f"tiny indexed edge case {case}")
    N = TINY.n_layers
    counts = {"all_pruned": (0, 0, 0), "block_off": (4, 4, 1024),
              "one_head_one_channel": (1, 1, 1), "no_self_heads": (0, 3, 640),
              "no_cross_no_ffn": (2, 0, 0)}[case]
    masks = synth.masks_from_counts(TINY.with_(ffn_chunk=1), [counts[0]] * N, [counts[1]] * N,
                                    [counts[2]] * N, seed=3,
                                    block_keep=[0] * N if case == "block_off" else None)
    x, ctx, e0 = inputs(TINY, 21)
    got, _ = run_block(model, TINY, masks, 1, x, ctx, e0, "indexed")
    if case == "block_off":
        assert np.array_equal(got, x)
    ref = oracle_block(TINY, w["layers"][1], masks, 1, x, ctx, e0)
    assert rel_err(got, ref) <= TOL["f32"]


def test_tiny_indexed_full_denoise(tiny_model):
    import torch
    w, model = tiny_model
    cfg = TINY
    say("tiny 4-step denoise, indexed plans")
    masks = [synth.make_masks(cfg, s) for s in range(4)]
    plans = [B.dif_plan_step(model, s, cfg.timesteps[s], masks[s], kind="indexed") for s in range(4)]
    z0 = synth.make_latents(cfg, seed=1)
    ctx = synth.make_context(cfg, seed=1)
    z = to_dev(z0, dtype=torch.float32)
    v = torch.empty_like(z)
    ws = B.workspace(model, 1, cfg.seq_len, cfg.text_len)
    sig = O.sigmas(cfg.timesteps)
    cd = to_dev(ctx, cfg)
    for s, t in enumerate(cfg.timesteps):
        B.dif_step_forward(plans[s], z, t, cd, v, ws)
        B.dif_euler(z, v, sig[s], sig[s + 1])
    torch.cuda.synchronize()
    ref = O.denoise(z0, ctx, w, masks, cfg)
    assert rel_err(to_np(z), ref) <= TOL["f32"]


def test_indexed_plan_memory_is_tables_only(tiny_model):
    _, model = tiny_model
    masks = synth.make_masks(TINY, 1)
    ni = B.dif_plan_bytes(model, masks, "indexed")
    nc = B.dif_plan_bytes(model, masks, "compact")
    say(f"tiny plan bytes indexed {ni} compact {nc}")
    assert ni < 64 * 1024 and nc > 10 * ni


@pytest.fixture(scope="module")
def mid14():
    w = synth.make_weights(MID14, seed=0)
    return w, make_model(MID14, w)


@pytest.mark.parametrize("step", [1, 3])
def test_wan14b_width_indexed_per_channel(mid14, step):
    """The 14B block structures keep a per-channel FFN count (11059, 8294)."""
    w, model = mid14
    say(f"wan14b-width indexed block step={step} L={MID14.seq_len}")
    masks = synth.make_masks(MID14, step)
    x, ctx, e0 = inputs(MID14, 50 + step)
    got, _ = run_block(model, MID14, masks, 0, x, ctx, e0, "indexed")
    ref = oracle_block(MID14, w["layers"][0], masks, 0, x, ctx, e0)
    err = rel_err(got, ref)
    say(f"  rel err {err:.3e}")
    assert err <= TOL["bf16"]


def test_wan14b_width_indexed_equals_compact_chunked(mid14):
    """C = 8 channel chunks (App. A): indexed and compact plans agree bit for bit."""
    w, model = mid14
    cfg8 = MID14.with_(ffn_chunk=8)
    say("wan14b-width indexed vs compact, C=8 chunked masks")
    masks = synth.masks_from_counts(cfg8, [28], [24], [9680], seed=5)
    assert chunk_aligned(masks, 8)
    x, ctx, e0 = inputs(MID14, 60)
    got, _ = run_block(model, MID14, masks, 0, x, ctx, e0, "indexed")
    ref_c, _ = run_block(model, MID14, masks, 0, x, ctx, e0, "compact")
    assert np.array_equal(got, ref_c)
