"""Teacher-forced parity on the 40-layer Wan-14B-shaped 480p stack.

For each of the four step structures the GPU runs the whole block stack in
sequence from patch-embedded latents, in the launch configuration the
benchmark times (32760 video tokens, 512 text tokens, the step's per-layer
keep masks from the depth-tilted recipe).  At layers 0, 13, 26 and 39 the
block's input -- the GPU's own residual stream after the layers before it --
goes to the oracle, which computes that block for sampled query rows (keys
and values over all L tokens) with the keep masks applied by zeroing dense
weights, and the GPU's block output must match within the bf16 tolerance.
The modulation e0 is the library's own time embedding of t_s (its parity is
checked at float32 on the tiny stack).  The oracle runs in float32 here to
keep the masked-dense projections within seconds.
"""
import numpy as np
import pytest

import oracle as O
from paper_2607_06631_amd import binding as B
from tests.gpu_util import rel_err, say, to_np
from workloads import get_config, synth

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

TOL = 2e-2
CHECK_LAYERS = (0, 13, 26, 39)


def _rows(L, seed, n=512):
    g = np.random.default_rng(seed)
    return np.unique(np.concatenate([np.arange(16), g.choice(L, n, replace=False),
                                     np.arange(L - 40, L)]))


@pytest.fixture(scope="module")
def stack():
    import torch
    cfg = get_config("wan14b_480p")
    say("generating the 40-layer Wan-14B-shaped stack in device memory")
    w = synth.make_weights_torch(cfg, "cuda", seed=0)
    model = B.dif_model_create(cfg, w)
    yield cfg, w, model
    del model
    torch.cuda.empty_cache()


@pytest.mark.parametrize("step", [0, 1, 2, 3])
def test_wan14b_480p_stack_teacher_forced(stack, step):
    import torch
    cfg, w, model = stack
    L, Lc, D, Cp = cfg.seq_len, cfg.text_len, cfg.dim, cfg.patch_dim
    masks = synth.make_masks(cfg, step)
    say(f"step {step}: plan ({int(masks['self_head_keep'].sum())} self heads, "
        f"{int(masks['ffn_keep'].sum())} FFN channels over {cfg.n_layers} layers)")
    plan = B.dif_plan_step(model, step, cfg.timesteps[step], masks)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(100 + step)
    z = torch.randn((L, Cp), generator=gen, device="cuda")
    ctx = torch.randn((1, Lc, D), generator=gen, device="cuda").to(torch.bfloat16)
    ws = B.workspace(model, 1, L, Lc)
    e = torch.empty(D, device="cuda")
    e0 = torch.empty(6 * D, device="cuda")
    B.dif_time_embed(model, cfg.timesteps[step], e, e0, ws)
    # the residual stream entering layer 0: patch embedding of the latents
    x = (z.to(torch.bfloat16).float() @ w["patch_w"].float().t() + w["patch_b"])
    x = x.to(torch.bfloat16).reshape(1, L, D).contiguous()
    saved = {}
    for layer in range(cfg.n_layers):
        if layer in CHECK_LAYERS:
            saved[layer] = [x.clone()]
        B.dif_block_forward(plan, layer, x, ctx, e0, ws)
        if layer in CHECK_LAYERS:
            saved[layer].append(x.clone())
    torch.cuda.synchronize()
    say(f"step {step}: GPU stack done; oracle on sampled rows of layers {CHECK_LAYERS}")
    ctx_np, e0_np = to_np(ctx)[0], to_np(e0).reshape(6, D)
    assert np.all(np.isfinite(to_np(x))), "non-finite residual stream"
    for layer in CHECK_LAYERS:
        x_in, x_out = (to_np(t)[0] for t in saved.pop(layer))
        wl = {k: v.float().cpu().numpy() for k, v in w["layers"][layer].items()}
        wz = O.apply_keep(wl, masks["self_head_keep"][layer], masks["cross_head_keep"][layer],
                          masks["ffn_keep"][layer], cfg.head_dim, np.float32)
        rows = _rows(L, 1000 * step + layer)
        ref = O.block(x_in, ctx_np, e0_np, wz, bool(masks["block_keep"][layer]), cfg.n_heads,
                      cfg.head_dim, cfg.grid, cfg.rope_theta, cfg.eps, rows=rows, dtype=np.float32)
        err = rel_err(x_out[rows], ref)
        say(f"  layer {layer}: {int(masks['self_head_keep'][layer].sum())} heads, "
            f"{int(masks['ffn_keep'][layer].sum())} channels: rel err {err:.3e} over {len(rows)} rows")
        assert err <= TOL
