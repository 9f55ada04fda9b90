"""Sampler updates and the rollout chain through the C ABI, against the oracle.

Tolerance 1e-4 (float32 configuration), as for the other float32 step tests.
"""
import numpy as np
import pytest

import oracle as O
from paper_2607_06631_amd import binding as B
from tests.gpu_util import make_model, rel_err, say, to_dev, to_np
from workloads import get_config, synth

pytestmark = pytest.mark.gpu

TOL = 1e-4
TINY = get_config("tiny")


@pytest.fixture(scope="module")
def tiny():
    w = synth.make_weights(TINY, seed=0, qk_gain=2.0)
    model = make_model(TINY, w)
    masks = [synth.make_masks(TINY, s) for s in range(4)]
    return w, model, masks


def test_renoise_kernel_matches_formula():
    import torch
    say("dif_renoise elementwise")
    g = np.random.default_rng(3)
    n = 3 * 1000 + 17
    z0, v, eps = (g.standard_normal(n).astype(np.float32) for _ in range(3))
    for sf, st, use_eps in [(0.999, 0.75, True), (0.5, 0.25, True), (0.25, 0.0, False)]:
        z = to_dev(z0, dtype=torch.float32)
        B.dif_renoise(z, to_dev(v, dtype=torch.float32), sf, st,
                      to_dev(eps, dtype=torch.float32) if use_eps else None)
        torch.cuda.synchronize()
        ref = O.renoise(O.predict_clean(z0.astype(np.float64), v, sf), st, eps)
        assert rel_err(to_np(z), ref) <= 1e-6


@pytest.mark.parametrize("kind", ["compact", "indexed"])
def test_rollout_renoise_matches_oracle(tiny, kind):
    import torch
    w, model, masks = tiny
    say(f"tiny 4-step rollout, re-noise sampler, {kind} plans")
    plans = [B.dif_plan_step(model, s, TINY.timesteps[s], masks[s], kind=kind) for s in range(4)]
    z0 = synth.make_latents(TINY, seed=11)
    ctx = synth.make_context(TINY, seed=11)
    eps = synth.make_renoise_eps(TINY, seed=11)
    z = to_dev(z0, dtype=torch.float32)
    v = torch.empty_like(z)
    ws = B.workspace(model, 1, TINY.seq_len, TINY.text_len)
    B.dif_rollout(plans, TINY.timesteps, z, to_dev(ctx, TINY), v, ws,
                  eps=[to_dev(e, dtype=torch.float32) for e in eps], sampler="renoise")
    torch.cuda.synchronize()
    ref = O.rollout(z0, ctx, w, masks, TINY, eps, sampler="renoise")
    err = rel_err(to_np(z), ref)
    say(f"  rel err {err:.3e}")
    assert err <= TOL


def test_rollout_from_an_intermediate_step(tiny):
    """The detached chain started at t2 from a given latent (Fig. 2(b))."""
    import torch
    w, model, masks = tiny
    say("tiny rollout from step 1")
    plans = [B.dif_plan_step(model, s, TINY.timesteps[s], masks[s]) for s in range(4)]
    z0 = synth.make_latents(TINY, seed=12)
    ctx = synth.make_context(TINY, seed=12)
    eps = synth.make_renoise_eps(TINY, seed=12)
    z = to_dev(z0, dtype=torch.float32)
    v = torch.empty_like(z)
    ws = B.workspace(model, 1, TINY.seq_len, TINY.text_len)
    B.dif_rollout(plans[1:], TINY.timesteps[1:], z, to_dev(ctx, TINY), v, ws,
                  eps=[to_dev(e, dtype=torch.float32) for e in eps[1:]], sampler="renoise")
    torch.cuda.synchronize()
    ref = O.rollout(z0, ctx, w, masks, TINY, eps, start=1, sampler="renoise")
    assert rel_err(to_np(z), ref) <= TOL


def test_rollout_euler_equals_step_by_step(tiny):
    """The Euler rollout runs the same kernels as step_forward + euler: same bits."""
    import torch
    w, model, masks = tiny
    say("tiny Euler rollout vs step-by-step")
    plans = [B.dif_plan_step(model, s, TINY.timesteps[s], masks[s]) for s in range(4)]
    z0 = synth.make_latents(TINY, seed=13)
    ctx = to_dev(synth.make_context(TINY, seed=13), TINY)
    ws = B.workspace(model, 1, TINY.seq_len, TINY.text_len)
    za = to_dev(z0, dtype=torch.float32)
    v = torch.empty_like(za)
    B.dif_rollout(plans, TINY.timesteps, za, ctx, v, ws, sampler="euler")
    zb = to_dev(z0, dtype=torch.float32)
    sig = O.sigmas(TINY.timesteps)
    for s, t in enumerate(TINY.timesteps):
        B.dif_step_forward(plans[s], zb, t, ctx, v, ws)
        B.dif_euler(zb, v, sig[s], sig[s + 1])
    torch.cuda.synchronize()
    assert np.array_equal(to_np(za), to_np(zb))
