"""Self-attention in the launch configuration the blocks use, against the oracle.

The blocks call the attention kernel with queries already multiplied by
log2(e)/sqrt(dh) (the QK-norm kernel writes them so), in workgroups of 256
queries for bfloat16 keys of 4096 and more (four waves of two 32-query
groups at head_dim 128, eight waves of 32 queries at 64), and -- when
the last round of workgroups on the device would run at most half full --
with that round's work items split along the keys and merged by a second
kernel.  dif_attention_ex runs exactly that launch.  Here it runs at the
benchmark's sequence length (32760 tokens = 127 * 256 + 248, so the last
query block is ragged) with sharp scores (standard deviation 4: the online
softmax's base moves often and a few keys dominate every row), and its
output O is compared element by element, on sampled query rows (the first
rows, random rows and the 248-row tail), with the oracle's attention on the
same bfloat16 inputs.  The kernel computes softmax(Qs K^T ln 2) V for the
pre-scaled Qs it is given, so the oracle receives Qs * sqrt(dh) / log2(e)
as its queries (its own scale 1/sqrt(dh) then gives the same scores).

Odd head counts at 32760 tokens leave 128 work items for the last round of
256 workgroups, which triggers the key split; even counts fill every round.
The tests read the device's compute-unit count and assert that the split
case really splits.  tests/test_attention_power.py shows on the CPU that a
uniform attention or a merge that keeps only one key half fails these
checks by far more than 3x the tolerance.
"""
import math

import numpy as np
import pytest

import oracle as O
from paper_2607_06631_amd import binding as B
from tests.gpu_util import rel_err, say
from workloads import synth

pytestmark = [pytest.mark.gpu]

TOL = 2e-2          # bfloat16 tolerance (max |g - r| / max |r|)
TOL_F32 = 1e-4
LOG2E = 1.4426950408889634
L_480P = 32760      # 21 x 30 x 52 latent tokens


def sample_rows(L, seed, n=320, head=32, tail=248):
    g = np.random.default_rng(seed)
    return np.unique(np.concatenate([np.arange(min(head, L)), g.choice(L, min(n, L), replace=False),
                                     np.arange(max(L - tail, 0), L)]))


def split_expected(Lq, Lk, heads, waves, ncu):
    """Mirror of the launch rule: items of the last round, and whether they split."""
    bmq = 32 * waves
    items = -(-Lq // bmq) * heads
    slots = ncu * (1 if waves == 8 else 2)
    rem = items % slots
    return rem > 0 and 2 * rem <= slots and rem <= 128 and Lk // 64 >= 4


def run_case(L, heads, dh, dtype, prescaled, split, q_std, k_std, seed, Lk=None):
    import torch
    Lk = L if Lk is None else Lk
    bf16 = dtype == "bf16"
    tdt = torch.bfloat16 if bf16 else torch.float32
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    waves = 8 if (bf16 and Lk >= 4096) else 4
    will_split = split and split_expected(L, Lk, heads, waves, ncu)
    say(f"attention L={L} Lk={Lk} heads={heads} dh={dh} {dtype} prescaled={prescaled} "
        f"split_ws={split} (splits: {will_split}, {ncu} CUs) q_std={q_std} k_std={k_std} seed={seed}")
    assert L == Lk, "self-attention cases"
    q, k, v = synth.make_attention_inputs(L, heads, dh, q_std, k_std, seed, bf16=bf16)
    c = LOG2E / math.sqrt(dh)
    if prescaled:
        qs = q * np.float32(c)
        qs = synth.bf16_round(qs) if bf16 else qs
    else:
        qs = q
    w = heads * dh
    ldvt = -(-Lk // 64) * 64
    Qd = torch.from_numpy(qs).cuda().to(tdt).contiguous()
    Kd = torch.from_numpy(k).cuda().to(tdt).contiguous()
    Vt = torch.zeros((w, ldvt), dtype=tdt, device="cuda")
    Vt[:, :Lk] = torch.from_numpy(v).cuda().to(tdt).t()
    Od = torch.empty((L, w), dtype=tdt, device="cuda")
    ws = None
    if split:
        ws = torch.empty(B.dif_attention_split_bytes(dh), dtype=torch.uint8, device="cuda")
    B.dif_attention_ex(Qd, Kd, Vt, Od, 1, L, Lk, heads, dh, w, w, ldvt, w,
                       flags=B.DIF_ATTN_Q_PRESCALED if prescaled else 0, split_ws=ws)
    torch.cuda.synchronize()
    rows = sample_rows(L, seed)
    got = Od[torch.from_numpy(rows).cuda()].float().cpu().numpy()
    say(f"  GPU done; oracle on {len(rows)} rows")
    q_or = qs[rows].astype(np.float64)
    if prescaled:
        q_or = q_or * (math.sqrt(dh) / LOG2E)
    ref = O.attention(q_or, k.astype(np.float64), v.astype(np.float64), heads, dh)
    err = rel_err(got, ref)
    say(f"  rel err {err:.3e} (max |O| {np.abs(ref).max():.3f})")
    return err, will_split


@pytest.mark.slow
def test_block_launch_480p_split():
    """29 kept heads at 32760 tokens: the block's exact launch, final round split."""
    err, split = run_case(L_480P, 29, 128, "bf16", True, True, 2.0, 2.0, seed=1)
    assert split, "the case must exercise the key split"
    assert err <= TOL


@pytest.mark.slow
def test_block_launch_480p_full_rounds():
    """30 kept heads: every round full, no split."""
    err, split = run_case(L_480P, 30, 128, "bf16", True, True, 2.0, 2.0, seed=2)
    assert not split
    assert err <= TOL


@pytest.mark.slow
def test_unscaled_queries_480p_no_workspace():
    """The plain operator's path (one multiply per score) at full length."""
    err, _ = run_case(L_480P, 29, 128, "bf16", False, False, 2.0, 2.0, seed=3)
    assert err <= TOL


def test_split_short_keys_four_waves():
    """bf16 below 4096 keys runs four waves; 120 items for 512 slots split."""
    err, split = run_case(3000, 5, 128, "bf16", True, True, 2.0, 2.0, seed=4)
    assert split
    assert err <= TOL


@pytest.mark.parametrize("dh", [64, 128])
def test_split_float32(dh):
    """float32, four waves, 99 items split; 1e-4 against the oracle."""
    err, split = run_case(4099, 3, dh, "f32", True, True, 1.5, 1.5, seed=5)
    assert split
    assert err <= TOL_F32


def test_attention_ex_errors():
    import torch
    q = torch.zeros((64, 128), dtype=torch.bfloat16, device="cuda")
    vt = torch.zeros((128, 64), dtype=torch.bfloat16, device="cuda")
    o = torch.empty_like(q)
    small = torch.empty(1024, dtype=torch.uint8, device="cuda")
    with pytest.raises(B.DifError):
        B.dif_attention_ex(q, q, vt, o, 1, 64, 64, 1, 128, 128, 128, 64, 128, flags=2)
    with pytest.raises(B.DifError):
        B.dif_attention_ex(q, q, vt, o, 1, 64, 64, 1, 128, 128, 128, 64, 128, split_ws=small)
    torch.cuda.synchronize()
