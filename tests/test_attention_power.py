"""Power of the full-length attention parity checks (CPU).

tests/test_gpu_attention_launch.py compares the blocks' attention launch
with the oracle at 32760 tokens with a tolerance of 2e-2 (max |g - r| /
max |r| over sampled rows).  A check that also passes a plausibly broken
kernel proves little, so this test takes the same inputs (the generator
draws each head from its own stream, so two heads suffice: head 0 and head
28, the one whose work items the 29-head launch splits along the keys at
key 254 * 64 = 16256) and shows that each of these mistakes moves the
result by more than three times the tolerance:
  * uniform attention (every probability 1 / Lk);
  * a key-split merge that keeps only the first or only the second half;
  * a merge that averages the two halves' normalised outputs instead of
    weighting them by their softmax mass.
"""
import math

import numpy as np
import pytest

import oracle as O
from workloads import synth

TOL = 2e-2
LOG2E = 1.4426950408889634
L, H, DH = 32760, 29, 128
SPLIT_HEAD, SPLIT_KEY = 28, 254 * 64


def _rel(got, ref):
    return float(np.max(np.abs(got - ref)) / np.max(np.abs(ref)))


@pytest.fixture(scope="module")
def inputs():
    q, k, v = synth.make_attention_inputs(L, H, DH, 2.0, 2.0, seed=1, heads=[0, SPLIT_HEAD])
    qs = synth.bf16_round(q * np.float32(LOG2E / math.sqrt(DH)))
    rows = np.random.default_rng(0).choice(L, 48, replace=False)
    q_or = qs[rows].astype(np.float64) * (math.sqrt(DH) / LOG2E)
    return q_or, k.astype(np.float64), v.astype(np.float64)


def _half(q, k, v, lo, hi):
    """Attention of every head over keys [lo, hi) only, plus each row's
    softmax mass there relative to its own maximum (for merges)."""
    return O.attention(q, k[lo:hi], v[lo:hi], 2, DH)


def test_reference_is_sharp(inputs):
    q, k, v = inputs
    s = (q[:, :DH] @ k[:, :DH].T) / math.sqrt(DH)
    p = O.softmax_rows(s)
    # a few keys dominate each row: the largest probability is far above 1/L
    assert np.median(p.max(axis=1)) > 0.1
    assert np.allclose(p.sum(axis=1), 1.0)


def test_uniform_attention_fails_by_far(inputs):
    q, k, v = inputs
    ref = O.attention(q, k, v, 2, DH)
    uni = np.tile(v.mean(axis=0), (q.shape[0], 1))
    assert _rel(uni, ref) > 3 * TOL


@pytest.mark.parametrize("keep", ["first", "second"])
def test_one_key_half_fails_by_far(inputs, keep):
    q, k, v = inputs
    ref = O.attention(q, k, v, 2, DH)
    lo, hi = (0, SPLIT_KEY) if keep == "first" else (SPLIT_KEY, L)
    bad = ref.copy()
    cs = slice(DH, 2 * DH)   # the split head only
    bad[:, cs] = _half(q, k, v, lo, hi)[:, cs]
    assert _rel(bad, ref) > 3 * TOL


def test_equal_weight_merge_fails_by_far(inputs):
    q, k, v = inputs
    ref = O.attention(q, k, v, 2, DH)
    a = _half(q, k, v, 0, SPLIT_KEY)
    b = _half(q, k, v, SPLIT_KEY, L)
    bad = ref.copy()
    cs = slice(DH, 2 * DH)
    bad[:, cs] = 0.5 * (a[:, cs] + b[:, cs])
    assert _rel(bad, ref) > 3 * TOL
