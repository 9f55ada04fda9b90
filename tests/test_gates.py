"""dif_hard_gates (host code behind the C ABI) against the oracle's rules."""
import numpy as np
import pytest

import oracle as O
from paper_2607_06631_amd import binding as B
from workloads import get_config


@pytest.mark.parametrize("name,chunk", [("tiny", 8), ("tiny", 4), ("wan14b_block", 8)])
def test_hard_gates_match_oracle(name, chunk):
    cfg = get_config(name).with_(n_layers=2)
    N, H, dh, D, F = cfg.n_layers, cfg.n_heads, cfg.head_dim, cfg.dim, cfg.ffn_dim
    g = np.random.default_rng(len(name) + chunk)
    m_block = g.standard_normal(N).astype(np.float32)
    m_self = (g.standard_normal((N, D)) + 0.02).astype(np.float32)
    m_cross = (g.standard_normal((N, D)) - 0.02).astype(np.float32)
    m_ffn = g.standard_normal((N, F // chunk)).astype(np.float32)
    # exact ties: a zero block mask, a head whose values cancel, zero chunks, NaN
    m_block[0] = 0.0
    m_self[0, :dh] = np.tile([1.0, -1.0], dh // 2)
    m_cross[1, dh:2 * dh] = 0.0
    m_ffn[0, :3] = 0.0
    m_ffn[1, 5] = np.nan
    got = B.dif_hard_gates(cfg, m_block, m_self, m_cross, m_ffn, chunk)
    ref = O.hard_gates(m_block, m_self, m_cross, m_ffn, H, dh, chunk)
    for k in ref:
        assert np.array_equal(got[k], ref[k]), k
    assert got["block_keep"][0] == 0 and got["self_head_keep"][0, 0] == 0
    assert got["cross_head_keep"][1, 1] == 0 and got["ffn_keep"][1, 5 * chunk] == 0


def test_hard_gates_reject_bad_chunk():
    cfg = get_config("tiny")
    z = np.zeros(10 ** 5, np.float32)
    with pytest.raises(RuntimeError):
        B.dif_hard_gates(cfg, z, z, z, z, chunk=7)
