"""Helpers shared by the GPU parity tests (device setup, error metric)."""
from __future__ import annotations

import sys

import numpy as np

from paper_2607_06631_amd import binding as B


def say(*a):
    """Progress line that names the case before a GPU step."""
    print(*a, flush=True)
    sys.stdout.flush()


def rel_err(got, ref) -> float:
    """max_i |g_i - r_i| / max_i |r_i| in float64."""
    g = np.asarray(got, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    assert np.all(np.isfinite(g)), "non-finite GPU output"
    return float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-30))


def torch_dtype(cfg):
    import torch
    return torch.bfloat16 if cfg.dtype == "bf16" else torch.float32


def to_dev(a, cfg=None, dtype=None):
    import torch
    dt = dtype if dtype is not None else torch_dtype(cfg)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda().to(dt).contiguous()


def to_np(t):
    return t.float().cpu().numpy()


def make_model(cfg, weights_np):
    dev_w = B.upload_weights(weights_np, cfg.dtype)
    return B.dif_model_create(cfg, dev_w)
