"""The C ABI on the host: the library loads, exports every entry point that
include/dif.h declares, and its host-only validation returns the documented
codes.  No device call is made here."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2607_06631_amd import binding as B
from workloads import get_config, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dif.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:dif_status|const char\*)\s+(dif_\w+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("libdif.so is not built (run __graft_entry__.build())")
    return B.lib()


def test_header_declares_the_contract():
    names = _declared()
    for want in ("dif_model_create", "dif_plan_step", "dif_block_forward", "dif_step_forward",
                 "dif_euler", "dif_plan_bytes", "dif_workspace_bytes", "dif_last_error",
                 "dif_validate_config", "dif_validate_masks", "dif_gemm", "dif_attention"):
        assert want in names


def test_library_exports_every_declared_symbol(lib):
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


def _cfg(**kw):
    return B.make_config(get_config("tiny").with_(**kw))


def _status(c):
    return B.lib().dif_validate_config(C.byref(c))


def test_validate_config_codes(lib):
    assert _status(_cfg()) == 0
    assert _status(B.make_config(get_config("wan14b_480p"))) == 0
    assert _status(_cfg(dim=250)) == -2                      # D != H * dh
    assert _status(_cfg(head_dim=32, dim=128)) == -4         # unsupported head_dim
    c = _cfg(); c.dtype = 7
    assert _status(c) == -1                                  # bad dtype enum
    assert _status(_cfg(patch_dim=48)) == -2
    assert _status(_cfg(n_layers=0)) == -2
    assert _status(_cfg(grid=(0, 8, 8))) == -2
    c = _cfg(); c.eps = 0.0
    assert _status(c) == -1
    assert lib.dif_validate_config(None) == -1
    assert b"null" in lib.dif_last_error()


def test_validate_masks_codes(lib):
    cfg = get_config("tiny")
    c = B.make_config(cfg)
    m = B._Masks(synth.make_masks(cfg, 1))
    assert lib.dif_validate_masks(C.byref(c), C.byref(m.struct)) == 0
    bad = synth.make_masks(cfg, 1)
    bad["ffn_keep"][1, 7] = 2
    mb = B._Masks(bad)
    assert lib.dif_validate_masks(C.byref(c), C.byref(mb.struct)) == -3
    assert b"ffn_keep" in lib.dif_last_error()
    empty = B.DifStepMasks()
    assert lib.dif_validate_masks(C.byref(c), C.byref(empty)) == -3


def test_python_wrappers_raise(lib):
    cfg = get_config("tiny")
    B.dif_validate_config(cfg)
    with pytest.raises(B.DifError) as ei:
        B.dif_validate_config(cfg.with_(dim=100))
    assert ei.value.code == -2
    bad = synth.make_masks(cfg, 0)
    bad["self_head_keep"][0, 0] = 9
    with pytest.raises(B.DifError):
        B.dif_validate_masks(cfg, bad)


def test_op_entry_points_reject_bad_arguments(lib):
    # rejected on the host before any device work
    assert lib.dif_gemm(5, 0, None, 0, None, 0, None, 0, 1, 1, 64, 0, None, None, None, None) == -1
    assert lib.dif_gemm(0, 0, None, 64, None, 64, None, 64, 4, 4, 48, 0, None, None, None, None) == -2
    # 256 rows of C (bf16, ldc = 2^22) or of A (lda = 2^22) span 2 GiB: more than
    # the kernels' 32-bit buffer descriptors address (the pointer is never used)
    fake = C.c_void_p(0x1000)
    big = 1 << 22
    assert lib.dif_gemm(0, 0, None, 64, None, 64, fake, big, 4, 4, 64, 0, None, None, None, None) == -2
    assert lib.dif_gemm(0, 0, None, big, None, 64, fake, 64, 4, 4, 64, 0, None, None, None, None) == -2
    assert b"2 GiB" in lib.dif_last_error()
    assert lib.dif_attention(0, 96, None, 0, None, 0, None, 0, None, 0, 1, 1, 1, 1, None) == -4
    assert lib.dif_attention(0, 128, None, 0, None, 0, None, 0, None, 0, 1, 1, 0, 1, None) == -2
    assert lib.dif_euler(None, None, 1.0, 0.5, 4, None) == -1
    assert lib.dif_model_create(None, None, None) == -1
    info = B.DifLayerInfo()
    assert lib.dif_plan_layer_info(None, 0, C.byref(info)) == -1


def test_sampler_entry_points_reject_bad_arguments(lib):
    # validation happens before any pointer is touched or kernel launched
    dummy = C.c_void_p(256)
    assert lib.dif_renoise(dummy, dummy, 0.75, 0.5, None, 4, None) == -1   # eps needed
    assert lib.dif_renoise(dummy, dummy, 0.75, 1.5, dummy, 4, None) == -1  # sigma_to > 1
    assert lib.dif_renoise(dummy, dummy, float("nan"), 0.0, None, 4, None) == -1
    assert lib.dif_renoise(dummy, dummy, 0.75, 0.0, None, -1, None) == -2
    assert lib.dif_renoise(None, dummy, 0.75, 0.0, None, 4, None) == -1
    P = (C.c_void_p * 1)(None)
    ts = (C.c_float * 1)(999.0)
    args = (dummy, None, dummy, 1, 16, 16, dummy, dummy, 0, None)
    assert lib.dif_rollout(P, ts, 0, 1, *args) == -1     # n_steps < 1
    assert lib.dif_rollout(P, ts, 1, 7, *args) == -1     # unknown sampler
    assert lib.dif_rollout(P, ts, 1, 1, *args) == -1     # null plan
    assert b"plan 0" in lib.dif_last_error()
    assert lib.dif_plan_bytes_ex(None, None, 0, None) == -1
