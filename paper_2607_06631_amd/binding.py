"""ctypes binding of libdif (include/dif.h): argument marshalling only.

Every computation runs in libdif's HIP kernels.  PyTorch supplies device
memory and the current HIP stream.  Functions carry the C entry points'
names; DifError is raised for a non-zero status with dif_last_error().
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdif.so")

DIF_BF16, DIF_F32 = 0, 1
EPI_STORE, EPI_GELU, EPI_RESIDUAL = 0, 1, 2
PROF_KINDS = 16

STATUS_NAMES = {0: "DIF_OK", -1: "DIF_E_ARG", -2: "DIF_E_SHAPE", -3: "DIF_E_MASK",
                -4: "DIF_E_UNSUPPORTED", -5: "DIF_E_WORKSPACE", -6: "DIF_E_HIP"}


class DifError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


class DifConfig(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("dim", "n_heads", "head_dim", "ffn_dim", "n_layers",
                                         "patch_dim", "freq_dim", "grid_f", "grid_h", "grid_w",
                                         "max_text_len", "dtype")] + \
               [("eps", C.c_float), ("rope_theta", C.c_float)]


LAYER_FIELDS = ("mod", "self_wq", "self_wk", "self_wv", "self_wo", "self_bq", "self_bk", "self_bv",
                "self_bo", "self_gq", "self_gk", "norm3_w", "norm3_b", "cross_wq", "cross_wk",
                "cross_wv", "cross_wo", "cross_bq", "cross_bk", "cross_bv", "cross_bo", "cross_gq",
                "cross_gk", "ffn_w1", "ffn_b1", "ffn_w2", "ffn_b2")
GLOBAL_FIELDS = ("patch_w", "patch_b", "t_w1", "t_b1", "t_w2", "t_b2", "t_w3", "t_b3", "head_mod",
                 "head_w", "head_b")
MATRIX_FIELDS = {"patch_w", "t_w1", "t_w2", "t_w3", "head_w", "self_wq", "self_wk", "self_wv",
                 "self_wo", "cross_wq", "cross_wk", "cross_wv", "cross_wo", "ffn_w1", "ffn_w2"}


class DifLayerWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in LAYER_FIELDS]


class DifWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in GLOBAL_FIELDS] + [("layers", C.POINTER(DifLayerWeights))]


class DifStepMasks(C.Structure):
    _fields_ = [("block_keep", C.c_void_p), ("self_head_keep", C.c_void_p),
                ("cross_head_keep", C.c_void_p), ("ffn_keep", C.c_void_p)]


class DifLayerInfo(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("block_keep", "self_heads", "cross_heads",
                                         "ffn_channels", "ffn_padded")]


_lib = None


def lib():
    """Load the in-tree libdif.so; fail loudly if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_06631_amd.build`")
        L = C.CDLL(LIB_PATH)
        vp, i32, i64, sz, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t, C.c_float
        sig = {
            "dif_last_error": (C.c_char_p, []),
            "dif_validate_config": (i32, [C.POINTER(DifConfig)]),
            "dif_validate_masks": (i32, [C.POINTER(DifConfig), C.POINTER(DifStepMasks)]),
            "dif_model_create": (i32, [C.POINTER(DifConfig), C.POINTER(DifWeights), C.POINTER(vp)]),
            "dif_model_destroy": (i32, [vp]),
            "dif_plan_bytes": (i32, [vp, C.POINTER(DifStepMasks), C.POINTER(sz)]),
            "dif_plan_step": (i32, [vp, i32, f32, C.POINTER(DifStepMasks), vp, sz, vp,
                                    C.POINTER(vp)]),
            "dif_plan_bytes_ex": (i32, [vp, C.POINTER(DifStepMasks), i32, C.POINTER(sz)]),
            "dif_plan_step_ex": (i32, [vp, i32, f32, C.POINTER(DifStepMasks), i32, i32, vp, sz, vp,
                                       C.POINTER(vp)]),
            "dif_plan_timestep": (i32, [vp, C.POINTER(f32), C.POINTER(i32)]),
            "dif_plan_destroy": (i32, [vp]),
            "dif_plan_layer_info": (i32, [vp, i32, C.POINTER(DifLayerInfo)]),
            "dif_workspace_bytes": (i32, [vp, i32, i32, i32, C.POINTER(sz)]),
            "dif_time_embed": (i32, [vp, f32, vp, vp, vp, sz, vp]),
            "dif_block_forward": (i32, [vp, i32, vp, vp, vp, i32, i32, i32, vp, sz, vp]),
            "dif_step_forward": (i32, [vp, vp, f32, vp, i32, i32, i32, vp, vp, sz, vp]),
            "dif_block_forward_cached": (i32, [vp, i32, vp, vp, sz, vp, i32, i32, i32, vp, sz, vp]),
            "dif_step_forward_cached": (i32, [vp, vp, f32, vp, sz, i32, i32, i32, vp, vp, sz, vp]),
            "dif_text_cache_bytes": (i32, [vp, i32, i32, C.POINTER(sz)]),
            "dif_text_cache_build": (i32, [vp, vp, i32, i32, vp, sz, vp]),
            "dif_euler": (i32, [vp, vp, f32, f32, i64, vp]),
            "dif_hard_gates": (i32, [C.POINTER(DifConfig), i32] + [vp] * 8),
            "dif_ffn_reorder": (i32, [vp, i32, vp, vp, vp, vp, vp, sz, vp]),
            "dif_renoise": (i32, [vp, vp, f32, f32, vp, i64, vp]),
            "dif_rollout": (i32, [C.POINTER(vp), C.POINTER(f32), i32, i32, vp, C.POINTER(vp), vp,
                                  i32, i32, i32, vp, vp, sz, vp]),
            "dif_rollout_cached": (i32, [C.POINTER(vp), C.POINTER(f32), i32, i32, vp, C.POINTER(vp),
                                         vp, sz, i32, i32, i32, vp, vp, sz, vp]),
            "dif_gemm": (i32, [i32, i32, vp, i64, vp, i64, vp, i64, i32, i32, i32, i32, vp, vp, vp, vp]),
            "dif_attention": (i32, [i32, i32, vp, i64, vp, i64, vp, i64, vp, i64, i32, i32, i32, i32, vp]),
            "dif_attention_split_bytes": (i32, [i32, C.POINTER(sz)]),
            "dif_attention_ex": (i32, [i32, i32, i32, vp, i64, vp, i64, vp, i64, vp, i64, i32, i32,
                                       i32, i32, vp, sz, vp]),
            "dif_attention_ex_static": (i32, [i32, i32, i32, vp, i64, vp, i64, vp, i64, vp, i64, i32,
                                              i32, i32, i32, vp]),
            "dif_mfma_probe": (i32, [i32, i32, vp, C.POINTER(C.c_double), vp]),
            "dif_profile_enable": (i32, [i32]),
            "dif_profile_reset": (i32, []),
            "dif_profile_kind_name": (C.c_char_p, [i32]),
            "dif_profile_collect": (i32, [C.POINTER(C.c_int64), C.POINTER(C.c_double),
                                          C.POINTER(C.c_double), C.POINTER(C.c_double)]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise DifError(status, lib().dif_last_error().decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must live in device memory")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _stream(stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _np_ptr(a: np.ndarray) -> int:
    return a.ctypes.data


# ---------------------------------------------------------------------------
# configuration, masks
# ---------------------------------------------------------------------------

def make_config(cfg) -> DifConfig:
    """DifConfig from any object with the model's attributes (dim, n_heads,
    head_dim, ffn_dim, n_layers, patch_dim, freq_dim, grid, text_len, dtype
    ("bf16"/"f32"), eps, rope_theta)."""
    gf, gh, gw = cfg.grid
    return DifConfig(cfg.dim, cfg.n_heads, cfg.head_dim, cfg.ffn_dim, cfg.n_layers, cfg.patch_dim,
                     cfg.freq_dim, gf, gh, gw, cfg.text_len,
                     DIF_BF16 if cfg.dtype == "bf16" else DIF_F32, cfg.eps, cfg.rope_theta)


class _Masks:
    """Host copies of one step's masks, kept alive while the C struct is used."""

    def __init__(self, masks: Dict[str, np.ndarray]):
        self.arrays = {k: np.ascontiguousarray(masks[k], dtype=np.uint8)
                       for k in ("block_keep", "self_head_keep", "cross_head_keep", "ffn_keep")}
        self.struct = DifStepMasks(*(_np_ptr(self.arrays[k]) for k in
                                     ("block_keep", "self_head_keep", "cross_head_keep", "ffn_keep")))


def dif_validate_config(cfg) -> None:
    c = make_config(cfg)
    _check(lib().dif_validate_config(C.byref(c)))


def dif_validate_masks(cfg, masks) -> None:
    c = make_config(cfg)
    m = _Masks(masks)
    _check(lib().dif_validate_masks(C.byref(c), C.byref(m.struct)))


# ---------------------------------------------------------------------------
# model and plans
# ---------------------------------------------------------------------------

def upload_weights(w: Dict, dtype: str, device="cuda"):
    """numpy weights (float32 arrays, see workloads.synth) -> device tensors:
    matrices in the model dtype, everything else float32."""
    import torch
    mdt = torch.bfloat16 if dtype == "bf16" else torch.float32

    def conv(k, a):
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
        return t.to(mdt) if k in MATRIX_FIELDS else t

    out = {k: conv(k, v) for k, v in w.items() if k != "layers"}
    out["layers"] = [{k: conv(k, v) for k, v in lw.items()} for lw in w["layers"]]
    return out


class Model:
    def __init__(self, cfg, weights: Dict):
        import torch
        self.cfg = cfg
        self.c = make_config(cfg)
        self.weights = weights   # keep device tensors alive
        mdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32

        def p(k, t):
            want = mdt if k in MATRIX_FIELDS else torch.float32
            if t.dtype != want:
                raise ValueError(f"{k}: dtype {t.dtype}, expected {want}")
            return _ptr(t)

        n = cfg.n_layers
        if len(weights["layers"]) != n:
            raise ValueError("layer count mismatch")
        self._layers = (DifLayerWeights * n)(*[
            DifLayerWeights(*(p(k, lw[k]) for k in LAYER_FIELDS)) for lw in weights["layers"]])
        self._w = DifWeights(*(p(k, weights[k]) for k in GLOBAL_FIELDS), self._layers)
        h = C.c_void_p()
        _check(lib().dif_model_create(C.byref(self.c), C.byref(self._w), C.byref(h)))
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.dif_model_destroy(self.handle)
            self.handle = None


class Plan:
    def __init__(self, model: Model, handle, mem, masks: _Masks, step: int):
        self.model, self.handle, self.mem, self._masks, self.step = model, handle, mem, masks, step

    def layer_info(self, layer: int) -> DifLayerInfo:
        info = DifLayerInfo()
        _check(lib().dif_plan_layer_info(self.handle, layer, C.byref(info)))
        return info

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.dif_plan_destroy(self.handle)
            self.handle = None


def dif_model_create(cfg, weights: Dict) -> Model:
    return Model(cfg, weights)


DIF_PLAN_COMPACT, DIF_PLAN_INDEXED = 0, 1
DIF_PLAN_ANY_T = 1
PLAN_KINDS = {"compact": DIF_PLAN_COMPACT, "indexed": DIF_PLAN_INDEXED}


def dif_plan_bytes(model: Model, masks, kind: str = "compact") -> int:
    m = _Masks(masks)
    n = C.c_size_t()
    _check(lib().dif_plan_bytes_ex(model.handle, C.byref(m.struct), PLAN_KINDS[kind], C.byref(n)))
    return n.value


def dif_plan_step(model: Model, step: int, t_s: float, masks, stream=None, kind: str = "compact",
                  any_t: bool = False) -> Plan:
    """Index tables (and, for kind="compact", the gather of the step's active
    parameters) in plan memory allocated here with torch (owned by the
    returned Plan).  The plan is bound to timestep t_s (any_t: unbound)."""
    import torch
    m = _Masks(masks)
    n = C.c_size_t()
    k = PLAN_KINDS[kind]
    _check(lib().dif_plan_bytes_ex(model.handle, C.byref(m.struct), k, C.byref(n)))
    mem = torch.empty(max(n.value, 256), dtype=torch.uint8, device="cuda")
    h = C.c_void_p()
    _check(lib().dif_plan_step_ex(model.handle, step, float(t_s), C.byref(m.struct), k,
                                  DIF_PLAN_ANY_T if any_t else 0, mem.data_ptr(), n.value,
                                  _stream(stream), C.byref(h)))
    plan = Plan(model, h, mem, m, step)
    plan.kind = kind
    return plan


def dif_plan_timestep(plan: Plan):
    """(t_s, flags) of a plan."""
    t, f = C.c_float(), C.c_int32()
    _check(lib().dif_plan_timestep(plan.handle, C.byref(t), C.byref(f)))
    return t.value, f.value


def dif_workspace_bytes(model: Model, B: int, L: int, Lc: int) -> int:
    n = C.c_size_t()
    _check(lib().dif_workspace_bytes(model.handle, B, L, Lc, C.byref(n)))
    return n.value


def workspace(model: Model, B: int, L: int, Lc: int):
    import torch
    return torch.empty(dif_workspace_bytes(model, B, L, Lc), dtype=torch.uint8, device="cuda")


def dif_time_embed(model: Model, t: float, e, e0, ws, stream=None) -> None:
    _check(lib().dif_time_embed(model.handle, float(t), _ptr(e), _ptr(e0), _ptr(ws),
                                ws.numel(), _stream(stream)))


def dif_block_forward(plan: Plan, layer: int, x, ctx, e0, ws, stream=None) -> None:
    B, L = x.shape[0], x.shape[1]
    Lc = ctx.shape[1]
    _check(lib().dif_block_forward(plan.handle, layer, _ptr(x), _ptr(ctx), _ptr(e0), B, L, Lc,
                                   _ptr(ws), ws.numel(), _stream(stream)))


def dif_step_forward(plan: Plan, z, t: float, ctx, v_out, ws, stream=None) -> None:
    B, L = z.shape[0], z.shape[1]
    Lc = ctx.shape[1]
    _check(lib().dif_step_forward(plan.handle, _ptr(z), float(t), _ptr(ctx), B, L, Lc, _ptr(v_out),
                                  _ptr(ws), ws.numel(), _stream(stream)))


class TextCache:
    """Device memory holding every layer's text keys and values for one
    context (B samples of Lc tokens); built by dif_text_cache_build."""

    def __init__(self, mem, B: int, Lc: int):
        self.mem, self.B, self.Lc = mem, B, Lc


def dif_text_cache_bytes(model: Model, B: int, Lc: int) -> int:
    n = C.c_size_t()
    _check(lib().dif_text_cache_bytes(model.handle, B, Lc, C.byref(n)))
    return n.value


def dif_text_cache_build(model: Model, ctx, stream=None) -> TextCache:
    import torch
    B, Lc = ctx.shape[0], ctx.shape[1]
    mem = torch.empty(dif_text_cache_bytes(model, B, Lc), dtype=torch.uint8, device=ctx.device)
    _check(lib().dif_text_cache_build(model.handle, _ptr(ctx), B, Lc, _ptr(mem), mem.numel(),
                                      _stream(stream)))
    return TextCache(mem, B, Lc)


def dif_block_forward_cached(plan: Plan, layer: int, x, cache: TextCache, e0, ws, stream=None) -> None:
    B, L = x.shape[0], x.shape[1]
    _check(lib().dif_block_forward_cached(plan.handle, layer, _ptr(x), _ptr(cache.mem),
                                          cache.mem.numel(), _ptr(e0), B, L, cache.Lc, _ptr(ws),
                                          ws.numel(), _stream(stream)))


def dif_step_forward_cached(plan: Plan, z, t: float, cache: TextCache, v_out, ws, stream=None) -> None:
    B, L = z.shape[0], z.shape[1]
    _check(lib().dif_step_forward_cached(plan.handle, _ptr(z), float(t), _ptr(cache.mem),
                                         cache.mem.numel(), B, L, cache.Lc, _ptr(v_out), _ptr(ws),
                                         ws.numel(), _stream(stream)))


def dif_hard_gates(cfg, m_block, m_self, m_cross, m_ffn, chunk: int = 8):
    """Keep masks of one step from its continuous masks (host arrays)."""
    import numpy as np
    N, H, F = cfg.n_layers, cfg.n_heads, cfg.ffn_dim
    c = make_config(cfg)
    ins = [np.ascontiguousarray(a, dtype=np.float32) for a in (m_block, m_self, m_cross, m_ffn)]
    out = {"block_keep": np.zeros(N, np.uint8), "self_head_keep": np.zeros((N, H), np.uint8),
           "cross_head_keep": np.zeros((N, H), np.uint8), "ffn_keep": np.zeros((N, F), np.uint8)}
    ptrs = [a.ctypes.data for a in ins] + [out[k].ctypes.data for k in
                                           ("block_keep", "self_head_keep", "cross_head_keep", "ffn_keep")]
    _check(lib().dif_hard_gates(C.byref(c), int(chunk), *ptrs))
    return out


def dif_ffn_reorder(model: "Model", layer: int, stream=None):
    """(perm, w1, b1, w2): the layer's FFN weights with hidden channels sorted
    by decreasing norm, as new device tensors."""
    import numpy as np
    import torch
    cfg = model.cfg
    D, F = cfg.dim, cfg.ffn_dim
    mdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    w1 = torch.empty((F, D), dtype=mdt, device="cuda")
    w2 = torch.empty((D, F), dtype=mdt, device="cuda")
    b1 = torch.empty((F,), dtype=torch.float32, device="cuda")
    scratch = torch.empty(F * 12 + 16, dtype=torch.uint8, device="cuda")
    perm = np.zeros(F, np.int32)
    _check(lib().dif_ffn_reorder(model.handle, layer, _ptr(w1), _ptr(b1), _ptr(w2),
                                 perm.ctypes.data, _ptr(scratch), scratch.numel(), _stream(stream)))
    return perm, w1, b1, w2


DIF_SAMPLER_EULER, DIF_SAMPLER_RENOISE = 0, 1
SAMPLERS = {"euler": DIF_SAMPLER_EULER, "renoise": DIF_SAMPLER_RENOISE}


def dif_renoise(z, v, sigma_from: float, sigma_to: float, eps=None, stream=None) -> None:
    _check(lib().dif_renoise(_ptr(z), _ptr(v), float(sigma_from), float(sigma_to),
                             _ptr(eps) if eps is not None else None, z.numel(), _stream(stream)))


def dif_rollout(plans, timesteps, z, ctx, v_scratch, ws, eps=None, sampler: str = "renoise",
                stream=None) -> None:
    """Steps plans[0..] from z (in place) to the clean estimate of the last one."""
    n = len(plans)
    P = (C.c_void_p * n)(*[p.handle for p in plans])
    ts = (C.c_float * n)(*[float(t) for t in timesteps])
    E = None
    if eps is not None:
        E = (C.c_void_p * n)(*[(_ptr(e) if e is not None else None) for e in eps])
    B, L = z.shape[0], z.shape[1]
    _check(lib().dif_rollout(P, ts, n, SAMPLERS[sampler], _ptr(z), E, _ptr(ctx), B, L, ctx.shape[1],
                             _ptr(v_scratch), _ptr(ws), ws.numel(), _stream(stream)))


def dif_rollout_cached(plans, timesteps, z, cache: TextCache, v_scratch, ws, eps=None,
                       sampler: str = "renoise", stream=None) -> None:
    """dif_rollout with the text keys and values read from `cache`."""
    n = len(plans)
    P = (C.c_void_p * n)(*[p.handle for p in plans])
    ts = (C.c_float * n)(*[float(t) for t in timesteps])
    E = None
    if eps is not None:
        E = (C.c_void_p * n)(*[(_ptr(e) if e is not None else None) for e in eps])
    B, L = z.shape[0], z.shape[1]
    _check(lib().dif_rollout_cached(P, ts, n, SAMPLERS[sampler], _ptr(z), E, _ptr(cache.mem),
                                    cache.mem.numel(), B, L, cache.Lc, _ptr(v_scratch), _ptr(ws),
                                    ws.numel(), _stream(stream)))


def dif_euler(z, v, sigma_from: float, sigma_to: float, stream=None) -> None:
    _check(lib().dif_euler(_ptr(z), _ptr(v), float(sigma_from), float(sigma_to), z.numel(),
                           _stream(stream)))


def _dt(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return DIF_BF16
    if t.dtype == torch.float32:
        return DIF_F32
    raise ValueError(f"unsupported dtype {t.dtype}")


def dif_gemm(A, B, C_out, epilogue=EPI_STORE, bias=None, gate0=None, gate1=None, M=None, N=None,
             K=None, lda=None, ldb=None, ldc=None, stream=None) -> None:
    """C = epilogue(A[M,K] B[N,K]^T); 2-D row-major tensors (strides as given)."""
    M = A.shape[0] if M is None else M
    N = B.shape[0] if N is None else N
    K = B.shape[1] if K is None else K
    lda = A.stride(0) if lda is None else lda
    ldb = B.stride(0) if ldb is None else ldb
    ldc = C_out.stride(0) if ldc is None else ldc
    _check(lib().dif_gemm(_dt(A), _dt(C_out), A.data_ptr(), lda, B.data_ptr(), ldb,
                          C_out.data_ptr(), ldc, M, N, K, epilogue, _ptr(bias), _ptr(gate0),
                          _ptr(gate1), _stream(stream)))


def dif_attention(Q, K, Vt, O, B: int, Lq: int, Lk: int, n_heads: int, head_dim: int,
                  ldq: int, ldk: int, ldvt: int, ldo: int, stream=None) -> None:
    _check(lib().dif_attention(_dt(Q), head_dim, Q.data_ptr(), ldq, K.data_ptr(), ldk,
                               Vt.data_ptr(), ldvt, O.data_ptr(), ldo, B, Lq, Lk, n_heads,
                               _stream(stream)))


DIF_ATTN_Q_PRESCALED = 1


MFMA_32X32X16, MFMA_16X16X32, PROBE_EXP_F32 = 0, 1, 2


def dif_mfma_probe(iters: int, sink, shape: int = MFMA_32X32X16, stream=None) -> float:
    """Launches the sustained-rate kernel for one bf16 MFMA shape (or, for
    PROBE_EXP_F32, the exponential); returns its FLOPs (the exponentials'
    count for PROBE_EXP_F32; time it with events on the same stream).
    `sink`: a float32 device tensor."""
    fl = C.c_double()
    _check(lib().dif_mfma_probe(shape, iters, sink.data_ptr(), C.byref(fl), _stream(stream)))
    return fl.value


def dif_attention_split_bytes(head_dim: int) -> int:
    n = C.c_size_t()
    _check(lib().dif_attention_split_bytes(head_dim, C.byref(n)))
    return n.value


def dif_attention_ex(Q, K, Vt, O, B: int, Lq: int, Lk: int, n_heads: int, head_dim: int,
                     ldq: int, ldk: int, ldvt: int, ldo: int, flags: int = 0, split_ws=None,
                     stream=None) -> None:
    """dif_attention with flags (DIF_ATTN_Q_PRESCALED) and an optional split
    workspace (a uint8 device tensor of >= dif_attention_split_bytes)."""
    _check(lib().dif_attention_ex(_dt(Q), head_dim, flags, Q.data_ptr(), ldq, K.data_ptr(), ldk,
                                  Vt.data_ptr(), ldvt, O.data_ptr(), ldo, B, Lq, Lk, n_heads,
                                  _ptr(split_ws), 0 if split_ws is None else split_ws.numel(),
                                  _stream(stream)))


def dif_attention_ex_static(Q, K, Vt, O, B: int, Lq: int, Lk: int, n_heads: int, head_dim: int,
                            ldq: int, ldk: int, ldvt: int, ldo: int, flags: int = 0,
                            stream=None) -> None:
    """dif_attention_ex with the library's static split workspace (allocates nothing)."""
    _check(lib().dif_attention_ex_static(_dt(Q), head_dim, flags, Q.data_ptr(), ldq, K.data_ptr(),
                                         ldk, Vt.data_ptr(), ldvt, O.data_ptr(), ldo, B, Lq, Lk,
                                         n_heads, _stream(stream)))


# ---------------------------------------------------------------------------
# kernel timing
# ---------------------------------------------------------------------------

def dif_profile_enable(on: bool = True) -> None:
    _check(lib().dif_profile_enable(1 if on else 0))


def dif_profile_reset() -> None:
    _check(lib().dif_profile_reset())


def dif_profile_collect() -> Dict[str, dict]:
    n = PROF_KINDS
    la, ms, fl, by = (C.c_int64 * n)(), (C.c_double * n)(), (C.c_double * n)(), (C.c_double * n)()
    _check(lib().dif_profile_collect(la, ms, fl, by))
    out = {}
    for k in range(n):
        if la[k]:
            out[lib().dif_profile_kind_name(k).decode()] = {
                "launches": la[k], "ms": ms[k], "flops": fl[k], "bytes": by[k]}
    return out
