"""Operator-level parity of the hot kernels through the C ABI.

GEMM: C = A B^T (its plain definition, numpy float64 matmul on the same
inputs).  Attention: the oracle's two-pass softmax attention on the same
inputs.  Shapes span several tiles with ragged tails in every dimension.
"""
import numpy as np
import pytest

import oracle as O
from paper_2607_06631_amd import binding as B
from tests.gpu_util import rel_err, say, to_np
from workloads.synth import bf16_round

pytestmark = pytest.mark.gpu


def _rand(g, shape, scale=1.0, bf16=True):
    a = g.standard_normal(shape, dtype=np.float32) * np.float32(scale)
    return bf16_round(a) if bf16 else a


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("M,N,K", [(1, 64, 64), (300, 200, 128), (517, 1152, 256), (1000, 640, 0),
                                   (2100, 768, 1536)])
def test_gemm_store_matches_matmul(dtype, M, N, K):
    import torch
    say(f"gemm store {dtype} M={M} N={N} K={K}")
    g = np.random.default_rng(M + N + K)
    bf = dtype == "bf16"
    tdt = torch.bfloat16 if bf else torch.float32
    a, b = _rand(g, (M, K), bf16=bf), _rand(g, (N, K), bf16=bf)
    bias = g.standard_normal(N).astype(np.float32)
    A = torch.from_numpy(a).cuda().to(tdt)
    Bm = torch.from_numpy(b).cuda().to(tdt)
    Cf = torch.full((M, N), float("nan"), device="cuda", dtype=torch.float32)
    B.dif_gemm(A, Bm, Cf, B.EPI_STORE, bias=torch.from_numpy(bias).cuda(), K=K)
    torch.cuda.synchronize()
    ref = a.astype(np.float64) @ b.astype(np.float64).T + bias
    tol = 1e-5 if K else 0.0
    assert rel_err(to_np(Cf), ref) <= tol
    if bf:  # bf16 output: one extra rounding
        Cb = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
        B.dif_gemm(A, Bm, Cb, B.EPI_STORE, bias=torch.from_numpy(bias).cuda(), K=K)
        torch.cuda.synchronize()
        assert rel_err(to_np(Cb), ref) <= 8e-3


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_gemm_gelu_and_residual_epilogues(dtype):
    import torch
    say(f"gemm epilogues {dtype}")
    g = np.random.default_rng(7)
    bf = dtype == "bf16"
    tdt = torch.bfloat16 if bf else torch.float32
    M, N, K = 777, 320, 192
    a, b = _rand(g, (M, K), 0.5, bf), _rand(g, (N, K), 0.5, bf)
    bias = g.standard_normal(N).astype(np.float32)
    g0, g1 = g.standard_normal(N).astype(np.float32), g.standard_normal(N).astype(np.float32)
    x0 = _rand(g, (M, N), 1.0, bf)
    A, Bm = torch.from_numpy(a).cuda().to(tdt), torch.from_numpy(b).cuda().to(tdt)
    acc = a.astype(np.float64) @ b.astype(np.float64).T + bias
    C = torch.empty((M, N), device="cuda", dtype=tdt)
    B.dif_gemm(A, Bm, C, B.EPI_GELU, bias=torch.from_numpy(bias).cuda())
    X = torch.from_numpy(x0).cuda().to(tdt)
    B.dif_gemm(A, Bm, X, B.EPI_RESIDUAL, bias=torch.from_numpy(bias).cuda(),
               gate0=torch.from_numpy(g0).cuda(), gate1=torch.from_numpy(g1).cuda())
    torch.cuda.synchronize()
    tol = 8e-3 if bf else 1e-5
    assert rel_err(to_np(C), O.gelu_tanh(acc)) <= tol
    assert rel_err(to_np(X), x0 + (g0 + g1) * acc) <= tol


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("ldc_pad", [0, 3])
def test_gemm_ragged_columns_and_unaligned_rows(dtype, ldc_pad):
    """N not a multiple of 4 and (ldc_pad = 3) rows that are not 4-element
    aligned: the epilogue's element-wise path; nothing outside C is written."""
    import torch
    say(f"gemm ragged {dtype} ldc_pad={ldc_pad}")
    g = np.random.default_rng(11 + ldc_pad)
    bf = dtype == "bf16"
    tdt = torch.bfloat16 if bf else torch.float32
    M, N, K = 300, 203, 64
    ldc = N + ldc_pad
    a, b = _rand(g, (M, K), 0.5, bf), _rand(g, (N, K), 0.5, bf)
    bias = g.standard_normal(N).astype(np.float32)
    g0 = g.standard_normal(N).astype(np.float32)
    x0 = _rand(g, (M, N), 1.0, bf)
    A, Bm = torch.from_numpy(a).cuda().to(tdt), torch.from_numpy(b).cuda().to(tdt)
    acc = a.astype(np.float64) @ b.astype(np.float64).T + bias
    tol = 8e-3 if bf else 1e-5
    for epi in (B.EPI_STORE, B.EPI_GELU, B.EPI_RESIDUAL):
        buf = torch.full((M + 1, ldc), 7.0, device="cuda", dtype=tdt)
        if epi == B.EPI_RESIDUAL:
            buf[:M, :N] = torch.from_numpy(x0).cuda().to(tdt)
        C = buf[:M]
        B.dif_gemm(A, Bm, C, epi, bias=torch.from_numpy(bias).cuda(),
                   gate0=torch.from_numpy(g0).cuda() if epi == B.EPI_RESIDUAL else None,
                   N=N, ldc=ldc)
        torch.cuda.synchronize()
        out = to_np(buf)
        ref = {B.EPI_STORE: acc, B.EPI_GELU: O.gelu_tanh(acc), B.EPI_RESIDUAL: x0 + g0 * acc}[epi]
        assert rel_err(out[:M, :N], ref) <= tol
        assert np.all(out[:M, N:] == 7.0) and np.all(out[M] == 7.0)


@pytest.mark.parametrize("M", [127 * 256 - 7, 127 * 256 + 37])
def test_gemm_store_either_side_of_the_small_problem_tiling(M):
    """Store-epilogue problems with fewer than 128 tiles of 256 x 256 run as
    128 x 128 tiles: M = 32505 and 32549 with N = 256 give 127 and 128 large
    tiles, one on each side of the switch; sampled rows incl. the ragged tail
    against the float64 product."""
    import torch
    N, K = 256, 192
    say(f"gemm store bf16 M={M} N={N} K={K}: {-(-M // 256) * (N // 256)} tiles of 256 x 256")
    g = np.random.default_rng(M)
    a, b = _rand(g, (M, K), 0.5), _rand(g, (N, K), 0.5)
    bias = g.standard_normal(N).astype(np.float32)
    C = torch.full((M, N), float("nan"), device="cuda", dtype=torch.float32)
    B.dif_gemm(torch.from_numpy(a).cuda().to(torch.bfloat16), torch.from_numpy(b).cuda().to(torch.bfloat16),
               C, B.EPI_STORE, bias=torch.from_numpy(bias).cuda())
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(64), g.choice(M, 512, replace=False), np.arange(M - 300, M)]))
    ref = a[rows].astype(np.float64) @ b.astype(np.float64).T + bias
    assert rel_err(to_np(C)[rows], ref) <= 1e-5


def _attn_case(dtype, dh, H, Lq, Lk, Bn=1, qscale=1.0, seed=0):
    import torch
    g = np.random.default_rng(seed)
    bf = dtype == "bf16"
    tdt = torch.bfloat16 if bf else torch.float32
    W = H * dh
    q = _rand(g, (Bn, Lq, W), qscale, bf)
    k = _rand(g, (Bn, Lk, W), 1.0, bf)
    v = _rand(g, (Bn, Lk, W), 1.0, bf)
    ldvt = -(-Lk // 64) * 64 + 64       # padded, garbage in the pad
    vt = np.full((Bn, W, ldvt), np.nan, np.float32)
    vt[:, :, :Lk] = v.transpose(0, 2, 1)
    Q, K = torch.from_numpy(q).cuda().to(tdt), torch.from_numpy(k).cuda().to(tdt)
    Vt = torch.from_numpy(vt).cuda().to(tdt)
    Ot = torch.full((Bn, Lq, W), float("nan"), device="cuda", dtype=tdt)
    B.dif_attention(Q, K, Vt, Ot, Bn, Lq, Lk, H, dh, W, W, ldvt, W)
    torch.cuda.synchronize()
    got = to_np(Ot)
    ref = np.stack([O.attention(q[b].astype(np.float64), k[b].astype(np.float64),
                                v[b].astype(np.float64), H, dh) for b in range(Bn)])
    return rel_err(got, ref)


@pytest.mark.parametrize("dtype,dh", [("bf16", 128), ("f32", 64), ("f32", 128), ("bf16", 64)])
@pytest.mark.parametrize("Lq,Lk", [(128, 64), (333, 517), (70, 5), (1, 1)])
def test_attention_matches_oracle(dtype, dh, Lq, Lk):
    say(f"attention {dtype} dh={dh} Lq={Lq} Lk={Lk}")
    err = _attn_case(dtype, dh, 3, Lq, Lk, Bn=2, qscale=3.0, seed=Lq + Lk)
    assert err <= (2e-2 if dtype == "bf16" else 1e-5)


@pytest.mark.parametrize("dh", [128, 64])
def test_attention_long_keys_online_softmax(dh):
    say(f"attention bf16 long keys dh={dh} (long-key kernels)")
    # sharp scores that keep moving the running max across many key tiles;
    # Lk >= 4096 takes the long-key kernels (two query groups per wave at
    # head_dim 128, eight waves at 64), Lq = 300 ends in a partial 256-query
    # block and Lk = 4099 in a 3-key tile
    err = _attn_case("bf16", dh, 2, 300, 4099, Bn=1, qscale=4.0, seed=11)
    assert err <= 2e-2


@pytest.mark.parametrize("Lk", [4160, 4165, 4257])
def test_attention_long_keys_ring_leftovers(Lk):
    """The two-group kernel runs its middle key tiles in groups of three
    (one per LDS ring slot) and the rest, with the last tile, through a
    run-time slot: 4160 keys (65 full tiles) leave none, 4165 (a 5-key
    tail) one, 4257 (a 33-key tail) two."""
    say(f"attention bf16 dh=128 Lk={Lk} (ring leftovers)")
    err = _attn_case("bf16", 128, 2, 300, Lk, Bn=2, qscale=4.0, seed=Lk)
    assert err <= 2e-2


@pytest.mark.gpu
def test_mfma_probe_rate_is_plausible():
    """dif_mfma_probe, both MFMA shapes and the exponential: counts as documented (iters rounded up
    to a multiple of 4; 2 workgroups x 4 waves per CU x 262144 FLOPs per
    iteration), a rate between a tenth and all of the 2.5 PFLOP/s nominal
    peak, and the guard store never taken; bad arguments are rejected."""
    import torch
    say("mfma probe")
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    sink = torch.zeros(1, device="cuda", dtype=torch.float32)
    for shape in (B.MFMA_32X32X16, B.MFMA_16X16X32):
        fl = B.dif_mfma_probe(1001, sink, shape)
        assert fl == 2 * ncu * 4 * 1004 * 8 * 2 * 32 * 32 * 16
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fl = B.dif_mfma_probe(2000, sink, shape)
        e1.record()
        torch.cuda.synchronize()
        tflops = fl / e0.elapsed_time(e1) / 1e9
        say(f"  shape {shape}: {tflops:.1f} TFLOP/s")
        assert 250.0 < tflops <= 2500.0
    # the exponential: 8 workgroups x 256 lanes per CU x 16 per iteration,
    # at a rate above 10^11 per second and no faster than every lane of
    # every SIMD finishing one per cycle at 2.4 GHz
    fl = B.dif_mfma_probe(1001, sink, B.PROBE_EXP_F32)
    assert fl == 8 * ncu * 256 * 1004 * 16
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    fl = B.dif_mfma_probe(20000, sink, B.PROBE_EXP_F32)
    e1.record()
    torch.cuda.synchronize()
    rate = fl / (e0.elapsed_time(e1) * 1e-3)
    say(f"  exp: {rate:.3e} per second")
    assert 1e11 < rate <= ncu * 64 * 2.4e9
    assert sink.item() == 0.0
    with pytest.raises(B.DifError):
        B.dif_mfma_probe(0, sink)
    with pytest.raises(B.DifError):
        B.dif_mfma_probe(10, sink, 3)
