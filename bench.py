"""Benchmark: pruned denoise steps of a Wan-14B-shaped 40-layer DiT at 480p.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A "step" is one denoise step of the 4-step sampler: timestep embedding,
patch embedding, 40 blocks under that step's structure, output head and the
Euler update; consecutive steps cycle through the four step structures
(t = 999, 750, 500, 250).  Weights (about 28 GB, random init), latents and
text context are synthetic and already resident in HBM when timing starts;
the four per-step compacted weight sets are built beforehand (plan time is
not step time).  Prints one JSON line.

The timed steps run twice: once with HIP events around every kernel launch
(per-kernel table and roofline; this pass gives `value`) and once without
(`ms_per_step_no_kernel_timing`).

--workload wan14b_block / wan1.3b_block time one full-length block per step
structure instead (ms per block, TFLOP/s, fraction of peak, t_s / t_1
against F_s / F_1).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 matrix
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E

# HBM bytes per self-attention launch over the four step structures, from
# rocprofv3 FETCH_SIZE and WRITE_SIZE passes scaled by a 2 GiB device copy
# (read factor 0.5, write factor 1.0).  Valid only for the workload and the
# kernel sources they were measured on; reported as null otherwise.
ATTN_TRAFFIC = {
    "kernel": "attn_self",
    "workload": "wan14b_480p",
    "sources": ("paper_2607_06631_amd/csrc/attention.hip", "paper_2607_06631_amd/csrc/common.h"),
    "sha256": "6464fc09cbbe108547641a49baaf2282ed1af408c8b706b33e64c5f012c99558",
    "fetch_bytes": 1103487.105078125 * 1024 / 0.500,
    "write_bytes": 255131.5083984375 * 1024 / 1.000,
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=8)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--workload", default="wan14b_480p",
                    choices=["wan14b_480p", "wan14b_720p", "tiny", "wan14b_block", "wan1.3b_block"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true",
                    help="skip the pass with per-kernel events (no kernel table / roofline)")
    ap.add_argument("--plan", default="compact", choices=["compact", "indexed"],
                    help="compact: per-step gathered weights; indexed: union weights read "
                         "in place through the index tables")
    ap.add_argument("--text-cache", action="store_true",
                    help="project every layer's text keys and values once per video "
                         "(timed apart, reported as text_cache_build_ms) and run the cached "
                         "step; the step's FLOP count then leaves out that projection")
    ap.add_argument("--gemm-vs-library", action="store_true",
                    help="instead of the step: time this library's GEMM (plain store "
                         "epilogue) against torch's bf16 linear (the platform BLAS) on the "
                         "step's projection shapes, and print one JSON line")
    ap.add_argument("--mfma-ceiling", action="store_true",
                    help="instead of the step: time the library's pure-MFMA probe (every CU "
                         "issuing the bf16 MFMA the kernels use, no memory traffic) and print "
                         "the sustained TFLOP/s as one JSON line")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="before the steps, run one plain device copy of this many MiB "
                         "(the reference dispatch that scales HBM byte counters)")
    return ap.parse_args()


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed counter passes, or
    None for another workload or when the kernel's sources differ from the
    ones measured."""
    import hashlib
    t = ATTN_TRAFFIC
    if kernel != t["kernel"] or workload != t["workload"]:
        return None
    h = hashlib.sha256()
    for f in t["sources"]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != t["sha256"]:
        return None
    return round(t["fetch_bytes"] + t["write_bytes"])


def kept_counts(plan, n_layers):
    infos = [plan.layer_info(l) for l in range(n_layers)]
    return ([i.self_heads for i in infos], [i.cross_heads for i in infos],
            [i.ffn_channels for i in infos], [i.block_keep for i in infos])


def host_info():
    """Cores this process may use, BLAS threads and the CPU model."""
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = int(os.environ.get("OMP_NUM_THREADS", "1"))
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return {"affinity_cores": len(os.sched_getaffinity(0)), "blas_threads": threads,
            "cpu_model": model}


def _oracle_block_rows(cfg, wl, m, layer, x, ctx, e0, rows):
    """Seconds of the oracle's masked-dense block (float32) for query rows
    `rows` (keys and values over all L tokens); weights zeroed beforehand."""
    import numpy as np

    import oracle as O
    wz = O.apply_keep(wl, m["self_head_keep"][layer], m["cross_head_keep"][layer],
                      m["ffn_keep"][layer], cfg.head_dim, np.float32)
    t0 = time.perf_counter()
    O.block(x, ctx, e0, wz, True, cfg.n_heads, cfg.head_dim, cfg.grid, cfg.rope_theta, cfg.eps,
            rows=rows, dtype=np.float32)
    return time.perf_counter() - t0


def _block_time_by_rows(cfg, wl, m, layer, r1, r2, seed):
    """Full-length block time of the oracle, from two timed runs on r1 and r2
    query rows: the oracle's row path costs a fixed part (LayerNorm, keys and
    values over all L tokens) plus a part per query row, so the time at L
    rows follows from the line through the two points."""
    import numpy as np

    from workloads import synth
    L = cfg.seq_len
    g = synth.rng(synth.SEED_INPUTS, seed, "cpu_sample", cfg.name)
    x = g.standard_normal((L, cfg.dim), dtype=np.float32) * np.float32(0.5)
    ctx = synth.bf16_round(g.standard_normal((cfg.text_len, cfg.dim), dtype=np.float32))
    e0 = g.standard_normal((6, cfg.dim), dtype=np.float32) * np.float32(0.1)
    rows = g.permutation(L)
    t1 = _oracle_block_rows(cfg, wl, m, layer, x, ctx, e0, np.sort(rows[:r1]))
    t2 = _oracle_block_rows(cfg, wl, m, layer, x, ctx, e0, np.sort(rows[:r2]))
    per_row = max(t2 - t1, 0.0) / (r2 - r1)
    return t1 + per_row * (L - r1), t1, t2


def cpu_baseline(cfg, w_dev, masks):
    """The oracle (numpy, masked-dense, as it stands) on the host cores:
    the tiny stack's 4-step denoise measured whole (float64); one
    full-length Wan-1.3B-width block and one block of this stack (layer 0)
    from two row samples each (float32).  `value` is the 40-layer step:
    40 x the stack's block time (masked-dense costs the same for every layer
    and structure; embedding and head are negligible)."""
    import numpy as np

    import oracle as O
    from workloads import get_config, synth
    info = host_info()
    t0 = time.perf_counter()
    tiny = get_config("tiny")
    wt = synth.make_weights(tiny, seed=0)
    O.denoise(synth.make_latents(tiny), synth.make_context(tiny), wt,
              [synth.make_masks(tiny, s) for s in range(4)], tiny)
    c1_ms = (time.perf_counter() - t0) * 1e3
    c2 = get_config("wan1.3b_block")
    c2_s, c2_t1, c2_t2 = _block_time_by_rows(c2, synth.make_layer_weights(c2, 0, 0),
                                             synth.make_masks(c2, 0), 0, 64, 256, 1)
    wl = {k: v.float().cpu().numpy() for k, v in w_dev["layers"][0].items()}
    c3_s, c3_t1, c3_t2 = _block_time_by_rows(cfg, wl, masks[0], 0, 32, 128, 2)
    step_ms = c3_s * 1e3 * cfg.n_layers
    return {
        "value": round(step_ms, 1), "unit": "ms per denoise step (extrapolated)",
        "cores": info["blas_threads"], "kind": "oracle",
        "affinity_cores": info["affinity_cores"], "cpu_model": info["cpu_model"],
        "c1_4step_ms_measured": round(c1_ms, 1),
        "c2_block_ms": round(c2_s * 1e3, 1), "c3_block_ms": round(c3_s * 1e3, 1),
        "sample": (f"float32 numpy oracle, {info['blas_threads']} BLAS threads on "
                   f"{info['affinity_cores']} cores ({info['cpu_model']}): one {cfg.dim}-wide "
                   f"block (layer 0, {cfg.seq_len} tokens, keys over all of them) timed on 32 "
                   f"and 128 query rows ({c3_t1:.1f} s, {c3_t2:.1f} s), the full block ({c3_s:.1f} s) "
                   f"from the line through them, x {cfg.n_layers} layers; Wan-1.3B-width block the "
                   f"same way on 64 / 256 rows ({c2_t1:.1f} s, {c2_t2:.1f} s -> {c2_s:.1f} s); tiny "
                   f"2-layer float64 4-step denoise measured whole ({c1_ms:.0f} ms)"),
    }


def kernel_table(prof, steps, peak, dh=128):
    """Per-kind launches, ms per step, TFLOP/s, GB/s and, for the attentions,
    softmax exponentials per second (one per (query, key, head): the kind's
    flops / (4 dh))."""
    kernels = {}
    for k, r in prof.items():
        ent = {"launches": r["launches"], "ms_per_step": round(r["ms"] / steps, 3)}
        if r["flops"] > 0:
            ent["tflops"] = round(r["flops"] / (r["ms"] * 1e-3) / 1e12, 1)
            ent["frac_peak"] = round(ent["tflops"] / peak, 4)
        if r["bytes"] > 0:
            ent["gbs"] = round(r["bytes"] / (r["ms"] * 1e-3) / 1e9, 1)
        if k.startswith("attn_") and r["flops"] > 0:
            ent["exp_per_s"] = float(f"{r['flops'] / (4 * dh) / (r['ms'] * 1e-3):.4g}")
        kernels[k] = ent
    return kernels


def roofline_of(prof, workload, peak, dh):
    if not prof:
        return None
    dom = max(prof, key=lambda k: prof[k]["ms"])
    r = prof[dom]
    per_launch_ms = r["ms"] / r["launches"]
    if r["flops"] > 0:
        ach = r["flops"] / r["launches"] / (per_launch_ms * 1e-3) / 1e12
        out = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 1), "peak": peak,
               "unit": "TFLOP/s", "frac": round(ach / peak, 4),
               "traffic": measured_traffic(dom, workload), "traffic_unit": "HBM bytes per launch",
               "avg_launch_ms": round(per_launch_ms, 4),
               "algorithmic_tflop_per_launch": round(r["flops"] / r["launches"] / 1e12, 4)}
        if dom.startswith("attn_"):
            out["exp_per_s"] = float(f"{r['flops'] / (4 * dh) / (r['ms'] * 1e-3):.4g}")
        return out
    ach = r["bytes"] / r["launches"] / (per_launch_ms * 1e-3) / 1e9
    return {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None,
            "avg_launch_ms": round(per_launch_ms, 4)}


def timed(B, run, n, offset, with_events):
    """Times n calls run(offset + i) on the current stream; returns the
    per-call ms (HIP events between calls), the wall time, and the kernel
    profile when with_events."""
    import torch
    stream = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    if with_events:
        B.dif_profile_reset()
        B.dif_profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(n):
        run(offset + i)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    B.dif_profile_enable(False)
    prof = B.dif_profile_collect() if with_events else {}
    return [evs[i].elapsed_time(evs[i + 1]) for i in range(n)], wall, prof


def run_blocks(args, cfg):
    """One full-length block per step structure (the block workloads)."""
    import numpy as np
    import torch

    from paper_2607_06631_amd import binding as B
    from paper_2607_06631_amd import flops
    from workloads import synth

    L, Lc, D, dh, H, F = cfg.seq_len, cfg.text_len, cfg.dim, cfg.head_dim, cfg.n_heads, cfg.ffn_dim
    w = synth.make_weights_torch(cfg, "cuda", seed=0)
    model = B.dif_model_create(cfg, w)
    n_struct = len(cfg.keep_heads)
    plans = [B.dif_plan_step(model, s, cfg.timesteps[s], synth.make_masks(cfg, s))
             for s in range(n_struct)]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1)
    x0 = (torch.randn((1, L, D), generator=gen, device="cuda") * 0.5).to(torch.bfloat16)
    x = x0.clone()
    ctx = torch.randn((1, Lc, D), generator=gen, device="cuda").to(torch.bfloat16)
    e0 = torch.randn(6 * D, generator=gen, device="cuda") * 0.1
    ws = B.workspace(model, 1, L, Lc)
    peak = PEAK_BF16_TFLOPS
    per = {}
    for s in range(n_struct):
        info = plans[s].layer_info(0)
        kept = flops.block_flops(L, Lc, D, dh, info.self_heads, info.cross_heads, info.ffn_channels)
        execd = sum(flops.block_executed_terms(L, Lc, D, dh, info.self_heads, info.cross_heads,
                                               info.ffn_padded).values())

        def run(i, s=s):
            x.copy_(x0)   # the same input every call (a block is applied in place)
            B.dif_block_forward(plans[s], 0, x, ctx, e0, ws)

        for i in range(args.warmup):
            run(i)
        torch.cuda.synchronize()
        ms, _, prof = timed(B, run, args.steps, 0, not args.no_kernel_timing)
        ms_clean, _, _ = timed(B, run, args.steps, 0, False)
        # the input copy each call makes, timed alone and subtracted
        copy_ms = float(np.median(timed(B, lambda i: x.copy_(x0), args.steps, 0, False)[0]))
        med = float(np.median(ms_clean)) - copy_ms
        per[f"t{s + 1}"] = {
            "heads": info.self_heads, "ffn_channels": info.ffn_channels,
            "ms_per_block": round(med, 3),
            "ms_per_block_with_kernel_events": round(float(np.median(ms)) - copy_ms, 3),
            "input_copy_ms_subtracted": round(copy_ms, 4),
            "kept_tflop": round(kept / 1e12, 3), "executed_tflop": round(execd / 1e12, 3),
            "tflops": round(kept / (med * 1e-3) / 1e12, 1),
            "frac_peak": round(kept / (med * 1e-3) / 1e12 / peak, 4),
            "kernels": kernel_table(prof, args.steps, peak, dh) if prof else None,
        }
        log(f"bench: structure t{s + 1}: {med:.3f} ms per block")
    t1 = per["t1"]
    for k, r in per.items():
        r["t_over_t1"] = round(r["ms_per_block"] / t1["ms_per_block"], 4)
        r["F_over_F1"] = round(r["kept_tflop"] / t1["kept_tflop"], 4)
        r["proportionality_r"] = round(r["t_over_t1"] / r["F_over_F1"], 4)
    mean_ms = float(np.mean([r["ms_per_block"] for r in per.values()]))
    kept_all = sum(r["kept_tflop"] for r in per.values())
    out = {
        "metric": "ms per full-length pruned block + effective TFLOP/s (frac. MFMA peak)",
        "value": round(mean_ms, 3), "unit": "ms", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(mean_ms, 3), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": (f"{cfg.name}: one DiT block, D={D}, {H} heads x {dh}, FFN {F}, "
                                f"{L} video tokens ({'x'.join(map(str, cfg.grid))}), {Lc} text "
                                f"tokens, batch 1, {n_struct} step structure(s)"),
                   "seq_len": L, "text_len": Lc, "dim": D, "heads": H, "ffn": F,
                   "parallelism": "none (1 GPU)"},
        "effective_tflops": round(kept_all / (mean_ms * n_struct * 1e-3), 1),
        "per_structure": per,
    }
    print(json.dumps(out))


def gemm_vs_library(args, cfg):
    """The step's projection GEMMs at full width (M = the video tokens; the
    first step structure keeps every head and FFN channel): this library's
    GEMM with the plain store epilogue against torch.nn.functional.linear
    in bf16, which calls the platform BLAS.  Same operands, alternating
    launches, HIP events; the outputs are compared (both accumulate in
    float32 and round to bf16)."""
    import torch
    import torch.nn.functional as F

    from paper_2607_06631_amd import binding as B

    M, D, Fd = cfg.seq_len, cfg.dim, cfg.ffn_dim
    shapes = [("qkv", 3 * D, D), ("out_proj", D, D), ("ffn1", Fd, D), ("ffn2", D, Fd)]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    reps = max(args.steps, 3)
    out = {}
    tot = {"dif": 0.0, "lib": 0.0, "flop": 0.0}
    for name, N, K in shapes:
        A = torch.randn((M, K), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
        W = (torch.randn((N, K), generator=gen, device="cuda", dtype=torch.float32) * 0.02).to(torch.bfloat16)
        C_dif = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
        runs = {"dif": lambda: B.dif_gemm(A, W, C_dif), "lib": lambda: F.linear(A, W)}
        for _ in range(max(args.warmup, 1)):
            for f in runs.values():
                f()
        times = {k: [] for k in runs}
        for _ in range(reps):
            for k, f in runs.items():
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                f()
                e1.record()
                torch.cuda.synchronize()
                times[k].append(e0.elapsed_time(e1))
        C_lib = F.linear(A, W)
        torch.cuda.synchronize()
        diff = ((C_dif.float() - C_lib.float()).abs().max() / C_lib.float().abs().max()).item()
        flop = 2.0 * M * N * K
        row = {"M": M, "N": N, "K": K, "max_rel_diff": diff}
        for k in runs:
            ms = sorted(times[k])[len(times[k]) // 2]
            row[f"{k}_ms"] = round(ms, 4)
            row[f"{k}_tflops"] = round(flop / ms / 1e9, 1)
            tot[k] += ms
        row["dif_over_lib"] = round(row["lib_ms"] / row["dif_ms"], 3)
        tot["flop"] += flop
        out[name] = row
        log(f"bench: {name} {row}")
        del A, W, C_dif, C_lib
    print(json.dumps({
        "metric": "projection GEMM TFLOP/s, this library against the platform BLAS",
        "library": f"torch.nn.functional.linear (bf16, blas backend "
                   f"{torch.backends.cuda.preferred_blas_library()})",
        "shapes": out,
        "dif_tflops": round(tot["flop"] / tot["dif"] / 1e9, 1),
        "lib_tflops": round(tot["flop"] / tot["lib"] / 1e9, 1),
        "dif_over_lib": round(tot["lib"] / tot["dif"], 3),
        "reps": reps, "data": "synthetic"}))


def mfma_ceiling(args):
    """The sustained rate of each bf16 MFMA shape the kernels use, with every
    CU busy and nothing else running (the chip's power limit sets the clock,
    and the shape changes it): the ceilings against which the kernels'
    fractions of the 2.5 PFLOP/s nominal peak are read."""
    import torch

    from paper_2607_06631_amd import binding as B

    sink = torch.zeros(1, device="cuda", dtype=torch.float32)
    iters = 300000   # about 0.1 s per launch
    out = {}
    for shape, name in ((B.MFMA_32X32X16, "32x32x16"), (B.MFMA_16X16X32, "16x16x32"),
                        (B.PROBE_EXP_F32, "exp_f32")):
        for _ in range(max(args.warmup, 1)):
            B.dif_mfma_probe(iters, sink, shape)
        torch.cuda.synchronize()
        rates = []
        for _ in range(max(args.steps, 3)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fl = B.dif_mfma_probe(iters, sink, shape)
            e1.record()
            torch.cuda.synchronize()
            rates.append(fl / e0.elapsed_time(e1) / 1e9)
        rates.sort()
        med = rates[len(rates) // 2]
        if shape == B.PROBE_EXP_F32:
            # rates are then 10^12 exponentials per second
            out[name] = {"exps_per_s_median": med * 1e12, "exps_per_s_min": rates[0] * 1e12,
                         "exps_per_s_max": rates[-1] * 1e12, "launches": len(rates),
                         "exps_per_launch": fl}
            continue
        out[name] = {"tflops_median": round(med, 1), "tflops_min": round(rates[0], 1),
                     "tflops_max": round(rates[-1], 1),
                     "frac_nominal_peak": round(med / PEAK_BF16_TFLOPS, 4),
                     "launches": len(rates), "flop_per_launch": fl}
    print(json.dumps({"metric": "sustained bf16 MFMA rate per instruction shape and v_exp_f32 "
                                "rate (all CUs, no memory traffic)", "shapes": out}))


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "bench.py measures one GPU: the library has no multi-GPU path "
                                   "(a step would shard over GPUs by sequence, with the kept "
                                   "heads' keys and values all-gathered per layer)",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_06631_amd import binding as B
    from paper_2607_06631_amd import flops
    from workloads import get_config, synth

    cfg = get_config(args.workload)
    torch.cuda.set_device(0)
    if args.gemm_vs_library:
        gemm_vs_library(args, cfg)
        return
    if args.mfma_ceiling:
        mfma_ceiling(args)
        return
    if cfg.name in ("wan14b_block", "wan1.3b_block"):
        run_blocks(args, cfg)
        return
    dev = "cuda"
    L, Lc, D, dh, H, F, N = (cfg.seq_len, cfg.text_len, cfg.dim, cfg.head_dim, cfg.n_heads,
                             cfg.ffn_dim, cfg.n_layers)
    t_setup = time.perf_counter()
    if cfg.dtype == "bf16":
        w = synth.make_weights_torch(cfg, dev, seed=0)
    else:
        w = B.upload_weights(synth.make_weights(cfg, seed=0), cfg.dtype)
    log(f"bench: weights ready ({time.perf_counter() - t_setup:.1f} s)")
    model = B.dif_model_create(cfg, w)
    masks = [synth.make_masks(cfg, s) for s in range(4)]
    plans = [B.dif_plan_step(model, s, cfg.timesteps[s], masks[s], kind=args.plan)
             for s in range(4)]
    plan_bytes = sum(p.mem.numel() for p in plans)
    gen = torch.Generator(device=dev)
    gen.manual_seed(1)
    z = torch.randn((1, L, cfg.patch_dim), generator=gen, device=dev, dtype=torch.float32)
    mdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    ctx = torch.randn((1, Lc, D), generator=gen, device=dev, dtype=torch.float32).to(mdt)
    v = torch.empty_like(z)
    ws = B.workspace(model, 1, L, Lc)
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup
    log(f"bench: plans ready ({setup_s:.1f} s)")

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 19   # bf16 elements
        src = torch.ones(n, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"bench: copy calibration {args.copy_calibration_mib} MiB read + write")
        del src, dst

    sig = [t / 1000.0 for t in cfg.timesteps] + [0.0]
    step_flops, step_exec, counts = [], [], []
    for s in range(4):
        h, hc, f, bk = kept_counts(plans[s], N)
        fp = [plans[s].layer_info(l).ffn_padded for l in range(N)]
        counts.append((h, hc, f))
        step_flops.append(flops.structure_flops(L, Lc, D, dh, h, hc, f, bk))
        step_exec.append(sum(sum(flops.block_executed_terms(L, Lc, D, dh, h[l], hc[l], fp[l]).values())
                             for l in range(N) if bk[l]))
    dense_flops = flops.structure_flops(L, Lc, D, dh, [H] * N, [H] * N, [F] * N)

    cache, cache_build_ms = None, None
    if args.text_cache:
        for s in range(4):   # the projection moves out of the step
            h, hc, f = counts[s]
            bk = kept_counts(plans[s], N)[3]
            step_flops[s] -= sum(4.0 * Lc * D * hc[l] * dh for l in range(N) if bk[l])
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        B.dif_text_cache_build(model, ctx)   # first build warms the GEMM code
        torch.cuda.synchronize()
        ev0.record()
        cache = B.dif_text_cache_build(model, ctx)
        ev1.record()
        torch.cuda.synchronize()
        cache_build_ms = ev0.elapsed_time(ev1)
        log(f"bench: text cache built ({cache_build_ms:.2f} ms, {cache.mem.numel() / 1e6:.0f} MB)")

    def one_step(i):
        s = i % 4
        if cache is None:
            B.dif_step_forward(plans[s], z, cfg.timesteps[s], ctx, v, ws)
        else:
            B.dif_step_forward_cached(plans[s], z, cfg.timesteps[s], cache, v, ws)
        B.dif_euler(z, v, sig[s], sig[s + 1])

    for i in range(args.warmup):
        one_step(i)
        torch.cuda.synchronize()
        log(f"bench: warmup step {i} done")

    # pass 1: HIP events around every kernel (kernel table, roofline) -> value
    step_ms, wall, prof = timed(B, one_step, args.steps, args.warmup,
                                not args.no_kernel_timing)
    log(f"bench: timed {args.steps} steps in {wall:.2f} s"
        f"{'' if args.no_kernel_timing else ' (with kernel events)'}")
    assert torch.isfinite(z).all().item(), "non-finite latents"
    # pass 2: the same steps without kernel events
    clean_ms, clean_wall, _ = ([], None, None) if args.no_kernel_timing else \
        timed(B, one_step, args.steps, args.warmup, False)
    if clean_ms:
        log(f"bench: timed {args.steps} steps in {clean_wall:.2f} s (no kernel events)")

    total_ms = sum(step_ms)
    ms_per_step = total_ms / args.steps
    kept_total = sum(step_flops[(args.warmup + i) % 4] for i in range(args.steps))
    exec_total = sum(step_exec[(args.warmup + i) % 4] for i in range(args.steps))
    tflops = kept_total / (total_ms * 1e-3) / 1e12
    per_struct = {}
    for i, ms in enumerate(step_ms):
        per_struct.setdefault((args.warmup + i) % 4, []).append(ms)
    per_struct_ms = {s: float(np.median(v_)) for s, v_ in sorted(per_struct.items())}
    prop = {}
    if 0 in per_struct_ms:
        for s, ms in per_struct_ms.items():
            prop[f"t{s + 1}"] = round((ms / per_struct_ms[0]) / (step_flops[s] / step_flops[0]), 4)

    peak = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_TFLOPS
    kernels = kernel_table(prof, args.steps, peak, dh)
    gemm_keys = [k for k in prof if k.startswith("gemm_")]
    gemm_ms = sum(prof[k]["ms"] for k in gemm_keys)
    gemm_fl = sum(prof[k]["flops"] for k in gemm_keys)
    roofline = roofline_of(prof, args.workload, peak, dh)

    out = {
        "metric": "ms per pruned denoise step + effective TFLOP/s (frac. MFMA peak), 14B 480p",
        "value": round(ms_per_step, 3),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": (f"{cfg.name}: {N}-layer DiT, D={D}, {H} heads x {dh}, FFN {F}, "
                                f"{L} video tokens ({'x'.join(map(str, cfg.grid))}), {Lc} text "
                                f"tokens, batch 1, 4 step structures"),
                   "layers": N, "seq_len": L, "text_len": Lc, "dim": D, "heads": H,
                   "ffn": F, "parallelism": "none (1 GPU)", "plan": args.plan,
                   "text_cache": bool(args.text_cache)},
        "ms_per_step_no_kernel_timing": round(sum(clean_ms) / len(clean_ms), 3) if clean_ms else None,
        "plan_gb_4_structures": round(plan_bytes / 1e9, 3),
        "text_cache_build_ms": None if cache_build_ms is None else round(cache_build_ms, 3),
        "effective_tflops": round(tflops, 1),
        "frac_mfma_peak": round(tflops / peak, 4),
        "executed_tflops": round(exec_total / (total_ms * 1e-3) / 1e12, 1),
        "kept_tflop_per_step": [round(f / 1e12, 2) for f in step_flops],
        "executed_tflop_per_step": [round(f / 1e12, 2) for f in step_exec],
        "flop_fraction_per_step": [round(f / dense_flops, 4) for f in step_flops],
        "ms_per_structure": {f"t{s + 1}": round(ms, 2) for s, ms in per_struct_ms.items()},
        "proportionality_r": prop,
        "gemm_tflops": round(gemm_fl / (gemm_ms * 1e-3) / 1e12, 1) if gemm_ms else None,
        "gemm_frac_peak": round(gemm_fl / (gemm_ms * 1e-3) / 1e12 / peak, 4) if gemm_ms else None,
        "kernels": kernels,
        "roofline": roofline,
        "wall_s_timed": round(wall, 3),
        "setup_s": round(setup_s, 1),
        "paper_context": ("paper: Wan-14B 4-step pruned denoise 40.72 s/video (10.18 s/step), 1.20x "
                          "over the dense 4-step distill, 30.01x over the 50-step teacher, on one "
                          "Kunlun P800 XPU in BF16 (different hardware; context, not the target)"),
    }
    if not args.no_cpu_baseline and args.workload != "tiny":
        log("bench: cpu oracle sample")
        out["cpu_baseline"] = cpu_baseline(cfg, w, masks)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
