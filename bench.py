"""Benchmark: pruned denoise steps of a Wan-14B-shaped 40-layer DiT at 480p.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A "step" is one denoise step of the 4-step sampler: timestep embedding,
patch embedding, 40 blocks under that step's structure, output head and the
Euler update; consecutive steps cycle through the four step structures
(t = 999, 750, 500, 250).  Weights (about 28 GB, random init), latents and
text context are synthetic and already resident in HBM when timing starts;
the four per-step compacted weight sets are built beforehand (plan time is
not step time).  Prints one JSON line.
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
    "sha256": "5ff35620f3e58b3ef6a133ca24869fe563c1761883c91083d417195d0e4a6dc7",
    "fetch_bytes": 1122453.0 * 1024 / 0.500,
    "write_bytes": 429584.5 * 1024 / 1.000,
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=8)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--workload", default="wan14b_480p",
                    choices=["wan14b_480p", "wan14b_720p", "tiny"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true",
                    help="time the steps without per-kernel events")
    ap.add_argument("--cpu-tokens", type=int, default=0,
                    help="token count of the CPU oracle sample (0: auto)")
    ap.add_argument("--plan", default="compact", choices=["compact", "indexed"],
                    help="compact: per-step gathered weights; indexed: union weights read "
                         "in place through the index tables")
    ap.add_argument("--text-cache", action="store_true",
                    help="project every layer's text keys and values once per video "
                         "(timed apart, reported as text_cache_build_ms) and run the cached "
                         "step; the step's FLOP count then leaves out that projection")
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


def cpu_baseline(cfg, w_dev, masks, step_flops_dense, tokens):
    """Time the oracle (float32 numpy, masked-dense) on one block over the
    first frames of the video and extrapolate by its measured FLOP rate."""
    import numpy as np

    import oracle as O
    from paper_2607_06631_amd import flops
    from workloads import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = int(os.environ.get("OMP_NUM_THREADS", "1"))
    gf, gh, gw = cfg.grid
    frames = max(1, min(gf, tokens // (gh * gw))) if tokens else 2
    grid = (frames, gh, gw)
    L = frames * gh * gw
    wl = {k: v.float().cpu().numpy() for k, v in w_dev["layers"][0].items()}
    g = synth.rng(synth.SEED_INPUTS, 0, "cpu_sample")
    x = g.standard_normal((L, cfg.dim), dtype=np.float32)
    ctx = synth.bf16_round(g.standard_normal((cfg.text_len, cfg.dim), dtype=np.float32))
    e0 = (g.standard_normal((6, cfg.dim), dtype=np.float32) * 0.1)
    m = masks[0]
    t0 = time.perf_counter()
    wz = O.apply_keep(wl, m["self_head_keep"][0], m["cross_head_keep"][0], m["ffn_keep"][0],
                      cfg.head_dim, np.float32)
    O.block(x, ctx, e0, wz, True, cfg.n_heads, cfg.head_dim, grid, cfg.rope_theta, cfg.eps,
            dtype=np.float32)
    dt = time.perf_counter() - t0
    H, F = cfg.n_heads, cfg.ffn_dim
    sample_flops = flops.block_flops(L, cfg.text_len, cfg.dim, cfg.head_dim, H, H, F)
    rate = sample_flops / dt
    return {
        "value": step_flops_dense / rate * 1e3, "unit": "ms per denoise step (extrapolated)",
        "cores": threads, "kind": "oracle",
        "sample": (f"one masked-dense block (float32 numpy) of the same model over the first "
                   f"{frames} latent frames ({L} tokens, {cfg.text_len} text tokens) took "
                   f"{dt:.2f} s = {rate / 1e12:.3f} TFLOP/s; a 40-layer {cfg.seq_len}-token step "
                   f"is {step_flops_dense / 1e12:.0f} TFLOP masked-dense"),
    }


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
    plans = [B.dif_plan_step(model, s, cfg.timesteps[s], masks[s], kind=args.plan) for s in range(4)]
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
    step_flops, counts = [], []
    for s in range(4):
        h, hc, f, bk = kept_counts(plans[s], N)
        counts.append((h, hc, f))
        step_flops.append(flops.structure_flops(L, Lc, D, dh, h, hc, f, bk))
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

    stream = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    if not args.no_kernel_timing:
        B.dif_profile_reset()
        B.dif_profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        one_step(args.warmup + i)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    B.dif_profile_enable(False)
    prof = {} if args.no_kernel_timing else B.dif_profile_collect()
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    log(f"bench: timed {args.steps} steps in {wall:.2f} s")
    assert torch.isfinite(z).all().item(), "non-finite latents"

    total_ms = sum(step_ms)
    ms_per_step = total_ms / args.steps
    kept_total = sum(step_flops[(args.warmup + i) % 4] for i in range(args.steps))
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
    kernels = {}
    for k, r in prof.items():
        ent = {"launches": r["launches"], "ms_per_step": round(r["ms"] / args.steps, 3)}
        if r["flops"] > 0:
            ent["tflops"] = round(r["flops"] / (r["ms"] * 1e-3) / 1e12, 1)
            ent["frac_peak"] = round(ent["tflops"] / peak, 4)
        if r["bytes"] > 0:
            ent["gbs"] = round(r["bytes"] / (r["ms"] * 1e-3) / 1e9, 1)
        kernels[k] = ent
    gemm_keys = [k for k in prof if k.startswith("gemm_")]
    gemm_ms = sum(prof[k]["ms"] for k in gemm_keys)
    gemm_fl = sum(prof[k]["flops"] for k in gemm_keys)
    roofline = None
    if prof:
        dom = max(prof, key=lambda k: prof[k]["ms"])
        r = prof[dom]
        per_launch_ms = r["ms"] / r["launches"]
        if r["flops"] > 0:
            ach = r["flops"] / r["launches"] / (per_launch_ms * 1e-3) / 1e12
            roofline = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 1), "peak": peak,
                        "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                        "traffic": measured_traffic(dom, args.workload), "traffic_unit": "HBM bytes per launch",
                        "avg_launch_ms": round(per_launch_ms, 4)}
        else:
            ach = r["bytes"] / r["launches"] / (per_launch_ms * 1e-3) / 1e9
            roofline = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                        "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None,
                        "avg_launch_ms": round(per_launch_ms, 4)}

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
        "plan_gb_4_structures": round(plan_bytes / 1e9, 3),
        "text_cache_build_ms": None if cache_build_ms is None else round(cache_build_ms, 3),
        "effective_tflops": round(tflops, 1),
        "frac_mfma_peak": round(tflops / peak, 4),
        "kept_tflop_per_step": [round(f / 1e12, 2) for f in step_flops],
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
        dense_step = float(dense_flops)
        out["cpu_baseline"] = cpu_baseline(cfg, w, masks, dense_step, args.cpu_tokens or 3 * 30 * 52)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
