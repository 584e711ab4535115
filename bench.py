"""Throughput of the selective partial-denoising step on one MI355X.

A step is one pass of the whole hot path over one batch: select + compact the
mask, gather with noise injection, the denoiser on the gathered tokens with the
DDIM update, and scatter back (all through the C ABI of libsphinx.so).  The
default workload is the headline configuration: 14 frames of a 4x72x128 bf16
latent (576x1024 views), 32256 tokens, Gaussian-blob uncertainty, 30 %
selected (9677 tokens), a 12-block D=1024 denoiser with 16 heads of 64 and an
MLP of 4096, 25 DDIM steps from t_start 0.5; step k runs schedule step
k mod 25.  Inputs are seeded synthetic latents and random-init weights.

Prints one JSON line: refined tokens*steps/s over the timed steps, the roofline
of the dominant kernel (attention) from HIP events recorded on its stream over
the timed region, per-kernel-class times, and the CPU oracle timed on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
METRIC = "refined tokens·steps/s + MFMA util, 14-frame 576×1024 latent, 30% selected"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=25)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="headline", choices=["headline", "small", "frame_region", "batched"])
    ap.add_argument("--rho", type=float, default=None, help="selected fraction (headline only)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--mode", default="step", choices=["step", "copy", "sweep", "peaks", "rho", "frontend"],
                    help="step: the hot path; copy: a plain 1 GiB fp32 copy through scatter_blend (no tokens), "
                         "used to calibrate HBM byte counters and to measure achievable bandwidth; sweep: "
                         "mask/compaction, gather and scatter at 2^20..2^26 tokens against the HBM roofline; "
                         "peaks: achievable dense bf16 MFMA rate and copy bandwidth; rho: step time of the "
                         "headline workload over the selected fraction; frontend: the mask front-end on the "
                         "headline views (14 x 576 x 1024) against the HBM roofline")
    ap.add_argument("--rhos", default="0.05,0.1,0.2,0.3,0.5,0.75,1.0", help="selected fractions of --mode rho")
    ap.add_argument("--layout", default="tokens", choices=["tokens", "nchw"],
                    help="layout of the fp32 state of record and the noise")
    ap.add_argument("--sweep-log2", default="20,22,24,26", help="token counts of the sweep (log2)")
    ap.add_argument("--attention", default="joint", choices=["joint", "factorised"],
                    help="denoiser attention: joint over the request, or spatial/temporal in alternating blocks")
    ap.add_argument("--per-frame-grid", action="store_true",
                    help="every frame on its own timestep grid from its own start (other reading of per-frame starts)")
    ap.add_argument("--cache-period", type=int, default=0,
                    help="latent cache with a full step every T steps (0: off, the default workload)")
    ap.add_argument("--select-every-step", type=int, default=1,
                    help="1: run mask+compaction in every step (default); 0: only when the active set changes")
    return ap.parse_args()


def traffic_entry(kernel: str, workload: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel source (else None)."""
    import hashlib

    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("|") and line.count("|") >= 3:
            parts = [p.strip() for p in line.strip().strip("|").split("|")]
            if len(parts) >= 2:
                fields[parts[0]] = parts[1]
    src = os.path.join(ROOT, "paper_2511_18672_amd", "csrc", fields.get("source", "attention.hip"))
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16] if os.path.exists(src) else None
    if fields.get("source_sha256_16") != digest:
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _oracle_e2e(O, wl, threads=None, min_s=1.0):
    """Refined tokens·steps/s of the unmodified oracle's whole loop on wl,
    repeated until at least min_s seconds have passed (tiny runs in ms)."""
    from threadpoolctl import threadpool_limits

    reps, n, t0 = 0, 0, time.perf_counter()
    while True:
        with threadpool_limits(limits=threads):
            _, trace = O.refine(wl, precision="model", trace=True)
        n += sum(r.n_sel for r in trace)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_s:
            return {"value": round(n / dt, 2), "runs": reps, "seconds": round(dt, 2),
                    "threads": "all" if threads is None else threads}


def cpu_baseline(wl) -> dict:
    """The oracle (numpy fp64, unmodified) on the host.  value: a bounded sample
    of the headline workload, one step through a one-block denoiser scaled to
    the full depth.  Also measured: the whole loop of the tiny and small
    workloads end to end, on all threads and on one."""
    import oracle as O
    import workloads as W

    try:
        from threadpoolctl import threadpool_info

        blas = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:
        blas = 1
    nproc = os.cpu_count() or 1
    try:
        affinity = len(os.sched_getaffinity(0))
    except Exception:
        affinity = nproc
    m = wl.model
    one = W.ModelCfg(D=m.D, heads=m.heads, head_dim=m.head_dim, mlp=m.mlp, L=1, dtype=m.dtype)
    sample = W.Workload(name=wl.name, model=one, requests=wl.requests, u=wl.u, thr=wl.thr, s_start=wl.s_start,
                        nsteps=wl.nsteps, z0=wl.z0, eps=wl.eps,
                        weights={k: v for k, v in wl.weights.items() if not k.startswith("b") or k.startswith("b0.")})
    plans = O.plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps)
    model = O.model_from_workload(sample)
    t0 = time.perf_counter()
    res = O.step(sample, model, wl.z0, plans[0], "model")
    dt = time.perf_counter() - t0
    per_step = dt * m.L  # blocks dominate; embedding and final projection counted L times (conservative)
    out = {"value": res.n_sel / per_step, "unit": "refined tokens·steps/s", "cores": int(blas),
           "kind": "oracle",
           "sample": f"one headline step ({res.n_sel} selected tokens) through a 1-block copy of the denoiser, "
                     f"{dt:.1f} s, scaled x{m.L} blocks (BLAS threads {blas}; elementwise numpy is one thread)",
           "nproc": int(nproc), "affinity_cpus": int(affinity), "blas_threads": int(blas)}
    runs = {}
    for name, ctor in (("tiny", W.tiny), ("small", W.small)):
        w = ctor()
        runs[name] = {"all_threads": _oracle_e2e(O, w), "one_thread": _oracle_e2e(O, w, threads=1)}
    out["end_to_end"] = runs
    out["end_to_end_unit"] = "refined tokens·steps/s over the whole loop (tiny: 1 step, small: 10 steps)"
    return out


def copy_mode(args):
    """Plain device copy of 2^28 fp32 values (1 GiB read + 1 GiB written) through
    scatter_blend with no selected tokens, which is one grid-stride copy kernel."""
    import torch

    import paper_2511_18672_amd as S
    import workloads as W

    reqs = S.make_requests([W.Request(256, 512, 512)])
    n = 16 * 256 * 256 * 256
    src = torch.randn(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        S.sphinx_scatter_blend(reqs, None, None, 0, src, S.F32, S.NCHW, dst, S.F32, S.NCHW)
    torch.cuda.synchronize()
    S.sphinx_timing_enable(True)
    for _ in range(args.steps):
        S.sphinx_scatter_blend(reqs, None, None, 0, src, S.F32, S.NCHW, dst, S.F32, S.NCHW)
    torch.cuda.synchronize()
    cnt, ms = S.sphinx_timing_read()["scatter"]
    S.sphinx_timing_enable(False)
    assert torch.equal(src, dst)
    nbytes = 2 * 4 * n
    avg_s = ms / cnt / 1e3
    print(json.dumps({"mode": "copy", "bytes_per_launch": nbytes, "launches": cnt, "avg_us": round(avg_s * 1e6, 2),
                      "GB/s": round(nbytes / avg_s / 1e9, 1), "frac_of_8TBs": round(nbytes / avg_s / 8e12, 4)}),
          flush=True)


def peaks_mode(args):
    """Achievable rates to read the roofline fractions against: a bf16 MFMA loop
    (four independent 32x32x16 chains per wave, 2048 workgroups of 4 waves) on
    constant and on random operands (the sustained rate depends on the data),
    and the 1 GiB fp32 copy."""
    import torch

    import paper_2511_18672_amd as S

    out = torch.empty(S.PEAK_BLOCKS, dtype=torch.float32, device="cuda")
    iters = 4096
    flop = float(S.PEAK_BLOCKS) * 4 * iters * 4 * 32768
    stream = torch.cuda.current_stream()
    rec = {"mode": "peaks", "flop_per_launch": flop}
    for name, kind in (("constant", S.PEAK_CONSTANT), ("random", S.PEAK_RANDOM)):
        for _ in range(3):
            S.sphinx_peak_mfma(iters, out, kind)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            S.sphinx_peak_mfma(iters, out, kind)
        e1.record(stream)
        torch.cuda.synchronize()
        avg_s = e0.elapsed_time(e1) / args.steps / 1e3
        tf = flop / avg_s / 1e12
        assert bool(torch.isfinite(out).all())
        rec[f"mfma_bf16_tflops_{name}"] = round(tf, 1)
        rec[f"frac_of_2500_{name}"] = round(tf / PEAK_BF16_TFLOPS, 4)
        rec[f"avg_us_{name}"] = round(avg_s * 1e6, 1)
    print(json.dumps(rec), flush=True)
    copy_mode(args)


def rho_mode(args):
    """Step time of the headline workload as the selected fraction grows; the
    same uncertainty map with its threshold moved (select runs every step)."""
    import torch

    import paper_2511_18672_amd as S
    import workloads as W

    base = None
    for rho in [float(x) for x in args.rhos.split(",")]:
        wl = W.headline(rho=rho)
        R = S.from_workload(wl, layout=S.TOKENS if args.layout == "tokens" else S.NCHW)
        R.reset()
        for i in range(args.warmup):
            R.step(i, force_select=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        refined = 0
        for i in range(args.warmup, args.warmup + args.steps):
            refined += R.step(i, force_select=True)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = 1e3 * wall / args.steps
        if base is None:
            base = (rho, ms)
        print(json.dumps({"mode": "rho", "rho": rho, "selected_tokens": int(R.n_sel), "tokens": int(wl.N),
                          "ms_per_step": round(ms, 4), "refined_tokens_steps_per_s": round(refined / wall, 1),
                          "ms_per_selected_ktoken": round(ms / (R.n_sel / 1e3), 4)}), flush=True)
        del R, wl
        torch.cuda.empty_cache()


def frontend_mode(args):
    """The mask front-end (luma, Laplacian variance, smoothing, per-frame Otsu,
    opacity, 16x16 pooling) over the 14 headline views of 576 x 1024.
    Algorithmic bytes: 3 (RGB) + 4 (opacity) per pixel read, 1 + 4 per token
    written (mask and uncertainty)."""
    import torch

    import paper_2511_18672_amd as S
    import workloads as W

    reqs_py = [W.Request(14, 72, 128)]
    rgb, opac = W.frontend_inputs(reqs_py)
    reqs = S.make_requests(reqs_py)
    N, G = reqs_py[0].tokens, reqs_py[0].frames
    d_rgb = torch.from_numpy(rgb[0].ravel()).cuda()
    d_op = torch.from_numpy(opac[0].ravel()).cuda()
    mask = torch.empty(N, dtype=torch.uint8, device="cuda")
    u = torch.empty(N, dtype=torch.float32, device="cuda")
    thr = torch.empty(G, dtype=torch.int32, device="cuda")
    ws = torch.empty(S.sphinx_mask_frontend_workspace_bytes(reqs), dtype=torch.uint8, device="cuda")
    for _ in range(max(args.warmup, 1)):
        S.sphinx_mask_frontend(reqs, d_rgb, d_op, 0.5, mask, u, thr, ws)
    torch.cuda.synchronize()
    S.sphinx_timing_enable(True, classes=["frontend"])
    for _ in range(args.steps):
        S.sphinx_mask_frontend(reqs, d_rgb, d_op, 0.5, mask, u, thr, ws)
    torch.cuda.synchronize()
    cnt, ms = S.sphinx_timing_read()["frontend"]
    S.sphinx_timing_enable(False)
    pixels = 256 * N
    nbytes = 7 * pixels + 5 * N
    avg_s = ms / cnt / 1e3
    print(json.dumps({"mode": "frontend", "frames": G, "image": "576x1024", "pixels": pixels, "tokens": N,
                      "masked_tokens": int(mask.sum().item()), "avg_us": round(avg_s * 1e6, 2),
                      "Mpix_per_s": round(pixels / avg_s / 1e6, 1), "algorithmic_bytes": nbytes,
                      "GB/s": round(nbytes / avg_s / 1e9, 1), "frac_of_8TBs": round(nbytes / avg_s / 8e12, 4)}),
          flush=True)


def sweep_mode(args):
    """HBM roofline of the memory-bound kernels at large token counts.

    One request of F frames of a 4x512x512 latent (2^16 tokens per frame),
    30 % selected, with two selection recipes: uniform random (worst case for
    the gathers: selected tokens are isolated) and Gaussian blobs at the
    headline map's density (clustered), for NCHW and token-major latents.
    Algorithmic bytes per launch:
      select  : 4 N (u) + N (mask) + 4 n_sel (idx)
      gather  : n_sel (4 idx + 64 state + 64 x_sel) [+ 32 n_sel bf16 noise when injecting]
      scatter : n_sel (4 idx + 64 x_sel + 64 state)
    """
    import torch

    import paper_2511_18672_amd as S
    import workloads as W

    torch.manual_seed(5)
    for lg in [int(x) for x in args.sweep_log2.split(",")]:
        N = 1 << lg
        F = N >> 16
        reqs = S.make_requests([W.Request(F, 512, 512)])
        state = torch.randn(16 * N, dtype=torch.float32, device="cuda")
        eps = torch.randn(16 * N, dtype=torch.bfloat16, device="cuda")
        mask = torch.empty(N, dtype=torch.uint8, device="cuda")
        idx = torch.empty(N, dtype=torch.int32, device="cuda")
        cu = torch.empty(2, dtype=torch.int32, device="cuda")
        ws = torch.empty(S.sphinx_select_workspace_bytes(N), dtype=torch.uint8, device="cuda")
        ones = torch.ones(F, dtype=torch.float32, device="cuda")
        zeros = torch.zeros(F, dtype=torch.float32, device="cuda")
        bvals = torch.full((F,), 0.5, dtype=torch.float32, device="cuda")
        for recipe in ("uniform", "blobs"):
            if recipe == "uniform":
                u = torch.rand(N, device="cuda")
            else:
                # the headline recipe (20 blobs of sigma 8 per 72x128 latent) at the
                # same density: 20 * (512*512)/(72*128) = 569 centres per frame
                yy = (2 * torch.arange(256, device="cuda", dtype=torch.float32) + 0.5)
                u = torch.zeros(F, 256, 256, device="cuda")
                for f in range(F):
                    c = torch.rand(569, 2, device="cuda") * 512
                    for c0 in range(0, 569, 64):
                        cc = c[c0:c0 + 64]
                        d2 = (yy[None, :, None] - cc[:, 0, None, None]) ** 2 + (yy[None, None, :] - cc[:, 1, None, None]) ** 2
                        u[f] += torch.exp(-d2 / 128.0).sum(0)
                u = (u + 0.1 * torch.rand_like(u)).reshape(-1)
            thr = torch.full((F,), float(torch.quantile(u[:1 << 24].float(), 0.7)), device="cuda")
            cu_host = S.sphinx_select_mask(reqs, u, thr, None, mask, idx, cu, ws)
            n = int(cu_host[-1])
            x = torch.empty(16 * n, dtype=torch.float32, device="cuda")
            reps = max(3, args.steps)

            def rate(tm, key, nbytes):
                cnt, ms = tm[key]
                us = 1e3 * ms / cnt
                gbs = nbytes / (us * 1e-6) / 1e9
                return {"avg_us": round(us, 2), "GB/s": round(gbs, 1), "frac_of_8TBs": round(gbs / PEAK_HBM_GBS, 4),
                        "bytes": nbytes}

            # one untimed call of every operation first (first-launch costs stay out of the rates)
            S.sphinx_select_mask(reqs, u, thr, None, mask, idx, cu, ws, readback=False)
            for lay in (S.NCHW, S.TOKENS):
                S.sphinx_gather(reqs, lay, state, S.F32, eps, S.BF16, idx, n, ones, bvals, x)
                S.sphinx_scatter_blend(reqs, x, idx, n, state, S.F32, lay, state, S.F32, lay)
            torch.cuda.synchronize()
            S.sphinx_timing_enable(True)
            for _ in range(reps):
                S.sphinx_select_mask(reqs, u, thr, None, mask, idx, cu, ws, readback=False)
            torch.cuda.synchronize()
            out = {"mode": "sweep", "N": N, "recipe": recipe, "selected": n,
                   "select": rate(S.sphinx_timing_read(), "select", 5 * N + 4 * n)}
            for lay_name, lay in (("nchw", S.NCHW), ("tokens", S.TOKENS)):
                S.sphinx_timing_enable(True)
                for _ in range(reps):
                    S.sphinx_gather(reqs, lay, state, S.F32, eps, S.BF16, idx, n, ones, zeros, x)
                torch.cuda.synchronize()
                t1 = S.sphinx_timing_read()
                S.sphinx_timing_enable(True)
                for _ in range(reps):
                    S.sphinx_gather(reqs, lay, state, S.F32, eps, S.BF16, idx, n, ones, bvals, x)
                torch.cuda.synchronize()
                t2 = S.sphinx_timing_read()
                S.sphinx_timing_enable(True)
                for _ in range(reps):
                    S.sphinx_scatter_blend(reqs, x, idx, n, state, S.F32, lay, state, S.F32, lay)
                torch.cuda.synchronize()
                t3 = S.sphinx_timing_read()
                out[lay_name] = {"gather": rate(t1, "gather", 132 * n), "gather_inject": rate(t2, "gather", 164 * n),
                                 "scatter": rate(t3, "scatter", 132 * n)}
            S.sphinx_timing_enable(False)
            print(json.dumps(out), flush=True)
            del x
        del state, eps, mask, idx, ws
        torch.cuda.empty_cache()


def main():
    args = parse()
    if args.mode == "sweep" and args.gpus == 1:
        return sweep_mode(args)
    if args.mode == "copy" and args.gpus == 1:
        return copy_mode(args)
    if args.mode == "peaks" and args.gpus == 1:
        return peaks_mode(args)
    if args.mode == "rho" and args.gpus == 1:
        return rho_mode(args)
    if args.mode == "frontend" and args.gpus == 1:
        return frontend_mode(args)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: --gpus {args.gpus} is not supported "
              f"(the selective-refinement step is built and measured on a single MI355X)", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2511_18672_amd as S
    import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    import dataclasses

    kw = {}
    if args.attention != "joint":
        base = W.XL_MODEL if args.config == "frame_region" else W.HEADLINE_MODEL
        kw["model"] = dataclasses.replace(base, attention=args.attention)
    if args.config == "headline":
        wl = W.headline(rho=args.rho, **kw) if args.rho is not None else W.headline(**kw)
    else:
        wl = W.CONFIGS[args.config](**kw)
    t_setup = time.perf_counter()
    R = S.from_workload(wl, layout=S.TOKENS if args.layout == "tokens" else S.NCHW,
                        cache_period=args.cache_period, per_frame_grid=args.per_frame_grid)
    R.reset()
    stream = torch.cuda.current_stream()
    D, L, mlp, hd = wl.model.D, wl.model.L, wl.model.mlp, wl.model.head_dim
    req_tokens = np.diff(np.asarray(wl.tok_offset)).astype(np.float64)
    force = bool(args.select_every_step)
    for i in range(args.warmup):
        R.step(i, force_select=force)
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup

    # timed region: only the dominant kernel (attention) is bracketed by events
    S.sphinx_timing_enable(True, classes=["attention"])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    refined = 0

    def joint_flop():  # one block's joint attention FLOPs of the step just run: 4 D sum_r n_r^2
        seg = np.diff(np.asarray(R.cu_host)).astype(np.float64)
        return 4.0 * D * float((seg ** 2).sum())

    # Attention FLOPs and selected tokens summed over the timed steps (the
    # selection can change from step to step, e.g. as frames reach their
    # start times); host-side values only, no extra synchronisation.
    attn_flop_timed = 0.0  # latent cache: queries x all keys of the request
    n_timed = 0.0
    for i in range(args.warmup, args.warmup + args.steps):
        refined += R.step(i, force_select=force)
        n_timed += R.n_sel
        if args.cache_period > 0:
            attn_flop_timed += 4.0 * D * float((np.diff(R.cu_fwd).astype(np.float64) * req_tokens).sum())
        else:
            attn_flop_timed += joint_flop()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    attn_timing = S.sphinx_timing_read()["attention"]
    # per-class breakdown from a few further, untimed steps with every class bracketed
    S.sphinx_timing_enable(True)
    n_breakdown = min(args.steps, 5)
    attn_flop_bd, n_bd = 0.0, 0.0
    for i in range(args.warmup + args.steps, args.warmup + args.steps + n_breakdown):
        R.step(i, force_select=force)
        attn_flop_bd += joint_flop()
        n_bd += R.n_sel
    torch.cuda.synchronize()
    timing = S.sphinx_timing_read()
    S.sphinx_timing_enable(False)

    ms_per_step = 1e3 * wall / args.steps
    value = refined / wall
    n = R.n_sel
    # FLOPs per attention launch, averaged over the timed steps (each step
    # launches attention once per block)
    attn_flop = attn_flop_timed * L / max(attn_timing[0], 1)
    bd_launch_flop = attn_flop_bd / n_breakdown  # the same for the breakdown steps
    if args.attention == "factorised":  # spatial (per frame) and temporal (per position) launches alternate
        idx = R.idx[:n].cpu().numpy().astype(np.int64)
        toff = np.asarray(wl.tok_offset)
        r_of = np.searchsorted(toff, idx, side="right") - 1
        tpf = np.array([q.hp * q.wp for q in wl.requests])[r_of]
        loc = idx - toff[r_of]
        frame_cnt = np.unique(np.stack([r_of, loc // tpf], 1), axis=0, return_counts=True)[1].astype(np.float64)
        col_cnt = np.unique(np.stack([r_of, loc % tpf], 1), axis=0, return_counts=True)[1].astype(np.float64)
        # (from the last step's selection; the headline selection is the same every step)
        attn_flop = bd_launch_flop = 4.0 * D * float((frame_cnt ** 2).sum() + (col_cnt ** 2).sum()) / 2.0

    def gemm_flops(nn):
        return {"gemm_qkv": 2.0 * nn * D * 3 * D, "gemm_out": 2.0 * nn * D * D, "gemm_mlp1": 2.0 * nn * D * mlp,
                "gemm_mlp2": 2.0 * nn * mlp * D}

    gemm_flop = gemm_flops(n_timed / args.steps)  # per launch, averaged over the timed steps
    gemm_flop_bd = gemm_flops(n_bd / n_breakdown)
    kernels = {}
    for k, (cnt, ms) in timing.items():
        if cnt == 0:
            continue
        avg_us = 1e3 * ms / cnt
        e = {"launches": cnt, "avg_us": round(avg_us, 2), "ms_per_step": round(ms / n_breakdown, 4)}
        if k == "attention" and args.cache_period == 0:
            e["tflops"] = round(bd_launch_flop / (avg_us * 1e-6) / 1e12, 1)
        if k in gemm_flop_bd:
            e["tflops"] = round(gemm_flop_bd[k] / (avg_us * 1e-6) / 1e12, 1)
        kernels[k] = e
    cnt, ms = attn_timing
    avg_s = ms / cnt / 1e3
    achieved = attn_flop / avg_s / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic_entry("attention", args.config) if args.cache_period == 0 else None,
                "kernel": (f"k_attn_bf16_dma{'' if hd == 64 else hd} (varlen flash attention, head_dim {hd})"
                           if wl.model.dtype == "bf16" else "k_attn_f32") if args.attention == "joint"
                else "attention class: k_attn_bf16_dma per frame and k_attn_temporal per position, alternating",
                "algorithmic_flop_per_launch": attn_flop}
    step_flop = L * (attn_flop + sum(gemm_flop.values()))
    mfma_util = step_flop / (ms_per_step * 1e-3) / (PEAK_BF16_TFLOPS * 1e12)

    out = {"metric": METRIC, "value": round(value, 1), "unit": "refined tokens·steps/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded latents, blob uncertainty map, random-init weights)",
           "config": {"workload": f"{wl.name}: {wl.G} frames, {wl.N} tokens, {n} selected, "
                                  f"D{D} H{wl.model.heads}x{wl.model.head_dim} L{L} MLP{mlp}, "
                                  f"{int(wl.max_steps)}-step DDIM schedule",
                      "selected_tokens": int(n), "tokens": int(wl.N), "select_every_step": force,
                      "state_layout": args.layout, "cache_period": args.cache_period,
                      "attention": args.attention, "per_frame_grid": args.per_frame_grid},
           "mfma_util_step": round(mfma_util, 4),
           "roofline": roofline, "kernels": kernels,
           "kernels_note": f"per-class HIP-event averages from {n_breakdown} further untimed steps; "
                           "only attention is bracketed inside the timed steps"
                           + ("; with the latent cache the GEMM rates assume the last step's write set and "
                              "mix full and partial steps" if args.cache_period > 0 else ""),
           "setup_s": round(setup_s, 1)}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
