#!/usr/bin/env python3
"""Throughput of the OPTIMA weight-update hot path on one MI355X.

One step prunes-and-reconstructs one synthetic Llama-3-8B-shaped q_proj layer
(d_in = 4096, 4096 output columns, 2:4 Wanda mask, 262144 bf16 calibration
tokens with heavy-tailed features and 8 outlier channels):

  Hessian H = X^T X over all 262144 tokens -> damping -> spectral norm
  (block-16 subspace iteration) ->
  batched rAPDHG solve of the 4096 column QPs at the paper's tolerance
  (relative = absolute = 0.01, at most 100000 iterations).

All inputs (X, W0, mask, start vector) are resident in HBM before timing.
`value` is QP columns solved per second for the whole step. The JSON line also
carries rAPDHG iterations/s, the roofline of the dominant kernel (the batched
H-product with the fused update, over the timed steps' own launches, timed with
HIP events on its stream inside the library) and the CPU oracle's throughput on
a bounded sample of the same workload. After the timed steps an untimed
full-batch leg runs all 4096 columns for a fixed number of iterations (the
iteration rate at B = C); --fixed-iters 0 leaves it out.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
                       [--precision bf16x3|fp32] [--fixed-iters N]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "QP columns solved/sec + rAPDHG iters/sec on 4096×4096 layer; MFMA % of peak"
# Published dense MFMA peaks of MI355X.
FP32_MFMA_PEAK_TFLOPS = 157.3
BF16_MFMA_PEAK_TFLOPS = 2500.0
# Rate of the 2:4-sparse bf16 instruction counted in the flops of the dense
# product it stands for (twice the dense instruction's).
BF16_SPARSE_MFMA_PEAK_TFLOPS = 5000.0
HBM_PEAK_GBS = 8000.0
# Start vectors of the subspace iteration that sets the step size.
SPECTRAL_BLOCK = 16

# HBM traffic of the product kernel from rocprofv3 FETCH_SIZE / WRITE_SIZE
# passes (profiles/), valid only for the kernel sources they were taken on.
TRAFFIC = {"sources_sha1": "83031e9020184cd01698e8f93ad9f1123919a061",
           "bytes_per_launch": 276962 * 1024,       # k_product_sparse<fused|store>
           "few_bytes_per_launch": 67072 * 1024}    # k_product_skinny_sparse<fused|store>


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def kernel_sources_sha1() -> str:
    h = hashlib.sha1()
    for f in ("gemm_core.h", "solver.hip"):
        with open(os.path.join(ROOT, "paper_2512_13886_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def cpu_baseline(cfg, X, W0, mask, sample_cols: int, sample_chunks: int) -> dict:
    """The oracle on a bounded sample of the same layer, scaled to columns/s."""
    import oracle
    import workloads
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    t0 = time.perf_counter()
    H = oracle.hessian(workloads.x_to_f64(X[c * cfg.chunk:(c + 1) * cfg.chunk])
                       for c in range(sample_chunks))
    t_hess = time.perf_counter() - t0
    H, _ = oracle.damp(H, cfg.rel_damp)
    t0 = time.perf_counter()
    lam, _ = oracle.subspace_iteration(H, workloads.power_start_block(cfg.d, SPECTRAL_BLOCK),
                                       1000, 1e-6)
    t_pow = time.perf_counter() - t0
    cols = np.linspace(0, cfg.n_cols - 1, sample_cols).astype(int)
    t0 = time.perf_counter()
    r = oracle.rapdhg(H, W0[cols], mask[cols], lam, oracle.SolverOptions())
    t_solve = time.perf_counter() - t0
    job_s = (t_hess * cfg.n_chunks / sample_chunks + t_pow
             + t_solve * cfg.n_cols / sample_cols)
    # The same work on one thread (BLAS limited to one), on a smaller sample:
    # one sequence for the Hessian and 16 columns for the solve.
    one = None
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            oracle.hessian([workloads.x_to_f64(X[:cfg.chunk])])
            t1_hess = time.perf_counter() - t0
            t0 = time.perf_counter()
            oracle.subspace_iteration(H, workloads.power_start_block(cfg.d, SPECTRAL_BLOCK),
                                      1000, 1e-6)
            t1_pow = time.perf_counter() - t0
            cols1 = cols[np.linspace(0, cols.size - 1, 16).astype(int)]
            t0 = time.perf_counter()
            oracle.rapdhg(H, W0[cols1], mask[cols1], lam, oracle.SolverOptions())
            t1_solve = time.perf_counter() - t0
        one = {"value": cfg.n_cols / (t1_hess * cfg.n_chunks + t1_pow
                                      + t1_solve * cfg.n_cols / cols1.size),
               "cores": 1,
               "sample": (f"one thread: Hessian over 1 sequence (time scaled x{cfg.n_chunks}), "
                          f"the same subspace iteration, rAPDHG on {cols1.size} of the sampled "
                          f"columns (time scaled x{cfg.n_cols // cols1.size}); measured "
                          f"{t1_hess + t1_pow + t1_solve:.1f} s")}
    except ImportError:  # pragma: no cover
        pass
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as fh:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in fh
                              if ln.startswith("model name")), "")
    except OSError:  # pragma: no cover
        pass
    return {
        "value": cfg.n_cols / job_s, "unit": "columns/s", "cores": int(threads),
        "affinity_cores": len(os.sched_getaffinity(0)), "cpu_model": cpu_model,
        "kind": "oracle",
        "sample": (f"fp64 NumPy oracle: Hessian over {sample_chunks} of {cfg.n_chunks} "
                   f"2048-token sequences (time scaled x{cfg.n_chunks // sample_chunks}), "
                   f"block-{SPECTRAL_BLOCK} subspace iteration, paper-tolerance rAPDHG on {sample_cols} of "
                   f"{cfg.n_cols} columns (time scaled x{cfg.n_cols // sample_cols}; "
                   f"max {int(r.iters.max())} iterations); measured "
                   f"{t_hess + t_pow + t_solve:.1f} s of CPU work"),
        "one_thread": one,
    }


def block_leg(L, torch, dev, precision) -> dict:
    """The streamed decoder block (Llama-3-8B shapes): for each calibration
    stream the Hessian, the Wanda masks of its matrices (from the undamped
    Hessian's diagonal, on the device), damping, the step size and the paper-
    mode solves. Tokens and weights are moved to the device before timing;
    the reported time is the device time of all of that work. The step size
    comes from the block iteration, or from Lanczos where the block iteration
    has not converged within a few passes (spectral_step_size)."""
    import workloads
    from paper_2512_13886_amd.pipeline import spectral_step_size
    total_ms = 0.0
    layers = {}
    streams = {}
    for sname, scfg in workloads.BLOCK_STREAMS.items():
        mats = [lc for lc, st in workloads.BLOCK_LAYERS if st == sname]
        X = workloads.x_all(scfg)
        Xd = torch.from_numpy(X.view(np.int16)).view(torch.bfloat16).to(dev)
        del X
        d = scfg.d
        W0s = [torch.from_numpy(workloads.w0(lc)).to(dev) for lc in mats]
        H = torch.empty((d, d), dtype=torch.float32, device=dev)
        lam = torch.empty(1, dtype=torch.float32, device=dev)
        lmax = torch.empty(1, dtype=torch.float32, device=dev)
        V0 = torch.from_numpy(workloads.power_start_block(d, SPECTRAL_BLOCK)).to(dev)
        masks = [torch.empty((lc.n_cols, d), dtype=torch.uint8, device=dev) for lc in mats]
        outs = [torch.empty_like(w) for w in W0s]
        stats = [{"iters": torch.zeros(lc.n_cols, dtype=torch.int32, device=dev),
                  "converged": torch.zeros(lc.n_cols, dtype=torch.uint8, device=dev),
                  "f_initial": torch.zeros(lc.n_cols, dtype=torch.float32, device=dev),
                  "f_final": torch.zeros(lc.n_cols, dtype=torch.float32, device=dev)}
                 for lc in mats]
        hws = torch.empty(L.optima_hessian_workspace_bytes(scfg.n_tok, d, L.DTYPE_BF16),
                          dtype=torch.uint8, device=dev)
        opts = L.SolverOpts.default()
        if precision is not None:
            opts.precision = precision
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3 + len(mats))]
        ev[0].record()
        L.optima_hessian_accumulate(Xd, H, ws=hws)
        for lc, W0d, M in zip(mats, W0s, masks):
            L.optima_wanda_mask(W0d, H, M, L.MASK_UNSTRUCTURED, lc.sparsity, col_sq_stride=d + 1)
        ev[1].record()
        L.optima_hessian_damp(H, scfg.rel_damp, lam)
        spec = spectral_step_size(H, V0, lmax)
        ev[2].record()
        infos = []
        for i, (lc, W0d, M, out, st) in enumerate(zip(mats, W0s, masks, outs, stats)):
            infos.append(L.optima_qp_solve_batched(H, lmax, W0d, M, out, opts=opts, stats=st))
            ev[3 + i].record()
        torch.cuda.synchronize()
        s_ms = ev[0].elapsed_time(ev[-1])
        total_ms += s_ms
        streams[sname] = {"d": d, "hessian_and_masks_ms": ev[0].elapsed_time(ev[1]),
                          "damp_spectral_ms": ev[1].elapsed_time(ev[2]),
                          "spectral": spec, "ms": s_ms}
        prev = ev[2]
        for i, (lc, st, inf) in enumerate(zip(mats, stats, infos)):
            layers[lc.name[len("block_"):]] = {
                "d": d, "columns": lc.n_cols, "solve_ms": prev.elapsed_time(ev[3 + i]),
                "iterations": inf["iterations"], "converged": int(st["converged"].sum().item()),
                "f_final_over_f_initial":
                    (st["f_final"].double().sum() / st["f_initial"].double().sum()).item()}
            prev = ev[3 + i]
        log(f"block stream {sname}: {s_ms:.1f} ms (step size: {spec['method']}, "
            f"{spec['block_passes']} block passes, {spec['lanczos_steps']} Lanczos steps)")
        del Xd, H, hws, W0s, outs, masks, stats
        torch.cuda.empty_cache()
    cols = sum(v["columns"] for v in layers.values())
    return {"block_prune_ms": total_ms, "columns": cols,
            "columns_per_s": cols / (total_ms * 1e-3), "streams": streams, "layers": layers}


def chain_leg(L, torch, dev, precision) -> dict:
    """The layer loop of Algorithm 1 on the chain of four 4096 x 4096 layers
    (SiLU between them) over 262144 bf16 tokens: per layer the Hessian of its
    (pruned) inputs, the device Wanda mask, the step size, the paper-mode solve,
    the skip rule, the layer-wise errors and the forward pass that feeds the
    next layer. Reported: device time per layer and the error ratios."""
    import workloads
    from paper_2512_13886_amd.pipeline import prune_chain
    X = workloads.x_all(workloads.CHAIN_STREAM)
    Xd = torch.from_numpy(X.view(np.int16)).view(torch.bfloat16).to(dev)
    del X
    W0s = [torch.from_numpy(workloads.w0(lc)).to(dev) for lc in workloads.CHAIN_LAYERS]
    starts = {}

    def start(d):
        if d not in starts:
            starts[d] = torch.from_numpy(workloads.power_start_block(d, SPECTRAL_BLOCK)).to(dev)
        return starts[d]

    opts = L.SolverOpts.default()
    if precision is not None:
        opts.precision = precision
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    _, _, reps, _ = prune_chain(Xd, W0s, start, sparsity=0.5, rel_damp=0.01, opts=opts,
                                timed=True)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3
    layers = []
    for r in reps:
        layers.append({"d_in": r.d_in, "d_out": r.d_out, "iterations": r.iterations,
                       "converged": r.converged, "skipped": r.skipped,
                       "error_ratio_vs_wanda": r.error_ratio, "ms": r.ms})
        log(f"chain layer: {r.iterations} iterations, {r.converged}/{r.d_out} converged, "
            f"skipped {r.skipped}, error ratio {r.error_ratio:.4f}, {r.ms['total']:.1f} ms")
    dev_ms = sum(r.ms["total"] for r in reps)
    return {"layers": layers, "device_ms": dev_ms, "wall_ms": wall,
            "tokens": int(Xd.shape[0]), "columns": sum(r.d_out for r in reps)}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-cols", type=int, default=256)
    ap.add_argument("--cpu-sample-chunks", type=int, default=32)
    ap.add_argument("--fixed-iters", type=int, default=1000,
                    help="iterations of the untimed full-batch leg (0: skip it)")
    ap.add_argument("--precision", choices=["fp32", "bf16x3"], default=None,
                    help="arithmetic of the per-iteration H-products (default: the "
                         "library's, bf16x3)")
    ap.add_argument("--block-config", action="store_true",
                    help="also prune the streamed Llama-3-8B-shaped decoder block (7 matrices, "
                         "4 calibration streams) and report its end-to-end device time")
    ap.add_argument("--chain-config", action="store_true",
                    help="also run the layer loop of Algorithm 1 on a chain of four 4096 x 4096 "
                         "layers (forward propagation of the pruned activations, skip rule, "
                         "layer-wise error ratios)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="first run one 256 MiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        log("bench.py measures one MI355X only: the library runs the hot path on a single GPU "
            "(columns would shard across GPUs with no per-iteration communication). "
            "Run it with --gpus 1.")
        return 2

    import torch
    import paper_2512_13886_amd as L
    from paper_2512_13886_amd.pipeline import spectral_step_size
    import workloads

    dev = torch.device("cuda:0")
    if args.calibration_copy:
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    cfg = workloads.Q_PROJ
    t0 = time.perf_counter()
    X = workloads.x_all(cfg)
    W0 = workloads.w0(cfg)
    col_sq = workloads.col_sq_norms(cfg, X)
    mask = workloads.layer_mask(cfg, W0, col_sq)
    V0 = workloads.power_start_block(cfg.d, SPECTRAL_BLOCK)
    log(f"inputs generated in {time.perf_counter() - t0:.1f} s")

    Xd = torch.from_numpy(X.view(np.int16)).view(torch.bfloat16).to(dev)
    W0d = torch.from_numpy(W0).to(dev)
    Md = torch.from_numpy(mask).to(dev)
    V0d = torch.from_numpy(V0).to(dev)
    d, C, N = cfg.d, cfg.n_cols, cfg.n_tok
    H = torch.empty((d, d), dtype=torch.float32, device=dev)
    lam = torch.empty(1, dtype=torch.float32, device=dev)
    lmax = torch.empty(1, dtype=torch.float32, device=dev)
    Wout = torch.empty_like(W0d)
    hws = torch.empty(L.optima_hessian_workspace_bytes(N, d, L.DTYPE_BF16), dtype=torch.uint8,
                      device=dev)
    sws = torch.empty(L.optima_spectral_norm_workspace_bytes(d, SPECTRAL_BLOCK),
                      dtype=torch.uint8, device=dev)
    qws = torch.empty(L.optima_qp_workspace_bytes(d, C), dtype=torch.uint8, device=dev)
    iters = torch.zeros(C, dtype=torch.int32, device=dev)
    conv = torch.zeros(C, dtype=torch.uint8, device=dev)
    f_init = torch.zeros(C, dtype=torch.float32, device=dev)
    f_fin = torch.zeros(C, dtype=torch.float32, device=dev)
    # Table 8: tol 0.01 / 0.01, 100000 iterations
    opts = L.SolverOpts.default()
    if args.precision is not None:
        opts.precision = {"fp32": L.PREC_FP32, "bf16x3": L.PREC_BF16X3}[args.precision]
    prec = opts.precision
    prec_name = "bf16x3" if prec == L.PREC_BF16X3 else "fp32"
    torch.cuda.reset_peak_memory_stats(dev)
    torch.cuda.synchronize()

    def step():
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record()
        L.optima_hessian_accumulate(Xd, H, accumulate=False, ws=hws)
        ev[1].record()
        L.optima_hessian_damp(H, cfg.rel_damp, lam)
        L.optima_spectral_norm(H, V0d, lmax, max_iters=1000, tol=1e-6, ws=sws)
        ev[2].record()
        info = L.optima_qp_solve_batched(H, lmax, W0d, Md, Wout, opts=opts, ws=qws,
                                         stats={"iters": iters, "converged": conv,
                                                "f_initial": f_init, "f_final": f_fin})
        ev[3].record()
        return ev, info

    for w in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"warmup step {w + 1}/{args.warmup} done")

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    recs = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    ms_step = wall * 1000.0 / args.steps
    hess_ms = np.mean([e[0].elapsed_time(e[1]) for e, _ in recs])
    spec_ms = np.mean([e[1].elapsed_time(e[2]) for e, _ in recs])
    solve_ms = np.mean([e[2].elapsed_time(e[3]) for e, _ in recs])
    solve_ms_median = float(np.median([e[2].elapsed_time(e[3]) for e, _ in recs]))
    it = np.mean([i["iterations"] for _, i in recs])
    col_it = np.mean([i["row_products"] for _, i in recs])
    all_launches = sum(i["timed_launches"] for _, i in recs)
    all_rows = sum(i["timed_row_products"] for _, i in recs)
    all_ms = sum(i["timed_product_ms"] for _, i in recs)
    sparse_products = all(i["sparse_products"] == 1 for _, i in recs)
    # The dominant kernel is the tiled product; the launches over at most 8
    # active columns run another kernel (H streamed once per launch), timed
    # and reported on their own.
    few_launches = sum(i["few_launches"] for _, i in recs)
    few_rows = sum(i["few_row_products"] for _, i in recs)
    few_ms = sum(i["few_product_ms"] for _, i in recs)
    launches = all_launches - few_launches
    rows = all_rows - few_rows
    prod_ms = all_ms - few_ms
    flops = 2.0 * d * d * rows
    achieved = flops / (prod_ms * 1e-3) / 1e12
    avg_launch_us = prod_ms * 1e3 / launches
    all_tflops = 2.0 * d * d * all_rows / (all_ms * 1e-3) / 1e12
    per_col_it = iters.cpu().numpy()
    f_ratio_rapdhg = float(f_fin.double().sum() / f_init.double().sum())
    log(f"step {ms_step:.1f} ms: hessian {hess_ms:.2f} ms, damp+spectral {spec_ms:.2f} ms, "
        f"solve {solve_ms:.1f} ms ({it:.0f} iterations, {conv.sum().item()}/{C} converged, "
        f"per-column iterations {per_col_it.min()}..{per_col_it.max()})")
    log(f"H-product (tiles): {launches} launches, avg {avg_launch_us:.1f} us, {achieved:.1f} TFLOP/s;"
        f" few-column: {few_launches} launches, avg "
        f"{(few_ms * 1e3 / few_launches) if few_launches else 0.0:.1f} us;"
        f" all: {all_launches} launches, {all_tflops:.1f} TFLOP/s")

    # Unconstrained-form leg (Eq. (7)-(11)): conjugate gradients on the same
    # layer and H at the same tolerances, tested every 8 iterations; no step
    # size is needed. Not part of the timed step.
    cg_opts = L.SolverOpts.default(method=L.METHOD_CG, check_every=8)
    if args.precision is not None:
        cg_opts.precision = prec
    cg_ms, cg_it = [], []
    for rep in range(4):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        cinfo = L.optima_qp_solve_batched(H, None, W0d, Md, Wout, opts=cg_opts, ws=qws,
                                          stats={"iters": iters, "converged": conv,
                                                 "f_initial": f_init, "f_final": f_fin})
        b.record()
        torch.cuda.synchronize()
        if rep:  # the first run is a warm-up
            cg_ms.append(a.elapsed_time(b))
            cg_it.append(cinfo["iterations"])
    cg_solve_ms = float(np.mean(cg_ms))
    cg_leg = {"solve_ms": cg_solve_ms, "iterations": float(np.mean(cg_it)), "check_every": 8,
              "converged": int(conv.sum().item()),
              "columns_per_s_solve_only": C / (cg_solve_ms * 1e-3),
              "step_ms_equivalent": hess_ms + cg_solve_ms,
              "columns_per_s_step_equivalent": C / ((hess_ms + cg_solve_ms) * 1e-3),
              "f_final_over_f_initial": float(f_fin.double().sum() / f_init.double().sum()),
              "rapdhg_f_final_over_f_initial": f_ratio_rapdhg}
    log(f"cg: solve {cg_solve_ms:.2f} ms ({cg_leg['iterations']:.0f} iterations, "
        f"{cg_leg['converged']}/{C} converged); sum f_final / sum f_initial "
        f"cg {cg_leg['f_final_over_f_initial']:.4f}, rapdhg {f_ratio_rapdhg:.4f}")

    # Preconditioned leg: Jacobi scaling of (a copy of) H, the spectral norm of
    # D H D and both solvers with the column scaling, at the paper's
    # tolerances and at a tight one (eps_rel 1e-4, eps_abs 0) beside the
    # unscaled solves. Not part of the timed step.
    Hs = torch.empty_like(H)
    Hs.copy_(H)
    Ds = torch.empty(d, dtype=torch.float32, device=dev)
    lmax_s = torch.empty(1, dtype=torch.float32, device=dev)
    stats_d = {"iters": iters, "converged": conv, "f_initial": f_init, "f_final": f_fin}

    def timed_solve(Hm, lm, o):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        inf = L.optima_qp_solve_batched(Hm, lm, W0d, Md, Wout, opts=o, ws=qws, stats=stats_d)
        b.record()
        torch.cuda.synchronize()
        return {"ms": a.elapsed_time(b), "iterations": inf["iterations"],
                "converged": int(conv.sum().item()),
                "f_final_over_f_initial": (f_fin.double().sum() / f_init.double().sum()).item()}

    e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    e[0].record()
    L.optima_hessian_jacobi(Hs, Ds)
    e[1].record()
    spec_s = spectral_step_size(Hs, V0d, lmax_s)
    e[2].record()
    torch.cuda.synchronize()

    def o_(**kw):
        o = L.SolverOpts.default(**kw)
        if args.precision is not None:
            o.precision = prec
        return o

    tight = dict(eps_rel=1e-4, eps_abs=0.0, max_iters=20000)
    pre = {"scale_ms": e[0].elapsed_time(e[1]), "spectral_ms": e[1].elapsed_time(e[2]),
           "spectral": spec_s,
           "paper_tolerance": {
               "rapdhg_scaled": timed_solve(Hs, lmax_s, o_(col_scale=Ds)),
               "cg_scaled": timed_solve(Hs, None, o_(method=L.METHOD_CG, check_every=8,
                                                      col_scale=Ds))},
           "tight_tolerance_eps_rel_1e-4": {
               "rapdhg": timed_solve(H, lmax, o_(**tight)),
               "rapdhg_scaled": timed_solve(Hs, lmax_s, o_(col_scale=Ds, **tight)),
               "cg": timed_solve(H, None, o_(method=L.METHOD_CG, check_every=8, **tight)),
               "cg_scaled": timed_solve(Hs, None, o_(method=L.METHOD_CG, check_every=8,
                                                     col_scale=Ds, **tight))}}
    tt = pre["tight_tolerance_eps_rel_1e-4"]
    log(f"jacobi-preconditioned: scale {pre['scale_ms']:.2f} ms, spectral {pre['spectral_ms']:.2f} ms "
        f"({spec_s['method']}: {spec_s['block_passes']} block passes, "
        f"{spec_s['lanczos_steps']} Lanczos steps); tight: rapdhg {tt['rapdhg']['iterations']} -> "
        f"{tt['rapdhg_scaled']['iterations']} it ({tt['rapdhg']['ms']:.1f} -> "
        f"{tt['rapdhg_scaled']['ms']:.1f} ms), cg {tt['cg']['iterations']} -> "
        f"{tt['cg_scaled']['iterations']} it ({tt['cg']['ms']:.1f} -> {tt['cg_scaled']['ms']:.1f} ms)")

    # Full-batch leg: all 4096 columns for a fixed number of iterations, the
    # iteration rate at B = C (not part of the timed step).
    fixed_batch = None
    if args.fixed_iters > 0:
        fixed = L.SolverOpts.default(max_iters=args.fixed_iters, fixed_iters=1, precision=prec)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        finfo = L.optima_qp_solve_batched(H, lmax, W0d, Md, Wout, opts=fixed, ws=qws)
        e1.record()
        torch.cuda.synchronize()
        fixed_ms = e0.elapsed_time(e1)
        f_flops = 2.0 * d * d * finfo["timed_row_products"]
        f_launch_us = finfo["timed_product_ms"] * 1e3 / finfo["timed_launches"]
        fixed_tflops = f_flops / (finfo["timed_product_ms"] * 1e-3) / 1e12
        log(f"fixed {args.fixed_iters} iterations x {C} columns: {fixed_ms:.1f} ms, H-product "
            f"{fixed_tflops:.1f} TFLOP/s, avg launch {f_launch_us:.1f} us")
        fixed_batch = {"iters": args.fixed_iters, "columns": C, "ms": fixed_ms,
                       "iters_per_s": args.fixed_iters / (fixed_ms * 1e-3),
                       "column_iters_per_s": args.fixed_iters * C / (fixed_ms * 1e-3),
                       "product_tflops": fixed_tflops, "product_avg_launch_us": f_launch_us}

    # Device mask selection (the selector ahead of the update; not part of
    # the step, whose mask is an input): both patterns on this layer's W0 and
    # fp64 column norms, 5 launches each.
    csd = torch.from_numpy(col_sq).to(dev)
    md = torch.empty_like(Md)

    def time_mask(pattern, sparsity, reps=5):
        L.optima_wanda_mask(W0d, csd, md, pattern, sparsity)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            L.optima_wanda_mask(W0d, csd, md, pattern, sparsity)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    m24_ms = time_mask(L.MASK_2TO4, 0.5)
    m24_same = bool(torch.equal(md, Md))
    mun_ms = time_mask(L.MASK_UNSTRUCTURED, 0.5)
    mask_bytes = 5.0 * C * d  # read W0 (4 B), write the mask (1 B) per element
    mask_select = {"two_four_ms": m24_ms, "unstructured_50_ms": mun_ms,
                   "two_four_gbps": mask_bytes / (m24_ms * 1e-3) / 1e9,
                   "unstructured_gbps": mask_bytes / (mun_ms * 1e-3) / 1e9,
                   "algorithmic_bytes_per_element": 5,
                   "two_four_equals_host_mask": m24_same}
    log(f"mask selection: 2:4 {m24_ms * 1e3:.1f} us, unstructured {mun_ms * 1e3:.1f} us, "
        f"2:4 equals the host mask: {m24_same}")

    block = None
    if args.block_config:
        block = block_leg(L, torch, dev, None if args.precision is None else prec)
        log(f"block prune: {block['block_prune_ms']:.1f} ms for {block['columns']} columns")

    chain = None
    if args.chain_config:
        chain = chain_leg(L, torch, dev, None if args.precision is None else prec)
        log(f"chain: {chain['device_ms']:.1f} ms device time for {len(chain['layers'])} layers")

    traffic = None  # the counter passes were taken on the bf16x3 kernels
    if (TRAFFIC and prec == L.PREC_BF16X3
            and TRAFFIC.get("sources_sha1") == kernel_sources_sha1()):
        traffic = TRAFFIC["bytes_per_launch"]

    # Roofline of the dominant kernel over the timed steps: algorithmic flops
    # (2 d^2 per column per iteration) over the device time of its launches.
    if prec == L.PREC_BF16X3 and sparse_products:
        # The 2:4 mask lets x travel compressed: each of the three bf16
        # products runs on v_smfmac_f32_16x16x64_bf16 and skips the pruned
        # half of K. achieved keeps the algorithmic count of the dense
        # product (2 d^2 per column and iteration) and frac compares it with
        # the dense bf16 peak; mfma_issued_frac compares the issued products
        # (3 x achieved) with the sparse instruction's own peak.
        roofline = {
            "kernel": "k_product_sparse<fused>: H-product x H over the active columns "
                      "(M = active columns, N = K = 4096), x 2:4-compressed, three bf16 "
                      "products per fp32 product on v_smfmac_f32_16x16x64_bf16 (256 x 128 "
                      "tiles), fused rAPDHG update in the epilogue",
            "bound": "mfma", "achieved": achieved, "peak": BF16_MFMA_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": achieved / BF16_MFMA_PEAK_TFLOPS,
            "traffic": traffic,
            "sparse_products": True,
            "mfma_issued_tflops": 3.0 * achieved,
            "mfma_issued_peak": BF16_SPARSE_MFMA_PEAK_TFLOPS,
            "mfma_issued_frac": 3.0 * achieved / BF16_SPARSE_MFMA_PEAK_TFLOPS,
            "fp32_equivalent_frac": achieved / FP32_MFMA_PEAK_TFLOPS,
        }
    elif prec == L.PREC_BF16X3:
        roofline = {
            "kernel": "k_product<fused, bf16x3>: H-product x H over the active columns "
                      "(M = active columns, N = K = 4096) on v_mfma_f32_16x16x32_bf16, three "
                      "bf16 products per fp32 product, fused rAPDHG update in the epilogue",
            "bound": "mfma", "achieved": achieved, "peak": BF16_MFMA_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": achieved / BF16_MFMA_PEAK_TFLOPS,
            "traffic": traffic,
            "mfma_issued_tflops": 3.0 * achieved,
            "mfma_issued_frac": 3.0 * achieved / BF16_MFMA_PEAK_TFLOPS,
            "fp32_equivalent_frac": achieved / FP32_MFMA_PEAK_TFLOPS,
        }
    else:
        roofline = {
            "kernel": "k_product<fused, fp32>: H-product over the active columns "
                      "(M = active columns, N = K = 4096) on v_mfma_f32_16x16x4_f32, fused "
                      "rAPDHG update in the epilogue",
            "bound": "mfma", "achieved": achieved, "peak": FP32_MFMA_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": achieved / FP32_MFMA_PEAK_TFLOPS,
            "traffic": traffic,
        }
    roofline.update({"avg_launch_us": avg_launch_us, "launches": launches,
                     "flops_per_launch": flops / launches})
    if few_launches:
        # H's split planes (4 d^2 bytes) dominate these launches; per active
        # column they add the compressed x planes (2 d bytes) and the packed
        # update (16.25 d bytes), or x in fp32 (4 d) and the update (33 d).
        per_col = (2.0 + 16.25) * d if sparse_products else (4.0 + 33.0) * d
        few_bytes = 4.0 * d * d * few_launches + per_col * few_rows
        few_gbs = few_bytes / (few_ms * 1e-3) / 1e9
        few_traffic = None
        if traffic is not None:
            few_traffic = TRAFFIC.get("few_bytes_per_launch")
        roofline["few_column_kernel"] = {
            "kernel": ("k_product_skinny_sparse" if sparse_products else "k_product_skinny") +
                      "<fused>: the same product when at most 8 columns are active, H's planes "
                      "streamed once per launch",
            "bound": "hbm", "achieved": few_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": few_gbs / HBM_PEAK_GBS, "traffic": few_traffic,
            "avg_launch_us": few_ms * 1e3 / few_launches, "launches": few_launches,
            "bytes_per_launch": few_bytes / few_launches}
    roofline["all_iteration_products"] = {
        "launches": all_launches, "avg_launch_us": all_ms * 1e3 / all_launches,
        "achieved": all_tflops, "unit": "TFLOP/s"}

    out = {
        "metric": METRIC,
        "value": C / (ms_step * 1e-3),
        "unit": "columns/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": prec_name,
        "data": "synthetic",
        "config": {
            "workload": ("q_proj layer d_in=4096 x 4096 columns: Hessian from 262144 bf16 "
                         "tokens (Student-t nu=4, 8 outlier channels x50), 2:4 Wanda mask, "
                         "rAPDHG at tol 0.01/0.01, max 100000 iterations"),
            "d": d, "n_cols": C, "n_tok": N, "x_dtype": "bf16", "mask": "2:4",
            "eps_rel": 0.01, "eps_abs": 0.01, "check_every": 64,
            "product_precision": prec_name,
        },
        "rapdhg_iters_per_s": it / (solve_ms * 1e-3),
        "column_iters_per_s": col_it / (solve_ms * 1e-3),
        "iterations": it,
        "phase_ms": {"hessian": hess_ms, "damp_spectral": spec_ms, "solve": solve_ms},
        "solve_only": {"solve_ms_median": solve_ms_median, "runs": args.steps,
                       "columns_per_s": C / (solve_ms_median * 1e-3)},
        "hessian_tflops": 2.0 * N * d * d / 2 / (hess_ms * 1e-3) / 1e12,
        "fixed_batch": fixed_batch,
        "mask_select": mask_select,
        "cg_unconstrained": cg_leg,
        "jacobi_preconditioned": pre,
        "decoder_block": block,
        "layer_chain": chain,
        "peak_device_memory_gib": torch.cuda.max_memory_allocated(dev) / 2**30,
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline(cfg, X, W0, mask, args.cpu_sample_cols,
                                           args.cpu_sample_chunks)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
