#!/usr/bin/env python3
"""Throughput of the OPTIMA weight-update hot path on one MI355X.

One step prunes-and-reconstructs one synthetic Llama-3-8B-shaped q_proj layer
(d_in = 4096, 4096 output columns, 2:4 Wanda mask, 262144 bf16 calibration
tokens with heavy-tailed features and 8 outlier channels):

  Hessian H = X^T X over all 262144 tokens -> damping -> spectral norm
  (block-16 subspace iteration) ->
  batched rAPDHG solve of the 4096 column QPs at the paper's tolerance
  (relative = absolute = 0.01, at most 100000 iterations).

All inputs (X, W0, mask, start vectors) are resident in HBM before timing.
`value` is QP columns solved per second for the whole step, over the K timed
steps. The JSON line also carries:
  - rapdhg_iters_per_s: the solver's iteration rate at B = C (all 4096
    columns for a fixed number of iterations, an untimed leg after the timed
    steps; --fixed-iters 0 leaves it out), and the paper-mode figures of the
    timed steps (loop passes/s, column-iterations/s, the fraction of columns
    that stop at the start-point check);
  - the roofline of the dominant kernel (the batched H-product with the fused
    update, over the timed steps' own launches, timed with HIP events on its
    stream inside the library);
  - per-configuration entries (tiny, GPT-2 fc, q_proj, down_proj): layer step
    time, columns/s, iterations/s at B = C, Hessian and product TFLOP/s, each
    product kernel's roofline, peak device memory;
  - the streamed decoder block's end-to-end prune time (--no-block skips it);
  - the CPU oracle's throughput on a bounded sample of the q_proj step.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
                       [--precision bf16x3|fp32] [--fixed-iters N] [--no-configs]
                       [--no-block] [--chain-config]
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
TRAFFIC = {"sources_sha1": "caba776757dbde68da49bb9b17ae5c4dba5b9493",
           "bytes_per_launch": 278758 * 1024,       # k_product_sparse<fused>
           "few_bytes_per_launch": 67098 * 1024}    # k_product_skinny_sparse<fused>
# The same for the Hessian's k_syrk_direct on the q_proj tokens (FETCH x 2 +
# WRITE of its one launch), valid for the Hessian sources it was taken on.
HESSIAN_TRAFFIC = {"sources_sha1": "74556267ecb4153098e1288c059f918b0d8584d1",
                   "bytes_per_launch": (2 * 5916560 + 382982) * 1024}

# Per-configuration legs after the headline: (config, untimed fixed-batch
# iterations, timed steps). The fixed-batch leg gives the iteration rate at
# B = C; down_proj runs fewer iterations (an iteration over 4096 columns at
# d = 14336 takes about 4 ms).
CONFIG_LEGS = (("tiny", 1000, 5), ("gpt2_fc", 1000, 3), ("down_proj", 100, 2))


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def kernel_sources_sha1(files=("gemm_core.h", "solver.hip")) -> str:
    h = hashlib.sha1()
    for f in files:
        with open(os.path.join(ROOT, "paper_2512_13886_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


HESSIAN_SOURCES = ("gemm_core.h", "hessian.hip")


def hessian_roofline(n_tok: int, d: int, hess_ms: float) -> dict:
    """The Hessian call (k_syrk_direct plus the fixed-order sum of its split
    partials) against the dense bf16 MFMA peak, in useful flops (one
    triangle, n_tok d^2), timed by the step's HIP events."""
    achieved = float(n_tok) * d * d / (hess_ms * 1e-3) / 1e12
    traffic = None
    if HESSIAN_TRAFFIC.get("sources_sha1") == kernel_sources_sha1(HESSIAN_SOURCES):
        traffic = HESSIAN_TRAFFIC["bytes_per_launch"]
    return {"kernel": "k_syrk_direct (256 x 256 lower tiles, token rows in place, ring of four "
                      "32-token LDS buffers, v_mfma_f32_16x16x32_bf16) + k_hess_reduce4",
            "bound": "mfma", "achieved": achieved, "peak": BF16_MFMA_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": achieved / BF16_MFMA_PEAK_TFLOPS, "traffic": traffic,
            "call_ms": hess_ms, "useful_flops": float(n_tok) * d * d}


def cpu_baseline(cfg, X, W0, mask, H_dev: np.ndarray, lam_dev: float, sample_cols: int,
                 sample_chunks: int) -> dict:
    """The oracle on a bounded sample of the same layer, scaled to columns/s.

    The Hessian is timed on a subset of the calibration sequences and scaled
    to all of them. The step size and the solve are timed on the damped H of
    the timed GPU steps (its fp32 values in fp64), so the sampled columns take
    the iteration counts the GPU's columns take.
    """
    import oracle
    import workloads
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    t0 = time.perf_counter()
    oracle.hessian(workloads.x_to_f64(X[c * cfg.chunk:(c + 1) * cfg.chunk])
                   for c in range(sample_chunks))
    t_hess = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.subspace_iteration(H_dev, workloads.power_start_block(cfg.d, SPECTRAL_BLOCK), 1000,
                              1e-6)
    t_pow = time.perf_counter() - t0
    cols = np.linspace(0, cfg.n_cols - 1, sample_cols).astype(int)
    t0 = time.perf_counter()
    r = oracle.rapdhg(H_dev, W0[cols], mask[cols], lam_dev, oracle.SolverOptions())
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
            oracle.subspace_iteration(H_dev, workloads.power_start_block(cfg.d, SPECTRAL_BLOCK),
                                      1000, 1e-6)
            t1_pow = time.perf_counter() - t0
            cols1 = cols[np.linspace(0, cols.size - 1, 16).astype(int)]
            t0 = time.perf_counter()
            oracle.rapdhg(H_dev, W0[cols1], mask[cols1], lam_dev, oracle.SolverOptions())
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
                   f"2048-token sequences (time scaled x{cfg.n_chunks // sample_chunks}); "
                   f"block-{SPECTRAL_BLOCK} subspace iteration and paper-tolerance rAPDHG on "
                   f"the damped H of the timed GPU steps, rAPDHG on {sample_cols} of "
                   f"{cfg.n_cols} columns (time scaled x{cfg.n_cols // sample_cols}; "
                   f"max {int(r.iters.max())} iterations); measured "
                   f"{t_hess + t_pow + t_solve:.1f} s of CPU work"),
        "one_thread": one,
    }


def product_kernel_name(d: int, rows: int, prec_name: str, sparse: bool) -> str:
    """The tiled H-product kernel the library runs for this shape."""
    if prec_name == "fp32":
        return "k_product<fused, fp32> (128 x 128 tiles, v_mfma_f32_16x16x4_f32)"
    if sparse:
        return ("k_product_sparse<fused> (256 x 128 tiles, x 2:4-compressed, "
                "v_smfmac_f32_16x16x64_bf16, three bf16 products per fp32 product)")
    if d >= 8192 and rows >= 256:
        return ("k_product_wide<fused, bf16x3> (256 x 128 tiles, v_mfma_f32_16x16x32_bf16, "
                "three bf16 products per fp32 product)")
    return ("k_product<fused, bf16x3> (128 x 128 tiles, v_mfma_f32_16x16x32_bf16, three "
            "bf16 products per fp32 product)")


def product_roofline(d: int, infos: list, prec_name: str, traffic=None,
                     few_traffic=None) -> dict:
    """Roofline of the iteration products over the given solves: algorithmic
    flops (2 d^2 per active column and iteration) over the device time of
    their launches, the tiled kernel and the few-column kernel apart."""
    sparse = all(i["sparse_products"] == 1 for i in infos)
    all_launches = sum(i["timed_launches"] for i in infos)
    all_rows = sum(i["timed_row_products"] for i in infos)
    all_ms = sum(i["timed_product_ms"] for i in infos)
    few_launches = sum(i["few_launches"] for i in infos)
    few_rows = sum(i["few_row_products"] for i in infos)
    few_ms = sum(i["few_product_ms"] for i in infos)
    launches, rows, ms = all_launches - few_launches, all_rows - few_rows, all_ms - few_ms
    out = {"sparse_products": sparse}
    if launches and ms > 0:
        achieved = 2.0 * d * d * rows / (ms * 1e-3) / 1e12
        peak = FP32_MFMA_PEAK_TFLOPS if prec_name == "fp32" else BF16_MFMA_PEAK_TFLOPS
        out.update({
            "kernel": product_kernel_name(d, rows // max(launches, 1), prec_name, sparse),
            "bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
            "frac": achieved / peak, "traffic": traffic,
            "avg_launch_us": ms * 1e3 / launches, "launches": launches,
            "avg_active_columns": rows / launches,
            "flops_per_launch": 2.0 * d * d * rows / launches})
        if prec_name != "fp32":
            out["mfma_issued_tflops"] = 3.0 * achieved
            out["mfma_issued_peak"] = (BF16_SPARSE_MFMA_PEAK_TFLOPS if sparse
                                       else BF16_MFMA_PEAK_TFLOPS)
            out["mfma_issued_frac"] = 3.0 * achieved / out["mfma_issued_peak"]
            out["fp32_equivalent_frac"] = achieved / FP32_MFMA_PEAK_TFLOPS
    if few_launches and few_ms > 0:
        # Iterations with at most 8 active columns. Launched one per iteration
        # they stream H's split planes (4 d^2 bytes) from HBM each time; per
        # active column they add the compressed x planes (2 d bytes) and the
        # packed update (16.25 d bytes), or x in fp32 (4 d) and the update
        # (33 d). Run as one cooperative launch per block of iterations they
        # keep H's planes in registers: then the figure below is the rate a
        # streaming kernel would need to match them (it can exceed the peak).
        persistent = sum(i.get("persistent_launches", 0) for i in infos)
        per_col = (2.0 + 16.25) * d if sparse else (4.0 + 33.0) * d
        few_bytes = 4.0 * d * d * few_launches + per_col * few_rows
        few_gbs = few_bytes / (few_ms * 1e-3) / 1e9
        if persistent:
            name = ("k_few_persistent<sparse>" if sparse else "k_few_persistent<bf16x3>") + \
                   (": at most 8 active columns, every iteration between two checks in one "
                    "cooperative launch with H's planes in registers and a grid barrier per "
                    "iteration")
            bound = "latency"
        else:
            name = ("k_product_skinny_sparse" if sparse else "k_product_skinny") + \
                   ("<fused>: the same product when at most 8 columns are active, H's planes "
                    "streamed once per launch")
            bound = "hbm"
        out["few_column_kernel"] = {
            "kernel": name, "bound": bound, "achieved": few_gbs, "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": few_gbs / HBM_PEAK_GBS,
            "traffic": None if persistent else few_traffic,
            "avg_launch_us": few_ms * 1e3 / few_launches, "launches": few_launches,
            "cooperative_launches": persistent,
            "bytes_per_launch": few_bytes / few_launches}
    if all_launches and all_ms > 0:
        out["all_iteration_products"] = {
            "launches": all_launches, "avg_launch_us": all_ms * 1e3 / all_launches,
            "achieved": 2.0 * d * d * all_rows / (all_ms * 1e-3) / 1e12, "unit": "TFLOP/s"}
    return out


class LayerRun:
    """Device buffers and one layer step (Hessian, damping, step size,
    paper-mode solve) for one synthetic layer."""

    def __init__(self, L, torch, dev, cfg, opts, spectral_policy: bool):
        import workloads
        self.L, self.torch, self.dev, self.cfg = L, torch, dev, cfg
        t0 = time.perf_counter()
        self.X = workloads.x_all(cfg)
        self.W0 = workloads.w0(cfg)
        self.col_sq = workloads.col_sq_norms(cfg, self.X)
        self.mask = workloads.layer_mask(cfg, self.W0, self.col_sq)
        self.V0 = workloads.power_start_block(cfg.d, SPECTRAL_BLOCK)
        self.gen_s = time.perf_counter() - t0
        if self.X.dtype == np.uint16:
            self.Xd = torch.from_numpy(self.X.view(np.int16)).view(torch.bfloat16).to(dev)
            xdt = L.DTYPE_BF16
        else:
            self.Xd = torch.from_numpy(self.X).to(dev)
            xdt = L.DTYPE_F32
        self.W0d = torch.from_numpy(self.W0).to(dev)
        self.Md = torch.from_numpy(self.mask).to(dev)
        self.V0d = torch.from_numpy(self.V0).to(dev)
        d, C, N = cfg.d, cfg.n_cols, cfg.n_tok
        self.H = torch.empty((d, d), dtype=torch.float32, device=dev)
        self.lam = torch.empty(1, dtype=torch.float32, device=dev)
        self.lmax = torch.empty(1, dtype=torch.float32, device=dev)
        self.Wout = torch.empty_like(self.W0d)
        self.hws = torch.empty(max(L.optima_hessian_workspace_bytes(N, d, xdt), 1),
                               dtype=torch.uint8, device=dev)
        self.sws = torch.empty(L.optima_spectral_norm_workspace_bytes(d, SPECTRAL_BLOCK),
                               dtype=torch.uint8, device=dev)
        self.qws = torch.empty(L.optima_qp_workspace_bytes(d, C), dtype=torch.uint8, device=dev)
        self.stats = {"iters": torch.zeros(C, dtype=torch.int32, device=dev),
                      "converged": torch.zeros(C, dtype=torch.uint8, device=dev),
                      "f_initial": torch.zeros(C, dtype=torch.float32, device=dev),
                      "f_final": torch.zeros(C, dtype=torch.float32, device=dev)}
        self.opts = opts
        self.policy = spectral_policy
        self.spectral = None

    def step(self):
        """Returns (events, solve info); events bracket Hessian, damping +
        step size and solve on the current stream."""
        L, torch = self.L, self.torch
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record()
        L.optima_hessian_accumulate(self.Xd, self.H, accumulate=False, ws=self.hws)
        ev[1].record()
        L.optima_hessian_damp(self.H, self.cfg.rel_damp, self.lam)
        if self.policy:
            from paper_2512_13886_amd.pipeline import spectral_step_size
            self.spectral = spectral_step_size(self.H, self.V0d, self.lmax)
        else:
            L.optima_spectral_norm(self.H, self.V0d, self.lmax, max_iters=1000, tol=1e-6,
                                   ws=self.sws)
        ev[2].record()
        info = L.optima_qp_solve_batched(self.H, self.lmax, self.W0d, self.Md, self.Wout,
                                         opts=self.opts, ws=self.qws, stats=self.stats)
        ev[3].record()
        return ev, info

    def fixed_batch(self, iters: int, prec: int, prec_name: str) -> dict:
        """All columns for a fixed number of iterations: the iteration rate at
        B = C (checks still restart, no column leaves)."""
        L, torch = self.L, self.torch
        C, d = self.cfg.n_cols, self.cfg.d
        fixed = L.SolverOpts.default(max_iters=iters, fixed_iters=1, precision=prec)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        finfo = L.optima_qp_solve_batched(self.H, self.lmax, self.W0d, self.Md, self.Wout,
                                          opts=fixed, ws=self.qws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        roof = product_roofline(d, [finfo], prec_name)
        return {"iters": iters, "columns": C, "ms": ms,
                "iters_per_s": iters / (ms * 1e-3),
                "column_iters_per_s": iters * C / (ms * 1e-3),
                "product_tflops": roof.get("achieved"),
                "product_frac": roof.get("frac"),
                "product_avg_launch_us": roof.get("avg_launch_us"),
                "product_kernel": roof.get("kernel")}

    def release(self):
        for k in ("Xd", "W0d", "Md", "V0d", "H", "Wout", "hws", "sws", "qws", "stats"):
            setattr(self, k, None)
        self.torch.cuda.empty_cache()


def summarize_steps(run: LayerRun, recs: list, prec_name: str, wall_ms_per_step=None,
                    traffic=None, few_traffic=None) -> dict:
    """Per-configuration figures of the timed steps of one layer."""
    cfg = run.cfg
    d, C, N = cfg.d, cfg.n_cols, cfg.n_tok
    hess = [e[0].elapsed_time(e[1]) for e, _ in recs]
    spec = [e[1].elapsed_time(e[2]) for e, _ in recs]
    solve = [e[2].elapsed_time(e[3]) for e, _ in recs]
    total = [e[0].elapsed_time(e[3]) for e, _ in recs]
    it = run.stats["iters"].cpu().numpy()
    step_ms = float(np.median(total))
    solve_ms = float(np.median(solve))
    out = {
        "d": d, "n_cols": C, "n_tok": N, "x_dtype": cfg.x_dtype,
        "mask": cfg.mask_kind if cfg.mask_kind == "2:4" else
        f"{int(round(cfg.sparsity * 100))}% unstructured",
        "steps": len(recs),
        "step_ms": step_ms,
        "columns_per_s": C / (step_ms * 1e-3),
        "phase_ms": {"hessian": float(np.median(hess)), "damp_spectral": float(np.median(spec)),
                     "solve": solve_ms},
        "solve_columns_per_s": C / (solve_ms * 1e-3),
        "hessian_tflops": 2.0 * N * d * d / 2 / (float(np.median(hess)) * 1e-3) / 1e12,
        "iterations_longest_column": int(it.max()),
        "mean_iterations_per_column": float(it.mean()),
        "start_check_fraction": float(np.mean(it == 0)),
        "converged": int(run.stats["converged"].sum().item()),
        "column_iters_per_s": float(it.sum()) / (solve_ms * 1e-3),
        "loop_passes_per_s": float(it.max()) / (solve_ms * 1e-3),
        "f_final_over_f_initial": float(run.stats["f_final"].double().sum()
                                        / run.stats["f_initial"].double().sum()),
        "roofline": product_roofline(d, [i for _, i in recs], prec_name, traffic, few_traffic),
    }
    if run.spectral is not None:
        out["spectral"] = run.spectral
    if wall_ms_per_step is not None:
        out["wall_ms_per_step"] = wall_ms_per_step
    return out


def config_leg(L, torch, dev, name, fixed_iters, steps, opts, prec, prec_name) -> dict:
    """One synthetic layer of another configuration: the same step (policy
    step size), 1 warm-up and `steps` timed steps, then the fixed-batch leg."""
    import workloads
    cfg = workloads.CONFIGS[name]
    torch.cuda.reset_peak_memory_stats(dev)
    run = LayerRun(L, torch, dev, cfg, opts, spectral_policy=True)
    torch.cuda.synchronize()
    run.step()
    torch.cuda.synchronize()
    recs = [run.step() for _ in range(steps)]
    torch.cuda.synchronize()
    out = summarize_steps(run, recs, prec_name)
    out["inputs_generated_s"] = run.gen_s
    out["fixed_batch"] = run.fixed_batch(fixed_iters, prec, prec_name)
    out["peak_device_memory_gib"] = torch.cuda.max_memory_allocated(dev) / 2**30
    log(f"{name}: step {out['step_ms']:.2f} ms ({out['columns_per_s']:.0f} columns/s), hessian "
        f"{out['phase_ms']['hessian']:.2f} ms, solve {out['phase_ms']['solve']:.2f} ms "
        f"({out['iterations_longest_column']} iterations, start-check fraction "
        f"{out['start_check_fraction']:.3f}); product "
        f"{out['roofline'].get('achieved', 0.0):.1f} TFLOP/s; fixed batch "
        f"{out['fixed_batch']['iters_per_s']:.0f} it/s")
    run.release()
    return out


def block_leg(L, torch, dev, opts, prec_name) -> dict:
    """The streamed decoder block (Llama-3-8B shapes): for each calibration
    stream the Hessian, the Wanda masks of its matrices (from the undamped
    Hessian's diagonal, on the device), damping, the step size and the paper-
    mode solves. Tokens and weights are moved to the device before timing;
    the reported time is the device time of all of that work. The step size
    comes from the block iteration, or from Lanczos where the block iteration
    has not converged within a few passes (spectral_step_size)."""
    import workloads
    from paper_2512_13886_amd.pipeline import spectral_step_size
    torch.cuda.reset_peak_memory_stats(dev)
    total_ms = 0.0
    layers = {}
    streams = {}
    gen_s = 0.0
    hess_flops = 0.0
    hess_ms = 0.0
    for sname, scfg in workloads.BLOCK_STREAMS.items():
        mats = [lc for lc, st in workloads.BLOCK_LAYERS if st == sname]
        t0 = time.perf_counter()
        X = workloads.x_all(scfg)
        W0h = [workloads.w0(lc) for lc in mats]
        gen_s += time.perf_counter() - t0
        Xd = torch.from_numpy(X.view(np.int16)).view(torch.bfloat16).to(dev)
        del X
        d = scfg.d
        W0s = [torch.from_numpy(w).to(dev) for w in W0h]
        del W0h
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
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4 + len(mats))]
        ev[0].record()
        L.optima_hessian_accumulate(Xd, H, ws=hws)
        ev[1].record()
        for lc, W0d, M in zip(mats, W0s, masks):
            L.optima_wanda_mask(W0d, H, M, L.MASK_UNSTRUCTURED, lc.sparsity, col_sq_stride=d + 1)
        ev[2].record()
        L.optima_hessian_damp(H, scfg.rel_damp, lam)
        spec = spectral_step_size(H, V0, lmax)
        ev[3].record()
        infos = []
        for i, (lc, W0d, M, out, st) in enumerate(zip(mats, W0s, masks, outs, stats)):
            infos.append(L.optima_qp_solve_batched(H, lmax, W0d, M, out, opts=opts, stats=st))
            ev[4 + i].record()
        torch.cuda.synchronize()
        s_ms = ev[0].elapsed_time(ev[-1])
        total_ms += s_ms
        h_ms = ev[0].elapsed_time(ev[1])
        hess_ms += h_ms
        hess_flops += float(scfg.n_tok) * d * d
        streams[sname] = {"d": d, "hessian_ms": h_ms,
                          "hessian_tflops": float(scfg.n_tok) * d * d / (h_ms * 1e-3) / 1e12,
                          "masks_ms": ev[1].elapsed_time(ev[2]),
                          "damp_spectral_ms": ev[2].elapsed_time(ev[3]),
                          "spectral": spec, "ms": s_ms}
        prev = ev[3]
        for i, (lc, st, inf) in enumerate(zip(mats, stats, infos)):
            it = st["iters"].cpu().numpy()
            sm = prev.elapsed_time(ev[4 + i])
            layers[lc.name[len("block_"):]] = {
                "d": d, "columns": lc.n_cols, "solve_ms": sm,
                "solve_columns_per_s": lc.n_cols / (sm * 1e-3),
                "iterations": inf["iterations"],
                "start_check_fraction": float(np.mean(it == 0)),
                "converged": int(st["converged"].sum().item()),
                "f_final_over_f_initial":
                    (st["f_final"].double().sum() / st["f_initial"].double().sum()).item(),
                "roofline": product_roofline(d, [inf], prec_name)}
            prev = ev[4 + i]
        log(f"block stream {sname}: {s_ms:.1f} ms (step size: {spec['method']}, "
            f"{spec['block_passes']} block passes, {spec['lanczos_steps']} Lanczos steps)")
        del Xd, H, hws, W0s, outs, masks, stats
        torch.cuda.empty_cache()
    cols = sum(v["columns"] for v in layers.values())
    return {"block_prune_ms": total_ms, "columns": cols,
            "columns_per_s": cols / (total_ms * 1e-3),
            "hessian_tflops": hess_flops / (hess_ms * 1e-3) / 1e12,
            "inputs_generated_s": gen_s,
            "peak_device_memory_gib": torch.cuda.max_memory_allocated(dev) / 2**30,
            "streams": streams, "layers": layers}


def chain_leg(L, torch, dev, opts) -> dict:
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


def read_phase_stamps(L):
    """Stamps of the instrumented library since the last call: tile-product
    rows (start, end of main loop, end, block | mode << 32 | rows << 40) and
    the cooperative launch's [4][256][6] per-iteration stamps."""
    import ctypes
    fn = ctypes.CDLL(L.library_path()).optima_phase_stamps
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    tile = np.zeros((1 << 16, 4), np.uint64)
    coop = np.zeros((4, 256, 6), np.uint64)
    n = fn(tile.ctypes.data, tile.shape[0], coop.ctypes.data)
    if n < 0:
        raise RuntimeError("optima_phase_stamps failed")
    return tile[:n].astype(np.int64), coop.astype(np.int64)


def summarize_phase_stamps(tile, coop) -> dict:
    """Per-launch phases of the 2:4 tile product over more than 8 active
    columns (fused update launches) and per-iteration phases of the last
    cooperative launch, in microseconds (the stamps count at 100 MHz)."""
    us = 0.01
    out = {}
    if len(tile):
        order = np.argsort(tile[:, 0])
        t = tile[order]
        mode = (t[:, 3] >> 32) & 0xff
        rows = t[:, 3] >> 40
        starts = np.where(np.diff(t[:, 0]) > 2000)[0] + 1  # launches start >20 us apart
        groups = np.split(np.arange(len(t)), starts)
        spans, loops, loop_max, epis, epi_max, gaps = [], [], [], [], [], []
        prev_end = None
        for g in groups:
            begin, end = t[g, 0].min(), t[g, 2].max()
            if mode[g[0]] == 3 and rows[g[0]] > 8:
                spans.append((end - begin) * us)
                loops.append(((t[g, 1] - t[g, 0]) * us).mean())
                loop_max.append(((t[g, 1] - t[g, 0]) * us).max())
                epis.append(((t[g, 2] - t[g, 1]) * us).mean())
                epi_max.append(((t[g, 2] - t[g, 1]) * us).max())
                if prev_end is not None:
                    gaps.append((begin - prev_end) * us)
            prev_end = end
        if spans:
            out["tile_fused"] = {
                "launches": len(spans), "span_us": float(np.mean(spans)),
                "main_loop_us": float(np.mean(loops)), "main_loop_max_us": float(np.mean(loop_max)),
                "epilogue_us": float(np.mean(epis)), "epilogue_max_us": float(np.mean(epi_max)),
                "gap_before_us_median": float(np.median(gaps)) if gaps else None}
    n_iter = int(coop[0, 0, 5])
    if n_iter > 1:
        c = coop[:, :n_iter - 1, :5] * us
        d = np.diff(c, axis=2)
        per = np.diff(c[:, :, 0], axis=1)
        out["cooperative"] = {
            "iterations": n_iter, "product_us": float(d[:, :, 0].mean()),
            "reduction_us": float(d[:, :, 1].mean()), "update_us": float(d[:, :, 2].mean()),
            "barrier_us": float(d[:, :, 3].mean()), "iteration_us": float(per.mean())}
    return out


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
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the tiny, GPT-2 fc and down_proj layers")
    ap.add_argument("--no-block", action="store_true",
                    help="skip the streamed Llama-3-8B-shaped decoder block (7 matrices, "
                         "4 calibration streams)")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the CG, Jacobi-preconditioned and mask-selection legs")
    ap.add_argument("--chain-config", action="store_true",
                    help="also run the layer loop of Algorithm 1 on a chain of four 4096 x 4096 "
                         "layers (forward propagation of the pruned activations, skip rule, "
                         "layer-wise error ratios)")
    ap.add_argument("--no-cooperative", action="store_true",
                    help="run the few-column iterations one launch per iteration instead of one "
                         "cooperative launch per block (rocprofv3 counter collection ends the "
                         "process with a crash after a cooperative launch)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="first run one 256 MiB device copy (reference for HBM byte counters)")
    ap.add_argument("--phase-stamps", action="store_true",
                    help="load the instrumented library (paper_2512_13886_amd/build.py phases) and "
                         "report the phases of the timed steps' sparse iteration products from its "
                         "clock stamps (the stamps add a little time to every product)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        log("bench.py measures one MI355X only: the library runs the hot path on a single GPU "
            "(columns would shard across GPUs with no per-iteration communication). "
            "Run it with --gpus 1.")
        return 2

    if args.phase_stamps:
        lib = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2512_13886_amd",
                           "liboptima_phases.so")
        if not os.path.exists(lib):
            log(f"--phase-stamps needs {lib}: run python paper_2512_13886_amd/build.py phases")
            return 1
        os.environ["OPTIMA_LIBRARY"] = lib
    import torch
    import paper_2512_13886_amd as L
    from paper_2512_13886_amd.pipeline import spectral_step_size
    import workloads

    dev = torch.device("cuda:0")
    torch.cuda.init()
    torch.cuda.set_device(dev)
    if args.calibration_copy:
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    # Table 8: tol 0.01 / 0.01, 100000 iterations
    opts = L.SolverOpts.default()
    if args.no_cooperative:
        opts.cooperative = 0
    if args.precision is not None:
        opts.precision = {"fp32": L.PREC_FP32, "bf16x3": L.PREC_BF16X3}[args.precision]
    prec = opts.precision
    prec_name = "bf16x3" if prec == L.PREC_BF16X3 else "fp32"

    cfg = workloads.Q_PROJ
    torch.cuda.reset_peak_memory_stats(dev)
    run = LayerRun(L, torch, dev, cfg, opts, spectral_policy=False)
    log(f"inputs generated in {run.gen_s:.1f} s")
    d, C, N = cfg.d, cfg.n_cols, cfg.n_tok
    H, lmax, W0d, Md, Wout, qws = run.H, run.lmax, run.W0d, run.Md, run.Wout, run.qws
    iters, conv = run.stats["iters"], run.stats["converged"]
    f_init, f_fin = run.stats["f_initial"], run.stats["f_final"]
    torch.cuda.synchronize()

    for w in range(args.warmup):
        run.step()
        torch.cuda.synchronize()
        log(f"warmup step {w + 1}/{args.warmup} done")

    torch.cuda.synchronize()
    if args.phase_stamps:
        read_phase_stamps(L)  # drop the warm-up steps' stamps
    t0 = time.perf_counter()
    recs = [run.step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    phases = summarize_phase_stamps(*read_phase_stamps(L)) if args.phase_stamps else None
    if phases:
        log(f"phase stamps: {json.dumps(phases)}")

    ms_step = wall * 1000.0 / args.steps
    hess_ms = np.mean([e[0].elapsed_time(e[1]) for e, _ in recs])
    spec_ms = np.mean([e[1].elapsed_time(e[2]) for e, _ in recs])
    solve_ms = np.mean([e[2].elapsed_time(e[3]) for e, _ in recs])
    solve_ms_median = float(np.median([e[2].elapsed_time(e[3]) for e, _ in recs]))
    it = np.mean([i["iterations"] for _, i in recs])
    per_col_it = iters.cpu().numpy()
    f_ratio_rapdhg = float(f_fin.double().sum() / f_init.double().sum())
    log(f"step {ms_step:.1f} ms: hessian {hess_ms:.2f} ms, damp+spectral {spec_ms:.2f} ms, "
        f"solve {solve_ms:.1f} ms ({it:.0f} iterations, {conv.sum().item()}/{C} converged, "
        f"per-column iterations {per_col_it.min()}..{per_col_it.max()}, "
        f"{np.mean(per_col_it == 0):.1%} stop at the start check)")

    traffic = few_traffic = None  # the counter passes were taken on the bf16x3 kernels
    if (TRAFFIC and prec == L.PREC_BF16X3
            and TRAFFIC.get("sources_sha1") == kernel_sources_sha1()):
        traffic = TRAFFIC["bytes_per_launch"]
        few_traffic = TRAFFIC.get("few_bytes_per_launch")
    qproj = summarize_steps(run, recs, prec_name, wall_ms_per_step=ms_step, traffic=traffic,
                            few_traffic=few_traffic)
    roofline = dict(qproj["roofline"])
    log(f"H-product (tiles): {roofline.get('launches')} launches, avg "
        f"{roofline.get('avg_launch_us', 0.0):.1f} us, {roofline.get('achieved', 0.0):.1f} "
        f"TFLOP/s (frac {roofline.get('frac', 0.0):.3f}); few-column: "
        f"{roofline.get('few_column_kernel', {}).get('avg_launch_us', 0.0):.1f} us per launch")

    # Full-batch leg: all 4096 columns for a fixed number of iterations, the
    # iteration rate at B = C (not part of the timed step).
    fixed_batch = None
    if args.fixed_iters > 0:
        fixed_batch = run.fixed_batch(args.fixed_iters, prec, prec_name)
        log(f"fixed {args.fixed_iters} iterations x {C} columns: {fixed_batch['ms']:.1f} ms "
            f"({fixed_batch['iters_per_s']:.0f} it/s), H-product "
            f"{fixed_batch['product_tflops']:.1f} TFLOP/s, avg launch "
            f"{fixed_batch['product_avg_launch_us']:.1f} us")
    qproj["fixed_batch"] = fixed_batch

    extras = {}
    if not args.no_extras:
        # Unconstrained-form leg (Eq. (7)-(11)): conjugate gradients on the
        # same layer and H at the same tolerances, tested every 8 iterations;
        # no step size is needed. Not part of the timed step.
        cg_opts = L.SolverOpts.default(method=L.METHOD_CG, check_every=8)
        if args.precision is not None:
            cg_opts.precision = prec
        cg_ms, cg_it = [], []
        for rep in range(4):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            cinfo = L.optima_qp_solve_batched(H, None, W0d, Md, Wout, opts=cg_opts, ws=qws,
                                              stats=run.stats)
            b.record()
            torch.cuda.synchronize()
            if rep:  # the first run is a warm-up
                cg_ms.append(a.elapsed_time(b))
                cg_it.append(cinfo["iterations"])
        cg_solve_ms = float(np.mean(cg_ms))
        extras["cg_unconstrained"] = {
            "solve_ms": cg_solve_ms, "iterations": float(np.mean(cg_it)), "check_every": 8,
            "converged": int(conv.sum().item()),
            "columns_per_s_solve_only": C / (cg_solve_ms * 1e-3),
            "step_ms_equivalent": hess_ms + cg_solve_ms,
            "columns_per_s_step_equivalent": C / ((hess_ms + cg_solve_ms) * 1e-3),
            "f_final_over_f_initial": float(f_fin.double().sum() / f_init.double().sum()),
            "rapdhg_f_final_over_f_initial": f_ratio_rapdhg}
        cgl = extras["cg_unconstrained"]
        log(f"cg: solve {cg_solve_ms:.2f} ms ({cgl['iterations']:.0f} iterations, "
            f"{cgl['converged']}/{C} converged); sum f_final / sum f_initial "
            f"cg {cgl['f_final_over_f_initial']:.4f}, rapdhg {f_ratio_rapdhg:.4f}")

        # Preconditioned leg: Jacobi scaling of (a copy of) H, the spectral
        # norm of D H D and both solvers with the column scaling, at the
        # paper's tolerances and at a tight one (eps_rel 1e-4, eps_abs 0)
        # beside the unscaled solves. Not part of the timed step.
        Hs = torch.empty_like(H)
        Hs.copy_(H)
        Ds = torch.empty(d, dtype=torch.float32, device=dev)
        lmax_s = torch.empty(1, dtype=torch.float32, device=dev)

        def timed_solve(Hm, lm, o):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            inf = L.optima_qp_solve_batched(Hm, lm, W0d, Md, Wout, opts=o, ws=qws,
                                            stats=run.stats)
            b.record()
            torch.cuda.synchronize()
            return {"ms": a.elapsed_time(b), "iterations": inf["iterations"],
                    "converged": int(conv.sum().item()),
                    "f_final_over_f_initial": (f_fin.double().sum()
                                               / f_init.double().sum()).item()}

        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record()
        L.optima_hessian_jacobi(Hs, Ds)
        e[1].record()
        spec_s = spectral_step_size(Hs, run.V0d, lmax_s)
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
        del Hs
        extras["jacobi_preconditioned"] = pre
        tt = pre["tight_tolerance_eps_rel_1e-4"]
        log(f"jacobi-preconditioned: scale {pre['scale_ms']:.2f} ms, spectral "
            f"{pre['spectral_ms']:.2f} ms ({spec_s['method']}: {spec_s['block_passes']} block "
            f"passes, {spec_s['lanczos_steps']} Lanczos steps); tight: rapdhg "
            f"{tt['rapdhg']['iterations']} -> {tt['rapdhg_scaled']['iterations']} it "
            f"({tt['rapdhg']['ms']:.1f} -> {tt['rapdhg_scaled']['ms']:.1f} ms), cg "
            f"{tt['cg']['iterations']} -> {tt['cg_scaled']['iterations']} it "
            f"({tt['cg']['ms']:.1f} -> {tt['cg_scaled']['ms']:.1f} ms)")

        # Device mask selection (the selector ahead of the update; not part
        # of the step, whose mask is an input): both patterns on this layer's
        # W0 and fp64 column norms, 5 launches each.
        csd = torch.from_numpy(run.col_sq).to(dev)
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
        extras["mask_select"] = {"two_four_ms": m24_ms, "unstructured_50_ms": mun_ms,
                                 "two_four_gbps": mask_bytes / (m24_ms * 1e-3) / 1e9,
                                 "unstructured_gbps": mask_bytes / (mun_ms * 1e-3) / 1e9,
                                 "algorithmic_bytes_per_element": 5,
                                 "two_four_equals_host_mask": m24_same}
        log(f"mask selection: 2:4 {m24_ms * 1e3:.1f} us, unstructured {mun_ms * 1e3:.1f} us, "
            f"2:4 equals the host mask: {m24_same}")
        del csd, md
    qproj["peak_device_memory_gib"] = torch.cuda.max_memory_allocated(dev) / 2**30

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        H_host = H.cpu().numpy().astype(np.float64)
        lam_host = float(lmax.item())
        cpu = cpu_baseline(cfg, run.X, run.W0, run.mask, H_host, lam_host,
                           args.cpu_sample_cols, args.cpu_sample_chunks)
        del H_host
    run.release()

    configs = {"q_proj": qproj}
    if not args.no_configs:
        for name, fixed_iters, steps in CONFIG_LEGS:
            configs[name] = config_leg(L, torch, dev, name, fixed_iters, steps, opts, prec,
                                       prec_name)
    configs = {k: configs[k] for k in ("tiny", "gpt2_fc", "q_proj", "down_proj")
               if k in configs}

    block = None
    if not args.no_block:
        block = block_leg(L, torch, dev, opts, prec_name)
        log(f"block prune: {block['block_prune_ms']:.1f} ms for {block['columns']} columns "
            f"({block['columns_per_s']:.0f} columns/s)")

    chain = None
    if args.chain_config:
        chain = chain_leg(L, torch, dev, opts)
        log(f"chain: {chain['device_ms']:.1f} ms device time for {len(chain['layers'])} layers")

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
        # The solver's iteration rate at B = C: all 4096 columns, a fixed
        # number of iterations (null when --fixed-iters 0).
        "rapdhg_iters_per_s": fixed_batch["iters_per_s"] if fixed_batch else None,
        "rapdhg_iters_per_s_batch_columns": C if fixed_batch else None,
        # The timed paper-mode solves, where the batch shrinks as columns stop.
        "paper_mode": {
            "loop_passes_per_s": float(it) / (solve_ms * 1e-3),
            "column_iters_per_s": qproj["column_iters_per_s"],
            "iterations_longest_column": qproj["iterations_longest_column"],
            "mean_iterations_per_column": qproj["mean_iterations_per_column"],
            "start_check_fraction": qproj["start_check_fraction"],
            "converged": qproj["converged"],
            "f_final_over_f_initial": f_ratio_rapdhg,
        },
        "phase_ms": {"hessian": hess_ms, "damp_spectral": spec_ms, "solve": solve_ms},
        "solve_only": {"solve_ms_median": solve_ms_median, "runs": args.steps,
                       "columns_per_s": C / (solve_ms_median * 1e-3)},
        "hessian_tflops": 2.0 * N * d * d / 2 / (hess_ms * 1e-3) / 1e12,
        "hessian_roofline": hessian_roofline(N, d, hess_ms),
        "fixed_batch": fixed_batch,
        "configs": configs,
        "decoder_block": block,
        "layer_chain": chain,
        "peak_device_memory_gib": qproj["peak_device_memory_gib"],
        "roofline": roofline,
    }
    out.update(extras)
    if phases is not None:
        out["phase_stamps"] = phases
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
