"""Benchmark: GP + EI candidates scored per second on one MI355X.

One step is one pass of the whole hot path over one batch: gp_fit on the n observed
configurations (encode, fp64 Gram, Cholesky, triangular inverse, alpha, K^-1, Laplace
probit classifier) followed by gp_score of the M candidates (encode, fp32 cross-kernel,
variance contraction on fp16 MFMA over high/low-split operands, EI/feasibility epilogue,
fp64 recomputation of ill-conditioned candidates, arg-max). Inputs are resident in HBM
before timing.

Prints one JSON line. The default workload is the FPGA-pragma-shaped space
(d = 20, n = 512 observations, 30% infeasible, M = 1,048,576 candidates).
"""
import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP64_PEAK_TFLOPS = 78.6        # MI355X dense fp64 (matrix and vector)
FP32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense fp32 matrix
FP16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 matrix
SPLIT_PRODUCTS = 3              # fp16 MFMA products per fp32-accurate multiply-add
HBM_PEAK_GBS = 8000.0           # MI355X HBM3E

WORKLOAD_TEXT = {
    "C1": "tiny mixed space d=5 (2 real, int, log2 ordinal, categorical)",
    "C2": "sparse-tensor-schedule space d=6 (ordinals, categorical, ints, Kendall permutation m=5)",
    "C3": "GPU-tile space d=10 log2 ordinals, known-constraint mask, 30% hidden-infeasible",
    "C4": "FPGA-pragma space d=20 (12 binary categorical, 6 log2 ordinal, 2 int), 30% infeasible",
    "C5": "stress space d=12 (6 ordinal, 2 real, 2 categorical, Spearman and Hamming permutations m=7)",
}


# Measured HBM traffic of a kernel: a JSON record under profiles/ with the rocprofv3
# FETCH_SIZE / WRITE_SIZE per dispatch, the factors that scale them to bytes (from a plain
# copy of known size) and the SHA-256 of the sources the kernel is built from. The figure
# is used only while those sources are unchanged.
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "contract_split_c4_counters.json")


def sources_digest(paths):
    h = hashlib.sha256()
    for rel in paths:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(record_path, workload):
    """HBM bytes of the contraction per step (all its launches) from the counter record,
    or None if there is no record for this workload or the kernel's sources changed
    since the counters were taken."""
    try:
        with open(record_path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None, "no counter record"
    if rec.get("workload") != workload:
        return None, f"counters were taken on {rec.get('workload')}"
    if sources_digest(rec["sources"]) != rec["sources_sha256"]:
        return None, "kernel sources changed since the counters were taken"
    fetch = rec["fetch_kib_per_step"] * 1024 * rec["fetch_scale"]
    write = rec["write_kib_per_step"] * 1024 * rec["write_scale"]
    return fetch + write, "rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated"


def calibrate_copy():
    """A plain device copy of 1 GiB, three times: the reference that scales FETCH_SIZE and
    WRITE_SIZE to bytes (profile this mode with one counter per run)."""
    import torch
    a = torch.empty(256 * 1024 * 1024, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1.0)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes_read": a.numel() * 4, "calibrate_copy_bytes_written":
                      b.numel() * 4, "copies": 3}), flush=True)


def contraction_flops_per_candidate(n, n_f, has_cls):
    """Algorithmic flops of the variance contraction for one candidate, the method's
    work counted once: the triangular product L_f^-1 k* (sum_{j<n_f} (j+1)
    multiply-adds), its squared norm and the mean k*.alpha (n_f(n_f+1) + 4 n_f), and the
    same for the classifier's n x n triangular factor with its latent mean
    (n(n+1) + 4n). C4 (n = 512, n_f = 359): 395,380."""
    f = n_f * (n_f + 1) + 4 * n_f
    if has_cls:
        f += n * (n + 1) + 4 * n
    return f


def contraction_executed_flops(model_tiles, M_rows):
    """MFMA flops the contraction issues: per 16-column sub-tile, k runs to the end of
    its triangle (or the tile's k-length), the sub-tile of a linear column to the
    tile's k-length; all-padding sub-tiles issue nothing."""
    per_rowblock = 0.0
    for kend, tri0, ncol, lin in model_tiles:
        for c in range(0, 128, 16):
            if lin >= 0 and c == lin // 16 * 16:
                per_rowblock += 2.0 * 128 * 16 * kend
            elif c < ncol:
                per_rowblock += 2.0 * 128 * 16 * min(kend, tri0 + c + 16)
    return per_rowblock * (M_rows / 128.0)


def cpu_baseline(w, sample):
    """The oracle as it stands, timed on this host: fit once, score `sample` candidates
    (all M by default), extrapolated linearly in the candidate count to the workload's M
    when the sample is smaller."""
    from oracle import gp_oracle as go
    try:
        from threadpoolctl import threadpool_info
        cores = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    t0 = time.perf_counter()
    om = go.fit(w.space, w.X, w.y, w.feasible, w.lengthscale, w.signal_var, w.noise_var,
                w.cls_signal_var)
    t1 = time.perf_counter()
    C = [c[:sample] for c in w.C]
    mask = None if w.mask is None else w.mask[:sample]
    go.score(om, C, mask, w.eps_f)
    t2 = time.perf_counter()
    t_step = (t1 - t0) + (t2 - t1) * (w.M / sample)
    return {"value": w.M / t_step, "unit": "candidates/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"fit on all n={w.n} observations ({t1 - t0:.2f} s) + score of all "
                       f"{w.M} candidates ({t2 - t1:.2f} s), no extrapolation"
                       if sample >= w.M else
                       f"fit on all n={w.n} observations ({t1 - t0:.2f} s) + score of the first "
                       f"{sample} of {w.M} candidates ({t2 - t1:.2f} s), extrapolated linearly to M"),
            "fit_s": t1 - t0, "score_sample_s": t2 - t1}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="C4", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--cpu-sample", type=int, default=0,
                    help="candidates the oracle scores for the CPU baseline (0: all M)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--unfused", action="store_true",
                    help="time gp_fit then gp_score instead of the fused gp_fit_score")
    ap.add_argument("--score-only-steps", type=int, default=0,
                    help="extra: also time this many gp_score calls alone (profiling aid)")
    ap.add_argument("--ls-starts", type=int, default=16,
                    help="extra: starts of the timed local search (0: skip it)")
    ap.add_argument("--ls-max-steps", type=int, default=200)
    ap.add_argument("--hyper-samples", type=int, default=256,
                    help="extra: samples of the timed hyperparameter fit (0: skip it)")
    ap.add_argument("--hyper-starts", type=int, default=8)
    ap.add_argument("--forest-trees", type=int, default=64,
                    help="extra: trees of the timed random-forest feasibility model (0: skip)")
    ap.add_argument("--cot-m", type=int, default=1 << 20,
                    help="extra: configurations of the timed Chain-of-Trees draw (0: skip it)")
    ap.add_argument("--other-workloads", default="C2,C3,C5",
                    help="extra: the fused step on these other full-size workloads "
                         "(comma-separated; empty to skip)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run the 1 GiB device copy that calibrates the HBM counters")
    args = ap.parse_args()
    if args.calibrate_copy:
        calibrate_copy()
        return

    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build runs the scorer on a single MI355X "
              f"(--gpus {args.gpus} is not supported; candidates would be sharded over GPUs "
              f"with a replicated model, see the design notes)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2212_11142_amd import gp
    from workloads import make_workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    gp.load()
    w = make_workload(args.workload)
    space = gp.Space(w.space)
    X = gp.to_device_columns(space, w.X)
    Cc = gp.to_device_columns(space, w.C)
    y = torch.from_numpy(np.nan_to_num(w.y, nan=0.0)).cuda()
    feas = torch.from_numpy(w.feasible).cuda()
    mask = torch.from_numpy(w.mask).cuda() if w.mask is not None else None

    def fit():
        return gp.fit(space, X, y, feas, w.lengthscale, w.signal_var, w.noise_var,
                      w.cls_signal_var)

    model = fit()
    bufs = gp.ScoreBuffers(model, w.M, want_p=True, want_argmax=True)
    fbufs = gp.FitScoreBuffers(space, len(w.y), w.M, w.cls_signal_var is not None,
                               want_p=True, want_argmax=True)

    def step():
        if args.unfused:
            m = fit()
            gp.score_into(m, Cc, bufs, mask, w.eps_f)
            return m
        # the fit, overlapped with the encoding and cross-kernel of the candidates
        return gp.fit_score_into(space, X, y, feas, w.lengthscale, w.signal_var, w.noise_var,
                                 w.cls_signal_var, Cc, fbufs, mask, w.eps_f)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # stage breakdown of the timed steps: HIP events recorded by the library on the
    # streams its scoring stages run on (the fit is timed alone below)
    gp.profile_start()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        keep = step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    prof = gp.profile_stop()
    calls = max(prof["calls"], 1)
    stage_ms = {s: prof[s] / calls for s in gp.STAGES}
    score_ms = sum(stage_ms.values())
    refined = gp.refined_count(keep, bufs if args.unfused else fbufs)

    torch.cuda.synchronize()
    tf0 = time.perf_counter()
    for _ in range(args.steps):
        fit()
    torch.cuda.synchronize()
    fit_ms = (time.perf_counter() - tf0) * 1e3 / args.steps

    info = keep.info()
    n, n_f, M = info["n"], info["n_feasible"], w.M
    has_cls = bool(info["has_classifier"])
    f_cand = contraction_flops_per_candidate(n, n_f, has_cls)
    alg_flops = f_cand * M
    t_con = stage_ms["contract"] * 1e-3
    # achieved: the method's flops (each multiply-add counted once) per second of the
    # contraction, against the peak of the unit it runs on (dense fp16 MFMA). It forms
    # each fp32-accurate product from three fp16 MFMA products (high x high, high x low,
    # low x high), so at most a third of that peak is reachable; the fp16 work it
    # issues is reported on its own.
    achieved_tf = alg_flops / t_con / 1e12
    kends = [t for t in keep_tiles(keep, not args.unfused)]
    exec_tf = SPLIT_PRODUCTS * contraction_executed_flops(kends, math.ceil(M / 128) * 128) / t_con / 1e12
    # contraction: K* read once (4 n bytes per candidate: fp16 high + low parts) + partial
    # sums written
    alg_bytes_contract = M * (4 * n + 4 * len(kends) + (4 if has_cls else 0))
    # a fused step contracts the value model's column tiles and the classifier's in two
    # launches (the first beside the classifier's fit)
    launches = 1 if args.unfused or not has_cls else 2
    traffic, traffic_note = measured_traffic(TRAFFIC_RECORD, args.workload)
    # cross-kernel: algorithmic bytes = K* row write (4 n) + encoded candidate read (4 R)
    xk_bytes = M * (4 * n + 4 * info["code_words"])
    xk_gbs = xk_bytes / (stage_ms["xkernel"] * 1e-3) / 1e9

    line = {
        "metric": "GP+EI candidates scored/sec (n=512, M=1M) + % HBM/MFMA peak",
        "value": M / (ms_step * 1e-3),
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32 scoring (split-fp16 MFMA contraction) / fp64 fit",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {WORKLOAD_TEXT[args.workload]}", "n": n,
                   "n_feasible": n_f, "M": M, "d": len(w.space), "classifier": has_cls,
                   "step": "gp_fit then gp_score" if args.unfused else
                           "gp_fit_score (fit overlapped with the first half of scoring)"},
        "roofline": {"kernel": "contract_split (variance contraction, fp16 MFMA on high/low split operands)",
                     "bound": "mfma", "achieved": achieved_tf, "peak": FP16_MFMA_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved_tf / FP16_MFMA_PEAK_TFLOPS,
                     "traffic": traffic, "traffic_unit": "bytes per step (all launches)",
                     "traffic_source": traffic_note,
                     "launches_per_step": launches,
                     "algorithmic_bytes_per_step": alg_bytes_contract,
                     "algorithmic_flops_per_candidate": f_cand,
                     "algorithmic_flops_per_step": alg_flops,
                     "frac_of_fp32_mfma_peak": achieved_tf / FP32_MFMA_PEAK_TFLOPS,
                     "issued_fp16_tflops": exec_tf,
                     "issued_frac_of_fp16_peak": exec_tf / FP16_MFMA_PEAK_TFLOPS,
                     "ms_per_step": stage_ms["contract"],
                     "avg_launch_ms": stage_ms["contract"] / launches},
        "xkernel": {"bound": "hbm", "achieved": xk_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": xk_gbs / HBM_PEAK_GBS, "bytes_per_launch": xk_bytes,
                    "avg_launch_ms": stage_ms["xkernel"]},
        "stages_ms": {**{k: round(v, 4) for k, v in stage_ms.items()}, "fit": round(fit_ms, 4)},
        "score_only_candidates_per_s": M / (score_ms * 1e-3),
        "refined_fp64": refined,
    }
    if args.ls_starts > 0:
        line["local_search"] = time_local_search(gp, keep, Cc, mask, w.eps_f, args.ls_starts,
                                                 args.ls_max_steps)
    if args.hyper_samples > 0:
        line["hyperfit"] = time_hyperfit(gp, w, space, X, y, feas, args.hyper_samples,
                                         args.hyper_starts, n_f)
    if args.forest_trees > 0:
        line["random_forest"] = time_forest(gp, space, X, feas, Cc, args.forest_trees)
    if args.cot_m > 0:
        line["chain_of_trees"] = time_cot(gp, args.cot_m)
    others = [x for x in args.other_workloads.split(",") if x and x != args.workload]
    if others:
        line["other_workloads"] = time_other_workloads(gp, others)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, M if args.cpu_sample <= 0 else min(args.cpu_sample, M))
    print(json.dumps(line), flush=True)


def time_local_search(gp, model, Cc, mask, eps_f, n_starts, max_steps, reps=3):
    """Extra (not part of the step): the multi-start local search from the full candidate
    set, wall time per call (one warm-up call first)."""
    import torch
    out = gp.local_search(model, Cc, mask, eps_f, n_starts, max_steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        out = gp.local_search(model, Cc, mask, eps_f, n_starts, max_steps)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / reps
    steps = out["steps"].cpu().tolist()
    return {"ms_per_call": ms, "n_starts": n_starts, "max_steps": max_steps,
            "moves_per_start": steps, "best_acq": float(out["acq"].max())}


def time_hyperfit(gp, w, space, X, y, feas, n_samples, n_starts, n_f, reps=3):
    """Extra (not part of the step): the multistart hyperparameter fit on the workload's
    observations (gamma(1.5, 1) lengthscale prior, noise floor 1e-6, 100 L-BFGS steps
    at most), and one batch of 64 objective + gradient evaluations with its fp64 rate
    (factorisation, triangular inverse and X^T X: n_f^3 / 3 multiply-adds each)."""
    import torch
    from workloads import hyper_starts
    d = len(w.space)
    th0 = torch.from_numpy(hyper_starts(d, n_samples, 7)).cuda()
    prior = (1.5, 1.0)
    out = gp.hyperfit(space, X, y, feas, th0, n_starts, prior, 1e-6, max_iter=100)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        out = gp.hyperfit(space, X, y, feas, th0, n_starts, prior, 1e-6, max_iter=100)
    torch.cuda.synchronize()
    fit_ms = (time.perf_counter() - t0) * 1e3 / reps
    batch = th0[:64]
    gp.log_posterior(space, X, y, feas, batch, prior, 1e-6)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        gp.log_posterior(space, X, y, feas, batch, prior, 1e-6)
    torch.cuda.synchronize()
    b_ms = (time.perf_counter() - t0) * 1e3 / reps
    flops = 64 * 3 * (2.0 * n_f ** 3 / 3.0)
    tf = flops / (b_ms * 1e-3) / 1e12
    return {"ms_per_call": fit_ms, "samples": n_samples, "starts": n_starts,
            "iterations": out["iters"].cpu().tolist(),
            "best_objective": float(out["value"].max()),
            "batch64_value_grad_ms": b_ms, "batch64_fp64_tflops": tf,
            "batch64_frac_of_fp64_peak": tf / FP64_PEAK_TFLOPS,
            "bound": "latency (one launch per 32-column block of the factorisation)"}


def time_forest(gp, space, X, feas, Cc, n_trees, reps=3):
    """Extra (not part of the step): the random-forest feasibility model on the
    workload's observations (depth <= 16), its fit and its prediction for every
    candidate, HIP events on the launch stream."""
    import torch
    M = int(Cc[0].shape[0])
    f = gp.Forest(space, X, feas, n_trees, 16, 2, 1)
    f.predict(Cc)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for r in range(reps):
        f = gp.Forest(space, X, feas, n_trees, 16, 2, r + 2)
    torch.cuda.synchronize()
    fit_ms = (time.perf_counter() - t0) * 1e3 / reps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(reps):
        p, _ = f.predict(Cc)
    ev[1].record()
    torch.cuda.synchronize()
    pr_ms = ev[0].elapsed_time(ev[1]) / reps
    nodes = sum(len(f.tree(t)[0]) for t in range(n_trees))
    return {"trees": n_trees, "max_depth": 16, "nodes": nodes, "fit_ms": fit_ms,
            "predict_M": M, "predict_ms": pr_ms, "predict_candidates_per_s": M / (pr_ms * 1e-3),
            "tree_walks_per_s": M * n_trees / (pr_ms * 1e-3), "mean_p": float(p.mean()),
            "bound": "latency of the dependent node loads (L2-resident trees)"}


def time_other_workloads(gp, names, steps=5, warmup=2):
    """Extra (parity configurations, not the headline): the same fused step (gp_fit_score)
    on the other full-size workloads, wall clock over `steps` steps, with the number of
    candidates the last step recomputed in fp64."""
    import torch
    from workloads import make_workload
    out = {}
    for name in names:
        w = make_workload(name)
        space = gp.Space(w.space)
        X = gp.to_device_columns(space, w.X)
        Cc = gp.to_device_columns(space, w.C)
        y = torch.from_numpy(np.nan_to_num(w.y, nan=0.0)).cuda()
        feas = torch.from_numpy(w.feasible).cuda()
        mask = torch.from_numpy(w.mask).cuda() if w.mask is not None else None
        fb = gp.FitScoreBuffers(space, len(w.y), w.M, w.cls_signal_var is not None,
                                want_p=True, want_argmax=True)

        def step():
            return gp.fit_score_into(space, X, y, feas, w.lengthscale, w.signal_var,
                                     w.noise_var, w.cls_signal_var, Cc, fb, mask, w.eps_f)

        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            m = step()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        info = m.info()
        out[name] = {"workload": WORKLOAD_TEXT[name], "n": info["n"],
                     "n_feasible": info["n_feasible"], "M": w.M, "ms_per_step": ms,
                     "candidates_per_s": w.M / (ms * 1e-3),
                     "refined_fp64": gp.refined_count(m, fb)}
        del fb, X, Cc
        torch.cuda.empty_cache()
    return out


def time_cot(gp, M, reps=5):
    """Extra (not part of the step): uniform-leaf draws and membership tests on the
    GPU-tile space's chain (one tree of ten ordinals, 9,339,902 leaves), HIP events on
    the launch stream. Algorithmic bytes per configuration: draw = 8 (its leaf key) +
    40 (ten int32 columns written); membership = 40 (columns read) + 8 (the matching
    key) + 1 (mask written)."""
    import torch
    from workloads import c3_chain_leaves, make_workload
    w = make_workload("C3", 4096)
    leaves = c3_chain_leaves()
    chain = gp.Chain(gp.Space(w.space), [list(range(10))], [leaves.astype(np.int32)])
    cols = chain.sample(M, seed=1)
    chain.member(cols)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    ev[0].record()
    for r in range(reps):
        cols = chain.sample(M, seed=r + 2)
    ev[1].record()
    for _ in range(reps):
        mask = chain.member(cols)
    ev[2].record()
    torch.cuda.synchronize()
    s_ms, m_ms = ev[0].elapsed_time(ev[1]) / reps, ev[1].elapsed_time(ev[2]) / reps
    assert bool(mask.all()), "every drawn configuration is in the chain"
    return {"workload": "C3 GPU-tile space: 1 tree of 10 ordinals, 9,339,902 leaves",
            "M": M, "sample_ms": s_ms, "member_ms": m_ms,
            "sample_configs_per_s": M / (s_ms * 1e-3), "member_configs_per_s": M / (m_ms * 1e-3),
            "sample_gbs": 48 * M / (s_ms * 1e-3) / 1e9, "member_gbs": 49 * M / (m_ms * 1e-3) / 1e9,
            "bound": "hbm (draw); latency of the binary search (membership)"}


def keep_tiles(model, fused):
    """(k-length, first column within its factor, non-padding columns, linear column or
    -1) of each column tile of the contraction, from the model's sizes: value tiles,
    classifier tiles, and the classifier's latent-mean column in a spare 16-column
    sub-tile of the last value tile (not for a model of gp_fit_score, whose value tiles
    are contracted ahead of the classifier), else of the last classifier tile, else a
    tile of its own."""
    info = model.info()
    n, n_f = info["n"], info["n_feasible"]
    r32 = lambda x: int(math.ceil(x / 32) * 32)
    out = [[r32(min(c0 + 128, n_f)), c0, min(128, n_f - c0), -1] for c0 in range(0, n_f, 128)]
    n_reg = len(out)
    if info["has_classifier"]:
        out += [[r32(min(c0 + 128, n)), c0, min(128, n - c0), -1] for c0 in range(0, n, 128)]
        up16 = lambda x: (x + 15) // 16 * 16
        if not fused and 0 < n_f % 128 and up16(n_f % 128) < 128:
            t, lin = n_reg - 1, up16(n_f % 128)
        elif 0 < n % 128 and up16(n % 128) < 128:
            t, lin = len(out) - 1, up16(n % 128)
        else:
            out.append([0, 0, 0, -1])
            t, lin = len(out) - 1, 0
        out[t][0], out[t][3] = r32(n), lin
    return [tuple(t) for t in out]


if __name__ == "__main__":
    main()
