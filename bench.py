#!/usr/bin/env python3
"""Throughput of the device-resident NUTS on one MI355X.

Default workload: the covtype-shaped logistic regression (N = 581,012 rows,
D = 55 columns with the intercept, synthetic iid N(0, 1) features, fp32),
one chain.  `--workload` selects another configured workload (see
workloads.py).

A "step" is one NUTS iteration of every chain: momentum, trajectory
doubling with the iterative tree builder, every leapfrog step's fused
potential and gradient over all rows, proposal selection.  --warmup W
iterations run first (untimed, NUTS warmup with the workload's settings);
the timed call resumes each chain from that state for exactly --steps K
iterations with the data already in HBM.  Defaults: the workload's own
warmup / sample counts.

The JSON line reports leapfrog gradient evaluations per second (`value`,
summed over chains) of that timed call and the roofline of its kernel
(algorithmic bytes = one read of X and y per gradient evaluation, over the
call's time from HIP events on the stream the kernel runs on).  Beside it:
  - ESS/s from the metric workload's full protocol (1000 warmup + 1000
    draws, fp32 and fp64), the only run long enough for an ESS;
  - the standalone gradient pass (the potential kernel alone, one position
    per call, back-to-back calls) for fp32 and fp64;
  - the other workloads' own lines (4,096 small per-chain models, 256
    chains on shared data on the matrix cores, the 4,000,000 x 257 stream),
    each with its roofline and CPU baseline;
  - the semi-supervised HMM;
  - the CPU oracle's gradient rate on the same data (one core, and all
    allowed cores up to 16) as a baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_F32_PEAK_TFLOPS = 157.3   # dense fp32 matrix-core peak of the MI355X
# vector ALU issue peak: 256 CUs x 4 SIMDs, one 64-lane instruction per SIMD
# every 4 clocks, 2.4 GHz -> 614.4 G wave-instructions/s (with one FMA per
# lane that is the 78.6 TFLOP/s fp64 vector peak)
VALU_PEAK_GIPS = 614.4
# plain vector arithmetic (a fused multiply-add counted as 2 flops) of the
# same 1,024 SIMDs at 2.4 GHz: fp64 78.6 TFLOP/s, fp32 157.3 TFLOP/s
VECTOR_PEAK_TFLOPS = {"f64": 78.6, "f32": 157.3}
METRIC = "leapfrog grad-evals/s + ESS/s, logistic N=581012 D=55; % HBM roofline"
SUB_WORKLOADS = ("chains4096_n500_d9_f64", "shared256_n200000_d129_f32", "stream_n4m_d257_f32")
# iterations (warmup, timed) of the other workloads' lines
SUB_STEPS = {"chains4096_n500_d9_f64": (100, 200), "shared256_n200000_d129_f32": (50, 50),
             "stream_n4m_d257_f32": (30, 20)}


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def _stream():
    """A torch stream of default priority that the library and the timing
    events share, so that the events bracket exactly the library's work."""
    import torch
    return torch.cuda.Stream()


def generate_on_device(wl):
    """The workload's recipe drawn on the device (torch's generator): used for
    the 4,000,000 x 257 set, whose numpy draw takes minutes.  w_true ~
    N(0, w_scale^2); features N(0, 1), zeroed with probability zero_frac; a
    ones column; y ~ Bernoulli(sigmoid(X w_true)).  Returns device X, y and
    host w_true."""
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(1000 + wl.data_seed)
    D = wl.D
    w = torch.randn(D, generator=g, device="cuda", dtype=torch.float64) * wl.w_scale
    dt = torch.float32 if wl.dtype == "f32" else torch.float64
    X = torch.empty((wl.N, D), dtype=dt, device="cuda")
    y = torch.empty(wl.N, dtype=torch.uint8, device="cuda")
    chunk = 1 << 18
    for r0 in range(0, wl.N, chunk):
        r1 = min(wl.N, r0 + chunk)
        f = torch.randn((r1 - r0, D - 1), generator=g, device="cuda", dtype=torch.float64)
        if wl.zero_frac > 0:
            f *= torch.rand(f.shape, generator=g, device="cuda", dtype=torch.float64) >= wl.zero_frac
        X[r0:r1, :D - 1] = f.to(dt)
        X[r0:r1, D - 1] = 1.0
        eta = X[r0:r1].double() @ w
        u = torch.rand(r1 - r0, generator=g, device="cuda", dtype=torch.float64)
        y[r0:r1] = (u < torch.sigmoid(eta)).to(torch.uint8)
    torch.cuda.synchronize()
    return X, y, w.cpu().numpy()


def load_workload(name):
    """(host X or None, host y or None, device X, device y, w_true)."""
    import torch

    import workloads

    wl = workloads.WORKLOADS[name]
    t0 = time.time()
    if wl.N * wl.D >= 100_000_000:
        Xd, yd, w_true = generate_on_device(wl)
        X = y = None
        log(f"{name}: drew X {tuple(Xd.shape)} {wl.dtype} on the device in {time.time() - t0:.1f}s")
    else:
        X, y = workloads.make_workload(wl)
        _, _, w_true = workloads.make_logistic(1, wl.D, w_scale=wl.w_scale, key=wl.data_seed)
        Xd = torch.from_numpy(X).cuda()
        yd = torch.from_numpy(y).cuda()
        log(f"{name}: generated X {X.shape} {X.dtype} in {time.time() - t0:.1f}s")
    torch.cuda.synchronize()
    return X, y, Xd, yd, w_true


def path_of(wl):
    """The path the library's AUTO rule takes for this shape, named
    explicitly, with its kernel and how it accumulates."""
    import paper_1912_11554_amd as nuts

    es = 8 if wl.dtype == "f64" else 4
    rows = "f32" if wl.dtype == "f32" else "f64"
    if wl.num_chains == 1 and wl.N * wl.D * es > 120 * 1024:
        return nuts.NUTS_PATH_GRID, "sampler_grid_kernel", f"{rows} row terms, f64 sums"
    if wl.num_chains == 1 or wl.per_chain_data or wl.dtype != "f32":
        return nuts.NUTS_PATH_WAVE, "sampler_wave_kernel", f"{rows} row terms, f64 sums"
    return (nuts.NUTS_PATH_BATCH, "sampler_batch_kernel",
            "f32 positions and f32 matrix-core products within each group's row range, "
            "f32 row terms, f64 sums across groups and of the loss")


def make_data(name, data, s):
    """The library's device layout of the workload's data, and its seconds."""
    import torch

    import workloads

    wl = workloads.WORKLOADS[name]
    _, _, Xd, yd, _ = data
    t0 = time.time()
    d = s.data(Xd, yd, per_chain=wl.per_chain_data)
    torch.cuda.synchronize()
    return d, time.time() - t0


def run_workload(name, data, s, stream, steps=None, warmup=None, adapt=False, variants=None, prepared=None):
    """--warmup untimed iterations, then exactly --steps timed ones resumed
    from that state, every buffer on the device.  `prepared`: (d, layout
    seconds) from make_data, else the layout is made here.  The line's rate
    is over the whole call (HIP events around it); the roofline uses the
    sampler kernel's own time (events the library records right around its
    launch, which is what a kernel trace measures)."""
    import torch

    import paper_1912_11554_amd as nuts
    import workloads
    from paper_1912_11554_amd.diagnostics import (effective_sample_size,
                                                  effective_sample_size_per_chain)

    wl = workloads.WORKLOADS[name]
    steps = wl.num_samples if steps is None else steps
    warmup = wl.num_warmup if warmup is None else warmup
    C, D = wl.num_chains, wl.D
    d, layout_s = prepared if prepared is not None else make_data(name, data, s)
    path, kernel, accumulate = path_of(wl)
    kw = dict(step_size=wl.step_size, max_tree_depth=wl.max_tree_depth, seed=wl.seed,
              prior_scale=wl.prior_scale, num_chains=C, path=path, **(variants or {}))
    if adapt and C != 1:
        sys.exit("--adapt takes single-chain workloads (the timed call shares one step size)")

    dev = dict(dtype=torch.float64, device="cuda")
    q = torch.empty((C, D), **dev)
    im = torch.empty((C, D), **dev)
    eps = torch.empty(C, **dev)
    t0 = time.time()
    r0 = d.sample(num_warmup=warmup, num_samples=1, adapt_diag_mass=wl.adapt_diag_mass,
                  adapt_step_size=adapt, out_final_q=q, out_inv_mass=im, out_step_size=eps, **kw)
    log(f"{name}: warmup {warmup} iterations x {C} chains, {r0['grad_evals']} gradient "
        f"evaluations, {time.time() - t0:.2f}s")
    inv_mass = im[0].contiguous() if wl.adapt_diag_mass else None
    if adapt:
        # the paper's covtype protocol: the step size from warmup adaptation
        kw["step_size"] = float(eps[0])
        log(f"{name}: step size adapted over {warmup} warmup iterations: {kw['step_size']:.6g}")

    samples = torch.empty((C, steps, D), **dev)
    stats = torch.empty((C, steps, nuts.STATS_DTYPE.itemsize), dtype=torch.uint8, device="cuda")
    outs = dict(out_final_q=torch.empty((C, D), **dev), out_inv_mass=torch.empty((C, D), **dev),
                out_step_size=torch.empty(C, **dev))
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record(stream)
    r = d.sample(num_warmup=0, num_samples=steps, init_q=q, first_iter=warmup + 1,
                 inv_mass=inv_mass, out_samples=samples, out_stats=stats, time_kernel=True, **outs, **kw)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    gpu_s = ev0.elapsed_time(ev1) / 1e3
    kernel_s = r["kernel_ms"] / 1e3
    st = stats.cpu().numpy().reshape(C, steps, -1).view(nuts.STATS_DTYPE)[..., 0]
    draws = samples.cpu().numpy()
    evals = r["grad_evals"]
    assert evals == int(st["num_steps"].sum()) + C
    # per-coordinate ESS: pooled over chains that share one target, per chain
    # (then the minimum over chains) when every chain has its own data
    ess = (effective_sample_size_per_chain(draws).min(axis=0) if wl.per_chain_data
           else effective_sample_size(draws))
    es = 8 if wl.dtype == "f64" else 4
    bytes_per_eval = wl.N * wl.D * es + wl.N
    achieved = evals * bytes_per_eval / kernel_s / 1e9
    # batched path: every chain of a 128-chain tile takes one leapfrog step
    # per pass until the tile's last chain is done; passes = the most
    # evaluations of any chain of the tile
    per_chain = 1 + st["num_steps"].sum(axis=1)
    passes = max(int(per_chain[t:t + 128].max()) for t in range(0, C, 128))
    flops_per_eval = 4.0 * wl.N * wl.D       # E = X q and G = X^T r, 2 flops per multiply-add
    tflops = evals * flops_per_eval / kernel_s / 1e12
    log(f"{name}: {steps} iterations x {C} chains, {evals} evaluations in {gpu_s * 1e3:.2f} ms GPU "
        f"({wall * 1e3:.2f} ms wall, sampler kernel {kernel_s * 1e3:.2f} ms): {evals / gpu_s:.0f} evals/s, "
        f"kernel {achieved:.0f} GB/s, {tflops:.1f} TFLOP/s")
    return d, dict(
        workload=name, N=wl.N, D=wl.D, dtype=wl.dtype, chains=C, step_size=kw["step_size"],
        step_size_adapted=bool(adapt), variants=sorted(k for k, v in (variants or {}).items() if v),
        max_tree_depth=wl.max_tree_depth, steps=steps, warmup=warmup, grad_evals=evals,
        gpu_seconds=gpu_s, kernel_seconds=kernel_s, wall_seconds=wall, layout_seconds=layout_s,
        evals_per_s=evals / gpu_s, ms_per_step=1e3 * wall / steps,
        ess_min_timed_call=float(ess.min()), bytes_per_eval=bytes_per_eval, achieved_gbs=achieved,
        mean_tree_depth=float(st["tree_depth"].mean()),
        mean_steps_per_iter=float(st["num_steps"].mean()),
        divergences=int(st["diverging"].sum()), accept_prob=float(st["accept_prob"].mean()),
        path=path, kernel=kernel, accumulate=accumulate, flops_per_eval=flops_per_eval,
        achieved_tflops=tflops, passes=passes, pass_fill=evals / (passes * C),
        ms_per_pass=1e3 * kernel_s / passes,
    )


def run_protocol(name, d, stream):
    """The workload's full single-chain protocol (num_warmup warmup + num_samples
    draws from q = 0, fixed step size) as two calls, all warmup iterations
    then all sampling iterations (resuming is exact: the counter-based draws
    make (q, t) the whole state), timed with HIP events; ESS over the draws."""
    import torch

    import paper_1912_11554_amd as nuts
    import workloads
    from paper_1912_11554_amd.diagnostics import effective_sample_size

    wl = workloads.WORKLOADS[name]
    W, S, D = wl.num_warmup, wl.num_samples, wl.D
    path, _, _ = path_of(wl)
    assert wl.num_chains == 1 and not wl.adapt_diag_mass and W >= 1
    kw = dict(step_size=wl.step_size, max_tree_depth=wl.max_tree_depth, seed=wl.seed,
              prior_scale=wl.prior_scale, path=path)
    dev = dict(dtype=torch.float64, device="cuda")
    q = torch.empty((1, D), **dev)
    sb = nuts.STATS_DTYPE.itemsize
    junk = dict(out_samples=torch.empty((1, 1, D), **dev), out_inv_mass=torch.empty((1, D), **dev),
                out_step_size=torch.empty(1, **dev),
                out_stats=torch.empty((1, 1, sb), dtype=torch.uint8, device="cuda"))
    samples = torch.empty((1, S, D), **dev)
    outs = dict(out_final_q=torch.empty((1, D), **dev), out_inv_mass=torch.empty((1, D), **dev),
                out_step_size=torch.empty(1, **dev),
                out_stats=torch.empty((1, S, sb), dtype=torch.uint8, device="cuda"))
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    r1 = d.sample(num_warmup=W - 1, num_samples=1, out_final_q=q, **junk, **kw)
    ev[1].record(stream)
    r2 = d.sample(num_warmup=0, num_samples=S, init_q=q, first_iter=W, out_samples=samples,
                  **outs, **kw)
    ev[2].record(stream)
    torch.cuda.synchronize()
    t_all = ev[0].elapsed_time(ev[2]) / 1e3
    t_samp = ev[1].elapsed_time(ev[2]) / 1e3
    ess = effective_sample_size(samples.cpu().numpy())
    evals = r1["grad_evals"] + r2["grad_evals"]
    log(f"{name}: protocol {W} + {S}: {evals} evaluations in {t_all * 1e3:.1f} ms, "
        f"min ESS {ess.min():.0f}, ESS/s {ess.min() / t_all:.0f}")
    return dict(workload=name, warmup=W, samples=S, grad_evals=evals, seconds=round(t_all, 4),
                sampling_seconds=round(t_samp, 4), sampling_grad_evals=r2["grad_evals"],
                ess_min=round(float(ess.min()), 1), ess_median=round(float(np.median(ess)), 1),
                ess_per_s=round(float(ess.min() / t_all), 1),
                ess_per_s_sampling=round(float(ess.min() / t_samp), 1),
                evals_per_s=round(evals / t_all, 1),
                note="ESS/s = min-coordinate ESS of the draws / GPU seconds of warmup and sampling")


def run_standalone(name, d, w_true, stream, launches=400):
    """The potential kernel alone: one position per call (the generating
    weights), back-to-back calls of the allocation-free entry point (which
    only enqueues), HIP events around all of them on the kernel's stream."""
    import torch

    import workloads

    wl = workloads.WORKLOADS[name]
    W = torch.from_numpy(np.ascontiguousarray(w_true[None, :])).cuda()
    U = torch.empty(1, dtype=torch.float64, device="cuda")
    G = torch.empty((1, wl.D), dtype=torch.float64, device="cuda")
    for _ in range(20):
        d.potential_grad(W, out_U=U, out_grad=G, no_alloc=True)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(launches):
        d.potential_grad(W, out_U=U, out_grad=G, no_alloc=True)
    ev1.record(stream)
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) * 1e3 / launches
    es = 8 if wl.dtype == "f64" else 4
    bytes_per_eval = wl.N * wl.D * es + wl.N
    gbs = bytes_per_eval / (us * 1e-6) / 1e9
    log(f"{name}: standalone gradient pass {us:.2f} us per call, {gbs:.0f} GB/s")
    return dict(workload=name, kernel="potential_grad_kernel", positions_per_call=1, calls=launches,
                us_per_call=round(us, 3), evals_per_s=round(1e6 / us, 1),
                roofline={"kernel": "potential_grad_kernel", "bound": "hbm", "achieved": round(gbs, 1),
                          "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                          "bytes_per_eval": bytes_per_eval},
                note="per call: the potential kernel alone (its exchange slots are left empty by "
                     "the previous call); back-to-back, so launch gaps are included")


def recorded_traffic(kernel, workload, evals):
    """HBM bytes of the timed launch from the PMC record in
    profiles/traffic.json (FETCH_SIZE + WRITE_SIZE per gradient evaluation,
    each scaled by the same counter's reading on a copy of known size), or
    None when there is no record for this kernel and workload or the sources
    the kernel is built from have changed since it was taken."""
    from paper_1912_11554_amd.profiling import source_fingerprint

    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    e = rec.get("kernels", {}).get(f"{kernel}/{workload}")
    if not e or e.get("fingerprint") != source_fingerprint(kernel):
        return None
    out = dict(bytes=round((e["fetch_bytes_per_eval"] + e["write_bytes_per_eval"]) * evals),
               fetch_bytes_per_eval=e["fetch_bytes_per_eval"],
               write_bytes_per_eval=e["write_bytes_per_eval"], source="profiles/traffic.json")
    if "valu_instructions_per_eval" in e:
        out["valu_instructions_per_eval"] = e["valu_instructions_per_eval"]
    return out


def roofline(res):
    """Roofline of a timed sampler call: HBM for the streaming paths, fp32
    matrix cores for the batched path, vector-ALU issue for the wave path
    with the data resident in LDS (from the recorded instruction count)."""
    kernel = res["kernel"]
    traffic = recorded_traffic(kernel, res["workload"], res["grad_evals"])
    if kernel == "sampler_batch_kernel":
        return {"kernel": kernel, "bound": "mfma", "achieved": round(res["achieved_tflops"], 2),
                "peak": MFMA_F32_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(res["achieved_tflops"] / MFMA_F32_PEAK_TFLOPS, 4),
                "traffic": traffic and traffic["bytes"], "traffic_detail": traffic,
                "flops_per_eval": res["flops_per_eval"], "passes": res["passes"],
                "pass_fill": round(res["pass_fill"], 4), "ms_per_pass": round(res["ms_per_pass"], 4)}
    if kernel == "sampler_wave_kernel" and traffic and "valu_instructions_per_eval" in traffic:
        rate = traffic["valu_instructions_per_eval"] * res["grad_evals"] / res["kernel_seconds"] / 1e9
        return {"kernel": kernel, "bound": "alu", "achieved": round(rate, 1), "peak": VALU_PEAK_GIPS,
                "unit": "G VALU wave-instructions/s", "frac": round(rate / VALU_PEAK_GIPS, 4),
                "traffic": traffic["bytes"], "traffic_detail": traffic,
                "valu_instructions_per_eval": traffic["valu_instructions_per_eval"],
                "bytes_per_eval": res["bytes_per_eval"], "algorithmic_gbs": round(res["achieved_gbs"], 1)}
    if kernel == "sampler_wave_kernel":
        # no instruction count recorded for these kernel sources: the
        # algorithmic flops (4 N D per evaluation) against the vector peak of
        # the kernel's arithmetic type; the data sit in LDS, so HBM is no bound
        peak = VECTOR_PEAK_TFLOPS[res["dtype"]]
        return {"kernel": kernel, "bound": "alu", "achieved": round(res["achieved_tflops"], 3), "peak": peak,
                "unit": "TFLOP/s", "frac": round(res["achieved_tflops"] / peak, 4),
                "traffic": traffic and traffic["bytes"], "traffic_detail": traffic,
                "flops_per_eval": res["flops_per_eval"], "note": "no instruction count recorded for these kernel sources"}
    return {"kernel": kernel, "bound": "hbm", "achieved": round(res["achieved_gbs"], 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(res["achieved_gbs"] / HBM_PEAK_GBS, 4),
            "traffic": traffic and traffic["bytes"], "traffic_detail": traffic,
            "bytes_per_eval": res["bytes_per_eval"]}


def cpu_baseline(name, data, seconds):
    """The oracle's fp64 gradient evaluations on the same data, one core,
    and on every allowed core up to 16.  For the 4,000,000-row set a slice of
    its first rows stands in (the time per evaluation is linear in N), and
    the rate is scaled to the full set."""
    import oracle
    import workloads

    wl = workloads.WORKLOADS[name]
    X, y, Xd, yd, w_true = data
    scale, what = 1.0, ""
    if X is None:
        rows = 400_000
        X = Xd[:rows].cpu().numpy()
        y = yd[:rows].cpu().numpy()
        scale = rows / wl.N
        what = f" on its first {rows} rows (rate scaled by {rows}/{wl.N})"
    if wl.per_chain_data:
        X, y = X[0], y[0]
    f = oracle.logistic_potential_grad_f32 if wl.dtype == "f32" else oracle.logistic_potential_grad
    U_check = f(X, y, w_true)[0]
    # the oracle's timing loop (about 10 ms of evaluations per call, or one
    # evaluation when that takes longer), so that small data sets are not
    # timed with the interpreter's share of each call
    Xc, yc = np.ascontiguousarray(X), np.ascontiguousarray(y, np.uint8)
    w, g = np.ascontiguousarray(w_true, np.float64), np.zeros(wl.D)
    reps = max(1, int(20_000_000 // (Xc.shape[0] * wl.D)))
    lib = oracle.lib()
    n = 0
    t0 = time.perf_counter()
    while True:
        U = lib.orc_logistic_ug_repeat(Xc.ctypes.data, yc.ctypes.data, Xc.shape[0], wl.D, wl.prior_scale,
                                       w.ctypes.data, g.ctypes.data, reps, 1 if wl.dtype == "f32" else 0)
        n += reps
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    assert U == U_check, (U, U_check)  # the loop evaluates what the entry point does
    log(f"cpu oracle {name}: {n} gradient evaluations in {el:.1f}s{what}")
    if wl.per_chain_data or wl.num_chains > 1 or wl.N * wl.D < 1_000_000:
        # many chains, or one small data set: independent evaluations on
        # every core (each thread its own chain's data set where chains have
        # their own, else its own position), as independent chains would run
        allc = cpu_independent(wl, min(seconds, 5.0))
    else:
        f_rows = oracle.logistic_potential_grad_f32 if wl.dtype == "f32" else oracle.logistic_potential_grad
        allc = cpu_all_cores(f_rows, Xc, yc, w_true, min(seconds, 5.0), scale)
    return dict(value=n / el * scale, unit="grad-evals/s", cores=1, kind="oracle", all_cores=allc,
                sample=f"{n} full potential+gradient evaluations of {name}"
                       f"{' (one chain data set)' if wl.per_chain_data else ''}{what} at w_true, "
                       f"single-threaded fp64 C, {el:.1f}s",
                host_cores_available=len(os.sched_getaffinity(0)))


HMM_SHAPE = dict(T=600, Tsup=100, K=3, V=10)


def run_hmm(chains, steps, warmup):
    """The semi-supervised HMM (T = 600 symbols, the first 100 hidden states
    observed, K = 3, V = 10).  (1) One chain under the paper's HMM protocol
    (1000 warmup iterations adapting the step size and the diagonal mass,
    then 1000 draws): milliseconds per leapfrog step, the paper's HMM metric.
    (2) `chains` chains at that step size and mass, `warmup` untimed
    iterations, then `steps` timed ones: gradient evaluations per second."""
    import torch

    import paper_1912_11554_amd as nuts
    import workloads
    from paper_1912_11554_amd.diagnostics import effective_sample_size

    sh = HMM_SHAPE
    K, V = sh["K"], sh["V"]
    w, z, _, _ = workloads.make_hmm(**sh)
    D = nuts.hmm_dim(K, V)
    stream = _stream()
    with torch.cuda.stream(stream):
        s = nuts.Sampler(0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r1 = s.hmm_sample(w, z, K, V, step_size=0.1, max_tree_depth=10, num_warmup=1000,
                      num_samples=1000, seed=1, adapt_step_size=True, adapt_diag_mass=True)
    one_s = time.perf_counter() - t0
    st1 = r1["stats"][0]
    ess1 = effective_sample_size(r1["samples"])
    eps, im = float(r1["step_size"][0]), r1["inv_mass"][0]
    log(f"hmm one chain: 2000 iterations, {r1['grad_evals']} gradient evaluations in "
        f"{one_s * 1e3:.1f} ms: {one_s * 1e3 / r1['grad_evals']:.5f} ms per leapfrog step, "
        f"adapted step {eps:.4g}, min ESS {ess1.min():.0f}")

    kw = dict(step_size=eps, inv_mass=im, max_tree_depth=10, seed=2, num_chains=chains)
    r0 = s.hmm_sample(w, z, K, V, num_warmup=warmup, num_samples=1, **kw)
    samples = torch.empty((chains, steps, D), dtype=torch.float64, device="cuda")
    stats = torch.empty((chains, steps, nuts.STATS_DTYPE.itemsize), dtype=torch.uint8, device="cuda")
    outs = dict(out_final_q=torch.empty((chains, D), dtype=torch.float64, device="cuda"),
                out_inv_mass=torch.empty((chains, D), dtype=torch.float64, device="cuda"),
                out_step_size=torch.empty(chains, dtype=torch.float64, device="cuda"))
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    q0 = torch.from_numpy(r0["final_q"]).cuda()
    kw["inv_mass"] = torch.from_numpy(np.ascontiguousarray(im)).cuda()
    torch.cuda.synchronize()
    ev0.record(stream)
    r = s.hmm_sample(w, z, K, V, num_warmup=0, num_samples=steps, init_q=q0,
                     first_iter=warmup + 1, out_samples=samples, out_stats=stats, time_kernel=True,
                     **outs, **kw)
    ev1.record(stream)
    torch.cuda.synchronize()
    gpu_s = ev0.elapsed_time(ev1) / 1e3
    kernel_s = r["kernel_ms"] / 1e3
    st = stats.cpu().numpy().reshape(chains, steps, -1).view(nuts.STATS_DTYPE)[..., 0]
    evals = r["grad_evals"]
    assert evals == int(st["num_steps"].sum()) + chains
    log(f"hmm {chains} chains: {steps} iterations, {evals} evaluations in {gpu_s * 1e3:.1f} ms: "
        f"{evals / gpu_s:.4g} evals/s, {st['num_steps'].mean():.1f} steps per iteration")
    s.close()
    return dict(workload="hmm_t600_tsup100_k3_v10", T=sh["T"], Tsup=sh["Tsup"], K=K, V=V, D=D,
                one_chain=dict(warmup=1000, samples=1000, adapt="step size + diagonal mass",
                               grad_evals=r1["grad_evals"], seconds=round(one_s, 4),
                               ms_per_leapfrog_step=round(one_s * 1e3 / r1["grad_evals"], 6),
                               step_size=round(eps, 6), ess_min=round(float(ess1.min()), 1),
                               mean_steps_per_iter=round(float(st1["num_steps"].mean()), 2),
                               divergences=int(st1["diverging"].sum())),
                chains=chains, steps=steps, warmup=warmup, grad_evals=evals,
                gpu_seconds=round(gpu_s, 4), kernel_seconds=round(kernel_s, 5),
                evals_per_s=round(evals / gpu_s, 1), kernel_evals_per_s=round(evals / kernel_s, 1),
                mean_steps_per_iter=round(float(st["num_steps"].mean()), 2),
                kernel="sampler_hmm_kernel")


def hmm_cpu_baseline(seconds):
    """The oracle's fp64 HMM gradient evaluations, one core and every
    allowed core up to 16."""
    import concurrent.futures

    import oracle
    import workloads

    w, z, _, _ = workloads.make_hmm(**HMM_SHAPE)
    D = oracle.hmm_dim(HMM_SHAPE["K"], HMM_SHAPE["V"])
    q = np.random.default_rng(3).normal(0.0, 0.5, D)
    U_check = oracle.hmm_potential_grad(w, z, HMM_SHAPE["K"], HMM_SHAPE["V"], q)[0]
    lib = oracle.lib()
    wu, zu = np.ascontiguousarray(w, np.uint8), np.ascontiguousarray(z, np.uint8)

    def loop(limit):
        # the oracle's timing loop, 500 evaluations per call, so that the
        # interpreter's share (which threads take in turn) stays small
        qq, gg = np.ascontiguousarray(q, np.float64), np.zeros(D)
        args = (wu.ctypes.data, wu.shape[0], zu.ctypes.data, zu.shape[0], HMM_SHAPE["K"], HMM_SHAPE["V"],
                qq.ctypes.data, gg.ctypes.data, 500)
        m, t1, U = 0, time.perf_counter(), None
        while time.perf_counter() - t1 < limit:
            U = lib.orc_hmm_ug_repeat(*args)
            m += 500
        return m, time.perf_counter() - t1, U

    n, el, U = loop(seconds)
    assert U == U_check, (U, U_check)
    log(f"cpu oracle hmm: {n} gradient evaluations in {el:.1f}s")
    cores = max(1, min(16, len(os.sched_getaffinity(0))))
    with concurrent.futures.ThreadPoolExecutor(max_workers=cores) as ex:
        res = list(ex.map(lambda _: loop(min(seconds, 5.0)), range(cores)))
    allc = dict(value=sum(m / t for m, t, _ in res), unit="grad-evals/s", cores=cores,
                sample=f"{sum(m for m, _, _ in res)} evaluations on {cores} threads")
    log(f"cpu oracle hmm, {cores} threads: {allc['value']:.0f} evaluations/s")
    return dict(value=n / el, unit="grad-evals/s", cores=1, kind="oracle", all_cores=allc,
                sample=f"{n} HMM potential+gradient evaluations (T 600, Tsup 100, K 3, V 10), "
                       f"single-threaded fp64 C, {el:.1f}s")


def hmm_line(h, cpu):
    """The HMM object of the JSON line, with its roofline: the wave-per-chain
    HMM kernel is bound by vector-ALU issue (the recursions run in
    registers, the symbols and occupancies in LDS)."""
    traffic = recorded_traffic(h["kernel"], h["workload"], h["grad_evals"])
    roof = None
    if traffic and "valu_instructions_per_eval" in traffic:
        rate = traffic["valu_instructions_per_eval"] * h["kernel_evals_per_s"] / 1e9
        roof = {"kernel": h["kernel"], "bound": "alu", "achieved": round(rate, 1),
                "peak": VALU_PEAK_GIPS, "unit": "G VALU wave-instructions/s",
                "frac": round(rate / VALU_PEAK_GIPS, 4), "traffic": traffic["bytes"],
                "valu_instructions_per_eval": traffic["valu_instructions_per_eval"]}
    out = dict(h)
    out["roofline"] = roof
    out["cpu_baseline"] = cpu
    # the paper's HMM figure (NumPyro, 32-bit, one CPU chain): context only
    out["paper_numpyro_cpu_ms_per_leapfrog_step"] = 0.09
    return out


def cpu_independent(wl, seconds):
    """The oracle's gradient on every allowed host core (at most 16), each
    thread evaluating on its own: chain t's data set for per-chain data,
    else the shared data at its own position.  Each call of the oracle's
    timing loop runs about 10 ms of evaluations, so the interpreter's share
    (which the threads take in turn) stays small."""
    import concurrent.futures

    import oracle
    import workloads

    cores = max(1, min(16, len(os.sched_getaffinity(0))))
    if wl.per_chain_data:
        Xs, ys = workloads.make_workload(wl, chains=list(range(cores)))
        sets = [(np.ascontiguousarray(Xs[t]), np.ascontiguousarray(ys[t])) for t in range(cores)]
    else:
        X, y = workloads.make_workload(wl)
        sets = [(X, y)] * cores
    _, _, w_true = workloads.make_logistic(1, wl.D, w_scale=wl.w_scale, key=wl.data_seed)
    lib = oracle.lib()
    f32 = 1 if wl.dtype == "f32" else 0
    rng = np.random.default_rng(11)
    pos = [np.ascontiguousarray(w_true + (0.01 * rng.normal(size=wl.D) if t else 0.0), np.float64)
           for t in range(cores)]

    def worker(t):
        Xt, yt = sets[t]
        w = pos[t]
        g = np.zeros(wl.D)
        reps = max(1, int(20_000_000 // (Xt.shape[0] * wl.D)))  # about 10 ms per call
        args = (Xt.ctypes.data, yt.ctypes.data, Xt.shape[0], wl.D, wl.prior_scale, w.ctypes.data,
                g.ctypes.data, reps, f32)
        m, t1 = 0, time.perf_counter()
        while time.perf_counter() - t1 < seconds:
            lib.orc_logistic_ug_repeat(*args)
            m += reps
        return m, time.perf_counter() - t1

    with concurrent.futures.ThreadPoolExecutor(max_workers=cores) as ex:
        res = list(ex.map(worker, range(cores)))
    v = sum(m / t for m, t in res)
    log(f"cpu oracle, {cores} threads, independent evaluations: {v:.0f} evaluations/s")
    what = "its own chain's data set" if wl.per_chain_data else "its own position"
    return dict(value=v, unit="grad-evals/s", cores=cores,
                sample=f"{sum(m for m, _ in res)} evaluations, each thread on {what}, "
                       f"{max(t for _, t in res):.1f}s")


def cpu_all_cores(f, X, y, w, seconds, scale=1.0):
    """The oracle's gradient on every allowed host core (at most 16): the rows
    in one fixed chunk per thread (ctypes releases the interpreter lock
    during the C call), the partial sums added in chunk order.  A timing
    mode only: each chunk's call also adds the prior, which this sum does not
    correct.  `scale` converts the rate on a row slice to the full set."""
    import concurrent.futures

    cores = max(1, min(16, len(os.sched_getaffinity(0))))
    N = X.shape[0]
    bounds = [(N * i // cores, N * (i + 1) // cores) for i in range(cores)]
    with concurrent.futures.ThreadPoolExecutor(max_workers=cores) as ex:
        n = 0
        t0 = time.perf_counter()
        while True:
            parts = list(ex.map(lambda b: f(X[b[0]:b[1]], y[b[0]:b[1]], w), bounds))
            g = parts[0][1].copy()
            for p in parts[1:]:
                g += p[1]
            n += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                break
    log(f"cpu oracle, {cores} threads: {n} gradient evaluations in {el:.1f}s")
    return dict(value=n / el * scale, unit="grad-evals/s", cores=cores,
                sample=f"{n} evaluations, rows in {cores} fixed chunks, {el:.1f}s")


def run_standalone_chains(name, d, chains, stream, launches=200):
    """The potential kernel alone on a per-chain workload: one position for
    every chain's data set per call (all data sets in one call, as the
    sampler evaluates them), back-to-back calls of the allocation-free entry
    point, HIP events around all of them.  The data sets stream from memory
    at every call; the sampler holds them in LDS for its whole launch."""
    import torch

    import workloads

    wl = workloads.WORKLOADS[name]
    rng = np.random.default_rng(3)
    W = torch.from_numpy(rng.normal(0.0, 0.1, size=(chains, wl.D))).cuda()
    U = torch.empty(chains, dtype=torch.float64, device="cuda")
    G = torch.empty((chains, wl.D), dtype=torch.float64, device="cuda")
    for _ in range(10):
        d.potential_grad(W, out_U=U, out_grad=G, no_alloc=True)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(launches):
        d.potential_grad(W, out_U=U, out_grad=G, no_alloc=True)
    ev1.record(stream)
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) * 1e3 / launches
    es = 8 if wl.dtype == "f64" else 4
    gbs = chains * (wl.N * wl.D * es + wl.N) / (us * 1e-6) / 1e9
    log(f"{name}: standalone gradient pass over {chains} data sets {us:.2f} us per call, "
        f"{chains / us:.1f} M evals/s, {gbs:.0f} GB/s")
    return dict(workload=name, entry_point="nuts_data_potential_grad_noalloc", positions_per_call=chains,
                calls=launches,
                us_per_call=round(us, 3), evals_per_s=round(chains / (us * 1e-6), 1),
                achieved_gbs=round(gbs, 1),
                note="per call: one position for each chain's data set, the data sets read from memory; "
                     "back-to-back, so launch gaps are included")


def sub_line(name, s, stream, cpu_seconds):
    """Another workload's line: its own short protocol, roofline and CPU
    baseline; for per-chain data also the standalone gradient pass over the
    same data sets."""
    import workloads

    data = load_workload(name)
    warmup, steps = SUB_STEPS[name]
    d, res = run_workload(name, data, s, stream, steps=steps, warmup=warmup)
    standalone = None
    if workloads.WORKLOADS[name].per_chain_data:
        standalone = run_standalone_chains(name, d, res["chains"], stream)
        standalone["sampler_evals_per_s_by_kernel_time"] = round(res["grad_evals"] / res["kernel_seconds"], 1)
        # the share of the sampler's vector instructions per evaluation that
        # are not the evaluation itself (the tree step, the draws), from the
        # recorded SQ_INSTS_VALU of both kernels on this workload
        items = recorded_traffic("potential_items_kernel", name, res["chains"])
        sampler_rec = recorded_traffic(res["kernel"], name, res["grad_evals"])
        if items and sampler_rec and "valu_instructions_per_eval" in items and \
                "valu_instructions_per_eval" in sampler_rec:
            vi, vs = items["valu_instructions_per_eval"], sampler_rec["valu_instructions_per_eval"]
            standalone["valu_instructions_per_eval"] = vi
            standalone["sampler_valu_instructions_per_eval"] = vs
            standalone["sampler_instruction_overhead"] = round(1.0 - vi / vs, 4)
    d.free()
    out = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in res.items()}
    if standalone:
        out["standalone_grad"] = standalone
    out["roofline"] = roofline(res)
    out["cpu_baseline"] = None if cpu_seconds <= 0 else cpu_baseline(name, data, cpu_seconds)
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default="covtype_n581012_d55_f32")
    ap.add_argument("--also", default="covtype_n581012_d55_f64",
                    help="second workload reported beside the first ('' for none)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-protocol", action="store_true",
                    help="skip the full-protocol ESS runs and the standalone gradient pass")
    ap.add_argument("--no-sub", action="store_true", help="skip the other workloads' lines")
    ap.add_argument("--adapt", action="store_true",
                    help="adapt the step size during warmup (dual averaging, target acceptance "
                         "0.8) and time the sampling at the adapted step size (the paper's covtype "
                         "protocol: 150 adaptation steps); single-chain workloads")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="also run a plain device copy of this many MiB (a known-size "
                         "kernel that calibrates rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    ap.add_argument("--uturn-generalized", action="store_true",
                    help="the generalised (momentum-sum) U-turn criterion")
    ap.add_argument("--subtree-merge", action="store_true",
                    help="subtree proposals chosen at the merges of halves")
    ap.add_argument("--hmm-chains", type=int, default=8192,
                    help="chains of the semi-supervised HMM reported beside the main workload "
                         "(0: no HMM line)")
    ap.add_argument("--hmm-steps", type=int, default=100)
    ap.add_argument("--hmm-only", action="store_true", help="run the HMM measurement alone")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1912_11554_amd as nuts
    import workloads

    if args.copy_mb:
        src = torch.ones(args.copy_mb << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {args.copy_mb} MiB read + {args.copy_mb} MiB written")
        del src, dst
    if args.hmm_only:
        h = run_hmm(args.hmm_chains, args.hmm_steps, 20)
        print(json.dumps(hmm_line(h, None)), flush=True)
        return
    cpu_s = 0.0 if args.no_cpu_baseline else args.cpu_seconds
    stream = _stream()
    with torch.cuda.stream(stream):
        s = nuts.Sampler(0)   # the library runs on `stream`
    variants = dict(uturn_generalized=args.uturn_generalized, subtree_merge=args.subtree_merge)

    def one(name):
        data = load_workload(name)
        wl = workloads.WORKLOADS[name]
        prepared = make_data(name, data, s)
        extra = {}
        # the full-protocol and standalone measurements first: the timed
        # call then finds the device at the clocks of sustained work, as in
        # any sampling run longer than the few milliseconds it lasts
        if not args.no_protocol and wl.num_chains == 1 and not wl.adapt_diag_mass:
            extra["protocol"] = run_protocol(name, prepared[0], stream)
            extra["standalone_grad"] = run_standalone(name, prepared[0], data[4], stream)
        d, res = run_workload(name, data, s, stream, args.steps, args.warmup, args.adapt, variants,
                              prepared=prepared)
        d.free()
        return data, res, extra

    main_data, main_res, main_extra = one(args.workload)
    other = None
    if args.also:
        _, other_res, other_extra = one(args.also)
        other = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in other_res.items()}
        other["frac_hbm"] = round(other_res["achieved_gbs"] / HBM_PEAK_GBS, 4)
        other.update(other_extra)
    cpu = None if cpu_s <= 0 else cpu_baseline(args.workload, main_data, cpu_s)
    del main_data

    proto = main_extra.get("protocol")
    line = {
        "metric": METRIC,
        "value": round(main_res["evals_per_s"], 1),
        "unit": "grad-evals/s",
        "n_gpus": 1,
        "steps": main_res["steps"],
        "warmup": main_res["warmup"],
        "ms_per_step": round(main_res["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": main_res["dtype"],
        "data": "synthetic",
        "config": {
            "workload": main_res["workload"], "N": main_res["N"], "D": main_res["D"],
            "chains": main_res["chains"], "step_size": main_res["step_size"],
            "step_size_adapted": main_res["step_size_adapted"], "variants": main_res["variants"],
            "max_tree_depth": main_res["max_tree_depth"], "accumulate": main_res["accumulate"],
            "path": main_res["kernel"],
        },
        # ESS needs the full protocol: the --steps timed iterations start in
        # the chain's transient (see ess_min_timed_call)
        "ess_per_s": proto and proto["ess_per_s"],
        "ess_min": proto and proto["ess_min"],
        "ess_protocol": proto,
        "ess_min_timed_call": round(main_res["ess_min_timed_call"], 1),
        "grad_evals": main_res["grad_evals"],
        "mean_steps_per_iter": round(main_res["mean_steps_per_iter"], 2),
        "divergences": main_res["divergences"],
        "layout_seconds": round(main_res["layout_seconds"], 4),
        "roofline": roofline(main_res),
        "cpu_baseline": cpu,
        "standalone_grad": main_extra.get("standalone_grad"),
    }
    if other:
        line["also"] = other
    if not args.no_sub:
        line["workloads"] = {name: sub_line(name, s, stream, min(cpu_s, 5.0))
                             for name in SUB_WORKLOADS if name != args.workload}
    s.close()
    if args.hmm_chains:
        h = run_hmm(args.hmm_chains, args.hmm_steps, 20)
        hc = None if cpu_s <= 0 else hmm_cpu_baseline(min(cpu_s, 10.0))
        line["hmm"] = hmm_line(h, hc)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
