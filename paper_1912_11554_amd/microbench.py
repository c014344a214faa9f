"""Time the fused potential+gradient kernels alone on a configured workload.

    python -m paper_1912_11554_amd.microbench --workload covtype_n581012_d55_f32 --positions 1
    python -m paper_1912_11554_amd.microbench --workload shared256_n200000_d129_f32 --positions 256 --batched
    python -m paper_1912_11554_amd.microbench --workload covtype_n581012_d55_f32 --positions 500 --loglik
    python -m paper_1912_11554_amd.microbench --workload covtype_n581012_d55_f32 --positions 500 --predictive

Each call evaluates U and grad U at K positions (around the data's generating
weights) with the data already in device memory (with --loglik: the
log-likelihood of the K positions as draws, the expected log-likelihood and
the predictive mean of every row); the outputs stay on the device.  Prints one JSON line: microseconds per call (HIP events on the
stream the kernels run on; the C-ABI call is synchronous, so this includes
its host side: pointer checks, launches, the final synchronisation), the
algorithmic rate at that time (bytes of X and y per position for the
streaming kernel, 4 N D flops per position for the batched matrix-core
kernel) and its fraction of the MI355X peak.  Run it under
`rocprofv3 --kernel-trace --stats` for the kernels' own durations.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_F32_PEAK_TFLOPS = 157.3


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", default="covtype_n581012_d55_f32")
    ap.add_argument("--positions", type=int, default=1)
    ap.add_argument("--batched", action="store_true",
                    help="nuts_data_potential_grad_batched (fp32 matrix cores)")
    ap.add_argument("--loglik", action="store_true",
                    help="nuts_data_log_likelihood at the positions as draws (with the expected "
                         "log-likelihood and the predictive mean)")
    ap.add_argument("--predictive", action="store_true",
                    help="nuts_data_posterior_predictive at the positions as draws (one byte per row "
                         "and draw)")
    ap.add_argument("--reps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="also run a plain device copy of this many MiB first (a known-size "
                         "kernel that calibrates rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()

    import torch

    if args.copy_mb:
        src = torch.ones(args.copy_mb << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    import paper_1912_11554_amd as nuts
    import workloads

    wl = workloads.WORKLOADS[args.workload]
    if wl.per_chain_data:
        sys.exit("microbench takes shared-data workloads")
    X, y, w_true = workloads.make_logistic(wl.N, wl.D, w_scale=wl.w_scale, key=wl.data_seed,
                                           dtype=wl.dtype, zero_frac=wl.zero_frac)
    K = args.positions
    rng = np.random.default_rng(0)
    W = torch.from_numpy(w_true[None, :] + rng.normal(0.0, 0.01, size=(K, wl.D))).cuda()
    s = nuts.Sampler(0)
    d = s.data(torch.from_numpy(X).cuda(), torch.from_numpy(y).cuda())
    U = torch.empty(K, dtype=torch.float64, device="cuda")
    G = torch.empty((K, wl.D), dtype=torch.float64, device="cuda")
    if args.predictive:
        Y = torch.empty((K, wl.N), dtype=torch.uint8, device="cuda")

        def call():
            d.posterior_predictive(W, seed=1, out_y=Y)
    elif args.loglik:
        pm = torch.empty(wl.N, dtype=torch.float64, device="cuda")
        el = torch.empty(1, dtype=torch.float64, device="cuda")

        def call():
            s._check(s._L.nuts_data_log_likelihood(s._h, d._d, W.data_ptr(), K, U.data_ptr(),
                                                   el.data_ptr(), pm.data_ptr()))
    else:
        def call():
            d.potential_grad(W, out_U=U, out_grad=G, batched=args.batched)
    for _ in range(args.warmup):
        call()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.reps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / args.reps
    es = 8 if wl.dtype == "f64" else 4
    kernel = ("batch_ll_kernel" if args.loglik or args.predictive else
              "batch_pass_kernel" if args.batched else "potential_grad_kernel")
    out = dict(workload=args.workload, N=wl.N, D=wl.D, dtype=wl.dtype, positions=K, kernel=kernel,
               reps=args.reps, us_per_call_with_host=round(us, 2))
    if args.predictive:
        # per (row, draw): the product row of E = X W^T, one sigmoid, a
        # quarter of a Philox4x64-10 block, one byte out
        pairs = wl.N * K
        tflops = 2.0 * wl.N * wl.D * K / (us * 1e-6) / 1e12
        out.update(pairs_per_s=round(pairs / (us * 1e-6), 1), bytes_out=pairs,
                   achieved_tflops=round(tflops, 2), peak=MFMA_F32_PEAK_TFLOPS,
                   frac=round(tflops / MFMA_F32_PEAK_TFLOPS, 4))
    elif args.loglik:
        tflops = 2.0 * wl.N * wl.D * K / (us * 1e-6) / 1e12   # E = X W^T only
        out.update(bound="mfma", achieved_tflops=round(tflops, 2), peak=MFMA_F32_PEAK_TFLOPS,
                   frac=round(tflops / MFMA_F32_PEAK_TFLOPS, 4))
    elif args.batched:
        tflops = 4.0 * wl.N * wl.D * K / (us * 1e-6) / 1e12
        out.update(bound="mfma", achieved_tflops=round(tflops, 2), peak=MFMA_F32_PEAK_TFLOPS,
                   frac=round(tflops / MFMA_F32_PEAK_TFLOPS, 4))
    else:
        gbs = (wl.N * wl.D * es + wl.N) * K / (us * 1e-6) / 1e9
        out.update(bound="hbm", achieved_gbs=round(gbs, 1), peak=HBM_PEAK_GBS,
                   frac=round(gbs / HBM_PEAK_GBS, 4))
    print(json.dumps(out), flush=True)
    d.free()
    s.close()


if __name__ == "__main__":
    main()
