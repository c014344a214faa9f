"""Summaries of rocprofv3 result databases, and the source fingerprint that
ties recorded HBM-traffic figures to the kernel code they were taken on.

    python -m paper_1912_11554_amd.profiling kernels RUN_results.db
        kernel-trace summary (calls, total, average, min, max per kernel)
    python -m paper_1912_11554_amd.profiling counters RUN_results.db
        PMC counter values per dispatch (summed over the counter instances)
    python -m paper_1912_11554_amd.profiling traffic FETCH.db WRITE.db BENCH.json
        the HBM-traffic record bench.py reads (profiles/traffic.json) from a
        FETCH_SIZE (+ SQ_INSTS_VALU) run and a WRITE_SIZE (+
        TCC_EA0_RDREQ_DRAM_32B_sum) run of bench.py --copy-mb 256 and that
        run's JSON line
    python -m paper_1912_11554_amd.profiling fingerprint [KERNEL]
        SHA-256 over the sources KERNEL is built from (its translation units,
        the csrc headers they include and include/nuts.h; default: all of
        csrc)

The databases are the SQLite files rocprofv3 writes (`-d DIR -o NAME`).
"""
from __future__ import annotations

import collections
import glob
import hashlib
import os
import sqlite3
import sys

HERE = os.path.dirname(os.path.abspath(__file__))


# The translation units each kernel is compiled in; its fingerprint covers
# them and every csrc header they include, directly or through another
# header (the include directive lines are followed, nothing else).
KERNEL_UNITS = {
    "potential_grad_kernel": ("potential.hip",),
    "potential_items_kernel": ("potential.hip",),
    "sampler_grid_kernel": ("sampler.hip", "sampler_f32.hip", "sampler_f64.hip", "sampler_ext_f32.hip",
                            "sampler_ext_f64.hip"),
    "sampler_wave_kernel": ("sampler.hip", "sampler_f32.hip", "sampler_f64.hip", "sampler_ext_f32.hip",
                            "sampler_ext_f64.hip"),
    "sampler_batch_kernel": ("batch.hip",),
    "batch_pass_kernel": ("batch.hip",),
    "batch_ll_kernel": ("batch.hip",),
    "sampler_hmm_kernel": ("hmm.hip", "hmm_ext.hip"),
    "hmm_potential_kernel": ("hmm.hip", "hmm_ext.hip"),
}


def kernel_sources(kernel: str) -> list[str]:
    """The csrc files a kernel is built from: its translation units and the
    closure of their local includes."""
    csrc = os.path.join(HERE, "csrc")
    todo = list(KERNEL_UNITS[kernel])
    seen = set()
    while todo:
        base = todo.pop()
        if base in seen or not os.path.exists(os.path.join(csrc, base)):
            continue
        seen.add(base)
        with open(os.path.join(csrc, base)) as f:
            for line in f:
                line = line.strip()
                if line.startswith("#include \""):
                    inc = line.split('"')[1]
                    if "/" not in inc:
                        todo.append(inc)
    # the public header's record layouts (nuts_stats) are written by the kernels
    return sorted(seen) + ["../../include/nuts.h"]


def source_fingerprint(kernel: str | None = None) -> str:
    """SHA-256 over the sources a kernel is built from (file names and
    contents, sorted): a change to any of them gives a new value, a change
    elsewhere does not.  With no kernel named, over all of csrc."""
    h = hashlib.sha256()
    if kernel is None:
        files = sorted(os.path.basename(p) for p in glob.glob(os.path.join(HERE, "csrc", "*")))
    else:
        files = kernel_sources(kernel)
    for base in files:
        h.update(base.encode())
        with open(os.path.normpath(os.path.join(HERE, "csrc", base)), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _short(name: str) -> str:
    name = name.replace("(anonymous namespace)::", "")
    cut = name.find("(")
    return (name[:cut] if cut > 0 else name).replace("void ", "")


def kernel_rows(db: str):
    """[(kernel, calls, total_ns, avg_ns, min_ns, max_ns)] by total time."""
    c = sqlite3.connect(db)
    agg = collections.OrderedDict()
    for name, dur in c.execute("select name, end - start from kernels order by start"):
        agg.setdefault(_short(name), []).append(int(dur))
    rows = [(k, len(v), sum(v), sum(v) / len(v), min(v), max(v)) for k, v in agg.items()]
    return sorted(rows, key=lambda r: -r[2])


def counter_rows(db: str):
    """[(dispatch_id, kernel, {counter: value summed over instances})]."""
    c = sqlite3.connect(db)
    per = collections.OrderedDict()
    for did, name, cn, cv in c.execute(
            "select dispatch_id, name, counter_name, counter_value from pmc_events order by dispatch_id"):
        d = per.setdefault(did, (_short(name), collections.defaultdict(float)))
        d[1][cn] += cv
    return [(did, k, dict(v)) for did, (k, v) in per.items()]


# The dispatch that times each workload in a run of bench.py: the last one
# of its kernel instantiation (the full-protocol calls, the warmup call and,
# for the standalone pass, the warmup launches all come before it).
TIMED_DISPATCH = {
    "covtype_n581012_d55_f32": ("sampler_grid_kernel", "sampler_grid_kernel<float, 8, 8, 1, false>"),
    "covtype_n581012_d55_f64": ("sampler_grid_kernel", "sampler_grid_kernel<double, 8, 8, 1, false>"),
    "stream_n4m_d257_f32": ("sampler_grid_kernel", "sampler_grid_kernel<float, 32, 10, 5, false>"),
    "shared256_n200000_d129_f32": ("sampler_batch_kernel", "sampler_batch_kernel<8, 3, false>"),
    "chains4096_n500_d9_f64": ("sampler_wave_kernel", "sampler_wave_kernel<double, 1, 16, true, false>"),
    "hmm_t600_tsup100_k3_v10": ("sampler_hmm_kernel", "sampler_hmm_kernel<3, false>"),
}
STANDALONE_DISPATCH = {
    "covtype_n581012_d55_f32": "potential_grad_kernel<float, 8, 8>",
    "covtype_n581012_d55_f64": "potential_grad_kernel<double, 8, 8>",
}
# the standalone pass beside a per-chain workload's line: one call, one
# position for every chain's data set
ITEMS_DISPATCH = {
    "chains4096_n500_d9_f64": "potential_items_kernel<double, 1, 16>",
}
KIB = 1024
TRAFFIC_NOTE = ("HBM bytes per gradient evaluation of each workload's timed dispatch in a run of bench.py "
                "(--copy-mb 256) under rocprofv3 --pmc: FETCH_SIZE and WRITE_SIZE (KiB, summed over instances) "
                "scaled by the same counter on the run's 256 MiB calibration copy; SQ_INSTS_VALU per evaluation; "
                "TCC_EA0_RDREQ_DRAM_32B_sum x 32 bytes (reads bound for the HBM side, Infinity Cache hits "
                "included) per evaluation; each entry holds the fingerprint of the sources its kernel is built "
                "from (python -m paper_1912_11554_amd.profiling fingerprint KERNEL)")


def _bench_evals(line: dict) -> dict:
    """Gradient evaluations of each workload's timed call in a bench.py line."""
    ev = {line["config"]["workload"]: line["grad_evals"]}
    if line.get("also"):
        ev[line["also"]["workload"]] = line["also"]["grad_evals"]
    for name, sub in (line.get("workloads") or {}).items():
        ev[name] = sub["grad_evals"]
    if line.get("hmm"):
        ev[line["hmm"]["workload"]] = line["hmm"]["grad_evals"]
    return ev


def traffic_record(fetch_db: str, write_db: str, bench_line: dict) -> dict:
    """HBM bytes per gradient evaluation of each timed dispatch: FETCH_SIZE
    and WRITE_SIZE (KiB) scaled by the same counter on the run's calibration
    copy (the first __amd_rocclr_copyBuffer: bench.py --copy-mb 256 moves 256
    MiB each way), SQ_INSTS_VALU per evaluation where the fetch run took it,
    and the 32-byte read requests bound for HBM (TCC_EA0_RDREQ_DRAM_32B_sum)
    where the write run took them."""
    fetch, write = counter_rows(fetch_db), counter_rows(write_db)

    def calib(rows, counter):
        for _, k, c in rows:
            if "copyBuffer" in k and counter in c:
                return c[counter]
        raise SystemExit(f"no calibration copy with {counter}")

    def last(rows, name):
        m = [c for _, k, c in rows if k.endswith(name)]
        if not m:
            raise SystemExit(f"no dispatch of {name}")
        return m[-1]

    known = 256 * 1024  # KiB each way
    fscale = known / calib(fetch, "FETCH_SIZE")
    wscale = known / calib(write, "WRITE_SIZE")
    dram_counter = "TCC_EA0_RDREQ_DRAM_32B_sum"
    entries = {}

    def add(kernel, workload, name, evals):
        f, w = last(fetch, name), last(write, name)
        e = dict(fetch_bytes_per_eval=round(f["FETCH_SIZE"] * fscale * KIB / evals),
                 write_bytes_per_eval=round(w["WRITE_SIZE"] * wscale * KIB / evals), evals=evals,
                 fetch_kib=f["FETCH_SIZE"], write_kib=w["WRITE_SIZE"], fetch_scale=round(fscale, 4),
                 write_scale=round(wscale, 4), fingerprint=source_fingerprint(kernel))
        if "SQ_INSTS_VALU" in f:
            e["valu_instructions_per_eval"] = round(f["SQ_INSTS_VALU"] / evals, 1)
        if dram_counter in w:
            e["hbm_read_requests_bytes_per_eval"] = round(w[dram_counter] * 32 / evals)
        entries[f"{kernel}/{workload}"] = e

    for workload, evals in _bench_evals(bench_line).items():
        if workload in TIMED_DISPATCH:
            kernel, name = TIMED_DISPATCH[workload]
            add(kernel, workload, name, evals)
        if workload in STANDALONE_DISPATCH and bench_line.get("standalone_grad") is not None:
            add("potential_grad_kernel", workload, STANDALONE_DISPATCH[workload], 1)
    for workload, sub in (bench_line.get("workloads") or {}).items():
        sa = sub.get("standalone_grad")
        if sa and workload in ITEMS_DISPATCH:
            add("potential_items_kernel", workload, ITEMS_DISPATCH[workload], sa["positions_per_call"])
    return entries


def main(argv):
    if len(argv) < 1:
        sys.exit(__doc__)
    cmd = argv[0]
    if cmd == "fingerprint":
        print(source_fingerprint(argv[1] if len(argv) > 1 else None))
    elif cmd == "kernels":
        print("| kernel | calls | total (us) | average (us) | min (us) | max (us) |")
        print("|---|---:|---:|---:|---:|---:|")
        for k, n, tot, avg, mn, mx in kernel_rows(argv[1]):
            print(f"| {k} | {n} | {tot / 1e3:.1f} | {avg / 1e3:.2f} | {mn / 1e3:.2f} | {mx / 1e3:.2f} |")
    elif cmd == "counters":
        rows = counter_rows(argv[1])
        names = sorted({cn for _, _, d in rows for cn in d})
        print("| dispatch | kernel | " + " | ".join(names) + " |")
        print("|---:|---|" + "---:|" * len(names))
        for did, k, d in rows:
            print(f"| {did} | {k} | " + " | ".join(f"{d.get(cn, 0):.0f}" for cn in names) + " |")
    elif cmd == "traffic":
        import json
        with open(argv[3]) as f:
            line = json.loads([x for x in f.read().splitlines() if x.startswith("{")][-1])
        rec = dict(note=TRAFFIC_NOTE, kernels=traffic_record(argv[1], argv[2], line))
        print(json.dumps(rec, indent=1))
    else:
        sys.exit(__doc__)


if __name__ == "__main__":

    main(sys.argv[1:])
