"""Summaries of rocprofv3 result databases, and the source fingerprint that
ties recorded HBM-traffic figures to the kernel code they were taken on.

    python -m paper_1912_11554_amd.profiling kernels RUN_results.db
        kernel-trace summary (calls, total, average, min, max per kernel)
    python -m paper_1912_11554_amd.profiling counters RUN_results.db
        PMC counter values per dispatch (summed over the counter instances)
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
    else:
        sys.exit(__doc__)


if __name__ == "__main__":
    main(sys.argv[1:])
