"""Summaries of rocprofv3 result databases, and the source fingerprint that
ties recorded HBM-traffic figures to the kernel code they were taken on.

    python -m paper_1912_11554_amd.profiling kernels RUN_results.db
        kernel-trace summary (calls, total, average, min, max per kernel)
    python -m paper_1912_11554_amd.profiling counters RUN_results.db
        PMC counter values per dispatch (summed over the counter instances)
    python -m paper_1912_11554_amd.profiling fingerprint [KERNEL]
        SHA-256 over the sources KERNEL is built from (default: all of csrc)

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


# Sources that only the HMM kernels are built from; the other kernels'
# fingerprint leaves them out (the HMM kernels include every shared header).
HMM_ONLY_SOURCES = ("hmm_impl.h", "hmm.hip", "hmm_ext.hip")
# Host-only sources (argument checks, staging, launch choices): no kernel is
# built from them, so no kernel's fingerprint covers them.
HOST_ONLY_SOURCES = ("api.cpp",)


def is_hmm_kernel(kernel: str) -> bool:
    return "hmm" in kernel


def source_fingerprint(kernel: str | None = None) -> str:
    """SHA-256 over the device and host sources a kernel is built from (file
    names and contents, sorted): any change to them gives a new value.  With
    no kernel named, over all of csrc."""
    h = hashlib.sha256()
    for path in sorted(glob.glob(os.path.join(HERE, "csrc", "*"))):
        base = os.path.basename(path)
        if kernel is not None and base in HOST_ONLY_SOURCES:
            continue
        if kernel is not None and not is_hmm_kernel(kernel) and base in HMM_ONLY_SOURCES:
            continue
        h.update(base.encode())
        with open(path, "rb") as f:
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
