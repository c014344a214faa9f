"""The C-ABI library (CPU-only checks): it loads, exports every function that
include/nuts.h declares, its record layout matches the header, and the
host-side argument checks fail cleanly without touching a GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_1912_11554_amd as nuts

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nuts.h")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(nuts_[a-z_]+)\s*\(", src)))


def test_library_built():
    assert os.path.exists(nuts.LIB_PATH), "run `python -m paper_1912_11554_amd.build` first"


def test_exports_every_declared_function():
    L = ctypes.CDLL(nuts.LIB_PATH)
    declared = _declared_functions()
    assert set(declared) == set(nuts.EXPORTED)
    for name in declared:
        assert hasattr(L, name), name


def test_stats_record_layout_matches_header():
    src = open(HEADER).read()
    body = src[src.index("typedef struct {\n    double potential_energy"):]
    body = body[: body.index("} nuts_stats;")]
    fields = re.findall(r"^\s*(\w+)\s+(\w+)(\[\d+\])?;", body, flags=re.M)
    names = [f[1] for f in fields]
    assert names == list(nuts.STATS_DTYPE.names)
    assert nuts.STATS_DTYPE.itemsize == 56


def test_null_handle_is_rejected():
    L = nuts.load_library()
    assert L.nuts_sample_data(None, None, 0, 1.0, 0.1, None, 5, 0, 1, 1, 0, None, None,
                              None) == nuts.NUTS_EINVAL
    assert L.nuts_data_potential_grad(None, None, 1.0, None, 1, None, None) == nuts.NUTS_EINVAL
    assert L.nuts_data_potential_grad_noalloc(None, None, 1.0, None, 1, None, None) == nuts.NUTS_EINVAL
    L.nuts_free(None)                    # no-op
    L.nuts_data_free(None, None)         # no-op
    assert L.nuts_last_error(None) is not None


def test_init_rejects_null_out():
    L = nuts.load_library()
    assert L.nuts_init(None, 0, None) == nuts.NUTS_EINVAL
    assert b"NULL" in L.nuts_last_error(None)
