"""CPU oracle for the iterative NUTS hot path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It wraps ``nuts_oracle.c`` (plain C,
fp64, sequential sums, no fused multiply-adds) with ctypes and adds the
numpy-side statistics (ESS, MCSE) in ``oracle.ess``.  It shares no code with
the HIP library and the library never imports it.

What each function follows is stated in ``nuts_oracle.c``: Appendix A
(Alg. 1 recursive BuildTree, Alg. 2 IterativeBuildTree) and Appendix B (the
logistic-regression model) of arXiv 1912.11554, Hoffman & Gelman (2014)
Alg. 6, Betancourt (2017) App. A, Salmon et al. (2011) for Philox.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "nuts_oracle.c")
# NUTS_ORACLE_LIB lets a test run load a deliberately broken copy (mutation checks).
_LIB = os.environ.get("NUTS_ORACLE_LIB", os.path.join(_HERE, "liboracle.so"))

# Per-sample statistics; same layout as the library's nuts_stats record.
STATS_DTYPE = np.dtype(
    [
        ("potential_energy", "<f8"),
        ("energy", "<f8"),
        ("accept_prob", "<f8"),
        ("tree_depth", "<i4"),
        ("num_steps", "<i4"),
        ("proposal_index", "<i4"),
        ("term_leaf", "<i4"),
        ("direction_bits", "<u4"),
        ("diverging", "u1"),
        ("turning", "u1"),
        ("hit_max_depth", "u1"),
        ("_pad", "u1", (9,)),
    ]
)
assert STATS_DTYPE.itemsize == 56

TARGET_LOGISTIC = 0
TARGET_LINGAUSS = 1
TARGET_HMM = 2
BUILDER_ITERATIVE = 0
BUILDER_RECURSIVE = 1


SANITIZED_LIB = os.path.join(_HERE, "liboracle_asan.so")


def build(force: bool = True, sanitize: bool = False) -> str:
    """Compile the oracle with gcc (plain C, -ffp-contract=off).  With
    sanitize=True, a separate copy with AddressSanitizer and
    UndefinedBehaviorSanitizer (liboracle_asan.so, aborting on the first
    report); load it by pointing NUTS_ORACLE_LIB at it, with libasan
    preloaded into the interpreter."""
    out = SANITIZED_LIB if sanitize else _LIB
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(_SRC):
        tmp = out + ".tmp%d" % os.getpid()
        extra = (["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=all"] if sanitize else ["-O2"])
        subprocess.check_call(
            ["gcc", *extra, "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
             "-Wall", "-o", tmp, _SRC, "-lm"]
        )
        os.replace(tmp, out)
    return out


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64, u64, dbl, i32 = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_int
        L.orc_philox4x64_10.argtypes = [P, P, P]
        L.orc_u53.argtypes = [u64]
        L.orc_u53.restype = dbl
        L.orc_normals.argtypes = [u64, u64, u64, i64, P]
        L.orc_direction.argtypes = [u64, u64, u64, u64]
        L.orc_direction.restype = i32
        L.orc_u_merge.argtypes = [u64, u64, u64, u64]
        L.orc_u_merge.restype = dbl
        L.orc_u_leaf.argtypes = [u64, u64, u64, u64, u64]
        L.orc_u_leaf.restype = dbl
        L.orc_logistic_ug.argtypes = [P, P, i64, i64, dbl, P, P]
        L.orc_logistic_ug.restype = dbl
        L.orc_logistic_ug_f32.argtypes = [P, P, i64, i64, dbl, P, P]
        L.orc_logistic_ug_f32.restype = dbl
        L.orc_logistic_ug_repeat.argtypes = [P, P, i64, i64, dbl, P, P, i64, i32]
        L.orc_logistic_ug_repeat.restype = dbl
        L.orc_lingauss_ug.argtypes = [P, P, i64, i64, dbl, dbl, P, P]
        L.orc_lingauss_ug.restype = dbl
        L.orc_bitcount.argtypes = [u64]
        L.orc_bitcount.restype = i32
        L.orc_trailing_ones.argtypes = [u64]
        L.orc_trailing_ones.restype = i32
        L.orc_check_range.argtypes = [u64, P, P]
        L.orc_nuts_chain.argtypes = [
            i32, P, P, P, i64, i64, dbl, dbl, dbl, P, i32, i64, i64, u64, u64, i32, i32, P,
            i64, P, P, P, P, P, i64, P, P, i64, P, u64, i32, dbl, P, i32, P, i64, i32, i32, i32,
        ]
        L.orc_nuts_chain.restype = i64
        L.orc_leapfrog_steps.argtypes = [i32, P, P, P, i64, i64, dbl, dbl, P, dbl, i64, P, P]
        L.orc_leapfrog_steps.restype = dbl
        L.orc_is_uturn_exported.argtypes = [P, P, P, P, i32, P, i64]
        L.orc_is_uturn_exported.restype = i32
        L.orc_is_uturn_gen_exported.argtypes = [P, P, P, P, i64]
        L.orc_is_uturn_gen_exported.restype = i32
        L.orc_normals_tagged.argtypes = [u64, u64, u64, u64, i64, P]
        L.orc_dual_avg_run.argtypes = [dbl, dbl, i64, P, P, P]
        L.orc_mass_windows.argtypes = [i64, P, i32]
        L.orc_mass_windows.restype = i32
        L.orc_find_step_size_at.argtypes = [i32, P, P, P, i64, i64, dbl, dbl, P, P, dbl, u64, u64,
                                            u64, P]
        L.orc_find_step_size_at.restype = dbl
        L.orc_log_likelihood.argtypes = [P, P, i64, i64, P, i64, P, P]
        L.orc_posterior_predictive.argtypes = [P, i64, i64, P, i64, u64, u64, P, P, P]
        L.orc_posterior_predictive.restype = None
        L.orc_hmm_ug.argtypes = [P, i64, P, i64, i32, i32, P, P]
        L.orc_hmm_ug.restype = dbl
        L.orc_hmm_ug_repeat.argtypes = [P, i64, P, i64, i32, i32, P, P, i64]
        L.orc_hmm_ug_repeat.restype = dbl
        L.orc_set_warmup_trace.argtypes = [P, i64]
        L.orc_logistic_laplace.argtypes = [P, i32, P, i64, i64, dbl, P, P, P]
        L.orc_logistic_laplace.restype = i64
        L.orc_expected_log_likelihood.argtypes = [P, i64]
        L.orc_expected_log_likelihood.restype = dbl
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _u8(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.uint8)


# ---------------------------------------------------------------- RNG ------
def philox4x64_10(counter, key):
    c = np.ascontiguousarray(counter, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib().orc_philox4x64_10(_p(c), _p(k), _p(out))
    return out


def u53(word: int) -> float:
    return lib().orc_u53(int(word))


def normals(seed, chain, t, D, tag=1):
    """D standard normals from the Philox stream (tag 1: the momentum of
    iteration t; tag 5: the step-size heuristic's momentum)."""
    out = np.zeros(D, dtype=np.float64)
    lib().orc_normals_tagged(seed, chain, t, tag, D, _p(out))
    return out


def direction(seed, chain, t, j):
    return lib().orc_direction(seed, chain, t, j)


def u_merge(seed, chain, t, j):
    return lib().orc_u_merge(seed, chain, t, j)


def u_leaf(seed, chain, t, j, n):
    return lib().orc_u_leaf(seed, chain, t, j, n)


# ------------------------------------------------------------ targets ------
def logistic_potential_grad(X, y, w, prior_scale=1.0):
    """U(w) and dU/dw of the logistic log-joint (Appendix B model), fp64."""
    X = _f64(X)
    y = _u8(y)
    w = _f64(w)
    N, D = X.shape
    g = np.zeros(D, dtype=np.float64)
    U = lib().orc_logistic_ug(_p(X), _p(y), N, D, prior_scale, _p(w), _p(g))
    return U, g


def logistic_potential_grad_f32(Xf, y, w, prior_scale=1.0):
    """Same values over an fp32 X, promoted to fp64 one row at a time."""
    Xf = np.ascontiguousarray(Xf, dtype=np.float32)
    y = _u8(y)
    w = _f64(w)
    N, D = Xf.shape
    g = np.zeros(D, dtype=np.float64)
    U = lib().orc_logistic_ug_f32(_p(Xf), _p(y), N, D, prior_scale, _p(w), _p(g))
    return U, g


def logistic_laplace(X, y, prior_scale=1.0):
    """Normal approximation of the logistic posterior: the MAP by Newton's
    method (iteratively reweighted least squares), the Laplace covariance
    (the inverse Hessian of U there) and the posterior mean to order 1/N^2
    (the mode moved by the skewness of U).  X may be fp64 or fp32 (promoted
    row by row).  Returns dict(w_map, cov, mean, newton_steps)."""
    f32 = X.dtype == np.float32
    X = np.ascontiguousarray(X, dtype=np.float32 if f32 else np.float64)
    y = _u8(y)
    N, D = X.shape
    w = np.zeros(D)
    cov = np.zeros((D, D))
    mean = np.zeros(D)
    steps = lib().orc_logistic_laplace(_p(X), 1 if f32 else 0, _p(y), N, D, prior_scale, _p(w),
                                       _p(cov), _p(mean))
    if steps < 0:
        raise RuntimeError("Newton's method did not converge")
    return dict(w_map=w, cov=cov, mean=mean, newton_steps=int(steps))


def lingauss_potential_grad(X, yv, w, prior_scale=1.0, noise_scale=1.0):
    X = _f64(X)
    yv = _f64(yv)
    w = _f64(w)
    N, D = X.shape
    g = np.zeros(D, dtype=np.float64)
    U = lib().orc_lingauss_ug(_p(X), _p(yv), N, D, prior_scale, noise_scale, _p(w), _p(g))
    return U, g


# ------------------------------------------------------ index logic --------
def bitcount(n):
    return lib().orc_bitcount(n)


def trailing_ones(n):
    return lib().orc_trailing_ones(n)


def check_range(n):
    a = ctypes.c_int()
    b = ctypes.c_int()
    lib().orc_check_range(n, ctypes.byref(a), ctypes.byref(b))
    return a.value, b.value


# ---------------------------------------------------------- sampler --------
def leapfrog(X, y, q, p, h, nsteps, inv_mass=None, prior_scale=1.0, target=TARGET_LOGISTIC,
             yv=None, noise_scale=1.0):
    X = _f64(X)
    N, D = X.shape
    q = _f64(q).copy()
    p = _f64(p).copy()
    im = _f64(np.ones(D) if inv_mass is None else inv_mass)
    U = lib().orc_leapfrog_steps(target, _p(X), _p(_u8(y)), _p(_f64(yv)), N, D, prior_scale,
                                 noise_scale, _p(im), h, nsteps, _p(q), _p(p))
    return q, p, U


def nuts(X, y, *, step_size, max_tree_depth, num_warmup, num_samples, seed, chain=0,
         prior_scale=1.0, inv_mass=None, builder=BUILDER_ITERATIVE, adapt_diag_mass=False,
         init_q=None, first_iter=0, target=TARGET_LOGISTIC, yv=None, noise_scale=1.0,
         trace_cap=0, leaves_cap=0, sel_salt=0, adapt_step_size=False, target_accept=0.8,
         uturn_generalized=False, hmm=None, subtree_merge=False, warmup_trace=False):
    """One chain of NUTS.  Returns a dict with samples [S, D], stats [S],
    final_q [D], inv_mass [D], step_size (the one in use at the end: the
    adapted one with adapt_step_size), grad_evals; with trace_cap the U-turn check
    trace as (first_leaf, last_leaf) pairs; with leaves_cap the generated
    leaves as records (j, n, position, H - H0).  ``sel_salt`` (test only)
    re-keys the proposal-selection draws and nothing else.  uturn_generalized
    selects the momentum-sum criterion (reading R20).  warmup_trace=True
    adds "warmup_q" [W, D] (the state after each warmup iteration) and
    "warmup_eps" [W] (the step size each warmup iteration ran with).  With hmm = dict(w, z,
    K, V) the target is the semi-supervised HMM (reading R21) and X, y are
    ignored.  subtree_merge chooses each subtree's proposal at the merges of
    its halves (reading R22) instead of by the streaming choice."""
    hz = None
    if hmm is not None:
        target = TARGET_HMM
        y = _u8(hmm["w"])
        hz = _u8(hmm["z"])
        N, D = y.shape[0], hmm_dim(hmm["K"], hmm["V"])
        X = np.zeros((1, D))
    else:
        X = _f64(X)
        N, D = X.shape
    samples = np.zeros((num_samples, D), dtype=np.float64)
    stats = np.zeros(num_samples, dtype=STATS_DTYPE)
    final_q = np.zeros(D, dtype=np.float64)
    out_im = np.zeros(D, dtype=np.float64)
    tr = np.zeros(max(2 * trace_cap, 1), dtype=np.int64)
    trlen = ctypes.c_int64(0)
    lv = np.zeros(max(4 * leaves_cap, 1), dtype=np.int64)
    lvlen = ctypes.c_int64(0)
    eps_out = ctypes.c_double(0.0)
    wt = np.zeros((max(num_warmup, 1), D + 1)) if warmup_trace else None
    if warmup_trace:
        lib().orc_set_warmup_trace(_p(wt), num_warmup)
    try:
        nev = lib().orc_nuts_chain(
            target, _p(X), _p(_u8(y)), _p(_f64(yv)), N, D, prior_scale, noise_scale, step_size,
            _p(_f64(inv_mass)), max_tree_depth, num_warmup, num_samples, seed, chain, builder,
            1 if adapt_diag_mass else 0, _p(_f64(init_q)), first_iter, _p(samples), _p(stats),
            _p(final_q), _p(out_im), _p(tr) if trace_cap else None, 2 * trace_cap,
            ctypes.byref(trlen), _p(lv) if leaves_cap else None, 4 * leaves_cap,
            ctypes.byref(lvlen), sel_salt, 1 if adapt_step_size else 0, target_accept,
            ctypes.byref(eps_out), 1 if uturn_generalized else 0, _p(hz),
            0 if hz is None else hz.shape[0], 0 if hmm is None else hmm["K"],
            0 if hmm is None else hmm["V"], 1 if subtree_merge else 0,
        )
    finally:
        if warmup_trace:
            lib().orc_set_warmup_trace(None, 0)
    out = dict(samples=samples, stats=stats, final_q=final_q, inv_mass=out_im,
               step_size=eps_out.value, grad_evals=nev)
    if warmup_trace:
        out["warmup_q"] = wt[:num_warmup, :D].copy()
        out["warmup_eps"] = wt[:num_warmup, D].copy()
    if trace_cap:
        out["trace"] = tr[: trlen.value].reshape(-1, 2)
    if leaves_cap:
        rec = lv[: lvlen.value].reshape(-1, 4)
        out["leaves"] = dict(j=rec[:, 0].copy(), n=rec[:, 1].copy(), pos=rec[:, 2].copy(),
                             dH=rec[:, 3].copy().view(np.float64))
    return out


def is_uturn(qa, pa, qb, pb, v, inv_mass=None):
    qa, pa, qb, pb = (_f64(a) for a in (qa, pa, qb, pb))
    D = qa.shape[0]
    im = _f64(np.ones(D) if inv_mass is None else inv_mass)
    return bool(lib().orc_is_uturn_exported(_p(qa), _p(pa), _p(qb), _p(pb), v, _p(im), D))


# --------------------------------------------------- warmup adaptation -----
def dual_averaging(eps0, delta, alphas):
    """The dual-averaging recursion (Hoffman & Gelman 2014, Section 3.2)
    driven by a given sequence of accept statistics; returns (log eps,
    log eps_bar) after each update."""
    a = _f64(alphas)
    n = a.shape[0]
    le = np.zeros(n)
    lb = np.zeros(n)
    lib().orc_dual_avg_run(eps0, delta, n, _p(a), _p(le), _p(lb))
    return le, lb


def mass_windows(num_warmup):
    """Slow windows [start, end) of the windowed diagonal-mass adaptation."""
    out = np.zeros(128, dtype=np.int64)
    n = lib().orc_mass_windows(num_warmup, _p(out), 64)
    return [(int(out[2 * i]), int(out[2 * i + 1])) for i in range(n)]


def find_step_size(X, y, q, eps, *, seed, chain=0, t=0, inv_mass=None, prior_scale=1.0,
                   target=TARGET_LOGISTIC, yv=None, noise_scale=1.0):
    """Hoffman & Gelman (2014) Alg. 4 from eps at q; returns (eps, gradient
    evaluations)."""
    X = _f64(X)
    N, D = X.shape
    im = _f64(np.ones(D) if inv_mass is None else inv_mass)
    ev = ctypes.c_int64(0)
    e = lib().orc_find_step_size_at(target, _p(X), _p(_u8(y)), _p(_f64(yv)), N, D, prior_scale,
                                    noise_scale, _p(im), _p(_f64(q)), eps, seed, chain, t,
                                    ctypes.byref(ev))
    return e, ev.value


# ------------------------------------------- log-likelihood over draws -----
def log_likelihood(X, y, W):
    """Per-draw log-likelihood ll [S] and posterior predictive mean
    P(y_i = 1) averaged over the draws [N] (Section 3.2), fp64 sums."""
    X = _f64(X)
    N, D = X.shape
    W = _f64(W).reshape(-1, D)
    S = W.shape[0]
    ll = np.zeros(S)
    pm = np.zeros(N)
    lib().orc_log_likelihood(_p(X), _p(_u8(y)), N, D, _p(W), S, _p(ll), _p(pm))
    return ll, pm


def posterior_predictive(X, W, seed, uniforms=False, first_draw=0):
    """Posterior predictive samples y [S, N] (uint8) at draws W [S, D] and
    the probabilities sigmoid(x_i . w_s) [S, N] they were drawn with
    (reading R23: one keyed uniform per (draw, row)); with uniforms=True
    also the uniforms [S, N].  Row s of W is keyed as draw first_draw + s."""
    X = _f64(X)
    N, D = X.shape
    W = _f64(W).reshape(-1, D)
    S = W.shape[0]
    y = np.zeros((S, N), dtype=np.uint8)
    p = np.zeros((S, N))
    u = np.zeros((S, N)) if uniforms else None
    lib().orc_posterior_predictive(_p(X), N, D, _p(W), S, seed, first_draw, _p(y), _p(p), _p(u))
    return (y, p, u) if uniforms else (y, p)


def expected_log_likelihood(ll):
    """logsumexp(ll) - log S."""
    ll = _f64(ll)
    return lib().orc_expected_log_likelihood(_p(ll), ll.shape[0])


def is_uturn_generalized(rho, pa, pb, inv_mass=None):
    """Reading R20's test on a (sub)trajectory with momentum sum rho and end
    momenta pa, pb."""
    rho, pa, pb = (_f64(a) for a in (rho, pa, pb))
    D = rho.shape[0]
    im = _f64(np.ones(D) if inv_mass is None else inv_mass)
    return bool(lib().orc_is_uturn_gen_exported(_p(rho), _p(pa), _p(pb), _p(im), D))


# ------------------------------------------------------------------- HMM ----
def hmm_dim(K, V):
    """Unconstrained dimension: K (K - 1) transition logits, K (V - 1)
    emission logits."""
    return K * (K - 1) + K * (V - 1)


def hmm_potential_grad(w, z, K, V, q):
    """U and grad U of the semi-supervised HMM (reading R21) at logits q."""
    w = _u8(w)
    z = _u8(z)
    q = _f64(q)
    g = np.zeros(q.shape[0])
    U = lib().orc_hmm_ug(_p(w), w.shape[0], _p(z), z.shape[0], K, V, _p(q), _p(g))
    return U, g
