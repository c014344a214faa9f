"""MI355X (gfx950) iterative NUTS for Bayesian logistic regression (and a
semi-supervised hidden Markov model, ``Sampler.hmm_sample``).

Thin ctypes binding over ``libnuts.so`` (C ABI in ``include/nuts.h``): it
marshals numpy arrays or torch tensors (host or device) into pointers and
passes torch's current HIP stream; every step of the sampler runs in the HIP
kernels.  Build the library with ``python -m paper_1912_11554_amd.build``.
There is no CPU fallback: without the built library every call raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnuts.so")

NUTS_OK, NUTS_EINVAL, NUTS_ENOMEM, NUTS_EDEVICE, NUTS_EUNSUPPORTED = 0, -1, -2, -3, -4
NUTS_F64, NUTS_F32 = 0, 1
NUTS_DATA_PER_CHAIN, NUTS_ADAPT_DIAG_MASS, NUTS_UTURN_GENERALIZED, NUTS_ADAPT_STEP_SIZE = 1, 2, 4, 8
NUTS_SUBTREE_MERGE = 16
NUTS_PATH_AUTO, NUTS_PATH_WAVE, NUTS_PATH_GRID, NUTS_PATH_BATCH = 0, 1, 2, 3

EXPORTED = [
    "nuts_init", "nuts_free", "nuts_last_error", "nuts_data_create", "nuts_data_free",
    "nuts_data_potential_grad", "nuts_data_potential_grad_batched", "nuts_potential_grad",
    "nuts_data_log_likelihood", "nuts_sample_data", "nuts_sample",
    "nuts_hmm_potential_grad", "nuts_hmm_sample", "nuts_data_posterior_predictive",
    "nuts_data_potential_grad_noalloc",
]

STATS_DTYPE = np.dtype([
    ("potential_energy", "<f8"), ("energy", "<f8"), ("accept_prob", "<f8"),
    ("tree_depth", "<i4"), ("num_steps", "<i4"), ("proposal_index", "<i4"),
    ("term_leaf", "<i4"), ("direction_bits", "<u4"), ("diverging", "u1"),
    ("turning", "u1"), ("hit_max_depth", "u1"), ("_pad", "u1", (9,)),
])
assert STATS_DTYPE.itemsize == 56


class NutsError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"NUTS error {code}: {msg}")
        self.code = code


class _Opts(ctypes.Structure):
    _fields_ = [
        ("init_q", ctypes.c_void_p),
        ("first_iter", ctypes.c_int64),
        ("out_final_q", ctypes.c_void_p),
        ("out_inv_mass", ctypes.c_void_p),
        ("out_grad_evals", ctypes.c_void_p),
        ("path", ctypes.c_int32),
        ("_reserved", ctypes.c_int32),
        ("target_accept", ctypes.c_double),
        ("out_step_size", ctypes.c_void_p),
        ("out_kernel_ms", ctypes.c_void_p),
    ]


_lib = None


def _torch_runtime_first():
    """With torch in the process there are two HIP runtimes (torch's bundled
    one and the one libnuts.so links).  They coexist when torch's is brought
    up on the device before libnuts.so is loaded; loaded the other way round,
    the second one to initialise has been seen to find no device."""
    try:
        import torch
        if torch.cuda.is_available():
            torch.empty(1, device="cuda")
    except Exception:
        pass


def load_library():
    """Load libnuts.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing; build it with "
                           "`python -m paper_1912_11554_amd.build`")
    _torch_runtime_first()
    L = ctypes.CDLL(LIB_PATH)
    P, i64, u64, i32, u32, dbl = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                  ctypes.c_int, ctypes.c_uint32, ctypes.c_double)
    L.nuts_init.argtypes = [ctypes.POINTER(P), i32, P]
    L.nuts_init.restype = i32
    L.nuts_free.argtypes = [P]
    L.nuts_free.restype = None
    L.nuts_last_error.argtypes = [P]
    L.nuts_last_error.restype = ctypes.c_char_p
    L.nuts_data_create.argtypes = [P, P, P, i64, i64, i32, i64, ctypes.POINTER(P)]
    L.nuts_data_create.restype = i32
    L.nuts_data_free.argtypes = [P, P]
    L.nuts_data_free.restype = None
    L.nuts_data_potential_grad.argtypes = [P, P, dbl, P, i64, P, P]
    L.nuts_data_potential_grad.restype = i32
    L.nuts_data_potential_grad_noalloc.argtypes = [P, P, dbl, P, i64, P, P]
    L.nuts_data_potential_grad_noalloc.restype = i32
    L.nuts_data_potential_grad_batched.argtypes = [P, P, dbl, P, i64, P, P]
    L.nuts_data_potential_grad_batched.restype = i32
    L.nuts_potential_grad.argtypes = [P, P, P, i64, i64, i32, dbl, P, P, P]
    L.nuts_potential_grad.restype = i32
    L.nuts_data_log_likelihood.argtypes = [P, P, P, i64, P, P, P]
    L.nuts_data_log_likelihood.restype = i32
    L.nuts_sample_data.argtypes = [P, P, u32, dbl, dbl, P, i32, i64, i64, i64, u64, P, P,
                                   ctypes.POINTER(_Opts)]
    L.nuts_sample_data.restype = i32
    L.nuts_sample.argtypes = [P, P, P, i64, i64, i32, u32, dbl, dbl, P, i32, i64, i64, i64,
                              u64, P, P]
    L.nuts_sample.restype = i32
    L.nuts_data_posterior_predictive.argtypes = [P, P, P, i64, u64, P]
    L.nuts_data_posterior_predictive.restype = i32
    L.nuts_hmm_potential_grad.argtypes = [P, P, i64, P, i64, i32, i32, P, i64, P, P]
    L.nuts_hmm_potential_grad.restype = i32
    L.nuts_hmm_sample.argtypes = [P, P, i64, P, i64, i32, i32, u32, dbl, P, i32, i64, i64, i64, u64,
                                  P, P, ctypes.POINTER(_Opts)]
    L.nuts_hmm_sample.restype = i32
    _lib = L
    return L


def _ptr(a):
    """Raw pointer of a numpy array or torch tensor (None stays None)."""
    if a is None:
        return None
    if isinstance(a, np.ndarray):
        assert a.flags.c_contiguous
        return a.ctypes.data
    assert a.is_contiguous()
    return a.data_ptr()


def _as_f64(a):
    """An fp64 input as a contiguous numpy array, or a device tensor as is
    (it must already be contiguous fp64)."""
    if a is None:
        return None
    if hasattr(a, "data_ptr") and not isinstance(a, np.ndarray):
        if str(a.dtype) != "torch.float64" or not a.is_contiguous():
            raise TypeError("device inputs must be contiguous float64 tensors")
        return a
    return np.ascontiguousarray(a, dtype=np.float64)


def _dtype_code(X):
    name = str(X.dtype)
    if name.endswith("float64"):
        return NUTS_F64
    if name.endswith("float32"):
        return NUTS_F32
    raise TypeError(f"X must be float64 or float32, got {X.dtype}")


def _current_stream(device: int = 0):
    """torch's current HIP stream on ``device`` (None without torch or GPU)."""
    try:
        import torch
        if torch.cuda.is_available():
            return torch.cuda.current_stream(device).cuda_stream
    except Exception:
        pass
    return None


class Sampler:
    """A handle on one GPU.  ``stream`` defaults to torch's current stream."""

    def __init__(self, device: int = 0, stream=None):
        L = load_library()
        h = ctypes.c_void_p()
        if stream is None:
            stream = _current_stream(device)
        rc = L.nuts_init(ctypes.byref(h), device, stream)
        if rc != NUTS_OK:
            raise NutsError(rc, L.nuts_last_error(None).decode())
        self._L = L
        self._h = h

    def close(self):
        if self._h:
            self._L.nuts_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, rc):
        if rc != NUTS_OK:
            raise NutsError(rc, self._L.nuts_last_error(self._h).decode())

    # ------------------------------------------------------------------
    def data(self, X, y, per_chain: bool = False):
        """Lay out X ([N, D] or, per chain, [C, N, D]) and y once."""
        if per_chain:
            C, N, D = X.shape
        else:
            (N, D), C = X.shape, 1
        out = ctypes.c_void_p()
        self._check(self._L.nuts_data_create(self._h, _ptr(X), _ptr(y), N, D, _dtype_code(X),
                                             C, ctypes.byref(out)))
        return Data(self, out, N, D, C)

    def potential_grad(self, X, y, w, prior_scale=1.0):
        """U and grad U at one position w [D] (float64)."""
        N, D = X.shape
        U = np.zeros(1)
        g = np.zeros(D)
        w = np.ascontiguousarray(w, dtype=np.float64)
        self._check(self._L.nuts_potential_grad(self._h, _ptr(X), _ptr(y), N, D, _dtype_code(X),
                                                prior_scale, _ptr(w), _ptr(U), _ptr(g)))
        return U[0], g

    def sample(self, X, y, *, step_size, max_tree_depth, num_warmup, num_samples,
               num_chains=1, seed=0, prior_scale=1.0, inv_mass=None, per_chain=False,
               adapt_diag_mass=False, **kw):
        """One-shot sampling; see ``Data.sample`` for the outputs."""
        d = self.data(X, y, per_chain=per_chain)
        try:
            return d.sample(step_size=step_size, max_tree_depth=max_tree_depth,
                            num_warmup=num_warmup, num_samples=num_samples,
                            num_chains=num_chains, seed=seed, prior_scale=prior_scale,
                            inv_mass=inv_mass, adapt_diag_mass=adapt_diag_mass, **kw)
        finally:
            d.free()


    # ------------------------------------------------------------------
    @staticmethod
    def _hmm_seq(w, z):
        w = np.ascontiguousarray(w, dtype=np.uint8)
        z = np.zeros(0, np.uint8) if z is None else np.ascontiguousarray(z, dtype=np.uint8)
        return w, z

    def hmm_potential_grad(self, w, z, K, V, Q):
        """Semi-supervised HMM: U [n] and grad U [n, D] at logits Q [n, D],
        D = K (K - 1) + K (V - 1), for symbols w [T] with the first len(z)
        hidden states z observed."""
        w, z = self._hmm_seq(w, z)
        D = hmm_dim(K, V)
        Q = np.ascontiguousarray(Q, dtype=np.float64).reshape(-1, D)
        n = Q.shape[0]
        U, g = np.zeros(n), np.zeros((n, D))
        self._check(self._L.nuts_hmm_potential_grad(self._h, _ptr(w), w.shape[0], _ptr(z), z.shape[0],
                                                    K, V, _ptr(Q), n, _ptr(U), _ptr(g)))
        return U, g

    def hmm_sample(self, w, z, K, V, *, step_size, max_tree_depth, num_warmup, num_samples,
                   num_chains=1, seed=0, inv_mass=None, adapt_diag_mass=False, init_q=None,
                   first_iter=0, adapt_step_size=False, target_accept=0.8,
                   uturn_generalized=False, subtree_merge=False, out_samples=None, out_stats=None,
                   out_final_q=None, out_inv_mass=None, out_step_size=None, time_kernel=False):
        """NUTS on the semi-supervised HMM (one wavefront per chain).  Returns
        the same dict as ``Data.sample``; samples hold the logits (numpy
        unless device tensors are passed in the out_* arguments, which are
        then filled and returned)."""
        w, z = self._hmm_seq(w, z)
        C, D = num_chains, hmm_dim(K, V)
        flags = (NUTS_ADAPT_DIAG_MASS if adapt_diag_mass else 0) | (
            NUTS_ADAPT_STEP_SIZE if adapt_step_size else 0) | (
            NUTS_UTURN_GENERALIZED if uturn_generalized else 0) | (
            NUTS_SUBTREE_MERGE if subtree_merge else 0)
        if out_samples is None:
            out_samples = np.zeros((C, num_samples, D))
        if out_stats is None:
            out_stats = np.zeros((C, num_samples), dtype=STATS_DTYPE)
        final_q = np.zeros((C, D)) if out_final_q is None else out_final_q
        out_im = np.zeros((C, D)) if out_inv_mass is None else out_inv_mass
        out_eps = np.zeros(C) if out_step_size is None else out_step_size
        gev = np.zeros(1, dtype=np.int64)
        im = _as_f64(inv_mass)
        iq = _as_f64(init_q)
        kms = np.zeros(1) if time_kernel else None
        opts = _Opts(_ptr(iq), first_iter, _ptr(final_q), _ptr(out_im), _ptr(gev), NUTS_PATH_AUTO,
                     0, target_accept, _ptr(out_eps), _ptr(kms))
        self._check(self._L.nuts_hmm_sample(
            self._h, _ptr(w), w.shape[0], _ptr(z), z.shape[0], K, V, flags, step_size, _ptr(im),
            max_tree_depth, num_warmup, num_samples, C, seed, _ptr(out_samples), _ptr(out_stats),
            ctypes.byref(opts)))
        return dict(samples=out_samples, stats=out_stats, final_q=final_q, inv_mass=out_im,
                    step_size=out_eps, grad_evals=int(gev[0]),
                    kernel_ms=None if kms is None else float(kms[0]))


def hmm_dim(K, V):
    """Number of logits of the semi-supervised HMM: K (K - 1) + K (V - 1)."""
    return K * (K - 1) + K * (V - 1)


class Data:
    """Data set in the library's device layout (owned by a Sampler)."""

    def __init__(self, sampler, handle, N, D, C):
        self.s, self._d, self.N, self.D, self.num_sets = sampler, handle, N, D, C

    def free(self):
        if self._d:
            self.s._L.nuts_data_free(self.s._h, self._d)
            self._d = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass

    def log_likelihood(self, W, pred_mean=False, out_ll=None):
        """Per-draw log-likelihood ll [S], the expected log-likelihood
        log mean exp(ll), and (pred_mean=True) the mean over the draws of
        P(y_i = 1) [N], for draws W [S, D] (numpy or device tensor)."""
        if isinstance(W, np.ndarray):
            W = np.ascontiguousarray(W, dtype=np.float64).reshape(-1, self.D)
        S = W.shape[0]
        if out_ll is None:
            out_ll = np.zeros(S)
        elpd = np.zeros(1)
        pm = np.zeros(self.N) if pred_mean else None
        self.s._check(self.s._L.nuts_data_log_likelihood(self.s._h, self._d, _ptr(W), S, _ptr(out_ll),
                                                         _ptr(elpd), _ptr(pm)))
        return out_ll, float(elpd[0]), pm

    def posterior_predictive(self, W, seed=0, out_y=None):
        """Posterior predictive samples y [S, N] (uint8) at draws W [S, D]:
        y_si ~ Bernoulli(sigmoid(x_i . w_s)) with keyed uniforms (fp32 data
        on the matrix cores)."""
        if isinstance(W, np.ndarray):
            W = np.ascontiguousarray(W, dtype=np.float64).reshape(-1, self.D)
        S = W.shape[0]
        if out_y is None:
            out_y = np.zeros((S, self.N), dtype=np.uint8)
        self.s._check(self.s._L.nuts_data_posterior_predictive(self.s._h, self._d, _ptr(W), S, seed,
                                                               _ptr(out_y)))
        return out_y

    def potential_grad(self, W, prior_scale=1.0, out_U=None, out_grad=None, batched=False,
                       no_alloc=False):
        """U [K] and grad [K, D] at positions W [K, D] (numpy or device tensor).
        batched=True uses nuts_data_potential_grad_batched (fp32 matrix cores).
        no_alloc=True uses nuts_data_potential_grad_noalloc: W, out_U and
        out_grad must then be device tensors, and the call returns once the
        work is enqueued on the handle's stream (synchronise before reading)."""
        if isinstance(W, np.ndarray):
            W = np.ascontiguousarray(W, dtype=np.float64).reshape(-1, self.D)
        K = W.shape[0]
        if out_U is None:
            out_U = np.zeros(K)
        if out_grad is None:
            out_grad = np.zeros((K, self.D))
        fn = (self.s._L.nuts_data_potential_grad_batched if batched
              else self.s._L.nuts_data_potential_grad_noalloc if no_alloc
              else self.s._L.nuts_data_potential_grad)
        self.s._check(fn(self.s._h, self._d, prior_scale, _ptr(W), K, _ptr(out_U),
                         _ptr(out_grad)))
        return out_U, out_grad

    def sample(self, *, step_size, max_tree_depth, num_warmup, num_samples, num_chains=1,
               seed=0, prior_scale=1.0, inv_mass=None, adapt_diag_mass=False, init_q=None,
               first_iter=0, path=NUTS_PATH_AUTO, out_samples=None, out_stats=None,
               adapt_step_size=False, target_accept=0.8, uturn_generalized=False,
               subtree_merge=False, out_final_q=None, out_inv_mass=None, out_step_size=None,
               time_kernel=False):
        """Run the chains.  Returns a dict: samples [C, S, D], stats [C, S]
        (STATS_DTYPE), final_q [C, D], inv_mass [C, D], step_size [C] (in use
        at the end: the adapted one with adapt_step_size), grad_evals, and
        with time_kernel the milliseconds of the sampler kernel launches
        (kernel_ms).  Outputs are numpy unless device tensors are passed in
        the out_* arguments (then those are filled and returned)."""
        C, D = num_chains, self.D
        flags = (NUTS_DATA_PER_CHAIN if self.num_sets > 1 else 0) | (
            NUTS_ADAPT_DIAG_MASS if adapt_diag_mass else 0) | (
            NUTS_ADAPT_STEP_SIZE if adapt_step_size else 0) | (
            NUTS_UTURN_GENERALIZED if uturn_generalized else 0) | (
            NUTS_SUBTREE_MERGE if subtree_merge else 0)
        if out_samples is None:
            out_samples = np.zeros((C, num_samples, D))
        if out_stats is None:
            out_stats = np.zeros((C, num_samples), dtype=STATS_DTYPE)
        final_q = np.zeros((C, D)) if out_final_q is None else out_final_q
        out_im = np.zeros((C, D)) if out_inv_mass is None else out_inv_mass
        out_eps = np.zeros(C) if out_step_size is None else out_step_size
        gev = np.zeros(1, dtype=np.int64)
        im = _as_f64(inv_mass)
        iq = _as_f64(init_q)
        kms = np.zeros(1) if time_kernel else None
        opts = _Opts(_ptr(iq), first_iter, _ptr(final_q), _ptr(out_im), _ptr(gev), path, 0,
                     target_accept, _ptr(out_eps), _ptr(kms))
        self.s._check(self.s._L.nuts_sample_data(
            self.s._h, self._d, flags, prior_scale, step_size, _ptr(im), max_tree_depth,
            num_warmup, num_samples, C, seed, _ptr(out_samples), _ptr(out_stats),
            ctypes.byref(opts)))
        return dict(samples=out_samples, stats=out_stats, final_q=final_q, inv_mass=out_im,
                    step_size=out_eps, grad_evals=int(gev[0]),
                    kernel_ms=None if kms is None else float(kms[0]))
