/*
 * nuts.h -- C ABI of the MI355X (gfx950) iterative No-U-Turn sampler for
 * Bayesian logistic regression (and a semi-supervised hidden Markov model,
 * declared at the end).
 *
 * What is computed (arXiv 1912.11554):
 *   - the model of Appendix B / Fig. 1a: weights m ~ N(0, 1), intercept
 *     b ~ N(0, 1), y_i ~ Bernoulli(logits = x_i . m + b).  Here the intercept
 *     is a column of ones inside X and every weight has prior N(0, s^2), so
 *       U(w)  = sum_i [softplus(eta_i) - y_i eta_i] + |w|^2 / (2 s^2)
 *               + D (ln s + ln(2 pi) / 2),                eta = X w,
 *       dU/dw = X^T (sigmoid(eta) - y) + w / s^2;
 *   - NUTS trajectory doubling with the iterative tree builder of
 *     Appendix A, Alg. 2 (even leaves kept in S[BitCount(n)], U-turn checks
 *     at odd leaves against the candidate set C(n)), the leapfrog integrator
 *     (Section 3.1), Hoffman & Gelman's endpoint U-turn criterion and
 *     divergence threshold 1000, multinomial selection inside subtrees and
 *     biased progressive selection between doublings (Betancourt 2017);
 *   - random draws from Philox4x64-10 keyed by (seed, chain) with counter
 *     (iteration, tag << 32 | doubling, leaf or block, 0), so every draw is
 *     reproducible per (chain, iteration, doubling, leaf).
 *
 * Conventions for every entry point:
 *   - X is row-major N x D (float64 or float32 as `dtype` says), D counting
 *     the ones column; y holds N bytes equal to 0 or 1.  With
 *     NUTS_DATA_PER_CHAIN, X is [C][N][D] and y is [C][N].
 *   - Every pointer argument may be host or device memory; the library
 *     finds out which.  Inputs are borrowed for the call only and never
 *     retained or freed.  Outputs are caller-allocated.
 *   - Calls are synchronous: they return after the outputs are written.  Work
 *     runs on the stream given to nuts_init.
 *   - Every call returns NUTS_OK or a negative code; nuts_last_error gives a
 *     message.  The library never aborts or exits.  A handle is used by one
 *     thread at a time.
 */
#ifndef NUTS_H
#define NUTS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct nuts_handle nuts_handle;
typedef struct nuts_data nuts_data;

enum {
    NUTS_OK = 0,
    NUTS_EINVAL = -1,       /* bad argument: null pointer, bad size, non-finite scale, y not 0/1 */
    NUTS_ENOMEM = -2,       /* device allocation failed */
    NUTS_EDEVICE = -3,      /* HIP runtime error, or a kernel reported a failure */
    NUTS_EUNSUPPORTED = -4  /* a shape no kernel path handles (see nuts_last_error) */
};

enum { NUTS_F64 = 0, NUTS_F32 = 1 };

enum {
    NUTS_DATA_PER_CHAIN = 1u << 0,  /* X is [C][N][D] and y is [C][N]; else one shared data set */
    NUTS_ADAPT_DIAG_MASS = 1u << 1,    /* set the diagonal inverse mass from warmup draws */
    NUTS_UTURN_GENERALIZED = 1u << 2,  /* U-turn on momentum sums (Betancourt 2017, App. A.4.2) */
    NUTS_ADAPT_STEP_SIZE = 1u << 3,    /* adapt the step size during warmup (dual averaging) */
    NUTS_SUBTREE_MERGE = 1u << 4       /* subtree proposals chosen at the merges of halves */
};

/* Kernel path selection for nuts_sample_data (opts->path). */
enum {
    NUTS_PATH_AUTO = 0,
    NUTS_PATH_WAVE = 1,  /* one wavefront per chain, whole tree on device */
    NUTS_PATH_GRID = 2,  /* one chain over the whole GPU, grid barrier per leapfrog step */
    NUTS_PATH_BATCH = 3  /* many chains on shared fp32 data: one leapfrog step of every chain
                            per pass, the gradients as a matrix product on the matrix cores */
};

/* One record per (chain, kept sample).  56 bytes, no implicit padding. */
typedef struct {
    double potential_energy;  /* U at the emitted sample */
    double energy;            /* U + K of the emitted sample and its momentum */
    double accept_prob;       /* mean over generated leaves of min(1, exp(H0 - H)) */
    int32_t tree_depth;       /* doublings performed, counting a rejected last one */
    int32_t num_steps;        /* leapfrog steps = gradient evaluations this iteration */
    int32_t proposal_index;   /* signed leapfrog offset of the sample from the start point */
    int32_t term_leaf;        /* leaf of the last subtree where it stopped; -1 none; -2 U-turn of the whole trajectory */
    uint32_t direction_bits;  /* bit j set iff doubling j went forward in time */
    uint8_t diverging;        /* the last subtree hit H - H0 > 1000 (or NaN) */
    uint8_t turning;          /* stopped by a U-turn (inside the last subtree or across the trajectory) */
    uint8_t hit_max_depth;    /* all max_tree_depth doublings completed */
    uint8_t _pad[9];
} nuts_stats;

/* Create a handle on device `device_ordinal`.  `hip_stream` is a hipStream_t
 * to run on (not owned), or NULL for a stream the handle creates. */
int nuts_init(nuts_handle** out, int device_ordinal, void* hip_stream);

/* Release a handle and every device buffer it owns.  NULL is a no-op. */
void nuts_free(nuts_handle* h);

/* Message describing the last failure on this handle ("" if none).  With a
 * NULL handle, the message of the last failed nuts_init. */
const char* nuts_last_error(const nuts_handle* h);

/* Copy X and y into the library's device layout (64-row column blocks, the
 * dtype kept) once, for repeated use.  num_datasets is 1 for shared data, or
 * C for per-chain data ([C][N][D] and [C][N]).  The result belongs to the
 * handle and must be released with nuts_data_free before nuts_free. */
int nuts_data_create(nuts_handle* h, const void* X, const uint8_t* y, int64_t N, int64_t D,
                     int dtype, int64_t num_datasets, nuts_data** out);
void nuts_data_free(nuts_handle* h, nuts_data* d);

/* Potential and gradient (Appendix B model) at K positions W [K][D].  With
 * shared data every row of W is evaluated on the same X; with per-chain data
 * row k uses data set k (K must equal num_datasets).  Writes out_U [K] and
 * out_grad [K][D] (fp64).  U and the gradient are accumulated in fp64 also
 * for fp32 X.  Large data sets are split over several workgroups per
 * position whose partial sums meet in device memory; many small items
 * (D <= 64, at most 32 row blocks of the layout each, K >= 64) take one
 * wavefront each. */
int nuts_data_potential_grad(nuts_handle* h, const nuts_data* d, double prior_scale,
                             const double* W, int64_t K, double* out_U, double* out_grad);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * quantities of nuts_data_potential_grad from the same kernel, with its
 * partial-sum slots in a fixed device array of the library (8 MiB per
 * device, held from nuts_init until the process ends) instead of handle
 * memory.  It allocates nothing, copies nothing and does not wait:
 *   - W [K][D], out_U [K] and out_grad [K][D] must be device memory
 *     (NUTS_EINVAL otherwise);
 *   - the call only enqueues the potential kernel on the handle's stream and
 *     returns; the outputs are ready once that stream has reached this
 *     point (synchronise it, or order later work after it);
 *   - 1 <= K <= 16384, and K x G x partial_width(D) doubles of partial sums
 *     must fit in the array's 8 MiB (G = groups per position, about
 *     num_CUs / K; one group per position for K >= num_CUs): with D <= 64 up
 *     to about 8 000 positions, with D <= 320 about 2 700; larger requests
 *     fail with NUTS_EINVAL and a message giving the sizes.  Many small items
 *     (D <= 64, data sets of at most 32 row blocks, K >= 64) are evaluated
 *     one wavefront an item and use no partial sums, so only K <= 16384
 *     applies to them;
 *   - every call on one device shares that device's array (each call leaves
 *     the slots it used empty for the next): calls that overlap on one
 *     device (different streams or handles, or host threads) race and give
 *     wrong results (a position whose partial sums another call took gets
 *     NaN after about 2 s); calls in one stream are ordered and safe.
 * Results are bitwise identical to nuts_data_potential_grad's. */
int nuts_data_potential_grad_noalloc(nuts_handle* h, const nuts_data* d, double prior_scale,
                                     const double* W, int64_t K, double* out_U, double* out_grad);

/* The same quantities for K positions on shared fp32 data, computed as one
 * contraction: E = X W^T (N x D by D x K) and G = X^T R (D x N by N x K) on
 * the fp32 matrix cores, with R = sigmoid(E) - y elementwise (the batched
 * form of the gradient in Section 3.1's vectorized setting).  X and W enter
 * the products as fp32 (W is rounded to fp32 for the likelihood terms; the
 * prior uses W in fp64), products accumulate in fp32 per row range, and the
 * per-position sums of the loss and of the partial rows are fp64.  Relative
 * error versus fp64 arithmetic on the same fp32 X is ~1e-6.  NUTS_EUNSUPPORTED
 * for fp64 data, per-chain data or D > 132.  The first call on a data set
 * builds a second device copy of X in the row-stage layout this path reads
 * (kept until nuts_data_free). */
int nuts_data_potential_grad_batched(nuts_handle* h, const nuts_data* d, double prior_scale,
                                     const double* W, int64_t K, double* out_U, double* out_grad);

/* One-shot form of the above for a single position w [D]: lays out X and y,
 * evaluates, releases.  N = 0 is allowed (the prior alone). */
int nuts_potential_grad(nuts_handle* h, const void* X, const uint8_t* y, int64_t N, int64_t D,
                        int dtype, double prior_scale, const double* w, double* out_U,
                        double* out_grad);

/* Log-likelihood of the model at S draws W [S][D] (Section 3.2: the
 * vectorised log-likelihood and posterior predictive of the Fig. 1 logistic
 * model, mapped over posterior draws):
 *   out_ll[s]        = sum_i log p(y_i | x_i, w_s) = -sum_i softplus((1 - 2 y_i) x_i . w_s),
 *   out_elpd[0]      = log((1/S) sum_s exp(out_ll[s]))        (may be NULL),
 *   out_pred_mean[i] = (1/S) sum_s sigmoid(x_i . w_s), [N]    (may be NULL).
 * fp32 data with D <= 132: one pass of matrix-core products over X per 128
 * draws (E = X W^T, fp32 products and row terms, fp64 sums); otherwise the
 * streaming potential kernel per draw (fp64 data keeps fp64 arithmetic),
 * and then out_pred_mean must be NULL (NUTS_EUNSUPPORTED).  One shared data
 * set (NUTS_EINVAL for per-chain data); 1 <= S <= 65535; W, out_ll and the
 * other outputs may be host or device memory. */
int nuts_data_log_likelihood(nuts_handle* h, const nuts_data* d, const double* W, int64_t S, double* out_ll,
                             double* out_elpd, double* out_pred_mean);

/* Posterior predictive samples at S draws W [S][D] (Section 3.2 / Fig. 1c:
 * the model run forward at each posterior draw, vectorised over the draws):
 *   out_y[s][i] = 1 if u_si < sigmoid(x_i . w_s) else 0,   [S][N] bytes,
 * u_si the 53-bit uniform from word i % 4 of the Philox4x64-10 block keyed
 * (seed, s) at counter (0, 7 << 32, i / 4, 0).  The prior predictive is the
 * same call with W drawn from the prior.  Computed in the matrix-core pass of
 * nuts_data_log_likelihood (fp32 products and fp32 sigmoid, compared with the
 * uniform in fp64), so fp32 data with D <= 132 only (else NUTS_EUNSUPPORTED);
 * one shared data set; 1 <= S <= 65535; W and out_y may be host or device
 * memory. */
int nuts_data_posterior_predictive(nuts_handle* h, const nuts_data* d, const double* W, int64_t S, uint64_t seed,
                                   uint8_t* out_y);

/* Options of nuts_sample_data; a NULL pointer means all defaults. */
typedef struct {
    const double* init_q;      /* [C][D] start positions, or NULL for zeros */
    int64_t first_iter;        /* global index of the first iteration (the RNG counter) */
    double* out_final_q;       /* [C][D] state after the last iteration, or NULL */
    double* out_inv_mass;      /* [C][D] inverse mass in use at the end, or NULL */
    int64_t* out_grad_evals;   /* [1] gradient evaluations of the whole call, or NULL */
    int32_t path;              /* NUTS_PATH_* */
    int32_t _reserved;
    double target_accept;      /* NUTS_ADAPT_STEP_SIZE: target acceptance in (0, 1); 0 = 0.8 */
    double* out_step_size;     /* [C] step size in use at the end (the adapted one), or NULL */
    double* out_kernel_ms;     /* [1] milliseconds between HIP events recorded on the handle's stream
                                  right before the first sampler kernel launch and right after the
                                  last (set-up kernels and read-backs excluded), or NULL */
} nuts_sample_opts;

/* Run num_chains chains for num_warmup + num_samples iterations on prepared
 * data, all on the device with no host round trip per leapfrog step.  Each
 * chain starts at init_q (zeros by default) with the gradient evaluated
 * there.  Iteration k of the call has global index first_iter + k; the first
 * num_warmup iterations are not emitted.  inv_mass_diag is [D] (shared by
 * all chains) or NULL for the identity.
 *
 * Warmup adaptation (the paper adapts step size and mass during warmup,
 * Section 2; its covtype step size came from 150 adaptation steps):
 *   - NUTS_ADAPT_DIAG_MASS alone: the inverse mass is re-set at the end of
 *     warmup from the variance of the warmup states in [num_warmup/2,
 *     num_warmup), shrunk towards 1e-3 with weight 5/(n+5) and scaled to
 *     mean one (the step size stays fixed).
 *   - NUTS_ADAPT_STEP_SIZE: before the first iteration the step size moves
 *     from step_size by Hoffman & Gelman's (2014) Alg. 4 heuristic (doubling
 *     or halving until one leapfrog step from a fresh momentum crosses half
 *     the density); every warmup iteration then updates it by their dual
 *     averaging (Section 3.2: gamma 0.05, t0 10, kappa 0.75, mu = log(10
 *     eps), target acceptance opts->target_accept, the accept statistic
 *     being the iteration's mean of min(1, exp(H0 - H)) over its leaves);
 *     sampling uses the averaged step size.  With NUTS_ADAPT_DIAG_MASS as
 *     well, the inverse mass comes from windowed warmup: slow windows of
 *     25, 50, 100, ... iterations after an initial buffer of 75 (the last
 *     stretched to a terminal buffer of 50; 15 % / 75 % / 10 % of warmup
 *     below 150 iterations; none below 20), each ending with the inverse mass
 *     set to the window's variance shrunk as above (not normalised) and the
 *     heuristic and dual averaging restarted.
 *   The step size in use at the end goes to opts->out_step_size.
 * Writes out_samples [C][S][D] fp64 and out_stats [C][S] (either may be
 * NULL).  Divergences are not errors.  NUTS_EINVAL for target_accept outside
 * (0, 1). */
/* NUTS_UTURN_GENERALIZED replaces Hoffman & Gelman's endpoint test (the
 * default; the paper's Alg. 1/2 leave the criterion open) by the
 * generalised one: a subtree or the whole trajectory turns when the
 * momentum sum rho over its points has rho . M^-1 p <= 0 at either end.  The
 * iterative builder then keeps in S[BitCount(n)] the leaf's momentum and the
 * subtree's momentum sum before the leaf; the candidate set C(n) is
 * unchanged. */
/* NUTS_SUBTREE_MERGE replaces the streaming choice of a subtree's proposal
 * (each new leaf taken with probability its share of the weight so far) by
 * the merge-structured one of Betancourt (2017, App. A.3): inside a subtree
 * every pair of completed equal halves merges, keeping the later half's
 * proposal with probability W_later / (W_earlier + W_later), one uniform per
 * merge under tag 6 indexed by the merge's ordinal among the subtree's
 * 2^j - 1 merges in completion order (the merge of the block of 2^d leaves
 * ending at leaf n is number n - BitCount(n) + d - 1).  The selection distribution is the same; the
 * draws differ.  The iterative builder keeps one waiting block per level
 * (its proposal and weight) in LDS beside S; NUTS_EUNSUPPORTED where a
 * path's tree state then no longer fits a CU. */
int nuts_sample_data(nuts_handle* h, const nuts_data* d, uint32_t flags, double prior_scale,
                     double step_size, const double* inv_mass_diag, int max_tree_depth,
                     int64_t num_warmup, int64_t num_samples, int64_t num_chains, uint64_t seed,
                     double* out_samples, nuts_stats* out_stats, const nuts_sample_opts* opts);

/* One-shot form: lays out X and y, samples, releases.  Argument order follows
 * the problem statement: data, prior, step size, mass, depth, iterations,
 * chains, seed, outputs. */
int nuts_sample(nuts_handle* h, const void* X, const uint8_t* y, int64_t N, int64_t D, int dtype,
                uint32_t flags, double prior_scale, double step_size, const double* inv_mass_diag,
                int max_tree_depth, int64_t num_warmup, int64_t num_samples, int64_t num_chains,
                uint64_t seed, double* out_samples, nuts_stats* out_stats);

/* Semi-supervised hidden Markov model (the HMM benchmark of Section 4 and
 * Appendix C, built as in Stan's semi-supervised example): K hidden states,
 * V observation symbols, one sequence w [T] (bytes < V) whose first Tsup
 * hidden states z [Tsup] (bytes < K) are observed.  The K transition rows
 * and K emission rows are simplexes with uniform Dirichlet priors, sampled
 * through additive log-ratios: a row is softmax(a_0, .., a_{n-2}, 0) and
 * its log Jacobian is the sum of the row's log entries.  A position q holds
 * D = K (K - 1) + K (V - 1) logits: the K - 1 free logits of transition row j
 * at j (K - 1), then those of emission row k at K (K - 1) + k (V - 1).
 *   U(q) = -[ sum over entries x of log x  +  sum_{t < Tsup} log phi_{z_t}(w_t)
 *             + sum_{0 < t < Tsup} log theta_{z_{t-1}}(z_t)
 *             + log p(w_Tsup .. w_{T-1} | z_{Tsup-1}) ],
 * the last term by the forward algorithm (from the uniform distribution,
 * without a transition, when Tsup = 0).  The gradient comes from the
 * backward recursion's expected counts.  Shapes: 2 <= K <= 4, V >= 2,
 * K*K + K*V <= 64, T - Tsup <= 512 (else NUTS_EUNSUPPORTED), T <= 2^30; w and z are
 * checked (NUTS_EINVAL for a symbol >= V or a state >= K).  fp64 throughout.
 *
 * nuts_hmm_potential_grad: U and grad U at num_points positions Q
 * [num_points][D]; writes out_U [num_points] and out_grad [num_points][D]. */
int nuts_hmm_potential_grad(nuts_handle* h, const uint8_t* w, int64_t T, const uint8_t* z, int64_t Tsup, int K,
                            int V, const double* Q, int64_t num_points, double* out_U, double* out_grad);

/* nuts_hmm_sample: NUTS on the model above, one wavefront per chain, with
 * the meaning of every other argument, flag and option as in
 * nuts_sample_data (flags NUTS_ADAPT_DIAG_MASS, NUTS_ADAPT_STEP_SIZE,
 * NUTS_UTURN_GENERALIZED and NUTS_SUBTREE_MERGE; opts->path NUTS_PATH_AUTO
 * or NUTS_PATH_WAVE).
 * Chains start at init_q or at q = 0 (uniform rows).  Writes out_samples
 * [C][S][D] (the logits) and out_stats [C][S]. */
int nuts_hmm_sample(nuts_handle* h, const uint8_t* w, int64_t T, const uint8_t* z, int64_t Tsup, int K, int V,
                    uint32_t flags, double step_size, const double* inv_mass_diag, int max_tree_depth,
                    int64_t num_warmup, int64_t num_samples, int64_t num_chains, uint64_t seed, double* out_samples,
                    nuts_stats* out_stats, const nuts_sample_opts* opts);

#ifdef __cplusplus
}
#endif

#endif /* NUTS_H */
