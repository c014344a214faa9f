/*
 * CPU oracle for the iterative No-U-Turn sampler on the Bayesian
 * logistic-regression log-joint.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain, obviously correct
 * reference that the GPU path is checked against.  Only the test suite, the
 * package smoke check and the benchmark's CPU-baseline leg may load it.  It
 * shares no source with the HIP library (no headers, no helpers, no tables)
 * and the library never calls it.
 *
 * Everything is fp64, summed sequentially in index order, built with
 * -ffp-contract=off so that no fused multiply-adds change the rounding.
 *
 * Sources restated here (no listing is copied):
 *   - Phan, Pradhan, Jankowiak, "Composable Effects for Flexible and
 *     Accelerated Probabilistic Programming in NumPyro" (arXiv 1912.11554):
 *       Appendix B / Fig. 1a   the logistic-regression model,
 *       Section 3.1            why the tree builder must be iterative,
 *       Appendix A, Alg. 1     recursive BuildTree,
 *       Appendix A, Alg. 2     IterativeBuildTree, the S array indexed by
 *                              BitCount and the candidate set C(n).
 *   - Hoffman & Gelman, "The No-U-Turn Sampler" (JMLR 2014), Alg. 6:
 *       U-turn criterion on the endpoints, random direction per doubling,
 *       divergence threshold Delta_max = 1000.
 *   - Betancourt, "A Conceptual Introduction to Hamiltonian Monte Carlo"
 *     (arXiv 1701.02434), App. A: multinomial trajectory sampling, biased
 *     progressive sampling across doublings.
 *   - Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2,
 *     3" (SC'11): Philox4x64 with 10 rounds.
 *   - Box & Muller (1958) for normal variates.
 *
 * Readings taken where the paper is silent (its Alg. 1/2 omit the proposal,
 * the direction and the step size):
 *   R1  TrailingBit(n) counts the trailing 1 bits of n (so C(11) = {10, 8}).
 *   R2  the check loop of Alg. 2 runs from i_max DOWN to i_min; S has
 *       max(d, 1) slots.
 *   R3  IsUTurn is Hoffman & Gelman's endpoint test on time-ordered ends,
 *       with velocities M^-1 p; a dot product of exactly 0 is not a U-turn.
 *   R4  multinomial weights exp(-H): streaming selection inside a subtree,
 *       biased progressive selection when a subtree is merged.
 *   R5  direction uniform on {-1, +1} per doubling; fixed step size.
 *   R6  a leaf diverges iff !(H - H0 <= 1000); that also catches NaN.
 *   R8  Philox4x64-10, key (seed, chain), counter (t, tag<<32 | j, n, 0).
 *   R13 optional diagonal inverse mass from warmup variance, normalised to
 *       mean one.
 *   R19 warmup adaptation (optional): the step-size heuristic of Hoffman &
 *       Gelman (2014) Alg. 4 from the given step size, then their dual
 *       averaging (Section 3.2, Alg. 5) with target acceptance delta,
 *       gamma = 0.05, t0 = 10, kappa = 0.75, mu = log(10 eps); the accept
 *       statistic of an iteration is the mean over its leaves of
 *       min(1, exp(H0 - H)); after warmup eps = exp(log eps_bar).  Together
 *       with the diagonal mass: the windowed scheme of the Stan reference
 *       manual (initial buffer 75, slow windows of 25, 50, 100, ...
 *       iterations with the last one stretched to the terminal buffer of
 *       50; 15 % / 75 % / 10 % when warmup is shorter than 150; no windows
 *       below 20); at each window end the inverse mass is the regularised
 *       variance of the window's states (weight 5/(n+5) towards 1e-3, not
 *       normalised) and the heuristic and dual averaging restart.
 *   R20 generalised U-turn criterion (optional; Betancourt 2017, App. A.4.2):
 *       a (sub)trajectory with momentum sum rho over all its points turns
 *       iff rho . M^-1 p <= 0 at either end.  The iterative builder keeps in
 *       S[BitCount(n)] the leaf's momentum and the subtree's momentum sum
 *       before that leaf, so the sum over leaves k..n is a difference of
 *       running sums; the trajectory test uses the sum over every point
 *       including the start.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Philox4x64-10 (Salmon et al. 2011).  Round: two 64x64->128 products of the
 * even words with the round multipliers; the odd words and the key are xored
 * into the high halves and the words are permuted.  The key is bumped by the
 * two Weyl constants between rounds.                                         */

#define ORC_PHILOX_M0 0xD2E7470EE14C6C93ULL
#define ORC_PHILOX_M1 0xCA5A826395121157ULL
#define ORC_PHILOX_W0 0x9E3779B97F4A7C15ULL
#define ORC_PHILOX_W1 0xBB67AE8584CAA73BULL

static void orc_mul128(uint64_t a, uint64_t b, uint64_t *hi, uint64_t *lo)
{
    unsigned __int128 p = (unsigned __int128)a * (unsigned __int128)b;
    *hi = (uint64_t)(p >> 64);
    *lo = (uint64_t)p;
}

void orc_philox4x64_10(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4])
{
    uint64_t x0 = ctr_in[0], x1 = ctr_in[1], x2 = ctr_in[2], x3 = ctr_in[3];
    uint64_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += ORC_PHILOX_W0;
            k1 += ORC_PHILOX_W1;
        }
        uint64_t hi0, lo0, hi1, lo1;
        orc_mul128(ORC_PHILOX_M0, x0, &hi0, &lo0);
        orc_mul128(ORC_PHILOX_M1, x2, &hi1, &lo1);
        uint64_t y0 = hi1 ^ x1 ^ k0;
        uint64_t y1 = lo1;
        uint64_t y2 = hi0 ^ x3 ^ k1;
        uint64_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* Draw tags: which random quantity a Philox block feeds (reading R8).
 * ORC_TAG_TREE block b of iteration t (counter {t, TREE << 32, b, 0}) holds
 * the direction of doubling b (word 0), the merge uniform of doubling b
 * (word 1) and the uniforms of leaves 2b and 2b + 1 (words 2, 3), leaves
 * numbered in the order the trajectory generates them: leaf n of doubling j
 * is number 2^j - 1 + n. */
enum { ORC_TAG_MOMENTUM = 1, ORC_TAG_TREE = 2, ORC_TAG_STEP = 5, ORC_TAG_SUBMERGE = 6,
       ORC_TAG_PREDICT = 7 };

static void orc_block(uint64_t seed, uint64_t chain, uint64_t t, uint64_t tag, uint64_t j,
                      uint64_t n, uint64_t out[4])
{
    uint64_t ctr[4] = { t, (tag << 32) | j, n, 0 };
    uint64_t key[2] = { seed, chain };
    orc_philox4x64_10(ctr, key, out);
}

/* 53 high bits of a word -> uniform on [0, 1). */
double orc_u53(uint64_t w) { return (double)(w >> 11) * (1.0 / 9007199254740992.0); }

/* D standard normals under a tag (the momentum of iteration t with
 * ORC_TAG_MOMENTUM): block b gives four uniforms, i.e. two Box-Muller pairs,
 * i.e. normals 4b .. 4b+3. */
void orc_normals_tagged(uint64_t seed, uint64_t chain, uint64_t t, uint64_t tag, int64_t D,
                        double *out)
{
    const double two_pi = 6.283185307179586476925286766559;
    for (int64_t b = 0; 4 * b < D; ++b) {
        uint64_t w[4];
        orc_block(seed, chain, t, tag, 0, (uint64_t)b, w);
        for (int pair = 0; pair < 2; ++pair) {
            double ua = orc_u53(w[2 * pair]);
            double ub = orc_u53(w[2 * pair + 1]);
            double r = sqrt(-2.0 * log(1.0 - ua));
            double th = two_pi * ub;
            int64_t i0 = 4 * b + 2 * pair;
            if (i0 < D) out[i0] = r * cos(th);
            if (i0 + 1 < D) out[i0 + 1] = r * sin(th);
        }
    }
}

void orc_normals(uint64_t seed, uint64_t chain, uint64_t t, int64_t D, double *out)
{
    orc_normals_tagged(seed, chain, t, ORC_TAG_MOMENTUM, D, out);
}

/* +1 or -1 for doubling j of iteration t. */
int orc_direction(uint64_t seed, uint64_t chain, uint64_t t, uint64_t j)
{
    uint64_t w[4];
    orc_block(seed, chain, t, ORC_TAG_TREE, 0, j, w);
    return (w[0] & 1ULL) ? +1 : -1;
}

double orc_u_merge(uint64_t seed, uint64_t chain, uint64_t t, uint64_t j)
{
    uint64_t w[4];
    orc_block(seed, chain, t, ORC_TAG_TREE, 0, j, w);
    return orc_u53(w[1]);
}

double orc_u_leaf(uint64_t seed, uint64_t chain, uint64_t t, uint64_t j, uint64_t n)
{
    const uint64_t g = (((uint64_t)1 << j) - 1) + n; /* the leaf's number in the iteration */
    uint64_t w[4];
    orc_block(seed, chain, t, ORC_TAG_TREE, 0, g >> 1, w);
    return orc_u53(w[2 + (g & 1)]);
}

/* Reading R22: the uniform of a merge of two halves inside subtree j, named
 * by its ordinal P among the subtree's 2^j - 1 merges in the order they
 * complete (the merge of the block of 2^d leaves ending at leaf n is number
 * n - BitCount(n) + d - 1). */
double orc_u_submerge(uint64_t seed, uint64_t chain, uint64_t t, uint64_t j, uint64_t P)
{
    uint64_t w[4];
    orc_block(seed, chain, t, ORC_TAG_SUBMERGE, j, P, w);
    return orc_u53(w[0]);
}

int orc_bitcount(uint64_t n);

static uint64_t orc_merge_ordinal(int64_t n, int d)
{
    return (uint64_t)(n - (int64_t)orc_bitcount((uint64_t)n) + d - 1);
}

/* ------------------------------------------------------------------------- */
/* Targets: U(w) = -log joint and its gradient.                              */

/* Bayesian logistic regression (Appendix B): weights m ~ N(0, 1) per feature,
 * intercept b ~ N(0, 1), y_i ~ Bernoulli(logits = x_i . m + b).  The intercept
 * is the last (or any) column of ones in X, sharing the N(0, s^2) prior, so
 *   U(w)  = sum_i [softplus(eta_i) - y_i eta_i] + sum_j w_j^2 / (2 s^2)
 *           + D (ln s + ln(2 pi) / 2),           eta = X w,
 *   dU/dw = X^T (sigmoid(eta) - y) + w / s^2.
 * Each row term is written as softplus((1 - 2 y_i) eta_i) >= 0 and the
 * residual as (1 - 2 y_i) sigmoid((1 - 2 y_i) eta_i), which are the same
 * numbers without cancellation.                                              */
static double orc_softplus(double x) { return fmax(x, 0.0) + log1p(exp(-fabs(x))); }

static double orc_sigmoid(double x)
{
    if (x >= 0.0) return 1.0 / (1.0 + exp(-x));
    double e = exp(x);
    return e / (1.0 + e);
}

double orc_logistic_ug(const double *X, const uint8_t *y, int64_t N, int64_t D, double s,
                       const double *w, double *grad)
{
    for (int64_t j = 0; j < D; ++j) grad[j] = 0.0;
    double U = 0.0;
    for (int64_t i = 0; i < N; ++i) {
        const double *xi = X + i * D;
        double eta = 0.0;
        for (int64_t j = 0; j < D; ++j) eta += xi[j] * w[j];
        double sgn = y[i] ? -1.0 : 1.0;
        double t = sgn * eta;
        U += orc_softplus(t);
        double r = sgn * orc_sigmoid(t);
        for (int64_t j = 0; j < D; ++j) grad[j] += r * xi[j];
    }
    const double half_log_2pi = 0.91893853320467274178032973640562;
    double inv_s2 = 1.0 / (s * s);
    for (int64_t j = 0; j < D; ++j) {
        U += 0.5 * w[j] * w[j] * inv_s2;
        grad[j] += w[j] * inv_s2;
    }
    U += (double)D * (log(s) + half_log_2pi);
    return U;
}

/* Log-likelihood over a batch of draws (Section 3.2, the vectorised
 * log-likelihood and posterior predictive of the Fig. 1 logistic model):
 *   ll[s]        = sum_i log p(y_i | x_i, w_s) = -sum_i softplus((1 - 2 y_i) eta_is),
 *   pred_mean[i] = (1/S) sum_s sigmoid(eta_is)   (may be NULL),
 * eta_is = x_i . w_s; W is [S][D].  Plain sums in index order.           */
void orc_log_likelihood(const double *X, const uint8_t *y, int64_t N, int64_t D, const double *W,
                        int64_t S, double *ll, double *pred_mean)
{
    for (int64_t s = 0; s < S; ++s) ll[s] = 0.0;
    for (int64_t i = 0; i < N; ++i) {
        const double *xi = X + i * D;
        double psum = 0.0;
        for (int64_t s = 0; s < S; ++s) {
            const double *w = W + s * D;
            double eta = 0.0;
            for (int64_t j = 0; j < D; ++j) eta += xi[j] * w[j];
            double sgn = y[i] ? -1.0 : 1.0;
            ll[s] -= orc_softplus(sgn * eta);
            psum += orc_sigmoid(eta);
        }
        if (pred_mean) pred_mean[i] = psum / (double)S;
    }
}

/* Posterior predictive samples (Section 3.2, Fig. 1c: the model run forward
 * at each posterior draw; reading R23): y_si = 1 iff u_si < sigmoid(x_i .
 * w_s), u_si the word i mod 4 of the Philox block keyed (seed, s) at counter
 * (0, 7 << 32, floor(i / 4), 0), s counted from s0 (the index of W's first
 * row among the draws).  Writes y [S][N] bytes and, where not NULL, the
 * probabilities p [S][N] and the uniforms u [S][N].                        */
void orc_posterior_predictive(const double *X, int64_t N, int64_t D, const double *W, int64_t S,
                              uint64_t seed, uint64_t s0, uint8_t *y, double *p, double *u)
{
    for (int64_t s = 0; s < S; ++s) {
        const double *w = W + s * D;
        uint64_t blk[4];
        for (int64_t i = 0; i < N; ++i) {
            const double *xi = X + i * D;
            double eta = 0.0;
            for (int64_t j = 0; j < D; ++j) eta += xi[j] * w[j];
            double prob = orc_sigmoid(eta);
            if ((i & 3) == 0) orc_block(seed, s0 + (uint64_t)s, 0, ORC_TAG_PREDICT, 0, (uint64_t)(i >> 2), blk);
            double ui = orc_u53(blk[i & 3]);
            y[s * N + i] = ui < prob ? 1 : 0;
            if (p) p[s * N + i] = prob;
            if (u) u[s * N + i] = ui;
        }
    }
}

/* The expected log-likelihood over the draws: log((1/S) sum_s exp(ll[s])),
 * i.e. logsumexp(ll) - log S, with the largest term factored out. */
double orc_expected_log_likelihood(const double *ll, int64_t S)
{
    double m = -INFINITY;
    for (int64_t s = 0; s < S; ++s) m = ll[s] > m ? ll[s] : m;
    double acc = 0.0;
    for (int64_t s = 0; s < S; ++s) acc += exp(ll[s] - m);
    return m + log(acc) - log((double)S);
}

/* Conjugate linear-Gaussian target used to pin the sampler's statistics:
 *   U(w) = sum_i (y_i - x_i . w)^2 / (2 sn^2) + sum_j w_j^2 / (2 s^2) + const,
 * whose posterior is N(mu, Sigma), Sigma = (X^T X / sn^2 + I / s^2)^-1,
 * mu = Sigma X^T y / sn^2.                                                   */
double orc_lingauss_ug(const double *X, const double *yv, int64_t N, int64_t D, double s,
                       double sn, const double *w, double *grad)
{
    for (int64_t j = 0; j < D; ++j) grad[j] = 0.0;
    double U = 0.0, inv_n2 = 1.0 / (sn * sn), inv_s2 = 1.0 / (s * s);
    for (int64_t i = 0; i < N; ++i) {
        const double *xi = X + i * D;
        double eta = 0.0;
        for (int64_t j = 0; j < D; ++j) eta += xi[j] * w[j];
        double res = yv[i] - eta;
        U += 0.5 * res * res * inv_n2;
        for (int64_t j = 0; j < D; ++j) grad[j] -= res * inv_n2 * xi[j];
    }
    for (int64_t j = 0; j < D; ++j) {
        U += 0.5 * w[j] * w[j] * inv_s2;
        grad[j] += w[j] * inv_s2;
    }
    return U;
}

/* Semi-supervised hidden Markov model (reading R21; the paper's HMM
 * benchmark, Appendix C, after Stan's semi-supervised example): K hidden
 * states, V observation symbols, one sequence w_1..w_T whose first Tsup
 * hidden states z_1..z_Tsup are observed.  Parameters: the K transition rows
 * theta_j and the K emission rows phi_k, each a simplex with a uniform
 * Dirichlet prior, sampled on the unconstrained space of additive log-ratios
 * (row x = softmax(a_0 .. a_{n-2}, 0), |Jacobian| = prod_i x_i).  q holds the
 * K (K - 1) transition logits (row j at j (K - 1)), then the K (V - 1)
 * emission logits (row k at K (K - 1) + k (V - 1)).  With
 *   f(q) = sum over rows of sum_i log x_i                       (Jacobians)
 *        + sum_{t <= Tsup} log phi_{z_t}(w_t) + sum_{2 <= t <= Tsup} log theta_{z_{t-1}}(z_t)
 *        + log p(w_{Tsup+1..T} | z_Tsup)                     (forward algorithm),
 * U = -f and grad U = -df/dq.  The forward recursion runs on scaled
 * probabilities (alpha_t normalised, log p = sum_t log c_t), starting from
 * theta_{z_Tsup} (uniform 1/K when Tsup = 0); the backward recursion gives
 * the expected transition counts xi and state occupancies gamma, which are
 * d log p / d log theta and d log p / d log phi.  Through the softmax,
 * df/da_i = G_i - x_i sum_m G_m with G = df/d log x.                        */
static void orc_softmax_row(const double *a, int n, double *x, double *lx)
{
    double m = 0.0;                               /* the fixed last logit */
    for (int i = 0; i < n - 1; ++i) m = a[i] > m ? a[i] : m;
    double tot = 0.0;
    for (int i = 0; i < n; ++i) tot += exp((i < n - 1 ? a[i] : 0.0) - m);
    double lse = m + log(tot);
    for (int i = 0; i < n; ++i) {
        lx[i] = (i < n - 1 ? a[i] : 0.0) - lse;
        x[i] = exp(lx[i]);
    }
}

double orc_hmm_ug(const uint8_t *w, int64_t T, const uint8_t *z, int64_t Tsup, int K, int V,
                  const double *q, double *grad)
{
    const int nt = K * (K - 1);
    double *th = (double *)malloc((size_t)K * K * sizeof(double));
    double *lth = (double *)malloc((size_t)K * K * sizeof(double));
    double *ph = (double *)malloc((size_t)K * V * sizeof(double));
    double *lph = (double *)malloc((size_t)K * V * sizeof(double));
    double *Gt = (double *)calloc((size_t)K * K, sizeof(double));
    double *Gp = (double *)calloc((size_t)K * V, sizeof(double));
    for (int j = 0; j < K; ++j) orc_softmax_row(q + j * (K - 1), K, th + j * K, lth + j * K);
    for (int k = 0; k < K; ++k) orc_softmax_row(q + nt + k * (V - 1), V, ph + k * V, lph + k * V);

    double f = 0.0;
    /* Jacobians: each entry contributes log x_i and d/d log x_i = 1 */
    for (int i = 0; i < K * K; ++i) { f += lth[i]; Gt[i] += 1.0; }
    for (int i = 0; i < K * V; ++i) { f += lph[i]; Gp[i] += 1.0; }
    /* the observed states */
    for (int64_t t = 0; t < Tsup; ++t) {
        f += lph[z[t] * V + w[t]];
        Gp[z[t] * V + w[t]] += 1.0;
        if (t > 0) {
            f += lth[z[t - 1] * K + z[t]];
            Gt[z[t - 1] * K + z[t]] += 1.0;
        }
    }
    /* forward over t = Tsup .. T-1 (0-based) */
    int64_t Tu = T - Tsup;
    if (Tu > 0) {
        double *al = (double *)malloc((size_t)(Tu + 1) * K * sizeof(double));
        double *be = (double *)malloc((size_t)Tu * K * sizeof(double));
        double *c = (double *)malloc((size_t)Tu * sizeof(double));
        for (int k = 0; k < K; ++k) al[k] = Tsup > 0 ? (z[Tsup - 1] == k ? 1.0 : 0.0) : 1.0 / K;
        for (int64_t s = 0; s < Tu; ++s) {
            const int ws = w[Tsup + s];
            const double *prev = al + s * K;
            double *cur = al + (s + 1) * K;
            double tot = 0.0;
            for (int k = 0; k < K; ++k) {
                double acc = 0.0;
                if (s == 0 && Tsup == 0) acc = prev[k];  /* initial distribution, no transition */
                else for (int j = 0; j < K; ++j) acc += prev[j] * th[j * K + k];
                cur[k] = acc * ph[k * V + ws];
                tot += cur[k];
            }
            c[s] = tot;
            for (int k = 0; k < K; ++k) cur[k] /= tot;
            f += log(tot);
        }
        /* backward (scaled by the same c) */
        for (int k = 0; k < K; ++k) be[(Tu - 1) * K + k] = 1.0;
        for (int64_t s = Tu - 2; s >= 0; --s) {
            const int wn = w[Tsup + s + 1];
            for (int j = 0; j < K; ++j) {
                double acc = 0.0;
                for (int k = 0; k < K; ++k) acc += th[j * K + k] * ph[k * V + wn] * be[(s + 1) * K + k];
                be[s * K + j] = acc / c[s + 1];
            }
        }
        /* expected counts */
        for (int64_t s = 0; s < Tu; ++s) {
            const int ws = w[Tsup + s];
            const double *prev = al + s * K;
            const double *cur = al + (s + 1) * K;
            for (int k = 0; k < K; ++k) Gp[k * V + ws] += cur[k] * be[s * K + k];
            if (s == 0 && Tsup == 0) continue;
            for (int j = 0; j < K; ++j)
                for (int k = 0; k < K; ++k)
                    Gt[j * K + k] += prev[j] * th[j * K + k] * ph[k * V + ws] * be[s * K + k] / c[s];
        }
        free(al); free(be); free(c);
    }
    /* through the softmax of each row, then U = -f */
    for (int j = 0; j < K; ++j) {
        double tot = 0.0;
        for (int k = 0; k < K; ++k) tot += Gt[j * K + k];
        for (int k = 0; k < K - 1; ++k) grad[j * (K - 1) + k] = -(Gt[j * K + k] - th[j * K + k] * tot);
    }
    for (int k = 0; k < K; ++k) {
        double tot = 0.0;
        for (int v = 0; v < V; ++v) tot += Gp[k * V + v];
        for (int v = 0; v < V - 1; ++v) grad[nt + k * (V - 1) + v] = -(Gp[k * V + v] - ph[k * V + v] * tot);
    }
    free(th); free(lth); free(ph); free(lph); free(Gt); free(Gp);
    return -f;
}

/* Timing loop for the benchmark's CPU baseline (no arithmetic of its own):
 * reps evaluations of orc_hmm_ug at the same point.  Returns the last U. */
double orc_hmm_ug_repeat(const uint8_t *w, int64_t T, const uint8_t *z, int64_t Tsup, int K, int V,
                         const double *q, double *grad, int64_t reps)
{
    double U = 0.0;
    for (int64_t r = 0; r < reps; ++r) U = orc_hmm_ug(w, T, z, Tsup, K, V, q, grad);
    return U;
}

enum { ORC_TARGET_LOGISTIC = 0, ORC_TARGET_LINGAUSS = 1, ORC_TARGET_HMM = 2 };

typedef struct {
    int kind;
    const double *X;      /* N x D row-major */
    const uint8_t *y;     /* logistic labels */
    const double *yv;     /* linear-Gaussian responses */
    int64_t N, D;
    double s;             /* prior scale */
    double sn;            /* noise scale (linear-Gaussian) */
    int64_t nevals;       /* gradient evaluations performed */
    /* HMM: the observations are y (N = T symbols), then these */
    const uint8_t *z;     /* the Tsup observed hidden states */
    int64_t Tsup;
    int K, V;
} orc_target;

static double orc_eval(orc_target *tg, const double *w, double *grad)
{
    tg->nevals++;
    if (tg->kind == ORC_TARGET_LINGAUSS)
        return orc_lingauss_ug(tg->X, tg->yv, tg->N, tg->D, tg->s, tg->sn, w, grad);
    if (tg->kind == ORC_TARGET_HMM)
        return orc_hmm_ug(tg->y, tg->N, tg->z, tg->Tsup, tg->K, tg->V, w, grad);
    return orc_logistic_ug(tg->X, tg->y, tg->N, tg->D, tg->s, w, grad);
}

/* ------------------------------------------------------------------------- */
/* Index arithmetic of Alg. 2.                                               */

int orc_bitcount(uint64_t n)
{
    int c = 0;
    while (n) { c += (int)(n & 1ULL); n >>= 1; }
    return c;
}

int orc_trailing_ones(uint64_t n)
{
    int c = 0;
    while (n & 1ULL) { ++c; n >>= 1; }
    return c;
}

/* For odd n: the S slots holding the first leaves of every balanced subtree
 * that ends at leaf n are i_max = BitCount(n-1) down to
 * i_min = i_max - TrailingBit(n) + 1. */
void orc_check_range(uint64_t n, int *i_max, int *i_min)
{
    int l = orc_trailing_ones(n);
    *i_max = orc_bitcount(n - 1);
    *i_min = *i_max - l + 1;
}

/* ------------------------------------------------------------------------- */
/* Phase-space nodes and the leapfrog integrator.                            */

typedef struct {
    double *q, *p, *g;
    double U;
} orc_node;

static void orc_node_alloc(orc_node *z, int64_t D)
{
    z->q = (double *)calloc((size_t)D, sizeof(double));
    z->p = (double *)calloc((size_t)D, sizeof(double));
    z->g = (double *)calloc((size_t)D, sizeof(double));
    z->U = 0.0;
}

static void orc_node_free(orc_node *z) { free(z->q); free(z->p); free(z->g); }

static void orc_node_copy(orc_node *dst, const orc_node *src, int64_t D)
{
    memcpy(dst->q, src->q, (size_t)D * sizeof(double));
    memcpy(dst->p, src->p, (size_t)D * sizeof(double));
    memcpy(dst->g, src->g, (size_t)D * sizeof(double));
    dst->U = src->U;
}

static double orc_kinetic(const double *p, const double *inv_mass, int64_t D)
{
    double k = 0.0;
    for (int64_t j = 0; j < D; ++j) k += inv_mass[j] * p[j] * p[j];
    return 0.5 * k;
}

/* Kick-drift-kick with the gradient carried in the node: one gradient
 * evaluation per step (the form the paper's LeapFrog calls through grad). */
static void orc_leapfrog(orc_target *tg, orc_node *z, double h, const double *inv_mass)
{
    int64_t D = tg->D;
    for (int64_t j = 0; j < D; ++j) z->p[j] = z->p[j] - 0.5 * h * z->g[j];
    for (int64_t j = 0; j < D; ++j) z->q[j] = z->q[j] + h * inv_mass[j] * z->p[j];
    z->U = orc_eval(tg, z->q, z->g);
    for (int64_t j = 0; j < D; ++j) z->p[j] = z->p[j] - 0.5 * h * z->g[j];
}

/* Hoffman & Gelman's endpoint criterion on time-ordered ends: a subtree whose
 * first-generated node is a and last-generated node is b, built in direction
 * v, has left end a and right end b if v > 0, else the reverse. */
static int orc_is_uturn(const double *qa, const double *pa, const double *qb, const double *pb,
                        int v, const double *inv_mass, int64_t D)
{
    const double *qL = v > 0 ? qa : qb, *pL = v > 0 ? pa : pb;
    const double *qR = v > 0 ? qb : qa, *pR = v > 0 ? pb : pa;
    double dl = 0.0, dr = 0.0;
    for (int64_t j = 0; j < D; ++j) {
        double dq = qR[j] - qL[j];
        dl += dq * inv_mass[j] * pL[j];
        dr += dq * inv_mass[j] * pR[j];
    }
    return (dl < 0.0) || (dr < 0.0);
}

/* Reading R20: rho . M^-1 p_a <= 0 or rho . M^-1 p_b <= 0 (either end). */
static int orc_is_uturn_gen(const double *rho, const double *pa, const double *pb,
                            const double *inv_mass, int64_t D)
{
    double da = 0.0, db = 0.0;
    for (int64_t j = 0; j < D; ++j) {
        da += rho[j] * inv_mass[j] * pa[j];
        db += rho[j] * inv_mass[j] * pb[j];
    }
    return (da <= 0.0) || (db <= 0.0);
}

int orc_is_uturn_gen_exported(const double *rho, const double *pa, const double *pb,
                              const double *inv_mass, int64_t D)
{
    return orc_is_uturn_gen(rho, pa, pb, inv_mass, D);
}

int orc_is_uturn_exported(const double *qa, const double *pa, const double *qb, const double *pb,
                          int v, const double *inv_mass, int64_t D)
{
    return orc_is_uturn(qa, pa, qb, pb, v, inv_mass, D);
}

static double orc_logaddexp(double a, double b)
{
    if (a == -INFINITY) return b;
    if (b == -INFINITY) return a;
    double m = fmax(a, b);
    return m + log1p(exp(-fabs(a - b)));
}

/* ------------------------------------------------------------------------- */
/* Tree building.                                                            */

enum { ORC_OK = 0, ORC_TURNING = 1, ORC_DIVERGENT = 2 };

/* Everything one iteration shares between the doubling loop and the two tree
 * builders. */
typedef struct {
    orc_target *tg;
    const double *inv_mass;
    double eps;
    uint64_t seed, chain, t;
    double H0;
    /* optional trace of U-turn checks inside subtrees: pairs (first, last) of
     * leaf indices within the current subtree, in the order performed */
    int64_t *trace;
    int64_t trace_cap, trace_len;
    /* optional trace of generated leaves: (doubling j, leaf n, signed
     * position, H - H0 as raw bits) per leaf */
    int64_t *leaves;
    int64_t leaves_cap, leaves_len;
    /* xored into the seed for the selection draws only (0 = the standard
     * protocol); lets a test re-draw the choices over a fixed trajectory */
    uint64_t sel_salt;
    /* per-iteration totals */
    int64_t nleaves;
    double sum_accept;
    /* reading R20: the generalised criterion instead of the endpoint one */
    int gen;
    /* reading R22: the subtree's proposal chosen at the merges of its halves
     * instead of by the streaming choice; -(H - H0) of the last leaf */
    int smerge;
    double last_lam;
} orc_iter;

/* What a subtree hands back: the streaming proposal and its log-weight. */
typedef struct {
    int status;
    int64_t term_leaf;
    double logw;          /* log of the summed exp(-(H - H0)) over the subtree */
    orc_node prop;
    int64_t prop_idx;     /* signed leaf offset of the proposal from q0 */
    int has_prop;
    double *rho;          /* momentum sum over the subtree's leaves (R20) */
} orc_sub;

static void orc_trace_check(orc_iter *it, int64_t first, int64_t last)
{
    if (it->trace && it->trace_len + 2 <= it->trace_cap) {
        it->trace[it->trace_len++] = first;
        it->trace[it->trace_len++] = last;
    }
}

/* Energy bookkeeping and the streaming multinomial choice for the leaf that
 * was just generated (leaf n of subtree j, whose start node sits at signed
 * offset e and which grows in direction v).  Returns ORC_DIVERGENT or ORC_OK. */
static int orc_leaf(orc_iter *it, orc_sub *sub, const orc_node *z, int j, int64_t n,
                    int64_t e, int v)
{
    int64_t D = it->tg->D;
    double H = z->U + orc_kinetic(z->p, it->inv_mass, D);
    double dH = H - it->H0;
    if (it->leaves && it->leaves_len + 4 <= it->leaves_cap) {
        int64_t bits;
        memcpy(&bits, &dH, sizeof(bits));
        it->leaves[it->leaves_len++] = j;
        it->leaves[it->leaves_len++] = n;
        it->leaves[it->leaves_len++] = e + (int64_t)v * (n + 1);
        it->leaves[it->leaves_len++] = bits;
    }
    it->nleaves++;
    if (dH == dH) it->sum_accept += (dH > 0.0) ? exp(-dH) : 1.0;
    if (!(dH <= 1000.0)) {
        sub->status = ORC_DIVERGENT;
        sub->term_leaf = n;
        return ORC_DIVERGENT;
    }
    double lam = -dH;
    if (it->smerge) {
        it->last_lam = lam;
        return ORC_OK;
    }
    double logw_new = orc_logaddexp(sub->logw, lam);
    double u = orc_u_leaf(it->seed ^ it->sel_salt, it->chain, it->t, (uint64_t)j, (uint64_t)n);
    if (u < exp(lam - logw_new)) {
        orc_node_copy(&sub->prop, z, D);
        sub->prop_idx = e + (int64_t)v * (n + 1);
        sub->has_prop = 1;
    }
    sub->logw = logw_new;
    return ORC_OK;
}

/* Alg. 2 (IterativeBuildTree): 2^j leapfrog steps from z in direction v.
 * Even leaves are kept in S[BitCount(n)]; at odd leaves the U-turn test runs
 * against the slots named by orc_check_range.  On return z holds the last
 * leaf generated. */
static void orc_build_iterative(orc_iter *it, orc_node *z, int j, int v, int64_t e,
                                orc_sub *sub)
{
    int64_t D = it->tg->D;
    int nslots = j > 0 ? j : 1;
    double *Sq = (double *)malloc((size_t)nslots * (size_t)D * sizeof(double));
    double *Sp = (double *)malloc((size_t)nslots * (size_t)D * sizeof(double));
    int64_t S_leaf[64];
    int64_t nleaf = (int64_t)1 << j;
    /* R20: running momentum sum of the subtree's leaves; the slots then hold
     * (sum before the leaf, the leaf's momentum) instead of (q, p) */
    double *rsum = sub->rho;
    double *rho = (double *)malloc((size_t)D * sizeof(double));
    for (int64_t k = 0; k < D; ++k) rsum[k] = 0.0;
    /* R22: the proposal, log-weight and offset of the completed left block
     * waiting at each level, and those of the block ending at this leaf */
    orc_node stk[64], cp;
    double stk_lw[64], c_lw = 0.0;
    int64_t stk_idx[64], c_idx = 0;
    if (it->smerge) {
        for (int k = 0; k < nslots; ++k) orc_node_alloc(&stk[k], D);
        orc_node_alloc(&cp, D);
    }
    for (int64_t n = 0; n < nleaf; ++n) {
        orc_leapfrog(it->tg, z, (double)v * it->eps, it->inv_mass);
        if (orc_leaf(it, sub, z, j, n, e, v) != ORC_OK) break;
        if (it->smerge) {
            /* the leaf is a block of one; every completed pair of equal
             * blocks merges, the later half's proposal kept with probability
             * its share of the weight */
            orc_node_copy(&cp, z, D);
            c_lw = it->last_lam;
            c_idx = e + (int64_t)v * (n + 1);
            int k = 0;
            while ((n >> k) & 1) {
                double lw = orc_logaddexp(stk_lw[k], c_lw);
                double u = orc_u_submerge(it->seed ^ it->sel_salt, it->chain, it->t, (uint64_t)j,
                                          orc_merge_ordinal(n, k + 1));
                if (!(u < exp(c_lw - lw))) {
                    orc_node_copy(&cp, &stk[k], D);
                    c_idx = stk_idx[k];
                }
                c_lw = lw;
                ++k;
            }
            if (n + 1 < nleaf) {
                orc_node_copy(&stk[k], &cp, D);
                stk_lw[k] = c_lw;
                stk_idx[k] = c_idx;
            } else {
                orc_node_copy(&sub->prop, &cp, D);
                sub->prop_idx = c_idx;
                sub->logw = c_lw;
                sub->has_prop = 1;
            }
        }
        for (int64_t k = 0; k < D; ++k) rsum[k] += z->p[k];
        if ((n & 1) == 0) {
            int i = orc_bitcount((uint64_t)n);
            if (it->gen) {
                for (int64_t k = 0; k < D; ++k) Sq[(int64_t)i * D + k] = rsum[k] - z->p[k];
            } else {
                memcpy(Sq + (int64_t)i * D, z->q, (size_t)D * sizeof(double));
            }
            memcpy(Sp + (int64_t)i * D, z->p, (size_t)D * sizeof(double));
            S_leaf[i] = n;
        } else {
            int i_max, i_min;
            orc_check_range((uint64_t)n, &i_max, &i_min);
            int turned = 0;
            for (int k = i_max; k >= i_min; --k) {
                orc_trace_check(it, S_leaf[k], n);
                int t;
                if (it->gen) {
                    for (int64_t c = 0; c < D; ++c) rho[c] = rsum[c] - Sq[(int64_t)k * D + c];
                    t = orc_is_uturn_gen(rho, Sp + (int64_t)k * D, z->p, it->inv_mass, D);
                } else {
                    t = orc_is_uturn(Sq + (int64_t)k * D, Sp + (int64_t)k * D, z->q, z->p, v,
                                     it->inv_mass, D);
                }
                if (t) {
                    turned = 1;
                    break;
                }
            }
            if (turned) {
                sub->status = ORC_TURNING;
                sub->term_leaf = n;
                break;
            }
        }
    }
    if (it->smerge) {
        for (int k = 0; k < nslots; ++k) orc_node_free(&stk[k]);
        orc_node_free(&cp);
    }
    free(rho);
    free(Sq);
    free(Sp);
}

/* Alg. 1 (BuildTree), recursive: a depth-d subtree is a depth-(d-1) subtree
 * followed by another one, then the U-turn test between the first leaf of
 * the left half and the last leaf of the right half.  Leaves are numbered
 * from `offset`; the first leaf's (q, p) is returned in fq/fp. */
static void orc_build_recursive(orc_iter *it, orc_node *z, int j, int d, int64_t offset, int v,
                                int64_t e, orc_sub *sub, double *fq, double *fp, double *rho,
                                orc_node *mp, double *mlw, int64_t *midx)
{
    int64_t D = it->tg->D;
    if (d == 0) {
        orc_leapfrog(it->tg, z, (double)v * it->eps, it->inv_mass);
        orc_leaf(it, sub, z, j, offset, e, v);
        memcpy(fq, z->q, (size_t)D * sizeof(double));
        memcpy(fp, z->p, (size_t)D * sizeof(double));
        memcpy(rho, z->p, (size_t)D * sizeof(double));
        if (it->smerge) {  /* R22: a leaf is its own block's proposal */
            orc_node_copy(mp, z, D);
            *mlw = it->last_lam;
            *midx = e + (int64_t)v * (offset + 1);
        }
        return;
    }
    orc_build_recursive(it, z, j, d - 1, offset, v, e, sub, fq, fp, rho, mp, mlw, midx);
    if (sub->status != ORC_OK) return;
    double *rq = (double *)malloc((size_t)D * sizeof(double));
    double *rp = (double *)malloc((size_t)D * sizeof(double));
    double *rr = (double *)malloc((size_t)D * sizeof(double));
    int64_t half = (int64_t)1 << (d - 1);
    orc_node rprop;
    double rlw = 0.0;
    int64_t ridx = 0;
    if (it->smerge) orc_node_alloc(&rprop, D);
    orc_build_recursive(it, z, j, d - 1, offset + half, v, e, sub, rq, rp, rr, &rprop, &rlw, &ridx);
    for (int64_t k = 0; k < D; ++k) rho[k] += rr[k];
    free(rq);
    free(rp);
    free(rr);
    if (it->smerge && sub->status == ORC_OK) {
        /* R22: merge the halves; the later one's proposal with probability
         * its share of the weight */
        double lw = orc_logaddexp(*mlw, rlw);
        double u = orc_u_submerge(it->seed ^ it->sel_salt, it->chain, it->t, (uint64_t)j,
                                  orc_merge_ordinal(offset + 2 * half - 1, d));
        if (u < exp(rlw - lw)) {
            orc_node_copy(mp, &rprop, D);
            *midx = ridx;
        }
        *mlw = lw;
    }
    if (it->smerge) orc_node_free(&rprop);
    if (sub->status != ORC_OK) return;
    int64_t last = offset + 2 * half - 1;
    orc_trace_check(it, offset, last);
    int t = it->gen ? orc_is_uturn_gen(rho, fp, z->p, it->inv_mass, D)
                    : orc_is_uturn(fq, fp, z->q, z->p, v, it->inv_mass, D);
    if (t) {
        sub->status = ORC_TURNING;
        sub->term_leaf = last;
    }
}

/* Per-sample statistics; the layout matches the library's nuts_stats. */
typedef struct {
    double potential_energy;
    double energy;
    double accept_prob;
    int32_t tree_depth;
    int32_t num_steps;
    int32_t proposal_index;
    int32_t term_leaf;
    uint32_t direction_bits;
    uint8_t diverging, turning, hit_max_depth, pad[9];
} orc_stats;

enum { ORC_BUILDER_ITERATIVE = 0, ORC_BUILDER_RECURSIVE = 1 };

/* One NUTS iteration from state (q, U, g) -- trajectory doubling (H&G Alg. 6
 * with multinomial selection).  On return `cur` holds the new state. */
static void orc_iteration(orc_iter *it, orc_node *cur, int max_depth, int builder,
                          orc_stats *st)
{
    orc_target *tg = it->tg;
    int64_t D = tg->D;
    const double *im = it->inv_mass;

    double *xi = (double *)malloc((size_t)D * sizeof(double));
    orc_normals(it->seed, it->chain, it->t, D, xi);
    for (int64_t j = 0; j < D; ++j) cur->p[j] = xi[j] / sqrt(im[j]);
    free(xi);
    it->H0 = cur->U + orc_kinetic(cur->p, im, D);
    it->nleaves = 0;
    it->sum_accept = 0.0;

    orc_node left, right, prop, z;
    orc_node_alloc(&left, D); orc_node_alloc(&right, D);
    orc_node_alloc(&prop, D); orc_node_alloc(&z, D);
    orc_node_copy(&left, cur, D);
    orc_node_copy(&right, cur, D);
    orc_node_copy(&prop, cur, D);
    int64_t prop_idx = 0, Lpos = 0, Rpos = 0;
    double logw_traj = 0.0;

    orc_sub sub;
    orc_node_alloc(&sub.prop, D);
    sub.rho = (double *)malloc((size_t)D * sizeof(double));
    double *fq = (double *)malloc((size_t)D * sizeof(double));
    double *fp = (double *)malloc((size_t)D * sizeof(double));
    /* R20: momentum sum over every point of the trajectory */
    double *rho_traj = (double *)malloc((size_t)D * sizeof(double));
    memcpy(rho_traj, cur->p, (size_t)D * sizeof(double));

    memset(st, 0, sizeof(*st));
    st->term_leaf = -1;
    for (int j = 0; j < max_depth; ++j) {
        int v = orc_direction(it->seed, it->chain, it->t, (uint64_t)j);
        if (v > 0) st->direction_bits |= (1u << j);
        orc_node_copy(&z, v > 0 ? &right : &left, D);
        int64_t e = v > 0 ? Rpos : Lpos;
        sub.status = ORC_OK;
        sub.term_leaf = -1;
        sub.logw = -INFINITY;
        sub.prop_idx = 0;
        sub.has_prop = 0;
        if (builder == ORC_BUILDER_RECURSIVE) {
            orc_build_recursive(it, &z, j, j, 0, v, e, &sub, fq, fp, sub.rho, &sub.prop, &sub.logw,
                                &sub.prop_idx);
            if (it->smerge) sub.has_prop = 1;
        } else
            orc_build_iterative(it, &z, j, v, e, &sub);
        st->tree_depth = j + 1;
        if (sub.status != ORC_OK) {
            st->term_leaf = (int32_t)sub.term_leaf;
            if (sub.status == ORC_DIVERGENT) st->diverging = 1;
            else st->turning = 1;
            break;
        }
        /* biased progressive selection between the old trajectory and the
         * new subtree */
        double u = orc_u_merge(it->seed ^ it->sel_salt, it->chain, it->t, (uint64_t)j);
        if (u < exp(sub.logw - logw_traj)) {
            orc_node_copy(&prop, &sub.prop, D);
            prop_idx = sub.prop_idx;
        }
        logw_traj = orc_logaddexp(logw_traj, sub.logw);
        if (v > 0) { orc_node_copy(&right, &z, D); Rpos += (int64_t)1 << j; }
        else       { orc_node_copy(&left, &z, D);  Lpos -= (int64_t)1 << j; }
        for (int64_t k = 0; k < D; ++k) rho_traj[k] += sub.rho[k];
        if (it->gen ? orc_is_uturn_gen(rho_traj, left.p, right.p, im, D)
                    : orc_is_uturn(left.q, left.p, right.q, right.p, +1, im, D)) {
            st->turning = 1;
            st->term_leaf = -2;
            break;
        }
        if (j == max_depth - 1) st->hit_max_depth = 1;
    }
    st->num_steps = (int32_t)it->nleaves;
    st->accept_prob = it->nleaves > 0 ? it->sum_accept / (double)it->nleaves : 0.0;
    st->proposal_index = (int32_t)prop_idx;
    orc_node_copy(cur, &prop, D);
    st->potential_energy = cur->U;
    st->energy = cur->U + orc_kinetic(cur->p, im, D);

    free(fq); free(fp);
    free(rho_traj);
    free(sub.rho);
    orc_node_free(&sub.prop);
    orc_node_free(&left); orc_node_free(&right);
    orc_node_free(&prop); orc_node_free(&z);
}

/* ------------------------------------------------------------------------- */
/* Warmup adaptation (reading R19).                                           */

#define ORC_LN2 0.69314718055994530942
#define ORC_STEP_TRIALS 100

/* Hoffman & Gelman (2014) Alg. 4: from eps, one leapfrog step with a fresh
 * momentum r ~ N(0, M) (drawn under ORC_TAG_STEP at counter t); a = +1 if
 * the step keeps more than half the density (H0 - H > -ln 2), else -1; then
 * eps is doubled (a = +1) or halved (a = -1) until that comparison flips.
 * A non-finite energy counts as density zero.  At most ORC_STEP_TRIALS
 * changes of eps. */
static double orc_log_ratio(orc_target *tg, const orc_node *cur, const double *r, double eps,
                            const double *im, double H0, orc_node *z)
{
    int64_t D = tg->D;
    orc_node_copy(z, cur, D);
    memcpy(z->p, r, (size_t)D * sizeof(double));
    orc_leapfrog(tg, z, eps, im);
    double d = H0 - (z->U + orc_kinetic(z->p, im, D));
    return d == d ? d : -INFINITY;
}

static double orc_find_step_size(orc_target *tg, const orc_node *cur, double eps,
                                 const double *im, uint64_t seed, uint64_t chain, uint64_t t)
{
    int64_t D = tg->D;
    double *r = (double *)malloc((size_t)D * sizeof(double));
    orc_normals_tagged(seed, chain, t, ORC_TAG_STEP, D, r);
    for (int64_t j = 0; j < D; ++j) r[j] = r[j] / sqrt(im[j]);
    double H0 = cur->U + orc_kinetic(r, im, D);
    orc_node z;
    orc_node_alloc(&z, D);
    double d = orc_log_ratio(tg, cur, r, eps, im, H0, &z);
    double a = d > -ORC_LN2 ? 1.0 : -1.0;
    for (int k = 0; k < ORC_STEP_TRIALS && a * (d + ORC_LN2) > 0.0; ++k) {
        eps = a > 0.0 ? eps * 2.0 : eps * 0.5;
        d = orc_log_ratio(tg, cur, r, eps, im, H0, &z);
    }
    orc_node_free(&z);
    free(r);
    return eps;
}

/* Dual averaging of log eps (Hoffman & Gelman 2014, Section 3.2). */
typedef struct {
    double mu, hbar, log_eps, log_eps_bar;
    int64_t m;
} orc_dual_avg;

#define ORC_DA_GAMMA 0.05
#define ORC_DA_T0 10.0
#define ORC_DA_KAPPA 0.75

static void orc_da_start(orc_dual_avg *da, double eps)
{
    da->mu = log(10.0 * eps);
    da->hbar = 0.0;
    da->log_eps = log(eps);
    da->log_eps_bar = 0.0;
    da->m = 0;
}

/* One update with the accept statistic alpha; returns the next eps. */
static double orc_da_update(orc_dual_avg *da, double alpha, double delta)
{
    da->m += 1;
    double m = (double)da->m;
    double w = 1.0 / (m + ORC_DA_T0);
    da->hbar = (1.0 - w) * da->hbar + w * (delta - alpha);
    da->log_eps = da->mu - (sqrt(m) / ORC_DA_GAMMA) * da->hbar;
    double eta = pow(m, -ORC_DA_KAPPA);
    da->log_eps_bar = eta * da->log_eps + (1.0 - eta) * da->log_eps_bar;
    return exp(da->log_eps);
}

/* Exposed for the tests: the recursion driven by a given accept sequence;
 * writes log eps and log eps_bar after each update. */
void orc_dual_avg_run(double eps0, double delta, int64_t n, const double *alpha,
                      double *out_log_eps, double *out_log_eps_bar)
{
    orc_dual_avg da = { 0.0, 0.0, 0.0, 0.0, 0 };
    orc_da_start(&da, eps0);
    for (int64_t i = 0; i < n; ++i) {
        orc_da_update(&da, alpha[i], delta);
        out_log_eps[i] = da.log_eps;
        out_log_eps_bar[i] = da.log_eps_bar;
    }
}

/* The slow windows of the windowed mass adaptation for W warmup
 * iterations: pairs [start, end) of iteration indices (0-based), at most
 * cap pairs; returns their number. */
int orc_mass_windows(int64_t W, int64_t *out, int cap)
{
    if (W < 20) return 0;
    int64_t init = 75, term = 50, base = 25;
    if (init + term + base > W) {
        init = (int64_t)(0.15 * (double)W);
        term = (int64_t)(0.10 * (double)W);
        base = W - (init + term);
    }
    int64_t slow_end = W - term;
    int n = 0;
    int64_t start = init, size = base;
    while (start < slow_end && n < cap) {
        int64_t end = start + size;
        /* stretch this window to the terminal buffer when the one after it
         * would not fit */
        if (end + 2 * size > slow_end) end = slow_end;
        out[2 * n] = start;
        out[2 * n + 1] = end;
        ++n;
        start = end;
        size *= 2;
    }
    return n;
}

/* Exposed for the tests: the step-size heuristic at q for one target. */
double orc_find_step_size_at(int kind, const double *X, const uint8_t *y, const double *yv,
                             int64_t N, int64_t D, double s, double sn, const double *inv_mass,
                             const double *q, double eps, uint64_t seed, uint64_t chain,
                             uint64_t t, int64_t *evals)
{
    orc_target tg = { kind, X, y, yv, N, D, s, sn, 0 };
    orc_node cur;
    orc_node_alloc(&cur, D);
    memcpy(cur.q, q, (size_t)D * sizeof(double));
    cur.U = orc_eval(&tg, cur.q, cur.g);
    double out = orc_find_step_size(&tg, &cur, eps, inv_mass, seed, chain, t);
    orc_node_free(&cur);
    if (evals) *evals = tg.nevals;
    return out;
}

/* Diagonal inverse mass from warmup draws (reading R13): Welford mean and
 * variance of the states after warmup iterations [W/2, W), shrunk towards
 * 1e-3 with weight 5/(n+5), then scaled to mean one. */
typedef struct {
    int64_t n;
    double *mean, *m2;
} orc_welford;

/* Test hook: when set, every warmup iteration k < cap writes the state after
 * it and the step size it ran with into buf [k][D + 1] (the state, then the
 * step size), so that tests can recompute the mass rule from the states. */
static double *orc_wtrace_buf = NULL;
static int64_t orc_wtrace_cap = 0;

void orc_set_warmup_trace(double *buf, int64_t cap)
{
    orc_wtrace_buf = buf;
    orc_wtrace_cap = buf ? cap : 0;
}

/* Full chain: init at q0, then num_warmup + num_samples iterations whose
 * global indices start at first_iter.  Kept samples go to out_samples
 * [num_samples][D] and out_stats [num_samples].  The final state goes to
 * out_q (may be NULL); out_inv_mass receives the inverse mass in use at the
 * end (may be NULL).  Returns the number of gradient evaluations. */
int64_t orc_nuts_chain(int kind, const double *X, const uint8_t *y, const double *yv, int64_t N,
                       int64_t D, double s, double sn, double eps, const double *inv_mass_in,
                       int max_depth, int64_t num_warmup, int64_t num_samples, uint64_t seed,
                       uint64_t chain, int builder, int adapt_diag, const double *q0,
                       int64_t first_iter, double *out_samples, orc_stats *out_stats,
                       double *out_q, double *out_inv_mass, int64_t *trace,
                       int64_t trace_cap, int64_t *trace_len, int64_t *leaves,
                       int64_t leaves_cap, int64_t *leaves_len, uint64_t sel_salt,
                       int adapt_step, double target_accept, double *out_step_size,
                       int uturn_gen, const uint8_t *hmm_z, int64_t hmm_tsup, int hmm_k, int hmm_v,
                       int sub_merge)
{
    orc_target tg = { kind, X, y, yv, N, D, s, sn, 0 };
    tg.z = hmm_z;
    tg.Tsup = hmm_tsup;
    tg.K = hmm_k;
    tg.V = hmm_v;
    double *im = (double *)malloc((size_t)D * sizeof(double));
    for (int64_t j = 0; j < D; ++j) im[j] = inv_mass_in ? inv_mass_in[j] : 1.0;

    orc_node cur;
    orc_node_alloc(&cur, D);
    for (int64_t j = 0; j < D; ++j) cur.q[j] = q0 ? q0[j] : 0.0;
    cur.U = orc_eval(&tg, cur.q, cur.g);

    orc_iter it;
    memset(&it, 0, sizeof(it));
    it.tg = &tg;
    it.inv_mass = im;
    it.eps = eps;
    it.seed = seed;
    it.chain = chain;
    it.trace = trace;
    it.trace_cap = trace_cap;
    it.leaves = leaves;
    it.leaves_cap = leaves_cap;
    it.sel_salt = sel_salt;
    it.gen = uturn_gen;
    it.smerge = sub_merge;

    orc_welford wf = { 0, (double *)calloc((size_t)D, sizeof(double)),
                       (double *)calloc((size_t)D, sizeof(double)) };

    /* reading R19: step size by dual averaging, windowed mass with it */
    int adapt = adapt_step && num_warmup > 0;
    orc_dual_avg da = { 0.0, 0.0, 0.0, 0.0, 0 };
    int64_t win[128];
    int nwin = 0, wi = 0;
    if (adapt) {
        it.eps = orc_find_step_size(&tg, &cur, it.eps, im, seed, chain, (uint64_t)first_iter);
        orc_da_start(&da, it.eps);
        if (adapt_diag) nwin = orc_mass_windows(num_warmup, win, 64);
    }

    orc_stats st;
    for (int64_t k = 0; k < num_warmup + num_samples; ++k) {
        it.t = (uint64_t)(first_iter + k);
        double eps_used = it.eps;
        orc_iteration(&it, &cur, max_depth, builder, &st);
        if (k < num_warmup && k < orc_wtrace_cap) {
            memcpy(orc_wtrace_buf + k * (D + 1), cur.q, (size_t)D * sizeof(double));
            orc_wtrace_buf[k * (D + 1) + D] = eps_used;
        }
        if (adapt && k < num_warmup) {
            it.eps = orc_da_update(&da, st.accept_prob, target_accept);
            if (wi < nwin && k >= win[2 * wi] && k < win[2 * wi + 1]) {
                wf.n++;
                for (int64_t j = 0; j < D; ++j) {
                    double d1 = cur.q[j] - wf.mean[j];
                    wf.mean[j] += d1 / (double)wf.n;
                    wf.m2[j] += d1 * (cur.q[j] - wf.mean[j]);
                }
            }
            if (wi < nwin && k == win[2 * wi + 1] - 1) {
                if (wf.n >= 2) {
                    double nn = (double)wf.n;
                    for (int64_t j = 0; j < D; ++j) {
                        double var = wf.m2[j] / (nn - 1.0);
                        im[j] = (nn / (nn + 5.0)) * var + 1e-3 * (5.0 / (nn + 5.0));
                    }
                }
                wf.n = 0;
                for (int64_t j = 0; j < D; ++j) wf.mean[j] = wf.m2[j] = 0.0;
                ++wi;
                it.eps = orc_find_step_size(&tg, &cur, it.eps, im, seed, chain,
                                            (uint64_t)(first_iter + k + 1));
                orc_da_start(&da, it.eps);
            }
            if (k == num_warmup - 1) it.eps = exp(da.log_eps_bar);
        }
        if (!adapt && adapt_diag && k < num_warmup && k >= num_warmup / 2) {
            wf.n++;
            for (int64_t j = 0; j < D; ++j) {
                double d1 = cur.q[j] - wf.mean[j];
                wf.mean[j] += d1 / (double)wf.n;
                wf.m2[j] += d1 * (cur.q[j] - wf.mean[j]);
            }
        }
        if (!adapt && adapt_diag && k == num_warmup - 1 && wf.n >= 2) {
            double nn = (double)wf.n, tot = 0.0;
            for (int64_t j = 0; j < D; ++j) {
                double var = wf.m2[j] / (nn - 1.0);
                im[j] = (nn / (nn + 5.0)) * var + 1e-3 * (5.0 / (nn + 5.0));
                tot += im[j];
            }
            double mean = tot / (double)D;
            for (int64_t j = 0; j < D; ++j) im[j] = im[j] / mean;
        }
        if (k >= num_warmup) {
            int64_t o = k - num_warmup;
            if (out_samples) memcpy(out_samples + o * D, cur.q, (size_t)D * sizeof(double));
            if (out_stats) out_stats[o] = st;
        }
    }
    if (out_q) memcpy(out_q, cur.q, (size_t)D * sizeof(double));
    if (out_inv_mass) memcpy(out_inv_mass, im, (size_t)D * sizeof(double));
    if (out_step_size) *out_step_size = it.eps;
    if (trace_len) *trace_len = it.trace_len;
    if (leaves_len) *leaves_len = it.leaves_len;
    free(wf.mean); free(wf.m2);
    orc_node_free(&cur);
    free(im);
    return tg.nevals;
}

/* Exposed single leapfrog step for the integrator tests (position, momentum
 * and gradient updated in place; returns the new potential). */
double orc_leapfrog_steps(int kind, const double *X, const uint8_t *y, const double *yv,
                          int64_t N, int64_t D, double s, double sn, const double *inv_mass,
                          double h, int64_t nsteps, double *q, double *p)
{
    orc_target tg = { kind, X, y, yv, N, D, s, sn, 0 };
    orc_node z;
    orc_node_alloc(&z, D);
    memcpy(z.q, q, (size_t)D * sizeof(double));
    memcpy(z.p, p, (size_t)D * sizeof(double));
    z.U = orc_eval(&tg, z.q, z.g);
    for (int64_t k = 0; k < nsteps; ++k) orc_leapfrog(&tg, &z, h, inv_mass);
    memcpy(q, z.q, (size_t)D * sizeof(double));
    memcpy(p, z.p, (size_t)D * sizeof(double));
    double U = z.U;
    orc_node_free(&z);
    return U;
}

/* Timing helper for the CPU baseline: `reps` gradient evaluations at w over
 * an fp32 X (promoted row by row, never copied whole), or fp64 X. */
double orc_logistic_ug_f32(const float *Xf, const uint8_t *y, int64_t N, int64_t D, double s,
                           const double *w, double *grad)
{
    double *row = (double *)malloc((size_t)D * sizeof(double));
    for (int64_t j = 0; j < D; ++j) grad[j] = 0.0;
    double U = 0.0;
    for (int64_t i = 0; i < N; ++i) {
        for (int64_t j = 0; j < D; ++j) row[j] = (double)Xf[i * D + j];
        double eta = 0.0;
        for (int64_t j = 0; j < D; ++j) eta += row[j] * w[j];
        double sgn = y[i] ? -1.0 : 1.0;
        double t = sgn * eta;
        U += orc_softplus(t);
        double r = sgn * orc_sigmoid(t);
        for (int64_t j = 0; j < D; ++j) grad[j] += r * row[j];
    }
    free(row);
    const double half_log_2pi = 0.91893853320467274178032973640562;
    double inv_s2 = 1.0 / (s * s);
    for (int64_t j = 0; j < D; ++j) {
        U += 0.5 * w[j] * w[j] * inv_s2;
        grad[j] += w[j] * inv_s2;
    }
    U += (double)D * (log(s) + half_log_2pi);
    return U;
}

/* Timing loop for the benchmark's CPU baseline (no arithmetic of its own):
 * reps evaluations of the logistic potential and gradient at the same point,
 * over fp64 rows, or fp32 rows promoted one at a time when f32 is nonzero,
 * so that a caller's threads spend their time here rather than in the
 * interpreter between calls.  Returns the last U. */
double orc_logistic_ug_repeat(const void *X, const uint8_t *y, int64_t N, int64_t D, double s,
                              const double *w, double *grad, int64_t reps, int f32)
{
    double U = 0.0;
    for (int64_t r = 0; r < reps; ++r)
        U = f32 ? orc_logistic_ug_f32((const float *)X, y, N, D, s, w, grad)
                : orc_logistic_ug((const double *)X, y, N, D, s, w, grad);
    return U;
}

/* ------------------------------------------------------------------------- */
/* Normal approximation of the logistic posterior (tests only): the sampler's
 * long runs are checked against it where no sampler of the oracle can run
 * long enough (hundreds of thousands of rows).
 *
 * MAP by Newton's method on U, which for this model is iteratively
 * reweighted least squares: with c_i = sigma(eta_i) sigma(-eta_i) the Hessian
 * is H(w) = X^T diag(c) X + I / s^2 and each step solves H d = grad U and
 * sets w <- w - d, from w = 0 until no coordinate moves by more than
 * 1e-13 (1 + |w_j|) (at most 100 steps).  The Laplace covariance is H^-1 at
 * the MAP.  The posterior mean differs from the mode at order 1/N through
 * the skewness of U: expanding exp(-U) around the mode to the cubic term
 * T_jkl = sum_i sigma''(eta_i) x_ij x_ik x_il (sigma'' = c (1 - 2 sigma), the
 * third derivative of U; the prior adds none) gives
 *   E[w] = w_map - (1/2) H^-1 b,   b_j = sum_kl T_jkl (H^-1)_kl
 *        = sum_i sigma''(eta_i) x_ij (x_i^T H^-1 x_i),
 * with an error of order 1/N^2.  X is fp64, or fp32 promoted one row at a
 * time when f32 is nonzero.  Plain loops, the Cholesky factorisation written
 * out. */
static void orc_row(const void *X, int f32, int64_t i, int64_t D, double *row)
{
    if (f32) {
        const float *xf = (const float *)X + i * D;
        for (int64_t j = 0; j < D; ++j) row[j] = (double)xf[j];
    } else {
        const double *xd = (const double *)X + i * D;
        for (int64_t j = 0; j < D; ++j) row[j] = xd[j];
    }
}

/* H = X^T diag(c) X + I / s^2 at w, and the gradient of U at w. */
static void orc_logistic_hessian(const void *X, int f32, const uint8_t *y, int64_t N, int64_t D,
                                 double s, const double *w, double *H, double *grad)
{
    double *row = (double *)malloc((size_t)D * sizeof(double));
    for (int64_t j = 0; j < D * D; ++j) H[j] = 0.0;
    for (int64_t j = 0; j < D; ++j) grad[j] = 0.0;
    for (int64_t i = 0; i < N; ++i) {
        orc_row(X, f32, i, D, row);
        double eta = 0.0;
        for (int64_t j = 0; j < D; ++j) eta += row[j] * w[j];
        double c = orc_sigmoid(eta) * orc_sigmoid(-eta);
        double sgn = y[i] ? -1.0 : 1.0;
        double r = sgn * orc_sigmoid(sgn * eta);
        for (int64_t j = 0; j < D; ++j) {
            grad[j] += r * row[j];
            double cj = c * row[j];
            for (int64_t k = 0; k <= j; ++k) H[j * D + k] += cj * row[k];
        }
    }
    double inv_s2 = 1.0 / (s * s);
    for (int64_t j = 0; j < D; ++j) {
        grad[j] += w[j] * inv_s2;
        H[j * D + j] += inv_s2;
        for (int64_t k = 0; k < j; ++k) H[k * D + j] = H[j * D + k];
    }
    free(row);
}

/* Lower Cholesky factor L of a symmetric positive definite A (in place of
 * the lower triangle of L); returns 0 if A is not positive definite. */
static int orc_cholesky(const double *A, int64_t D, double *L)
{
    for (int64_t j = 0; j < D * D; ++j) L[j] = 0.0;
    for (int64_t j = 0; j < D; ++j) {
        double d = A[j * D + j];
        for (int64_t k = 0; k < j; ++k) d -= L[j * D + k] * L[j * D + k];
        if (!(d > 0.0)) return 0;
        double ljj = sqrt(d);
        L[j * D + j] = ljj;
        for (int64_t i = j + 1; i < D; ++i) {
            double v = A[i * D + j];
            for (int64_t k = 0; k < j; ++k) v -= L[i * D + k] * L[j * D + k];
            L[i * D + j] = v / ljj;
        }
    }
    return 1;
}

/* x = A^-1 b with A = L L^T (forward, then backward substitution). */
static void orc_chol_solve(const double *L, int64_t D, const double *b, double *x)
{
    for (int64_t i = 0; i < D; ++i) {
        double v = b[i];
        for (int64_t k = 0; k < i; ++k) v -= L[i * D + k] * x[k];
        x[i] = v / L[i * D + i];
    }
    for (int64_t i = D - 1; i >= 0; --i) {
        double v = x[i];
        for (int64_t k = i + 1; k < D; ++k) v -= L[k * D + i] * x[k];
        x[i] = v / L[i * D + i];
    }
}

/* Writes w_map [D], cov [D][D] (H^-1 at the MAP) and mean [D] (the
 * skewness-corrected mean); returns the Newton steps taken, or -1 if a
 * Hessian was not positive definite or the steps did not converge. */
int64_t orc_logistic_laplace(const void *X, int f32, const uint8_t *y, int64_t N, int64_t D,
                             double s, double *w_map, double *cov, double *mean)
{
    double *H = (double *)malloc((size_t)(D * D) * sizeof(double));
    double *L = (double *)malloc((size_t)(D * D) * sizeof(double));
    double *g = (double *)malloc((size_t)D * sizeof(double));
    double *d = (double *)malloc((size_t)D * sizeof(double));
    double *e = (double *)calloc((size_t)D, sizeof(double));
    double *row = (double *)malloc((size_t)D * sizeof(double));
    double *b = (double *)calloc((size_t)D, sizeof(double));
    int64_t steps = -1;
    for (int64_t j = 0; j < D; ++j) w_map[j] = 0.0;
    for (int64_t it = 1; it <= 100; ++it) {
        orc_logistic_hessian(X, f32, y, N, D, s, w_map, H, g);
        if (!orc_cholesky(H, D, L)) goto done;
        orc_chol_solve(L, D, g, d);
        int moved = 0;
        for (int64_t j = 0; j < D; ++j) {
            w_map[j] -= d[j];
            if (fabs(d[j]) > 1e-13 * (1.0 + fabs(w_map[j]))) moved = 1;
        }
        if (!moved) {
            steps = it;
            break;
        }
    }
    if (steps < 0) goto done;
    /* H^-1 at the MAP, column by column */
    orc_logistic_hessian(X, f32, y, N, D, s, w_map, H, g);
    if (!orc_cholesky(H, D, L)) {
        steps = -1;
        goto done;
    }
    for (int64_t k = 0; k < D; ++k) {
        for (int64_t j = 0; j < D; ++j) e[j] = (j == k) ? 1.0 : 0.0;
        orc_chol_solve(L, D, e, d);
        for (int64_t j = 0; j < D; ++j) cov[j * D + k] = d[j];
    }
    /* b_j = sum_i sigma''(eta_i) x_ij (x_i^T cov x_i) */
    for (int64_t i = 0; i < N; ++i) {
        orc_row(X, f32, i, D, row);
        double eta = 0.0;
        for (int64_t j = 0; j < D; ++j) eta += row[j] * w_map[j];
        double sp = orc_sigmoid(eta), sm = orc_sigmoid(-eta);
        double s2 = sp * sm * (sm - sp);
        double quad = 0.0;
        for (int64_t j = 0; j < D; ++j) {
            double cj = 0.0;
            for (int64_t k = 0; k < D; ++k) cj += cov[j * D + k] * row[k];
            quad += row[j] * cj;
        }
        for (int64_t j = 0; j < D; ++j) b[j] += s2 * quad * row[j];
    }
    for (int64_t j = 0; j < D; ++j) {
        double cb = 0.0;
        for (int64_t k = 0; k < D; ++k) cb += cov[j * D + k] * b[k];
        mean[j] = w_map[j] - 0.5 * cb;
    }
done:
    free(H); free(L); free(g); free(d); free(e); free(row); free(b);
    return steps;
}
