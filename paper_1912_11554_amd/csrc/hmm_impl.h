// Semi-supervised hidden Markov model as a sampler target: one wavefront per
// chain, the whole tree builder of sampler_impl.h around an evaluator that
// runs the forward-backward recursions in parallel over time.
//
// Model (the HMM benchmark of arXiv 1912.11554, Section 4 and Appendix C,
// set up as in Stan's semi-supervised HMM example): K hidden states, V symbols, one
// sequence w_0 .. w_{T-1} whose first Tsup hidden states z_t are observed.
// The parameters are the K transition rows theta_j and the K emission rows
// phi_k, each a simplex under a uniform Dirichlet prior, sampled on the
// scale of additive log-ratios: a row is the softmax of its free logits and
// a fixed 0, and its Jacobian is the product of its entries.  With
//   f = sum over entries x of (1 + n_x) log x + log p(w_Tsup .. | z_{Tsup-1}),
// n_x the entry's count among the observed transitions and emissions and
// the last term from the forward algorithm, U = -f.  Through the softmax,
// df/da_i = G_i - x_i sum_row G with G = df/d log x = 1 + n_x + expected
// counts (transitions xi, occupancies gamma) from the backward recursion.
//
// Lanes.  Entry lanes: lane e < K*K holds transition entry (e / K, e % K),
// lane K*K + k*V + v emission entry (k, v).  Dimension lanes hold q and
// grad U as the tree builder keeps them: the K - 1 free logits of
// transition row j at j (K - 1), those of emission row k at K (K - 1) +
// k (V - 1).
//
// Time.  Lane l owns the unobserved steps s in [l Ls, (l + 1) Ls), Ls =
// ceil(Tu / 64) <= kHmmSteps, Tu = T - Tsup.  Step s maps the filtered
// distribution a_s to a_{s+1} proportional to a_s M_s, M_s = Theta
// diag(phi(w_s)) (diag(phi(w_0)) alone when no state is observed: the
// chain then starts from the uniform distribution).
//   1. Each lane multiplies its steps' matrices, rescaled by powers of two
//      (exact), so only directions carry rounding.
//   2. A prefix product over the lanes gives each lane the direction of its
//      first forward vector, a suffix product that of its last backward
//      vector.
//   3. Each lane re-runs the scaled forward recursion over its steps (a
//      normalised to sum 1, c_s its normaliser, log p = sum_s log c_s), then
//      the scaled backward recursion (b_{s-1} = M_s b_s / c_s, starting
//      from the direction of step 2 with a_{s+1} . b_s = 1), adding the
//      expected transition counts a_s(j) Theta_jk phi_k(w_s) b_s(k) / c_s
//      in registers and storing the occupancies a_{s+1}(k) b_s(k) in LDS,
//      grouped by symbol.
//   4. Emission lanes add their symbol's run of occupancies (in time order),
//      transition lanes take wave sums of the transition counts.
#pragma once

#include "sampler_impl.h"

namespace nuts {
namespace hmm {

using sampler::run_chain;

constexpr int kHmmChainsPerGroup = 4;
constexpr double kLn2 = 0.69314718055994530942;

// Orders this wave's LDS stores before its later LDS loads of other lanes'
// data (and the loads before later stores).
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    __builtin_amdgcn_wave_barrier();
}

template <int K>
__device__ __forceinline__ void set_identity(double (&P)[K][K])
{
#pragma unroll
    for (int r = 0; r < K; ++r)
#pragma unroll
        for (int c = 0; c < K; ++c) P[r][c] = r == c ? 1.0 : 0.0;
}

// Scale a non-negative matrix by a power of two so its largest entry lies in
// [0.5, 1): exact, so the direction is untouched.
template <int K>
__device__ __forceinline__ void unit_scale(double (&P)[K][K])
{
    // the maximum as a tree (short dependency chains)
    double m[K * K];
#pragma unroll
    for (int r = 0; r < K; ++r)
#pragma unroll
        for (int c = 0; c < K; ++c) m[r * K + c] = P[r][c];
#pragma unroll
    for (int w = 1; w < K * K; w *= 2)
#pragma unroll
        for (int i = 0; i + w < K * K; i += 2 * w) m[i] = fmax(m[i], m[i + w]);
    const double mx = m[0];
    int e = 0;
    (void)frexp(mx, &e);
#pragma unroll
    for (int r = 0; r < K; ++r)
#pragma unroll
        for (int c = 0; c < K; ++c) P[r][c] = ldexp(P[r][c], -e);
}

template <int K>
__device__ __forceinline__ void mat_mul(const double (&A)[K][K], const double (&B)[K][K], double (&C)[K][K])
{
#pragma unroll
    for (int r = 0; r < K; ++r)
#pragma unroll
        for (int c = 0; c < K; ++c) {
            double s = 0.0;
#pragma unroll
            for (int j = 0; j < K; ++j) s += A[r][j] * B[j][c];
            C[r][c] = s;
        }
}

// Sums over the wave of N values per lane at once (a reduce-scatter
// butterfly): at the stage of lane bit M each lane keeps the lower or the
// upper part of its current values, by that bit, and adds its partner's copy
// of them; once one value is left the butterfly goes on over the remaining
// bits.  Returns this lane's final value: the total of value index
// scatter_index(e) == this lane for some e, see scatter_lane.
template <int M, int C>
__device__ __forceinline__ double scatter_stage(const double (&cur)[C])
{
    if constexpr (C == 1) {
        const double s = cur[0] + xor_move<M>(cur[0]);
        if constexpr (M > 1) {
            double n[1] = {s};
            return scatter_stage<M / 2, 1>(n);
        } else {
            return s;
        }
    } else {
        constexpr int lo = (C + 1) / 2, hi = C - lo;
        const bool upper = (lane() & M) != 0;
        double n[lo];
#pragma unroll
        for (int i = 0; i < lo; ++i) {
            const double up = i < hi ? cur[lo + i] : 0.0;
            const double send = upper ? cur[i] : up;
            const double keep = upper ? up : cur[i];
            n[i] = keep + xor_move<M>(send);
        }
        if constexpr (M > 1) {
            return scatter_stage<M / 2, lo>(n);
        } else {
            static_assert(lo == 1, "more values than lanes");
            return n[0];
        }
    }
}

// The lane left holding the total of value e by scatter_stage<32, C>.
__host__ __device__ inline int scatter_lane(int e, int C)
{
    int lanebits = 0;
    for (int M = 32; M >= 1; M >>= 1) {
        if (C == 1) break;
        const int lo = (C + 1) / 2;
        if (e >= lo) {
            lanebits |= M;
            e -= lo;
        }
        C = lo;
    }
    return lanebits;
}

// LDS of one wave, in doubles: the checkpoint array S, the occupancies
// (Tu x K, symbol-sorted; first used to sort the symbols), the emission
// table (V x K), the row table (2K rows of row_width, zero-padded).
struct HmmLds {
    int s_off, gam_off, phi_off, row_off, wave;
};

// Slots of one simplex row in the row table: the longer row length, even.
__host__ __device__ inline int hmm_row_width(int K, int V) { return ((K > V ? K : V) + 1) & ~1; }

__host__ __device__ inline HmmLds hmm_lds(int K, int V, int T, int Tsup, int D, int max_depth, int sub_merge)
{
    HmmLds L;
    const int tu = T - Tsup > 1 ? T - Tsup : 1;
    L.s_off = 0;
    L.gam_off = (int)chain_lds_doubles(D, max_depth, sub_merge, false);
    L.phi_off = L.gam_off + tu * K;
    L.row_off = L.phi_off + V * K;
    L.wave = (L.row_off + 2 * K * hmm_row_width(K, V) + 1) & ~1;  // 16-byte aligned waves
    return L;
}

template <int K>
struct HmmEval {
    static constexpr bool kSpeculative = false;
    static constexpr bool kNodesInLds = false;
    int V, D, Tsup, Tu;
    // this lane's entry
    int src;       // dimension lane of its logit; -1 for a row's fixed logit or no entry
    int RW;        // row table: slots per row
    int slot;      // this entry's slot in the row table (-1 off the entries)
    int row0;      // first slot of its row (0 off the entries)
    double cnt1;   // 1 + its count among the observed states (0 off the entries)
    // the gather of occupancies: gather lane L takes piece L % GP of the
    // symbol run of emission entry L / GP (GP lanes per entry)
    int GP, g_k, g_start, g_count, g_max;  // g_max: the longest piece (wave-uniform)
    int dst;       // dimension lanes: the entry lane of the logit
    int xi_src;    // transition lanes: the lane the wave's sum of its count ends in
    // this lane's steps: first, count, and per step symbol | position << 8
    int s0, ns;
    int sp[kHmmSteps];
    double init[K];  // distribution before the first unobserved step
    bool no_transition0;  // Tsup == 0: step 0 emits from the initial distribution
    double* gam;
    double* phi;
    double* rowt;

    __device__ bool s_writer() const { return true; }
    __device__ bool out_writer() const { return true; }
    __device__ bool aborted() const { return false; }

    __device__ void init_chain(const HmmView& hv, int D_, double* gam_, double* phi_, double* rowt_)
    {
        const int l = lane();
        V = hv.V;
        D = D_;
        Tsup = hv.Tsup;
        Tu = hv.T - hv.Tsup;
        gam = gam_;
        phi = phi_;
        rowt = rowt_;
        RW = hmm_row_width(K, V);
        const int KK = K * K, E = KK + K * V, nt = K * (K - 1);
        if (l < KK) {
            const int j = l / K, k = l % K;
            src = k < K - 1 ? j * (K - 1) + k : -1;
            row0 = j * RW;
            slot = row0 + k;
        } else if (l < E) {
            const int e = l - KK, k = e / V, v = e % V;
            src = v < V - 1 ? nt + k * (V - 1) + v : -1;
            row0 = (K + k) * RW;
            slot = row0 + v;
        } else {
            src = -1;
            row0 = 0;
            slot = -1;
        }
        // the pads of the row table stay zero (a neutral entry for the sums,
        // and for the maximum, which starts from the fixed logit 0)
        for (int i = l; i < 2 * K * RW; i += kWave) rowt[i] = 0.0;
        xi_src = scatter_lane(l < KK ? l : 0, KK);
        if (l < nt) {
            dst = (l / (K - 1)) * K + l % (K - 1);
        } else if (l < D) {
            const int d = l - nt;
            dst = KK + (d / (V - 1)) * V + d % (V - 1);
        } else {
            dst = l;
        }
        const int Ls = (Tu + kWave - 1) / kWave;
        s0 = l * Ls < Tu ? l * Ls : Tu;
        ns = (s0 + Ls < Tu ? s0 + Ls : Tu) - s0;

        // stable counting sort of the unobserved symbols: lane v counts
        // symbol v, then every step gets its place in its symbol's run
        const uint8_t* wu = hv.w + Tsup;
        uint16_t* place = reinterpret_cast<uint16_t*>(gam);
        int cnt = 0;
        for (int c0 = 0; c0 < Tu; c0 += kWave) {
            const int s = c0 + l;
            const int sy = s < Tu ? (int)wu[s] : -1;
            for (int v = 0; v < V; ++v) {
                const unsigned long long m = __ballot(sy == v);
                if (l == v) cnt += __popcll(m);
            }
        }
        int start = 0;
        for (int v = 0; v < V; ++v) {
            const int cv = __builtin_amdgcn_readlane(cnt, v);
            if (v < l) start += cv;
        }
        const unsigned long long below = (1ull << l) - 1ull;
        int run = start;
        for (int c0 = 0; c0 < Tu; c0 += kWave) {
            const int s = c0 + l;
            const int sy = s < Tu ? (int)wu[s] : -1;
            for (int v = 0; v < V; ++v) {
                const unsigned long long m = __ballot(sy == v);
                const int base = __builtin_amdgcn_readlane(run, v);
                if (sy == v) place[s] = (uint16_t)(base + __popcll(m & below));
                if (l == v) run += __popcll(m);
            }
        }
        GP = K * V * 4 <= kWave ? 4 : (K * V * 2 <= kWave ? 2 : 1);
        int cmax = 0;
        for (int v = 0; v < V; ++v) {
            const int cv = __builtin_amdgcn_readlane(cnt, v);
            cmax = cv > cmax ? cv : cmax;
        }
        const int piece = (cmax + GP - 1) / GP;  // run length per piece
        g_max = piece;
        const int ge = l / GP, gh = l % GP;
        const bool gl = ge < K * V;
        const int gv = gl ? ge % V : 0;
        g_k = gl ? ge / V : 0;
        // (cross-lane reads with every lane active: a lane outside the
        // condition would read as zero)
        const int st = __shfl(start, gv);
        const int gc = __shfl(cnt, gv);
        const int lo = gh * piece < gc ? gh * piece : gc;
        const int hi = (gh + 1) * piece < gc ? (gh + 1) * piece : gc;
        g_start = st + lo;
        g_count = gl ? hi - lo : 0;
        wave_lds_sync();
#pragma unroll
        for (int i = 0; i < kHmmSteps; ++i) {
            int v = 0, p = 0;
            if (i < ns) {
                v = wu[s0 + i];
                p = place[s0 + i];
            }
            sp[i] = v | (p << 8);
        }
        wave_lds_sync();  // the sort's scratch is read before evaluations reuse it

        // counts of the observed transitions and emissions per entry
        int ce = 0;
        for (int t0 = 0; t0 < Tsup; t0 += kWave) {
            const int t = t0 + l;
            int eth = -1, eph = -1;
            if (t < Tsup) {
                const int zt = hv.z[t];
                eph = KK + zt * V + hv.w[t];
                if (t > 0) eth = hv.z[t - 1] * K + zt;
            }
            for (int e = 0; e < E; ++e) {
                const unsigned long long m1 = __ballot(eth == e), m2 = __ballot(eph == e);
                if (l == e) ce += __popcll(m1) + __popcll(m2);
            }
        }
        cnt1 = l < E ? 1.0 + (double)ce : 0.0;
        no_transition0 = Tsup == 0;
        const int z0 = Tsup > 0 ? hv.z[Tsup - 1] : 0;
#pragma unroll
        for (int k = 0; k < K; ++k) init[k] = Tsup > 0 ? (k == z0 ? 1.0 : 0.0) : 1.0 / K;
    }

    // Every entry lane's value into its row slot, then over this lane's row
    // in slot order: the maximum (from 0) or the sum (from 0).
    template <bool MAX>
    __device__ double row_reduce(double v)
    {
        wave_lds_sync();  // earlier reads of the table are done
        if (slot >= 0) rowt[slot] = v;
        wave_lds_sync();
        const double* r = rowt + row0;
        double acc = 0.0;
        for (int i = 0; i < RW; i += 2) {
            const double v0 = r[i], v1 = r[i + 1];
            if constexpr (MAX) {
                acc = v0 > acc ? v0 : acc;
                acc = v1 > acc ? v1 : acc;
            } else {
                acc += v0;
                acc += v1;
            }
        }
        return acc;
    }

    __device__ void eval(const double (&q)[1], double& U, double (&g)[1])
    {
        const int l = lane();
        const int KK = K * K, E = KK + K * V;

        // the rows' softmax: max with the fixed 0, then exps summed in row order
        double a = __shfl(q[0], src < 0 ? 0 : src);
        a = src < 0 ? 0.0 : a;
        const double m = row_reduce<true>(a);
        const double ex = exp_nonpos(a - m);
        const double tot = row_reduce<false>(ex);
        const double lx = a - (m + log(tot));
        const double x = exp_nonpos(lx);

        // Theta in every lane's registers, phi in LDS as [symbol][state]
        double th[K][K];
#pragma unroll
        for (int j = 0; j < K; ++j)
#pragma unroll
            for (int k = 0; k < K; ++k) th[j][k] = readlane_f64(x, j * K + k);
        wave_lds_sync();
        if (l >= KK && l < E) {
            const int e = l - KK;
            phi[(e % V) * K + e / V] = x;
        }
        wave_lds_sync();

        // 1. this lane's product of step matrices
        double P[K][K];
        set_identity<K>(P);
#pragma unroll
        for (int i = 0; i < kHmmSteps; ++i) {
            if (i < ns) {
                const double* f = phi + (sp[i] & 255) * K;
                const bool diag = no_transition0 && s0 + i == 0;
                double N[K][K];
#pragma unroll
                for (int r = 0; r < K; ++r)
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        double s = 0.0;
#pragma unroll
                        for (int j = 0; j < K; ++j) s += P[r][j] * th[j][k];
                        N[r][k] = (diag ? P[r][k] : s) * f[k];
                    }
                unit_scale<K>(N);
#pragma unroll
                for (int r = 0; r < K; ++r)
#pragma unroll
                    for (int k = 0; k < K; ++k) P[r][k] = N[r][k];
            }
        }
        double Pown[K][K];
#pragma unroll
        for (int r = 0; r < K; ++r)
#pragma unroll
            for (int k = 0; k < K; ++k) Pown[r][k] = P[r][k];

        // 2a. inclusive prefix product over lanes; the forward start of lane
        // l is init times the product of lanes 0 .. l-1, normalised
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
            double O[K][K], N[K][K];
#pragma unroll
            for (int r = 0; r < K; ++r)
#pragma unroll
                for (int k = 0; k < K; ++k) O[r][k] = __shfl_up(P[r][k], off);
            if (l >= off) {
                mat_mul<K>(O, P, N);
                unit_scale<K>(N);
#pragma unroll
                for (int r = 0; r < K; ++r)
#pragma unroll
                    for (int k = 0; k < K; ++k) P[r][k] = N[r][k];
            }
        }
        double alpha[K];
        {
            double wv[K];
#pragma unroll
            for (int k = 0; k < K; ++k) {
                double s = 0.0;
#pragma unroll
                for (int j = 0; j < K; ++j) s += init[j] * P[j][k];
                wv[k] = s;
            }
            double st = 0.0;
#pragma unroll
            for (int k = 0; k < K; ++k) {
                wv[k] = __shfl_up(wv[k], 1);
                st += wv[k];
            }
            const double r = recip(st);
#pragma unroll
            for (int k = 0; k < K; ++k) alpha[k] = l == 0 ? init[k] : wv[k] * r;
        }

        // 2b. inclusive suffix product; the backward direction at the last
        // step of lane l is the product of lanes l+1 .. 63 times ones
#pragma unroll
        for (int r = 0; r < K; ++r)
#pragma unroll
            for (int k = 0; k < K; ++k) P[r][k] = Pown[r][k];
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
            double O[K][K], N[K][K];
#pragma unroll
            for (int r = 0; r < K; ++r)
#pragma unroll
                for (int k = 0; k < K; ++k) O[r][k] = __shfl_down(P[r][k], off);
            if (l + off < kWave) {
                mat_mul<K>(P, O, N);
                unit_scale<K>(N);
#pragma unroll
                for (int r = 0; r < K; ++r)
#pragma unroll
                    for (int k = 0; k < K; ++k) P[r][k] = N[r][k];
            }
        }
        double bdir[K];
#pragma unroll
        for (int j = 0; j < K; ++j) {
            double s = 0.0;
#pragma unroll
            for (int k = 0; k < K; ++k) s += P[j][k];
            bdir[j] = __shfl_down(s, 1);
        }

        // 3a. scaled forward over this lane's steps
        double ah[kHmmSteps][K];  // a_s before each step
        double rc[kHmmSteps];     // 1 / c_s
        double lm = 1.0;          // product of the c_s as mantissa and exponent
        int le = 0;
#pragma unroll
        for (int i = 0; i < kHmmSteps; ++i) {
            if (i < ns) {
                const double* f = phi + (sp[i] & 255) * K;
                const bool diag = no_transition0 && s0 + i == 0;
                double u[K], c = 0.0;
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    ah[i][k] = alpha[k];
                    double s = 0.0;
#pragma unroll
                    for (int j = 0; j < K; ++j) s += alpha[j] * th[j][k];
                    u[k] = (diag ? alpha[k] : s) * f[k];
                    c += u[k];
                }
                const double r = recip(c);
                rc[i] = r;
#pragma unroll
                for (int k = 0; k < K; ++k) alpha[k] = u[k] * r;
                int e = 0;
                lm = frexp(lm * c, &e);
                le += e;
            }
        }
        const double logp = ns > 0 ? log(lm) + (double)le * kLn2 : 0.0;

        // 3b. scaled backward, expected counts
        double beta[K];
        {
            const bool last = s0 + ns == Tu;
            double d = 0.0;
#pragma unroll
            for (int k = 0; k < K; ++k) d += alpha[k] * bdir[k];
            const double r = recip(d);
#pragma unroll
            for (int k = 0; k < K; ++k) beta[k] = last ? 1.0 : bdir[k] * r;
        }
        double xi[K][K];
#pragma unroll
        for (int j = 0; j < K; ++j)
#pragma unroll
            for (int k = 0; k < K; ++k) xi[j][k] = 0.0;
#pragma unroll
        for (int i = kHmmSteps - 1; i >= 0; --i) {
            if (i < ns) {
                const double* f = phi + (sp[i] & 255) * K;
                double* gp = gam + (sp[i] >> 8) * K;
                double v[K];
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    gp[k] = alpha[k] * beta[k];
                    v[k] = f[k] * beta[k] * rc[i];
                }
                if (!(no_transition0 && s0 + i == 0)) {
#pragma unroll
                    for (int j = 0; j < K; ++j)
#pragma unroll
                        for (int k = 0; k < K; ++k) xi[j][k] += ah[i][j] * th[j][k] * v[k];
                }
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    double s = 0.0;
#pragma unroll
                    for (int k = 0; k < K; ++k) s += th[j][k] * v[k];
                    beta[j] = s;
                    alpha[j] = ah[i][j];
                }
            }
        }
        wave_lds_sync();

        // 4. G = df/d log x on the entry lanes
        double G = cnt1;
        {
            double flat[K * K];
#pragma unroll
            for (int j = 0; j < K; ++j)
#pragma unroll
                for (int k = 0; k < K; ++k) flat[j * K + k] = xi[j][k];
            const double tot = scatter_stage<32, K * K>(flat);
            const double sx = __shfl(tot, xi_src);
            if (l < KK) G += sx;
        }
        double gs = 0.0;
        for (int i0 = 0; i0 < g_max; i0 += 4) {
            double t4[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) t4[u] = i0 + u < g_count ? gam[(g_start + i0 + u) * K + g_k] : 0.0;
#pragma unroll
            for (int u = 0; u < 4; ++u) gs += t4[u];
        }
        // an emission entry's pieces, in time order
        const int gbase = ((l - KK) * GP) & (kWave - 1);
        for (int h = 0; h < GP; ++h) {
            const double ph = __shfl(gs, (gbase + h) & (kWave - 1));
            if (l >= KK && l < E) G += ph;
        }

        // 5. through the softmax, then onto the dimension lanes
        const double rowG = row_reduce<false>(G);
        const double ga = -(G - x * rowG);
        const double gd = __shfl(ga, dst);
        g[0] = l < D ? gd : 0.0;
        U = -wave_sum((l < E ? cnt1 * lx : 0.0) + logp);
    }
};

template <int K, bool EXT>
__global__ void __launch_bounds__(kHmmChainsPerGroup * kWave, 2) sampler_hmm_kernel(SamplerArgs A, HmmView hv,
                                                                                     int cpg)
{
    extern __shared__ double lds[];
    const int wave = threadIdx.x / kWave;
    const int64_t chain = (int64_t)blockIdx.x * cpg + wave;
    if (wave >= cpg || chain >= A.num_chains) return;
    const HmmLds L = hmm_lds(K, hv.V, hv.T, hv.Tsup, A.data.D, A.max_depth, EXT ? A.sub_merge : 0);
    double* base = lds + (int64_t)wave * L.wave;
    HmmEval<K> ev;
    ev.init_chain(hv, A.data.D, base + L.gam_off, base + L.phi_off, base + L.row_off);
    run_chain<1, EXT>(A, ev, chain, base + L.s_off);
}

template <int K>
__global__ void __launch_bounds__(kHmmChainsPerGroup * kWave, 2) hmm_potential_kernel(HmmView hv, int D,
                                                                                       const double* Q, int64_t n,
                                                                                       double* out_U,
                                                                                       double* out_grad, int cpg)
{
    extern __shared__ double lds[];
    const int wave = threadIdx.x / kWave;
    const int64_t p = (int64_t)blockIdx.x * cpg + wave;
    if (wave >= cpg || p >= n) return;
    const int l = lane();
    const HmmLds L = hmm_lds(K, hv.V, hv.T, hv.Tsup, D, 1, 0);
    double* base = lds + (int64_t)wave * L.wave;
    HmmEval<K> ev;
    ev.init_chain(hv, D, base + L.gam_off, base + L.phi_off, base + L.row_off);
    double q[1] = {l < D ? Q[p * D + l] : 0.0}, U, g[1];
    ev.eval(q, U, g);
    if (l < D) out_grad[p * D + l] = g[0];
    if (l == 0) out_U[p] = U;
}

// Chains (waves) per group whose LDS fits, from 4 down to 1; 0 if none.
inline int hmm_chains_per_group(const HmmLds& L, int64_t n)
{
    for (int cpg = kHmmChainsPerGroup; cpg >= 1; cpg /= 2) {
        if (cpg > n && cpg > 1) continue;
        if ((size_t)cpg * L.wave * sizeof(double) <= sampler::kMaxGroupLds) return cpg;
    }
    return 0;
}

template <int K, bool EXT>
hipError_t hmm_sampler_launch(const SamplerArgs& a, const HmmView& hv, hipStream_t stream)
{
    const HmmLds L = hmm_lds(K, hv.V, hv.T, hv.Tsup, a.data.D, a.max_depth, a.sub_merge);
    const int cpg = hmm_chains_per_group(L, a.num_chains);
    if (cpg == 0) return hipErrorInvalidValue;
    const size_t lds = (size_t)cpg * L.wave * sizeof(double);
    const void* k = (const void*)sampler_hmm_kernel<K, EXT>;
    hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    const unsigned grid = (unsigned)((a.num_chains + cpg - 1) / cpg);
    hipLaunchKernelGGL((sampler_hmm_kernel<K, EXT>), dim3(grid), dim3(kHmmChainsPerGroup * kWave), lds, stream, a,
                       hv, cpg);
    return hipGetLastError();
}

template <bool EXT>
hipError_t hmm_sampler_dispatch(const SamplerArgs& a, const HmmView& hv, hipStream_t stream)
{
    switch (hv.K) {
    case 2: return hmm_sampler_launch<2, EXT>(a, hv, stream);
    case 3: return hmm_sampler_launch<3, EXT>(a, hv, stream);
    case 4: return hmm_sampler_launch<4, EXT>(a, hv, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace hmm
}  // namespace nuts
