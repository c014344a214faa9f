// Device-resident NUTS: trajectory doubling with the iterative tree builder,
// leapfrog steps, multinomial / biased-progressive proposal selection, U-turn
// and divergence checks, all inside one kernel launch.
//
// Tree state is held lane-per-dimension: lane d of a wave keeps component d
// of every phase-space vector (position q, momentum p, gradient g) of the
// current leaf, both trajectory edges, the proposal and the subtree proposal.
// Dot products are wave butterflies, so every lane (and, on the grid path,
// the controller wave of every group) holds bit-identical scalars and takes
// identical decisions.  Lanes >= D carry zeros.
//
// Two evaluators supply U and grad U at a position:
//   WaveEval -- one wave streams its chain's data set (small data; one wave
//               per chain, thousands of chains per launch);
//   GridEval -- one chain on the whole device.  In every group, wave 0 is the
//               controller (it runs the tree logic) and the other waves are
//               workers (they stream a slice of the rows).  Group partials
//               meet at a grid barrier whose last arriver adds them in group
//               order.  Controller and workers run the same collective with
//               the same workgroup barriers; only the workers' copy contains
//               the data pass, so tree state and data-pass registers are never
//               live together.
//
// Algorithmic sources: Appendix A of arXiv 1912.11554 (Alg. 2 iterative tree,
// the S array indexed by BitCount, candidate set C(n)); Hoffman & Gelman 2014,
// Alg. 6 (direction per doubling, endpoint U-turn rule, Delta_max = 1000);
// Betancourt 2017, App. A (multinomial and biased progressive selection).
#include "launch.h"
#include "rows.h"

namespace nuts {

namespace {

constexpr int kTreeOk = 0, kTreeTurning = 1, kTreeDivergent = 2;
constexpr double kHalfLog2Pi = 0.91893853320467274178032973640562;

// Endpoint U-turn test on time-ordered ends: (a, b) are the first- and
// last-generated nodes of a subtree built in direction v.
__device__ __forceinline__ bool is_uturn(double qa, double pa, double qb, double pb, int v, double im)
{
    const double qL = v > 0 ? qa : qb, pL = v > 0 ? pa : pb;
    const double qR = v > 0 ? qb : qa, pR = v > 0 ? pb : pa;
    const double dq = qR - qL;
    const double dl = wave_sum(dq * im * pL);
    const double dr = wave_sum(dq * im * pR);
    return uni((dl < 0.0) || (dr < 0.0));
}

struct Node {
    double q, p, g;  // this lane's component
    double U;        // wave-uniform
};

// Evaluator interface: eval(q_lane, U, g_lane); s_writer() says whether this
// wave stores the checkpoint array S, out_writer() whether it stores the
// chain's outputs; aborted() reports a failed grid barrier.

template <typename T, int S>
struct WaveEval {
    const T* X;
    const uint8_t* y;
    int64_t N, nb;
    int D;
    double inv_s2, prior_const;

    __device__ bool s_writer() const { return true; }
    __device__ bool out_writer() const { return true; }
    __device__ bool aborted() const { return false; }

    __device__ void eval(double q, double& U, double& g)
    {
        constexpr int CPS = kColsPerLane;
        double qv[CPS];
        spread_position<CPS, S>(q, qv);
        double acc[CPS];
#pragma unroll
        for (int c = 0; c < CPS; ++c) acc[c] = 0.0;
        double loss = 0.0;
        stream_blocks<T, CPS, S>(X, y, D, N, nb, 0, 1, qv, acc, loss);
        const double col = finish_pass<CPS, S>(acc, loss);
        const double prior = wave_sum(0.5 * q * q * inv_s2);
        U = loss + prior + prior_const;
        g = (lane() < D) ? col + q * inv_s2 : 0.0;
    }
};

// ---------------------------------------------------------------------------
// Grid path.

constexpr int kCmdEval = 1, kCmdExit = 2;

template <int NW>
struct GridShared {
    double qbuf[kWave];
    double red[NW][kWave];
    int cmd;
    int last;
};

struct GridCtx {
    const void* X;
    const uint8_t* y;
    int64_t N, nb;
    int D;
    int groups;
    double* partials;  // [2][groups][64]
    double* result;    // [2][64]
    GridSync* sync;
};

// Cross-group exchange.  Everything that one group publishes for another
// (partials, the result, counters, the flag) is written and read with
// agent-scope atomic accesses, which the L2 keeps coherent across the XCDs one
// access at a time.  Ordering between them comes from waiting for the
// group's outstanding memory operations (s_waitcnt) before the next one is
// issued.  No whole-cache write-back or invalidate (what a device-scope
// fence does) is needed: no ordinary store has to become visible to another
// group, and no ordinary load may observe another group's writes.
__device__ __forceinline__ void store_shared(double* p, double v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double load_shared(const double* p)
{
    return __hip_atomic_load(const_cast<double*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void drain_memory_ops()
{
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// The result slots hold this bit pattern (a signalling NaN, which no
// arithmetic produces) until the step's result is written.
constexpr unsigned long long kEmptySlot = 0x7FF4DEADBEEF0001ull;

__device__ __forceinline__ unsigned long long slot_bits(const double* p)
{
    return __hip_atomic_load(reinterpret_cast<unsigned long long*>(const_cast<double*>(p)), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
}

// One collective evaluation for the whole group.  Wave 0 passes the position
// (lane per dimension) and the command; with kCmdEval every worker streams its
// blocks and the group joins the grid-wide sum.  Returns the command; on
// return wave 0 finds the full sums (columns, loss in slot 63) in *out_r.
// Controller and workers execute the same workgroup barriers; the workers
// return as soon as their part is handed over.
//
// Step s uses parity buffer s & 1.  Each group stores its partial and counts
// itself in; the group that completes the count adds all partials in group
// order, re-arms the other parity's result slots (every controller has read
// them: it arrived at this step after reading them) and stores the result.
// Controllers poll their own lane's result slot until it is no longer empty.
template <typename T, int S, int NW, bool WORKER>
__device__ int grid_collective(const GridCtx& c, GridShared<NW>& sh, unsigned long long step, double q,
                               int cmd_in, double* out_r, bool* aborted)
{
    constexpr int CPS = kColsPerLane;
    const int l = lane();
    const int wave = threadIdx.x / kWave;
    const int par = (int)(step & 1);
    if (wave == 0) {
        sh.qbuf[l] = q;
        if (l == 0) sh.cmd = cmd_in;
    }
    __syncthreads();  // position and command published
    const int cmd = sh.cmd;
    if (cmd == kCmdExit) return cmd;

    double mine = 0.0;
    if (WORKER) {
        double qv[CPS];
        const int p = l & (S - 1);
#pragma unroll
        for (int k = 0; k < CPS; ++k) qv[k] = sh.qbuf[(k * S + p) & (kWave - 1)];
        double acc[CPS];
#pragma unroll
        for (int k = 0; k < CPS; ++k) acc[k] = 0.0;
        double loss = 0.0;
        const int workers = NW - 1;
        stream_blocks<T, CPS, S>((const T*)c.X, c.y, c.D, c.N, c.nb, (int64_t)blockIdx.x * workers + (wave - 1),
                                 (int64_t)c.groups * workers, qv, acc, loss);
        const double col = finish_pass<CPS, S>(acc, loss);
        mine = (l < c.D) ? col : (l == kWave - 1 ? loss : 0.0);
    }
    sh.red[wave][l] = mine;
    __syncthreads();  // group partials in LDS

    if (wave == 0) {
        double s = 0.0;
#pragma unroll
        for (int w = 1; w < NW; ++w) s += sh.red[w][l];
        store_shared(&c.partials[((int64_t)par * c.groups + blockIdx.x) * kWave + l], s);
        drain_memory_ops();
        // arrival: per group slot (group index mod 8) first, so that the
        // atomics spread over eight addresses; the group completing its slot
        // counts the slot in at the top counter; the group completing the top
        // count reduces
        int last = 0;
        if (l == 0) {
            const int slot = blockIdx.x & 7;
            const unsigned long long per = (unsigned long long)((c.groups - slot + 7) / 8);
            const unsigned long long o =
                __hip_atomic_fetch_add(&c.sync->slot[slot][0], 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (o + 1 == (step + 1) * per) {
                const unsigned long long slots = c.groups < 8 ? (unsigned long long)c.groups : 8ull;
                const unsigned long long t =
                    __hip_atomic_fetch_add(&c.sync->counter, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                last = (t + 1 == (step + 1) * slots) ? 1 : 0;
            }
        }
        last = __shfl(last, 0);
        if (l == 0) sh.last = last;
    }
    __syncthreads();  // arrival recorded
    if (sh.last) {
        // every controller has read the other parity's result by now: re-arm
        // those slots while the partials load
        if (wave == 0)
            __hip_atomic_store(reinterpret_cast<unsigned long long*>(&c.result[(par ^ 1) * kWave + l]), kEmptySlot,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // add the group partials in group order, spread over the waves, then
        // in wave order
        double s = 0.0;
        const double* src = c.partials + (int64_t)par * c.groups * kWave + l;
        int gg = wave;
        for (; gg + 7 * NW < c.groups; gg += 8 * NW) {
            double v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = load_shared(src + (int64_t)(gg + i * NW) * kWave);
#pragma unroll
            for (int i = 0; i < 8; ++i) s += v[i];
        }
        for (; gg < c.groups; gg += NW) s += load_shared(src + (int64_t)gg * kWave);
        sh.red[wave][l] = s;
        __syncthreads();  // per-wave sums in LDS
        if (wave == 0) {
            double tot = 0.0;
#pragma unroll
            for (int w = 0; w < NW; ++w) tot += sh.red[w][l];
            drain_memory_ops();  // the re-arm above lands before this result
            store_shared(&c.result[par * kWave + l], tot);
        }
    }
    if (WORKER) return cmd;

    // controller: wait for this lane's result slot; give up (and tell every
    // group) after about 10 s so that a broken invariant can never hang the
    // device
    const double* slot = &c.result[par * kWave + l];
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    bool bad = false;
    unsigned long long bits = kEmptySlot;
    for (;;) {
        if (bits == kEmptySlot) bits = slot_bits(slot);
        if (__all(bits != kEmptySlot)) break;
        if (__hip_atomic_load(&c.sync->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
            bad = true;
            break;
        }
        if (__builtin_amdgcn_s_memrealtime() - t0 > 1000000000ull) {
            if (l == 0) __hip_atomic_store(&c.sync->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            bad = true;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    *aborted = bad;
    *out_r = bad ? 0.0 : __builtin_bit_cast(double, bits);
    return cmd;
}

template <typename T, int S, int NW>
struct GridEval {
    GridCtx c;
    GridShared<NW>* sh;
    double inv_s2, prior_const;
    unsigned long long step;
    bool abort;

    __device__ bool s_writer() const { return true; }  // only the controller runs the chain
    __device__ bool out_writer() const { return blockIdx.x == 0; }
    __device__ bool aborted() const { return abort; }

    __device__ void eval(double q, double& U, double& g)
    {
        double r = 0.0;
        bool ab = false;
        grid_collective<T, S, NW, false>(c, *sh, step, q, kCmdEval, &r, &ab);
        abort = ab;
        step++;
        const double prior = wave_sum(0.5 * q * q * inv_s2);
        U = __shfl(r, kWave - 1) + prior + prior_const;
        g = (lane() < c.D) ? r + q * inv_s2 : 0.0;
    }

    __device__ void finish()
    {
        double r;
        bool ab;
        grid_collective<T, S, NW, false>(c, *sh, step, 0.0, kCmdExit, &r, &ab);
    }
};

// The whole chain: init, warmup + sampling iterations, outputs.  S points to
// this chain's checkpoint array in LDS: [max(max_depth, 1)][2][D].
template <class Eval>
__device__ void run_chain(const SamplerArgs& A, Eval& ev, int64_t chain, double* S)
{
    const int l = lane();
    const int D = A.data.D;
    const bool act = l < D;
    const int maxd = A.max_depth;
    const double eps = A.step_size;
    const uint64_t seed = A.seed;
    const int64_t cidx = A.chain_offset + chain;
    const uint64_t key_chain = (uint64_t)cidx;
    const bool out = ev.out_writer();
    const bool s_out = ev.s_writer();

    double im = (act && A.inv_mass) ? A.inv_mass[l] : 1.0;

    Node cur;
    cur.q = (act && A.init_q) ? A.init_q[cidx * D + l] : 0.0;
    cur.p = 0.0;
    ev.eval(cur.q, cur.U, cur.g);
    unsigned long long evals = 1;

    double wmean = 0.0, wm2 = 0.0;
    int64_t wn = 0;
    const int64_t iters = A.num_warmup + A.num_samples;

    for (int64_t k = 0; k < iters && !ev.aborted(); ++k) {
        const uint64_t t = (uint64_t)(A.first_iter + k);

        // momentum and initial energy
        const double xi = act ? momentum_normal(seed, key_chain, t, l) : 0.0;
        cur.p = act ? xi / sqrt(im) : 0.0;
        const double H0 = cur.U + 0.5 * wave_sum(im * cur.p * cur.p);

        // per-iteration draws, one doubling per lane: direction bits and the
        // merge uniforms
        int dir_bit = 0;
        double u_merge = 0.0;
        if (l < maxd) {
            dir_bit = (int)(draw(seed, key_chain, t, kTagDirection, (uint64_t)l, 0).w0 & 1ull);
            u_merge = unit53(draw(seed, key_chain, t, kTagMerge, (uint64_t)l, 0).w0);
        }
        const uint64_t dirmask = __ballot(dir_bit);

        Node left = cur, right = cur, prop = cur;
        int64_t prop_idx = 0, Lpos = 0, Rpos = 0;
        double logw_traj = 0.0;
        int nleaves = 0;
        double sum_acc = 0.0;
        int depth = 0, term = -1;
        uint32_t dirbits = 0;
        int diverging = 0, turning = 0, maxhit = 0;

        for (int j = 0; j < maxd; ++j) {
            const int v = ((dirmask >> j) & 1ull) ? 1 : -1;
            if (v > 0) dirbits |= 1u << j;
            Node z = v > 0 ? right : left;
            const int64_t e = v > 0 ? Rpos : Lpos;
            const double h = v * eps;
            double logw = -INFINITY;
            Node sprop = z;
            int64_t sprop_idx = 0;
            int status = kTreeOk;
            depth = j + 1;
            const int64_t nleaf = 1ll << j;
            double u_leaf = 0.0;

            for (int64_t n = 0; n < nleaf; ++n) {
                if ((n & (kWave - 1)) == 0)
                    u_leaf = (n + l < nleaf)
                                 ? unit53(draw(seed, key_chain, t, kTagLeaf, (uint64_t)j, (uint64_t)(n + l)).w0)
                                 : 0.0;
                // leapfrog: half kick, drift, gradient, half kick
                const double ph = z.p - 0.5 * h * z.g;
                z.q = z.q + h * im * ph;
                ev.eval(z.q, z.U, z.g);
                if (ev.aborted()) break;
                z.p = ph - 0.5 * h * z.g;
                ++nleaves;

                const double dH = (z.U + 0.5 * wave_sum(im * z.p * z.p)) - H0;
                if (dH == dH) sum_acc += dH > 0.0 ? exp(-dH) : 1.0;
                if (uni(!(dH <= 1000.0))) {
                    status = kTreeDivergent;
                    term = (int)n;
                    break;
                }
                // streaming multinomial choice inside the subtree
                const double lam = -dH;
                const double lw = logaddexp(logw, lam);
                const double u = __shfl(u_leaf, (int)(n & (kWave - 1)));
                if (uni(u < exp(lam - lw))) {
                    sprop = z;
                    sprop_idx = e + v * (n + 1);
                }
                logw = lw;

                if ((n & 1) == 0) {
                    // even leaf: checkpoint into S[BitCount(n)]
                    const int i = __popcll((unsigned long long)n);
                    if (s_out && act) {
                        S[(2 * i) * D + l] = z.q;
                        S[(2 * i + 1) * D + l] = z.p;
                    }
                } else {
                    // odd leaf: test the subtrees that end here, smallest first
                    const int nl = __builtin_ctzll(~(unsigned long long)n);
                    const int imax = __popcll((unsigned long long)(n - 1));
                    const int imin = imax - nl + 1;
                    bool turned = false;
                    for (int kk = imax; kk >= imin; --kk) {
                        const double sq = act ? S[(2 * kk) * D + l] : 0.0;
                        const double sp = act ? S[(2 * kk + 1) * D + l] : 0.0;
                        if (is_uturn(sq, sp, z.q, z.p, v, im)) {
                            turned = true;
                            break;
                        }
                    }
                    if (turned) {
                        status = kTreeTurning;
                        term = (int)n;
                        break;
                    }
                }
            }
            if (ev.aborted()) break;
            if (status != kTreeOk) {
                if (status == kTreeDivergent) diverging = 1;
                else turning = 1;
                break;
            }
            // biased progressive choice between trajectory and new subtree
            const double um = __shfl(u_merge, j);
            if (uni(um < exp(logw - logw_traj))) {
                prop = sprop;
                prop_idx = sprop_idx;
            }
            logw_traj = logaddexp(logw_traj, logw);
            if (v > 0) {
                right = z;
                Rpos += nleaf;
            } else {
                left = z;
                Lpos -= nleaf;
            }
            if (is_uturn(left.q, left.p, right.q, right.p, 1, im)) {
                turning = 1;
                term = -2;
                break;
            }
            if (j == maxd - 1) maxhit = 1;
        }
        evals += (unsigned long long)nleaves;
        cur = prop;

        // diagonal inverse mass from warmup states in [W/2, W)
        if (A.adapt_diag && k < A.num_warmup && k >= A.num_warmup / 2) {
            ++wn;
            const double d1 = cur.q - wmean;
            wmean += d1 / (double)wn;
            wm2 += d1 * (cur.q - wmean);
        }
        if (A.adapt_diag && k == A.num_warmup - 1 && wn >= 2) {
            const double nn = (double)wn;
            double var = (nn / (nn + 5.0)) * (wm2 / (nn - 1.0)) + 1e-3 * (5.0 / (nn + 5.0));
            var = act ? var : 0.0;
            const double mean = wave_sum(var) / (double)D;
            im = act ? var / mean : 1.0;
        }

        if (k >= A.num_warmup && out) {
            const int64_t s = k - A.num_warmup;
            if (A.out_samples && act) A.out_samples[(cidx * A.num_samples + s) * D + l] = cur.q;
            if (A.out_stats) {
                const double K = 0.5 * wave_sum(im * cur.p * cur.p);
                if (l == 0) {
                    nuts_stats st;
                    st.potential_energy = cur.U;
                    st.energy = cur.U + K;
                    st.accept_prob = nleaves > 0 ? sum_acc / (double)nleaves : 0.0;
                    st.tree_depth = depth;
                    st.num_steps = nleaves;
                    st.proposal_index = (int32_t)prop_idx;
                    st.term_leaf = term;
                    st.direction_bits = dirbits;
                    st.diverging = (uint8_t)diverging;
                    st.turning = (uint8_t)turning;
                    st.hit_max_depth = (uint8_t)maxhit;
                    for (int i = 0; i < 9; ++i) st._pad[i] = 0;
                    A.out_stats[cidx * A.num_samples + s] = st;
                }
            }
        }
    }
    if (out) {
        if (A.out_final_q && act) A.out_final_q[cidx * D + l] = cur.q;
        if (A.out_inv_mass && act) A.out_inv_mass[cidx * D + l] = im;
        if (l == 0) A.grad_evals[cidx] = evals;
    }
}

constexpr int kWaveChainsPerGroup = 4;

template <typename T, int S>
__global__ void __launch_bounds__(kWaveChainsPerGroup * kWave, 3) sampler_wave_kernel(SamplerArgs A)
{
    constexpr int R = BlockShape<T, S>::R;
    extern __shared__ double lds[];
    const int wave = threadIdx.x / kWave;
    const int64_t chain = (int64_t)blockIdx.x * kWaveChainsPerGroup + wave;
    if (chain >= A.num_chains) return;
    const int D = A.data.D;
    const int slots = A.max_depth > 1 ? A.max_depth : 1;
    double* S_arr = lds + (int64_t)wave * slots * 2 * D;
    const int64_t c = A.chain_offset + chain;
    const int64_t ds = A.per_chain_data ? c : 0;
    WaveEval<T, S> ev;
    ev.X = (const T*)A.data.X + ds * A.data.nb * (int64_t)D * R;
    ev.y = A.data.y + ds * A.data.nb * R;
    ev.N = A.data.N;
    ev.nb = A.data.nb;
    ev.D = D;
    ev.inv_s2 = 1.0 / (A.prior_scale * A.prior_scale);
    ev.prior_const = (double)D * (log(A.prior_scale) + kHalfLog2Pi);
    run_chain(A, ev, chain, S_arr);
}

constexpr int kGridWaves = 16;  // 1 controller + 15 workers

template <typename T, int S>
__global__ void __launch_bounds__(kGridWaves * kWave, 1) sampler_grid_kernel(SamplerArgs A, int groups,
                                                                         double* partials,
                                                                         double* result,
                                                                         GridSync* sync)
{
    extern __shared__ double lds[];
    __shared__ GridShared<kGridWaves> sh;
    GridCtx c;
    c.X = A.data.X;
    c.y = A.data.y;
    c.N = A.data.N;
    c.nb = A.data.nb;
    c.D = A.data.D;
    c.groups = groups;
    c.partials = partials;
    c.result = result;
    c.sync = sync;
    const int wave = threadIdx.x / kWave;
    if (wave == 0) {
        GridEval<T, S, kGridWaves> ev;
        ev.c = c;
        ev.sh = &sh;
        ev.inv_s2 = 1.0 / (A.prior_scale * A.prior_scale);
        ev.prior_const = (double)A.data.D * (log(A.prior_scale) + kHalfLog2Pi);
        ev.step = 0;
        ev.abort = false;
        run_chain(A, ev, 0, lds);
        ev.finish();
    } else {
        unsigned long long step = 0;
        for (;;) {
            double r;
            bool ab;
            if (grid_collective<T, S, kGridWaves, true>(c, sh, step, 0.0, 0, &r, &ab) == kCmdExit) break;
            step++;
        }
    }
}

}  // namespace

__global__ void fill_empty_slots(double* result)
{
    reinterpret_cast<unsigned long long*>(result)[threadIdx.x] = kEmptySlot;
}

template <typename T, int S>
static hipError_t wave_launch(const SamplerArgs& a, hipStream_t stream)
{
    const int slots = a.max_depth > 1 ? a.max_depth : 1;
    const size_t lds = (size_t)kWaveChainsPerGroup * slots * 2 * a.data.D * sizeof(double);
    const unsigned grid = (unsigned)((a.num_chains + kWaveChainsPerGroup - 1) / kWaveChainsPerGroup);
    hipLaunchKernelGGL((sampler_wave_kernel<T, S>), dim3(grid), dim3(kWaveChainsPerGroup * kWave), lds,
                       stream, a);
    return hipGetLastError();
}

template <typename T>
static hipError_t wave_launch_split(const SamplerArgs& a, hipStream_t stream)
{
    if (a.data.split == 1) return wave_launch<T, 1>(a, stream);
    if (a.data.split == 2) return wave_launch<T, 2>(a, stream);
    if (a.data.split == 4) return wave_launch<T, 4>(a, stream);
    return wave_launch<T, 8>(a, stream);
}

hipError_t launch_sampler_wave(const SamplerArgs& a, hipStream_t stream)
{
    return a.data.dtype == NUTS_F64 ? wave_launch_split<double>(a, stream) : wave_launch_split<float>(a, stream);
}

static void* pick_grid_kernel(int dtype, int split)
{
    if (dtype == NUTS_F64) {
        if (split == 1) return (void*)sampler_grid_kernel<double, 1>;
        if (split == 2) return (void*)sampler_grid_kernel<double, 2>;
        if (split == 4) return (void*)sampler_grid_kernel<double, 4>;
        return (void*)sampler_grid_kernel<double, 8>;
    }
    if (split == 1) return (void*)sampler_grid_kernel<float, 1>;
    if (split == 2) return (void*)sampler_grid_kernel<float, 2>;
    if (split == 4) return (void*)sampler_grid_kernel<float, 4>;
    return (void*)sampler_grid_kernel<float, 8>;
}

int grid_sampler_groups(const DataView& dv, int max_depth, int num_cu)
{
    void* k = pick_grid_kernel(dv.dtype, dv.split);
    int per_cu = 0;
    const int slots = max_depth > 1 ? max_depth : 1;
    const size_t lds = (size_t)slots * 2 * dv.D * sizeof(double);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, kGridWaves * kWave, lds) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    if (per_cu > 1) per_cu = 1;
    int64_t groups = (int64_t)num_cu * per_cu;
    const int64_t most = (dv.nb + kGridWaves - 2) / (kGridWaves - 1);
    if (groups > most) groups = most;
    if (groups < 1) groups = 1;
    return (int)groups;
}

hipError_t launch_sampler_grid(const SamplerArgs& a, int groups, double* partials, double* result,
                               GridSync* sync, hipStream_t stream)
{
    hipError_t e = hipMemsetAsync(sync, 0, sizeof(GridSync), stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fill_empty_slots, dim3(1), dim3(2 * kWave), 0, stream, result);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int slots = a.max_depth > 1 ? a.max_depth : 1;
    const size_t lds = (size_t)slots * 2 * a.data.D * sizeof(double);
    void* k = pick_grid_kernel(a.data.dtype, a.data.split);
    SamplerArgs A = a;
    void* args[] = {&A, &groups, &partials, &result, &sync};
    return hipLaunchCooperativeKernel(k, dim3(groups), dim3(kGridWaves * kWave), args, (unsigned)lds, stream);
}

}  // namespace nuts
