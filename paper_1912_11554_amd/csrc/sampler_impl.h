// Device-resident NUTS: trajectory doubling with the iterative tree builder,
// leapfrog steps, multinomial / biased-progressive proposal selection, U-turn
// and divergence checks, all inside one kernel launch.
//
// Tree state is held lane-per-dimension: dimension d lives in lane d % 64,
// component d / 64 (DPL = ceil(D / 64) components per lane).  Every lane
// keeps its components of the phase-space vectors (position q, momentum p,
// gradient g) of the current leaf, both trajectory edges, the proposal and
// the subtree proposal.  Dot products are DPP wave sums, so every lane (and,
// on the grid path, the controller wave of every group) holds bit-identical
// scalars and takes identical decisions.  Dimensions >= D carry zeros.
//
// Two evaluators supply U and grad U at a position:
//   WaveEval -- one wave streams its chain's data set (small data; one wave
//               per chain, thousands of chains per launch; D <= 64);
//   GridEval -- one chain on the whole device.  In every group, wave 0 is the
//               controller (it runs the tree logic) and the other waves are
//               workers (they stream a slice of the rows).  Group partials
//               meet in a grid-wide exchange where each column has an owner
//               group that adds its partials in a fixed order.  Controller and workers run the same collective
//               with the same workgroup barriers; only the workers' copy
//               contains the data pass, so tree state and data-pass
//               registers are never live together.
//
// Algorithmic sources: Appendix A of arXiv 1912.11554 (Alg. 2 iterative tree,
// the S array indexed by BitCount, candidate set C(n)); Hoffman & Gelman 2014,
// Alg. 6 (direction per doubling, endpoint U-turn rule, Delta_max = 1000);
// Betancourt 2017, App. A (multinomial and biased progressive selection).
#pragma once

#include "launch.h"
#include "rows.h"

namespace nuts {
namespace sampler {

constexpr int kTreeOk = 0, kTreeTurning = 1, kTreeDivergent = 2;
constexpr double kHalfLog2Pi = 0.91893853320467274178032973640562;

template <int DPL>
struct Node {
    double q[DPL], p[DPL], g[DPL];  // this lane's components
    double U;                       // wave-uniform
};

// The trajectory's two edges, its proposal and the current subtree's
// proposal.  In registers, or (LDS: the wide shapes of the grid and batch
// paths, whose controller would otherwise spill them to scratch memory) in
// a region of the chain's LDS: node k at base + k * kStride holds q, p and
// grad U (lane l's component m at l + 64 m of each of the three vectors),
// then U.  Only the chain's own wave reads and writes the region.
template <int DPL, bool LDS>
struct EdgeNodes;

template <int DPL>
struct EdgeNodes<DPL, false> {
    Node<DPL> left, right, prop, sprop;
    __device__ void bind(double*) {}
    __device__ void reset(const Node<DPL>& c) { left = right = prop = c; }
    __device__ Node<DPL> edge(bool r) const { return r ? right : left; }
    __device__ void set_edge(bool r, const Node<DPL>& z)
    {
        if (r) right = z;
        else left = z;
    }
    __device__ double edge_q(bool r, int m) const { return r ? right.q[m] : left.q[m]; }
    __device__ double edge_p(bool r, int m) const { return r ? right.p[m] : left.p[m]; }
    __device__ double edge_g(bool r, int m) const { return r ? right.g[m] : left.g[m]; }
    __device__ void set_sprop(const Node<DPL>& z) { sprop = z; }
    __device__ void accept_sprop() { prop = sprop; }
    __device__ Node<DPL> get_prop() const { return prop; }
};

template <int DPL>
struct EdgeNodes<DPL, true> {
    static constexpr int kVec = 64 * DPL;
    static constexpr int kStride = 3 * kVec + 1;
    static constexpr int kLeft = 0, kRight = 1, kProp = 2, kSprop = 3;
    double* base;
    __device__ void bind(double* b) { base = b; }
    __device__ void store(int k, const Node<DPL>& n)
    {
        const int l = lane();
        double* b = base + k * kStride;
#pragma unroll
        for (int m = 0; m < DPL; ++m) {
            b[l + 64 * m] = n.q[m];
            b[kVec + l + 64 * m] = n.p[m];
            b[2 * kVec + l + 64 * m] = n.g[m];
        }
        if (l == 0) b[3 * kVec] = n.U;
    }
    __device__ Node<DPL> load(int k) const
    {
        const int l = lane();
        const double* b = base + k * kStride;
        Node<DPL> n;
#pragma unroll
        for (int m = 0; m < DPL; ++m) {
            n.q[m] = b[l + 64 * m];
            n.p[m] = b[kVec + l + 64 * m];
            n.g[m] = b[2 * kVec + l + 64 * m];
        }
        n.U = b[3 * kVec];
        return n;
    }
    __device__ void reset(const Node<DPL>& c)
    {
        store(kLeft, c);
        store(kRight, c);
        store(kProp, c);
    }
    __device__ Node<DPL> edge(bool r) const { return load(r ? kRight : kLeft); }
    __device__ void set_edge(bool r, const Node<DPL>& z) { store(r ? kRight : kLeft, z); }
    __device__ double edge_q(bool r, int m) const { return base[(r ? kRight : kLeft) * kStride + lane() + 64 * m]; }
    __device__ double edge_p(bool r, int m) const
    {
        return base[(r ? kRight : kLeft) * kStride + kVec + lane() + 64 * m];
    }
    __device__ double edge_g(bool r, int m) const
    {
        return base[(r ? kRight : kLeft) * kStride + 2 * kVec + lane() + 64 * m];
    }
    __device__ void set_sprop(const Node<DPL>& z) { store(kSprop, z); }
    __device__ void accept_sprop() { store(kProp, load(kSprop)); }
    __device__ Node<DPL> get_prop() const { return load(kProp); }
};

// Endpoint U-turn test on time-ordered ends: (a, b) are the first- and
// last-generated nodes of a subtree built in direction v.  one_row: D <= 16
// (the lanes past D hold zeros, see wave_sum_rows).
template <int DPL>
__device__ __forceinline__ bool is_uturn(const double (&qa)[DPL], const double (&pa)[DPL], const double (&qb)[DPL],
                                         const double (&pb)[DPL], int v, const double (&im)[DPL], bool one_row)
{
    double sl = 0.0, sr = 0.0;
#pragma unroll
    for (int m = 0; m < DPL; ++m) {
        const double qL = v > 0 ? qa[m] : qb[m], pL = v > 0 ? pa[m] : pb[m];
        const double qR = v > 0 ? qb[m] : qa[m], pR = v > 0 ? pb[m] : pa[m];
        const double dq = qR - qL;
        sl += dq * im[m] * pL;
        sr += dq * im[m] * pR;
    }
    const double dl = wave_sum_rows(sl, one_row);
    const double dr = wave_sum_rows(sr, one_row);
    return uni((dl < 0.0) || (dr < 0.0));
}

// Generalised criterion (Betancourt 2017, App. A.4.2): a (sub)trajectory
// with momentum sum rho turns iff rho . M^-1 p <= 0 at either end.
template <int DPL>
__device__ __forceinline__ bool is_uturn_gen(const double (&rho)[DPL], const double (&pa)[DPL],
                                             const double (&pb)[DPL], const double (&im)[DPL], bool one_row)
{
    double sa = 0.0, sb = 0.0;
#pragma unroll
    for (int m = 0; m < DPL; ++m) {
        sa += rho[m] * im[m] * pa[m];
        sb += rho[m] * im[m] * pb[m];
    }
    const double da = wave_sum_rows(sa, one_row);
    const double db = wave_sum_rows(sb, one_row);
    return uni((da <= 0.0) || (db <= 0.0));
}

// Evaluator interface: eval(q, U, g) with q, g lane-per-dimension arrays;
// s_writer() says whether this wave stores the checkpoint array S,
// out_writer() whether it stores the chain's outputs; aborted() reports a
// failed grid exchange.

template <typename T, int S, int CPS>
struct WaveEval {
    static constexpr bool kSpeculative = false;
    static constexpr bool kNodesInLds = false;
    const T* X;
    const uint8_t* y;
    int64_t N, nb;
    int D;
    double inv_s2, prior_const;

    __device__ bool s_writer() const { return true; }
    __device__ bool out_writer() const { return true; }
    __device__ bool aborted() const { return false; }

    __device__ void eval(const double (&q)[1], double& U, double (&g)[1])
    {
        double qv[CPS];
        spread_position<CPS, S>(q[0], qv);
        double acc[CPS];
#pragma unroll
        for (int c = 0; c < CPS; ++c) acc[c] = 0.0;
        double loss = 0.0;
        stream_blocks<T, CPS, S, false, false>(X, y, D, N, nb, 0, 1, qv, acc, loss);
        const double col = finish_pass<CPS, S>(acc, loss);
        const double prior = wave_sum(0.5 * q[0] * q[0] * inv_s2);
        U = loss + prior + prior_const;
        g[0] = (lane() < D) ? col + q[0] * inv_s2 : 0.0;
    }
};

// ---------------------------------------------------------------------------
// Grid path.

constexpr int kCmdEval = 1, kCmdExit = 2;

// The grid workers' stream: two block register sets and lane-masked loads of
// the last column slots for fp32 data; fp64 keeps one set (with two, its
// kernels spill registers in the stream).
template <typename T>
constexpr bool kGridPipe = sizeof(T) == 4;

// The grid workers load the first block of their share before the position
// arrives (fp32: 0.7 % faster per evaluation on the 581,012 x 55 set; fp64:
// 3 % slower, the held block costs registers beside the exchange code).
template <typename T>
constexpr bool kGridPrefetch = sizeof(T) == 4;

template <int DPL, int NW>
struct GridShared {
    static constexpr int W = 64 * (DPL + 1);  // partial_width(D)
    double qbuf[64 * DPL];
    union {
        double red[NW][W];                  // per-wave column sums of the group
        double red_flat[(NW - 1) * kWave];  // the gathered partials of the group's columns
    };
    int cmd;
    int gen;   // number of the current collective (counted by wave 0 from 1)
    int stop;  // number of the last collective wave 0 called off (0: none)
};

struct GridCtx {
    const void* X;
    const uint8_t* y;
    int64_t N, nb;
    int D;
    int groups;
    double* partials;  // [kGridPhases][D + 1][groups]
    double* result;    // [kGridPhases][kGridReplicas][kReplicaStride], W used of each row
    GridSync* sync;
};

// Cross-group exchange.  Everything that one group publishes for another
// (partials, results, the error flag) is written and read with agent-scope
// atomic accesses, which the L2 keeps coherent across the XCDs one access at
// a time.  A slot that carries a value holds kEmptySlot until the value is
// written, so a reader needs no separate flag: it waits for the slot itself.
// Ordering between accesses comes from waiting for the wave's outstanding
// memory operations (s_waitcnt) before the next one is issued.  No
// whole-cache write-back or invalidate (what a device-scope fence does) is
// needed: no ordinary store has to become visible to another group, and no
// ordinary load may observe another group's writes.
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

// The slot bit pattern meaning "not written yet" (a signalling NaN, which no
// arithmetic produces).
constexpr unsigned long long kEmptySlot = 0x7FF4DEADBEEF0001ull;

__device__ __forceinline__ unsigned long long slot_bits(const double* p)
{
    return __hip_atomic_load(reinterpret_cast<unsigned long long*>(const_cast<double*>(p)), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void empty_slot(double* p)
{
    __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), kEmptySlot, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool grid_error(const GridCtx& c)
{
    return __hip_atomic_load(&c.sync->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
}
__device__ __forceinline__ void raise_grid_error(const GridCtx& c)
{
    __hip_atomic_store(&c.sync->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// about 10 s of the 100 MHz constant clock: a wait that long means a broken
// invariant, and every group then gives up instead of hanging the device
constexpr uint64_t kGridWaitTicks = 1000000000ull;
// Waits look at the error flag (which another group raises when its own wait
// timed out) only after 20 us, and then every 16th poll: on the short waits
// of every step its loads would only queue beside the slot polls of every
// group at the one channel that holds the flag.
constexpr uint64_t kErrorPollTicks = 2000ull;

__device__ __forceinline__ bool error_poll_due(uint64_t waited, unsigned polls)
{
    return waited > kErrorPollTicks && (polls & 15u) == 0u;
}

// Wait until *p holds a value; false if the exchange failed meanwhile.
__device__ __forceinline__ bool wait_slot(const GridCtx& c, const double* p, double& v)
{
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    for (unsigned polls = 1;; ++polls) {
        const unsigned long long b = slot_bits(p);
        if (b != kEmptySlot) {
            v = __builtin_bit_cast(double, b);
            return true;
        }
        const uint64_t waited = __builtin_amdgcn_s_memrealtime() - t0;
        if (error_poll_due(waited, polls) && grid_error(c)) return false;
        if (waited > kGridWaitTicks) {
            raise_grid_error(c);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// A worker's share of the data blocks: first, first + stride, ... < nb.
// The last res.count of them sit in LDS for the whole launch; the others,
// those below nb_mem, stream from memory at every evaluation.  Every wave
// keeps at least one block in memory (the one it loads ahead of the
// position).
struct WaveShare {
    int64_t first, stride, nb_mem;
    ResidentBlocks res;
};

__device__ inline WaveShare grid_wave_share(int64_t nb, int groups, int wave, int resident, const char* res_base)
{
    WaveShare w;
    w.stride = (int64_t)groups * (kGridWaves - 1);
    w.first = (int64_t)blockIdx.x * (kGridWaves - 1) + (wave - 1);
    const int64_t count = w.first < nb ? (nb - 1 - w.first) / w.stride + 1 : 0;
    const int nres = count >= 2 ? (int)(count - 1 < resident ? count - 1 : resident) : 0;
    w.nb_mem = count > 0 ? w.first + (count - nres - 1) * w.stride + 1 : nb;
    w.res.base = res_base;
    w.res.count = nres;
    w.res.first_block = w.first + (count - nres) * w.stride;
    return w;
}

// Position of the loss in a result row: right after the D gradient columns
// when the row has room there (so that it shares their cache lines), else
// the first slot of the extra lane-row.
__device__ __forceinline__ int loss_pos(int D, int DPL) { return D < 64 * DPL ? D : 64 * DPL; }
// Position in a result row of used column ci (0..D-1, or D for the loss).
__device__ __forceinline__ int result_pos(int ci, int D, int DPL) { return ci < D ? ci : loss_pos(D, DPL); }

// One collective evaluation for the whole group, in two halves so that wave
// 0 (the controller) can work between them while the workers stream.
//
// grid_begin: wave 0 passes the position, the command and the collective's
// number; with kCmdEval every worker streams its blocks and leaves its column
// sums in LDS.  Returns the command (and, to the workers, the number).
//
// grid_end: wave 0 says whether the evaluation still counts.  If it called
// it off (a speculative next position the tree logic turned out not to
// need), the workers stop streaming at their next block and the whole group
// returns false from here: nothing is published and the step does not
// advance, identically in every group since every controller takes the same
// decisions.  Otherwise the group joins the grid-wide sum and wave 0 finds
// the full sums in out_r: component m of lane l is column l + 64 m, and
// component DPL of lane 0 is the loss.  Controller and workers execute the
// same workgroup barriers; the workers return as soon as their part is done.
// The numbers make the stop word unambiguous: wave 0 writes a collective's
// number into it before that collective's second barrier, and a worker
// compares it with the number it read after the first one.
//
// Step s uses phase s mod 3 of the buffers.  Each group stores its partial of
// every used column (the D gradient columns and the loss) into that column's
// row of group slots.  Group g owns the used columns g, g + G, ...: its
// workers wait for the G slots of each, empty them again, add them in a fixed
// order (lane l takes groups l, l + 64, ... in increasing order, then the
// lanes in butterfly order), store the column's result slot in every copy of
// the result row and empty the same slots of the previous phase.  The
// controller of group g waits for the result slots of its lanes in copy
// g mod kGridReplicas.  Emptying is safe: a group's partial of step s is written
// after its controller read all of step s - 1's results, and the next write
// of an emptied slot comes only after the worker that emptied it has waited
// for its own stores (s_waitcnt at its next step, before it stores the next
// result that every writer must first read).  A called-off collective writes
// and empties nothing, so the next one reuses its step.
template <typename T, int S, int CPS, int DPL, int NW, bool WORKER>
__device__ int grid_begin(const GridCtx& c, GridShared<DPL, NW>& sh, const double (&q)[DPL], int cmd_in,
                          int gen_in, int* gen_out, const WaveShare* share = nullptr,
                          const BlockRegs<T, CPS, S>* first_block = nullptr)
{
    const int l = lane();
    const int wave = threadIdx.x / kWave;
    if (wave == 0) {
#pragma unroll
        for (int m = 0; m < DPL; ++m) sh.qbuf[l + 64 * m] = q[m];
        if (l == 0) {
            sh.cmd = cmd_in;
            sh.gen = gen_in;
        }
    }
    __syncthreads();  // position, command and number published
    const int cmd = sh.cmd;
    *gen_out = sh.gen;
    if (cmd == kCmdExit) return cmd;
    if (WORKER) {
        const int D = c.D;
        double qv[CPS];
        spread_position_lds<CPS, S>(sh.qbuf, D, qv);
        double acc[CPS];
#pragma unroll
        for (int k = 0; k < CPS; ++k) acc[k] = 0.0;
        double loss = 0.0;
        const WaveShare& ws = *share;
        if constexpr (kGridPrefetch<T>)
            stream_blocks_from<T, CPS, S, kGridPipe<T>, kGridPipe<T>, true, true>(
                *first_block, (const T*)c.X, c.y, D, c.N, ws.nb_mem, ws.first, ws.stride, qv, acc, loss, &sh.stop,
                *gen_out, ws.res);
        else
            stream_blocks<T, CPS, S, kGridPipe<T>, kGridPipe<T>, true, true>((const T*)c.X, c.y, D, c.N, ws.nb_mem,
                                                                            ws.first, ws.stride, qv, acc, loss,
                                                                            &sh.stop, *gen_out, ws.res);
        if constexpr (S <= 8 && CPS == 8) {
            const double col = finish_pass<CPS, S>(acc, loss);
            if (l < D) sh.red[wave][l] = col;
            if (l == 0) sh.red[wave][64 * DPL] = loss;
        } else {
            finish_pass_to_row<CPS, S>(acc, loss, sh.red[wave], D, 64 * DPL);
        }
    }
    return cmd;
}

template <typename T, int S, int CPS, int DPL, int NW, bool WORKER>
__device__ bool grid_end(const GridCtx& c, GridShared<DPL, NW>& sh, unsigned long long step, int gen, bool stop,
                         double (&out_r)[DPL + 1], bool* aborted)
{
    static_assert(GridShared<DPL, NW>::W <= kReplicaStride, "a result row fits its copy");
    const int l = lane();
    const int wave = threadIdx.x / kWave;
    if (!WORKER && stop && l == 0)
        __hip_atomic_store(&sh.stop, gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __syncthreads();  // per-worker sums in LDS, or the pass called off
    if (__hip_atomic_load(&sh.stop, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) == gen) return false;

    const int ph = (int)(step % kGridPhases);
    const int D = c.D;
    const int used = D + 1;
    const int G = c.groups;
    const int g = blockIdx.x;
    double* part = c.partials + (int64_t)ph * used * G;

    if (WORKER && wave == 1) {
        // the group's partial of each used column, workers in wave order
#pragma unroll
        for (int m = 0; m <= DPL; ++m) {
            const int colw = l + 64 * m;
            const int ci = m < DPL ? colw : (l == 0 ? D : -1);
            if (ci >= 0 && (m == DPL || colw < D)) {
                double s = 0.0;
#pragma unroll
                for (int w = 1; w < NW; ++w) s += sh.red[w][colw];
                store_shared(&part[(int64_t)ci * G + g], s);
            }
        }
    }

    const int mine = g < used ? (used - 1 - g) / G + 1 : 0;  // used columns this group owns
    if (mine > 0) {                                           // uniform over the group
        __syncthreads();  // the per-worker sums are consumed
        if (WORKER) {
            drain_memory_ops();  // this lane's emptying stores of earlier steps have landed
            bool ok = true;
            for (int i = (wave - 1) * kWave + l; i < mine * G; i += (NW - 1) * kWave) {
                const int jc = i / G;
                const int src = i - jc * G;
                double* slot = &part[(int64_t)(g + jc * G) * G + src];
                double v = 0.0;
                if (ok) ok = wait_slot(c, slot, v);
                sh.red_flat[i] = v;
                empty_slot(slot);
            }
        }
        __syncthreads();  // the group's columns gathered
        if (WORKER) {
            for (int jc = wave - 1; jc < mine; jc += NW - 1) {
                const int ci = g + jc * G;
                double s = 0.0;
                for (int t = l; t < G; t += kWave) s += sh.red_flat[jc * G + t];
                s = wave_sum(s);  // the same bits in every lane
                if (l < kGridReplicas) {
                    const int pos = result_pos(ci, D, DPL);
                    const int prev = (ph + kGridPhases - 1) % kGridPhases;
                    store_shared(&c.result[(ph * kGridReplicas + l) * kReplicaStride + pos], s);
                    empty_slot(&c.result[(prev * kGridReplicas + l) * kReplicaStride + pos]);
                }
            }
        }
    }
    if (WORKER) return true;

    // controller: wait for this lane's result slots, all at once
    const double* row = &c.result[(ph * kGridReplicas + g % kGridReplicas) * kReplicaStride];
    const int lp = loss_pos(D, DPL);
    unsigned long long bits[DPL + 1];
#pragma unroll
    for (int m = 0; m <= DPL; ++m) {
        const int pos = l + 64 * m;
        const bool used_slot = pos < D || pos == lp;
        bits[m] = used_slot ? kEmptySlot : 0ull;  // 0ull: +0.0, nothing to wait for
    }
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    bool bad = false;
    for (unsigned polls = 1;; ++polls) {
#pragma unroll
        for (int m = 0; m <= DPL; ++m)
            if (bits[m] == kEmptySlot) bits[m] = slot_bits(row + l + 64 * m);
        bool ready = true;
#pragma unroll
        for (int m = 0; m <= DPL; ++m) ready = ready && bits[m] != kEmptySlot;
        if (__all(ready)) break;
        const uint64_t waited = __builtin_amdgcn_s_memrealtime() - t0;
        if (error_poll_due(waited, polls) && grid_error(c)) {
            bad = true;
            break;
        }
        if (waited > kGridWaitTicks) {
            if (l == 0) raise_grid_error(c);
            bad = true;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    *aborted = bad;
#pragma unroll
    for (int m = 0; m <= DPL; ++m) out_r[m] = bad ? 0.0 : __builtin_bit_cast(double, bits[m]);
    return true;
}

// The grid path's evaluator.  Besides eval(), it can start an evaluation
// (begin) and collect it later (end), so that run_chain hands the workers the
// next leapfrog position before it does the tree logic of the current leaf;
// cancel() calls a started evaluation off.
template <typename T, int S, int CPS, int DPL, int NW>
struct GridEval {
    static constexpr bool kSpeculative = true;
    static constexpr bool kNodesInLds = DPL >= 3;  // the edge and proposal nodes in LDS (see EdgeNodes)
    GridCtx c;
    GridShared<DPL, NW>* sh;
    double inv_s2, prior_const;
    unsigned long long step;
    int gen;
    bool abort;

    __device__ bool s_writer() const { return true; }  // only the controller runs the chain
    __device__ bool out_writer() const { return blockIdx.x == 0; }
    __device__ bool aborted() const { return abort; }

    // A called-off collective's second barrier, which the workers wait at
    // once they have stopped: the controller takes it at its next command
    // (it finishes the iteration meanwhile), never before the workers could
    // read the stop word.
    bool owed = false;

    __device__ void pay_barrier()
    {
        if (owed) {
            __syncthreads();
            owed = false;
        }
    }

    __device__ void begin(const double (&q)[DPL])
    {
        pay_barrier();
        int gn;
        grid_begin<T, S, CPS, DPL, NW, false>(c, *sh, q, kCmdEval, ++gen, &gn);
    }

    // U and grad U of the started evaluation, at the position q it was
    // started with
    __device__ void end(const double (&q)[DPL], double& U, double (&g)[DPL])
    {
        double r[DPL + 1];
        bool ab = false;
        grid_end<T, S, CPS, DPL, NW, false>(c, *sh, step, gen, false, r, &ab);
        abort = ab;
        step++;
        double pr = 0.0;
#pragma unroll
        for (int m = 0; m < DPL; ++m) pr += 0.5 * q[m] * q[m] * inv_s2;
        const double prior = wave_sum(pr);
        const int lp = loss_pos(c.D, DPL);
        double loss = r[DPL];
#pragma unroll
        for (int m = 0; m < DPL; ++m)
            if (m == lp / 64) loss = r[m];
        U = readlane_f64(loss, lp % 64) + prior + prior_const;
        const int l = lane();
#pragma unroll
        for (int m = 0; m < DPL; ++m) g[m] = (l + 64 * m < c.D) ? r[m] + q[m] * inv_s2 : 0.0;
    }

    __device__ void cancel()
    {
        // the stop word, as grid_end stores it for a called-off collective;
        // the barrier after it is taken at the next command
        if (lane() == 0) __hip_atomic_store(&sh->stop, gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        owed = true;
    }

    __device__ void eval(const double (&q)[DPL], double& U, double (&g)[DPL])
    {
        begin(q);
        end(q, U, g);
    }

    __device__ void finish()
    {
        pay_barrier();
        double q[DPL];
#pragma unroll
        for (int m = 0; m < DPL; ++m) q[m] = 0.0;
        int gn;
        grid_begin<T, S, CPS, DPL, NW, false>(c, *sh, q, kCmdExit, ++gen, &gn);
    }
};

template <int DPL>
__device__ __forceinline__ void copy_node(Node<DPL>& dst, const Node<DPL>& src)
{
    dst = src;
}

// ---------------------------------------------------------------------------
// Warmup adaptation of the step size (Hoffman & Gelman 2014: Alg. 4 to start,
// dual averaging of Section 3.2 per warmup iteration) and the windowed
// diagonal mass that goes with it.  Scalars are wave-uniform; every lane (and
// every controller of the grid path) computes the same bits.

constexpr double kLn2 = 0.69314718055994530942;
constexpr int kStepTrials = 100;
constexpr double kDaGamma = 0.05, kDaT0 = 10.0, kDaKappa = 0.75;

struct DualAvg {
    double mu, hbar, log_eps, log_eps_bar;
    int64_t m;

    __device__ void start(double eps)
    {
        mu = log(10.0 * eps);
        hbar = 0.0;
        log_eps = log(eps);
        log_eps_bar = 0.0;
        m = 0;
    }
    // One update with accept statistic alpha; returns the next step size.
    __device__ double update(double alpha, double delta)
    {
#pragma clang fp contract(off)
        m += 1;
        const double mm = (double)m;
        const double w = 1.0 / (mm + kDaT0);
        hbar = (1.0 - w) * hbar + w * (delta - alpha);
        log_eps = mu - (sqrt(mm) / kDaGamma) * hbar;
        const double eta = pow(mm, -kDaKappa);
        log_eps_bar = eta * log_eps + (1.0 - eta) * log_eps_bar;
        return exp(log_eps);
    }
};

// log of the density kept by one leapfrog step of size e from (cur.q, r):
// H0 - H', or -inf when H' is not a number.
template <int DPL, class Eval>
__device__ double step_log_ratio(Eval& ev, const Node<DPL>& cur, const double (&r)[DPL], double e,
                                 const double (&im)[DPL], double H0)
{
    Node<DPL> z = cur;
    double ph[DPL];
#pragma unroll
    for (int m = 0; m < DPL; ++m) {
        ph[m] = r[m] - 0.5 * e * z.g[m];
        z.q[m] = z.q[m] + e * im[m] * ph[m];
    }
    ev.eval(z.q, z.U, z.g);
    double k2 = 0.0;
#pragma unroll
    for (int m = 0; m < DPL; ++m) {
        z.p[m] = ph[m] - 0.5 * e * z.g[m];
        k2 += im[m] * z.p[m] * z.p[m];
    }
    const double d = H0 - (z.U + 0.5 * wave_sum(k2));
    return d == d ? d : -INFINITY;
}

// Alg. 4: from eps, double (the step keeps more than half the density) or
// halve (it does not) until that flips; the momentum is drawn under
// kTagStepSize at counter t.  Adds the gradient evaluations to *evals.
template <int DPL, class Eval>
__device__ double find_step_size(Eval& ev, const Node<DPL>& cur, double eps, const double (&im)[DPL],
                                 const bool (&act)[DPL], uint64_t seed, uint64_t chain, uint64_t t,
                                 unsigned long long* evals)
{
    const int l = lane();
    double r[DPL], kin = 0.0;
#pragma unroll
    for (int m = 0; m < DPL; ++m) {
        const double xi = act[m] ? momentum_normal(seed, chain, t, l + 64 * m, kTagStepSize) : 0.0;
        r[m] = act[m] ? xi / sqrt(im[m]) : 0.0;
        kin += im[m] * r[m] * r[m];
    }
    const double H0 = cur.U + 0.5 * wave_sum(kin);
    double d = step_log_ratio<DPL>(ev, cur, r, eps, im, H0);
    *evals += 1;
    const double a = d > -kLn2 ? 1.0 : -1.0;
    for (int k = 0; k < kStepTrials && a * (d + kLn2) > 0.0 && !ev.aborted(); ++k) {
        eps = a > 0.0 ? eps * 2.0 : eps * 0.5;
        d = step_log_ratio<DPL>(ev, cur, r, eps, im, H0);
        *evals += 1;
    }
    return eps;
}

// The slow windows of the windowed mass adaptation for W warmup iterations:
// an initial buffer, windows of base, 2 base, ... iterations, the last one
// stretched to the terminal buffer when a doubled window after it would not
// fit.  next() moves to the following window.
struct MassWindows {
    int64_t start, end, size, slow_end;
    bool any;

    __device__ void init(int64_t W)
    {
        int64_t init = 75, term = 50, base = 25;
        if (init + term + base > W) {
            init = (int64_t)(0.15 * (double)W);
            term = (int64_t)(0.10 * (double)W);
            base = W - (init + term);
        }
        any = W >= 20;
        slow_end = W - term;
        start = init;
        size = base;
        end = stretch(start + size);
    }
    __device__ int64_t stretch(int64_t e) const { return e + 2 * size > slow_end ? slow_end : e; }
    __device__ void next()
    {
        start = end;
        size *= 2;
        end = stretch(start + size);
        any = start < slow_end;
    }
};

// First half of a leapfrog step from (q, p, grad U = g) with step h: the
// half-kicked momentum ph and the drifted position q_out (which may alias
// q).  Contraction is off, so every call site rounds alike: the grid path
// computes a position once to start its evaluation and again when it takes
// the results, and both must give the same bits.
template <int DPL>
__device__ __forceinline__ void leapfrog_drift(const double (&q)[DPL], const double (&p)[DPL],
                                               const double (&g)[DPL], double h, const double (&im)[DPL],
                                               double (&ph)[DPL], double (&q_out)[DPL])
{
#pragma clang fp contract(off)
#pragma unroll
    for (int m = 0; m < DPL; ++m) {
        ph[m] = p[m] - 0.5 * h * g[m];
        q_out[m] = q[m] + h * im[m] * ph[m];
    }
}

// The whole chain: init, warmup + sampling iterations, outputs.  S_arr points
// to this chain's checkpoint array in LDS: [max(max_depth, 1)][2][D].
// EXT = false compiles the optional features out (warmup adaptation of the
// step size, the generalised U-turn criterion): the kernels without them keep
// their registers for the tree and the data pass.
template <int DPL, bool EXT, class Eval>
__device__ void run_chain(const SamplerArgs& A, Eval& ev, int64_t chain, double* S_arr)
{
    const int l = lane();
    const int D = A.data.D;
    bool act[DPL];
#pragma unroll
    for (int m = 0; m < DPL; ++m) act[m] = l + 64 * m < D;
    // every dimension in the first 16 lanes: the tree's sums take one row
    const bool one_row = uni(D <= 16);
    const int maxd = A.max_depth;
    double eps = A.step_size;
    const uint64_t seed = A.seed;
    const int64_t cidx = A.chain_offset + chain;
    const uint64_t key_chain = (uint64_t)cidx;
    const bool out = ev.out_writer();
    const bool s_out = ev.s_writer();

    double im[DPL];
#pragma unroll
    for (int m = 0; m < DPL; ++m) im[m] = (act[m] && A.inv_mass) ? A.inv_mass[l + 64 * m] : 1.0;

    Node<DPL> cur;
#pragma unroll
    for (int m = 0; m < DPL; ++m) {
        cur.q[m] = (act[m] && A.init_q) ? A.init_q[cidx * D + l + 64 * m] : 0.0;
        cur.p[m] = 0.0;
    }
    ev.eval(cur.q, cur.U, cur.g);
    unsigned long long evals = 1;

    double wmean[DPL], wm2[DPL];
#pragma unroll
    for (int m = 0; m < DPL; ++m) wmean[m] = wm2[m] = 0.0;
    int64_t wn = 0;
    const int64_t iters = A.num_warmup + A.num_samples;

    // warmup adaptation of the step size, with windowed mass if asked
    const bool adapt = EXT && A.adapt_step && A.num_warmup > 0;
    // generalised criterion: the slots of S hold (momentum sum of the subtree
    // before the leaf, the leaf's momentum) instead of (q, p)
    const bool gen = EXT && A.uturn_gen;
    // merge-structured subtree proposals: the waiting block of each level
    // sits after S (proposal q, p, grad U per level, then per level the
    // log-weight, offset and U)
    const bool smerge = EXT && A.sub_merge;
    double* stk = S_arr + (int64_t)(maxd > 1 ? maxd : 1) * 2 * D;
    double* stk_sc = stk + (int64_t)merge_levels(maxd) * 3 * D;
    EdgeNodes<DPL, Eval::kNodesInLds> nodes;
    nodes.bind(S_arr + chain_lds_doubles(D, maxd, smerge ? 1 : 0, false));
    DualAvg da;
    MassWindows win;
    win.any = false;
    if (adapt) {
        eps = find_step_size<DPL>(ev, cur, eps, im, act, seed, key_chain, (uint64_t)A.first_iter, &evals);
        da.start(eps);
        if (A.adapt_diag) win.init(A.num_warmup);
    }

    // An iteration's draws: the momentum's standard normals (component l +
    // 64 m in lane l) and tree block l (kTagTree): the direction bit and the
    // merge uniform of doubling l, the uniforms of the iteration's leaves 2l
    // and 2l + 1.  None depends on the chain's state, so with a speculative
    // evaluator the next iteration's are drawn while the first leaf of this
    // one is evaluated, off the path between iterations.
    struct IterDraws {
        double xi[DPL];
        int dir_bit;
        double u_merge;
        double u_leaf_a, u_leaf_b;
    };
    const auto draw_iteration = [&](uint64_t t, IterDraws& dr) {
#pragma unroll
        for (int m = 0; m < DPL; ++m) dr.xi[m] = act[m] ? momentum_normal(seed, key_chain, t, l + 64 * m) : 0.0;
        const Block4 b = draw(seed, key_chain, t, kTagTree, 0, (uint64_t)l);
        dr.dir_bit = l < maxd ? (int)(b.w0 & 1ull) : 0;
        dr.u_merge = l < maxd ? unit53(b.w1) : 0.0;
        dr.u_leaf_a = unit53(b.w2);
        dr.u_leaf_b = unit53(b.w3);
    };
    IterDraws next_draws;
    bool have_next = false;

    for (int64_t k = 0; k < iters && !ev.aborted(); ++k) {
        const uint64_t t = (uint64_t)(A.first_iter + k);
        IterDraws dr;
        if (Eval::kSpeculative && have_next) dr = next_draws;
        else draw_iteration(t, dr);
        have_next = false;

        // momentum and initial energy
        double kin = 0.0;
#pragma unroll
        for (int m = 0; m < DPL; ++m) {
            cur.p[m] = act[m] ? dr.xi[m] / sqrt(im[m]) : 0.0;
            kin += im[m] * cur.p[m] * cur.p[m];
        }
        const double H0 = cur.U + 0.5 * wave_sum_rows(kin, one_row);
        double rho_traj[DPL];  // momentum sum over the trajectory's points
#pragma unroll
        for (int m = 0; m < DPL; ++m) rho_traj[m] = cur.p[m];

        const double u_merge = dr.u_merge;
        const uint64_t dirmask = __ballot(dr.dir_bit);
        // uniforms of the leaves 128 c .. 128 c + 127 (c = leaf_chunk): lane l
        // holds those of leaves 128 c + 2 l and 128 c + 2 l + 1
        double u_la = dr.u_leaf_a, u_lb = dr.u_leaf_b;
        int64_t leaf_chunk = 0;

        nodes.reset(cur);
        // a speculative evaluation: the next leapfrog position, handed to the
        // evaluator before the bookkeeping of the current leaf decides
        // whether the trajectory goes on (evaluators that can start one)
        bool pend = false;
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
            Node<DPL> z = nodes.edge(v > 0);
            const int64_t e = v > 0 ? Rpos : Lpos;
            const double h = v * eps;
            double logw = -INFINITY;
            nodes.set_sprop(z);
            int64_t sprop_idx = 0;
            int status = kTreeOk;
            depth = j + 1;
            const int64_t nleaf = 1ll << j;
            double u_sm = 0.0;    // merge-structured: uniforms of merges [msub & ~63, + 64)
            int64_t msub = 0;     // merges completed in this subtree
            double rsum[DPL];  // momentum sum over the subtree's leaves so far
#pragma unroll
            for (int m = 0; m < DPL; ++m) rsum[m] = 0.0;

            for (int64_t n = 0; n < nleaf; ++n) {
                const int64_t gleaf = nleaf - 1 + n;  // the leaf's number in the iteration
                if (!smerge && uni((gleaf >> 7) != leaf_chunk)) {
                    leaf_chunk = gleaf >> 7;
                    const Block4 b = draw(seed, key_chain, t, kTagTree, 0, (uint64_t)(leaf_chunk * 64 + l));
                    u_la = unit53(b.w2);
                    u_lb = unit53(b.w3);
                }
                // leapfrog: half kick, drift, gradient, half kick
                double ph[DPL];
                if constexpr (Eval::kSpeculative) {
                    // the same bits the speculative start computed from
                    // this node (or the edge it was started from)
                    leapfrog_drift<DPL>(z.q, z.p, z.g, h, im, ph, z.q);
                    if (!pend) ev.begin(z.q);
                    pend = false;
                    if (nleaves == 0 && k + 1 < iters) {
                        draw_iteration(t + 1, next_draws);  // while the first leaf streams
                        have_next = true;
                    }
                    ev.end(z.q, z.U, z.g);
                } else {
#pragma unroll
                    for (int m = 0; m < DPL; ++m) {
                        ph[m] = z.p[m] - 0.5 * h * z.g[m];
                        z.q[m] = z.q[m] + h * im[m] * ph[m];
                    }
                    ev.eval(z.q, z.U, z.g);
                }
                if (ev.aborted()) break;
                double k2 = 0.0;
#pragma unroll
                for (int m = 0; m < DPL; ++m) {
                    z.p[m] = ph[m] - 0.5 * h * z.g[m];
                    k2 += im[m] * z.p[m] * z.p[m];
                }
                ++nleaves;
                if constexpr (Eval::kSpeculative) {
                    // Start the next evaluation now, so that the workers
                    // stream while the bookkeeping below runs: the next leaf
                    // of this subtree, or else the first leaf of the next
                    // doubling from the trajectory edge it starts at (this
                    // leaf, once merged, if it goes the same way).  If the
                    // bookkeeping ends the trajectory it is called off.
                    const bool more = n + 1 < nleaf;
                    if (more || j + 1 < maxd) {
                        const int vn = more ? v : (((dirmask >> (j + 1)) & 1ull) ? 1 : -1);
                        const bool from_z = more || vn == v;
                        const double hn = vn * eps;
                        double bq[DPL], bp[DPL], bg[DPL], nph[DPL], nq[DPL];
#pragma unroll
                        for (int m = 0; m < DPL; ++m) {
                            bq[m] = from_z ? z.q[m] : nodes.edge_q(vn > 0, m);
                            bp[m] = from_z ? z.p[m] : nodes.edge_p(vn > 0, m);
                            bg[m] = from_z ? z.g[m] : nodes.edge_g(vn > 0, m);
                        }
                        leapfrog_drift<DPL>(bq, bp, bg, hn, im, nph, nq);
                        ev.begin(nq);
                        pend = true;
                    }
                }
                if (gen) {
#pragma unroll
                    for (int m = 0; m < DPL; ++m) rsum[m] += z.p[m];
                }

                const double dH = (z.U + 0.5 * wave_sum_rows(k2, one_row)) - H0;
                if (dH == dH) sum_acc += dH > 0.0 ? exp_nonpos(-dH) : 1.0;
                if (uni(!(dH <= 1000.0))) {
                    status = kTreeDivergent;
                    term = (int)n;
                    break;
                }
                const double lam = -dH;
                if (smerge) {
                    // the leaf is a block of one; every completed pair of
                    // equal blocks merges, keeping the later block's proposal
                    // with probability its share of the weight (the merges'
                    // uniforms are keyed by their ordinal in completion
                    // order, drawn 64 at a time)
                    const int nm = __builtin_ctzll(~(unsigned long long)n);
                    Node<DPL> cp = z;
                    double clw = lam;
                    int64_t cix = e + v * (n + 1);
                    for (int k2 = 0; k2 < nm; ++k2) {
                        if ((msub & (kWave - 1)) == 0)
                            u_sm = (msub + l < nleaf - 1)
                                       ? unit53(draw(seed, key_chain, t, kTagSubMerge, (uint64_t)j,
                                                     (uint64_t)(msub + l)).w0)
                                       : 0.0;
                        const double um = readlane_f64(u_sm, (int)(msub & (kWave - 1)));
                        ++msub;
                        const double* lv = stk + (int64_t)k2 * 3 * D;
                        const double* sc = stk_sc + 3 * k2;
                        double share;  // the later block's share of the weight
                        const double lw = logaddexp_share(sc[0], clw, share);
                        if (!uni(um < share)) {
#pragma unroll
                            for (int m = 0; m < DPL; ++m) {
                                cp.q[m] = act[m] ? lv[l + 64 * m] : 0.0;
                                cp.p[m] = act[m] ? lv[D + l + 64 * m] : 0.0;
                                cp.g[m] = act[m] ? lv[2 * D + l + 64 * m] : 0.0;
                            }
                            cp.U = sc[2];
                            cix = (int64_t)sc[1];
                        }
                        clw = lw;
                    }
                    if (n + 1 < nleaf) {
                        if (s_out) {
                            double* lv = stk + (int64_t)nm * 3 * D;
#pragma unroll
                            for (int m = 0; m < DPL; ++m) {
                                if (act[m]) {
                                    lv[l + 64 * m] = cp.q[m];
                                    lv[D + l + 64 * m] = cp.p[m];
                                    lv[2 * D + l + 64 * m] = cp.g[m];
                                }
                            }
                            if (l == 0) {
                                stk_sc[3 * nm] = clw;
                                stk_sc[3 * nm + 1] = (double)cix;
                                stk_sc[3 * nm + 2] = cp.U;
                            }
                        }
                    } else {
                        nodes.set_sprop(cp);
                        sprop_idx = cix;
                        logw = clw;
                    }
                } else {
                    // streaming multinomial choice inside the subtree
                    double share;  // the leaf's share of the subtree's weight
                    const double lw = logaddexp_share(logw, lam, share);
                    const int gi = (int)(gleaf & 127);
                    const double u = readlane_f64((gi & 1) ? u_lb : u_la, gi >> 1);
                    if (uni(u < share)) {
                        nodes.set_sprop(z);
                        sprop_idx = e + v * (n + 1);
                    }
                    logw = lw;
                }

                if ((n & 1) == 0) {
                    // even leaf: checkpoint into S[BitCount(n)]
                    const int i = __popcll((unsigned long long)n);
                    if (s_out) {
#pragma unroll
                        for (int m = 0; m < DPL; ++m) {
                            if (act[m]) {
                                S_arr[(2 * i) * D + l + 64 * m] = gen ? rsum[m] - z.p[m] : z.q[m];
                                S_arr[(2 * i + 1) * D + l + 64 * m] = z.p[m];
                            }
                        }
                    }
                } else {
                    // odd leaf: test the subtrees that end here, smallest first
                    const int nl = __builtin_ctzll(~(unsigned long long)n);
                    const int imax = __popcll((unsigned long long)(n - 1));
                    const int imin = imax - nl + 1;
                    bool turned = false;
                    for (int kk = imax; kk >= imin; --kk) {
                        double sq[DPL], sp[DPL];
#pragma unroll
                        for (int m = 0; m < DPL; ++m) {
                            sq[m] = act[m] ? S_arr[(2 * kk) * D + l + 64 * m] : 0.0;
                            sp[m] = act[m] ? S_arr[(2 * kk + 1) * D + l + 64 * m] : 0.0;
                        }
                        bool t_;
                        if (gen) {
                            double rho[DPL];
#pragma unroll
                            for (int m = 0; m < DPL; ++m) rho[m] = rsum[m] - sq[m];
                            t_ = is_uturn_gen<DPL>(rho, sp, z.p, im, one_row);
                        } else {
                            t_ = is_uturn<DPL>(sq, sp, z.q, z.p, v, im, one_row);
                        }
                        if (t_) {
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
            const double um = readlane_f64(u_merge, j);
            const double dw = logw - logw_traj;
            if (uni(um < (dw >= 0.0 ? 1.0 : exp_nonpos(dw)))) {
                nodes.accept_sprop();
                prop_idx = sprop_idx;
            }
            logw_traj = logaddexp(logw_traj, logw);
            nodes.set_edge(v > 0, z);
            if (v > 0) Rpos += nleaf;
            else Lpos -= nleaf;
            if (gen) {
#pragma unroll
                for (int m = 0; m < DPL; ++m) rho_traj[m] += rsum[m];
            }
            bool traj_turn;
            if constexpr (Eval::kNodesInLds) {
                // the edge just extended is z, the other one is read back; the
                // pair (other, z) is the trajectory's ends in the order of a
                // subtree built in direction v, which is_uturn puts in time
                // order element by element (is_uturn_gen is symmetric in its
                // ends).  (References chosen between the two nodes at run
                // time put both in scratch memory.)
                const Node<DPL> other = nodes.edge(v < 0);
                traj_turn = gen ? is_uturn_gen<DPL>(rho_traj, other.p, z.p, im, one_row)
                                : is_uturn<DPL>(other.q, other.p, z.q, z.p, v, im, one_row);
            } else {
                traj_turn = gen ? is_uturn_gen<DPL>(rho_traj, nodes.left.p, nodes.right.p, im, one_row)
                                : is_uturn<DPL>(nodes.left.q, nodes.left.p, nodes.right.q, nodes.right.p, 1, im,
                                                one_row);
            }
            if (traj_turn) {
                turning = 1;
                term = -2;
                break;
            }
            if (j == maxd - 1) maxhit = 1;
        }
        if constexpr (Eval::kSpeculative) {
            if (pend) ev.cancel();  // the trajectory ended before that position
        }
        evals += (unsigned long long)nleaves;
        cur = nodes.get_prop();

        if (adapt && k < A.num_warmup) {
            const double alpha = nleaves > 0 ? sum_acc / (double)nleaves : 0.0;
            eps = da.update(alpha, A.target_accept);
            if (win.any && k >= win.start && k < win.end) {
                ++wn;
#pragma unroll
                for (int m = 0; m < DPL; ++m) {
                    const double d1 = cur.q[m] - wmean[m];
                    wmean[m] += d1 / (double)wn;
                    wm2[m] += d1 * (cur.q[m] - wmean[m]);
                }
            }
            if (win.any && k == win.end - 1) {
                if (wn >= 2) {
                    const double nn = (double)wn;
#pragma unroll
                    for (int m = 0; m < DPL; ++m)
                        im[m] = act[m] ? (nn / (nn + 5.0)) * (wm2[m] / (nn - 1.0)) + 1e-3 * (5.0 / (nn + 5.0))
                                       : 1.0;
                }
                wn = 0;
#pragma unroll
                for (int m = 0; m < DPL; ++m) wmean[m] = wm2[m] = 0.0;
                win.next();
                eps = find_step_size<DPL>(ev, cur, eps, im, act, seed, key_chain,
                                          (uint64_t)(A.first_iter + k + 1), &evals);
                da.start(eps);
            }
            if (k == A.num_warmup - 1) eps = exp(da.log_eps_bar);
        }

        // diagonal inverse mass from warmup states in [W/2, W)
        if (!adapt && A.adapt_diag && k < A.num_warmup && k >= A.num_warmup / 2) {
            ++wn;
#pragma unroll
            for (int m = 0; m < DPL; ++m) {
                const double d1 = cur.q[m] - wmean[m];
                wmean[m] += d1 / (double)wn;
                wm2[m] += d1 * (cur.q[m] - wmean[m]);
            }
        }
        if (!adapt && A.adapt_diag && k == A.num_warmup - 1 && wn >= 2) {
            const double nn = (double)wn;
            double var[DPL], tot = 0.0;
#pragma unroll
            for (int m = 0; m < DPL; ++m) {
                var[m] = (nn / (nn + 5.0)) * (wm2[m] / (nn - 1.0)) + 1e-3 * (5.0 / (nn + 5.0));
                var[m] = act[m] ? var[m] : 0.0;
                tot += var[m];
            }
            const double mean = wave_sum(tot) / (double)D;
#pragma unroll
            for (int m = 0; m < DPL; ++m) im[m] = act[m] ? var[m] / mean : 1.0;
        }

        if (k >= A.num_warmup && out) {
            const int64_t s = k - A.num_warmup;
            if (A.out_samples) {
#pragma unroll
                for (int m = 0; m < DPL; ++m)
                    if (act[m]) A.out_samples[(cidx * A.num_samples + s) * D + l + 64 * m] = cur.q[m];
            }
            if (A.out_stats) {
                double kk2 = 0.0;
#pragma unroll
                for (int m = 0; m < DPL; ++m) kk2 += im[m] * cur.p[m] * cur.p[m];
                const double K = 0.5 * wave_sum(kk2);
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
#pragma unroll
        for (int m = 0; m < DPL; ++m) {
            if (act[m] && A.out_final_q) A.out_final_q[cidx * D + l + 64 * m] = cur.q[m];
            if (act[m] && A.out_inv_mass) A.out_inv_mass[cidx * D + l + 64 * m] = im[m];
        }
        if (l == 0) A.grad_evals[cidx] = evals;
        if (l == 0 && A.out_step_size) A.out_step_size[cidx] = eps;
    }
}

constexpr int kWaveChainsPerGroup = 4;
// LDS a workgroup may use on gfx950.
constexpr size_t kMaxGroupLds = 160 * 1024;

// LDS bytes of one group of the wave path with `cpg` chains: their
// checkpoint arrays and, when RESIDENT, their data sets (column blocks back
// to back, then a zero pad for the last chain's over-read, then the labels).
template <typename T, int S, int CPS>
struct WaveLds {
    static constexpr int R = BlockShape<T, S>::R;
    __host__ __device__ static size_t s_bytes(int D, int max_depth, int sub_merge, int cpg)
    {
        return (size_t)cpg * chain_lds_doubles(D, max_depth, sub_merge, false) * sizeof(double);
    }
    __host__ __device__ static int64_t x_elems(int D, int64_t nb) { return nb * D * R; }
    __host__ __device__ static int64_t pad_elems(int D) { return (int64_t)(CPS * S - D) * R; }
    static size_t bytes(int D, int64_t nb, int max_depth, int sub_merge, bool resident, int cpg)
    {
        size_t b = s_bytes(D, max_depth, sub_merge, cpg);
        if (resident)
            b += (size_t)(cpg * x_elems(D, nb) + pad_elems(D)) * sizeof(T) + (size_t)cpg * nb * R;
        return b;
    }
};

// One wavefront per chain, `cpg` chains (waves) per group.  RESIDENT: the
// group first copies its chains' data sets into LDS (one barrier) and every
// gradient evaluation then streams from LDS; a group is then one per CU, so
// the register budget is the whole wave's share of the SIMD.
template <typename T, int S, int CPS, bool RESIDENT, bool EXT>
__global__ void __launch_bounds__(kWaveChainsPerGroup * kWave, RESIDENT ? 1 : 3) sampler_wave_kernel(SamplerArgs A,
                                                                                                   int cpg)
{
    using G = WaveLds<T, S, CPS>;
    constexpr int R = G::R;
    extern __shared__ double lds[];
    const int wave = threadIdx.x / kWave;
    const bool idle = wave >= cpg;  // a group of fewer than four chains
    if (!RESIDENT && idle) return;   // (no group barrier on this variant)
    const int l = lane();
    const int64_t chain = (int64_t)blockIdx.x * cpg + wave;
    const int D = A.data.D;
    const int64_t nb = A.data.nb;
    double* S_arr = lds + (int64_t)wave * chain_lds_doubles(D, A.max_depth, EXT ? A.sub_merge : 0, false);
    const int64_t c = A.chain_offset + chain;
    const int64_t ds = A.per_chain_data ? c : 0;
    const T* Xg = (const T*)A.data.X + ds * nb * (int64_t)D * R;
    const uint8_t* yg = A.data.y + ds * nb * R;
    WaveEval<T, S, CPS> ev;
    if constexpr (RESIDENT) {
        const int64_t xe = G::x_elems(D, nb);
        T* Xl = reinterpret_cast<T*>(reinterpret_cast<char*>(lds) + G::s_bytes(D, A.max_depth, EXT ? A.sub_merge : 0, cpg));
        T* Xw = Xl + wave * xe;
        uint8_t* yl = reinterpret_cast<uint8_t*>(Xl + cpg * xe + G::pad_elems(D));
        uint8_t* yw = yl + wave * nb * R;
        // 16-byte pieces: a chain's X is nb * D * R * sizeof(T) bytes, a
        // multiple of 16 since R * sizeof(T) is 512 / S or 1024 and S <= 8
        const int64_t n16 = xe * (int64_t)sizeof(T) / 16;
        uint4* dst = reinterpret_cast<uint4*>(Xw);
        if (idle) {
            // an idle wave only takes part in the barrier below
        } else if (chain < A.num_chains) {
            const uint4* src = reinterpret_cast<const uint4*>(Xg);
            for (int64_t i = l; i < n16; i += kWave) dst[i] = src[i];
            const int64_t n8 = nb * R / 8;
            for (int64_t i = l; i < n8; i += kWave)
                reinterpret_cast<uint2*>(yw)[i] = reinterpret_cast<const uint2*>(yg)[i];
        } else {
            // a neighbour's last block over-reads into this region: zeros
            for (int64_t i = l; i < n16; i += kWave) dst[i] = uint4{0u, 0u, 0u, 0u};
        }
        if (!idle && wave == cpg - 1) {
            T* pad = Xl + cpg * xe;
            for (int64_t i = l; i < G::pad_elems(D); i += kWave) pad[i] = T(0);
        }
        __syncthreads();
        if (idle || chain >= A.num_chains) return;
        ev.X = Xw;
        ev.y = yw;
    } else {
        if (chain >= A.num_chains) return;
        ev.X = Xg;
        ev.y = yg;
    }
    ev.N = A.data.N;
    ev.nb = nb;
    ev.D = D;
    ev.inv_s2 = 1.0 / (A.prior_scale * A.prior_scale);
    ev.prior_const = (double)D * (log(A.prior_scale) + kHalfLog2Pi);
    run_chain<1, EXT>(A, ev, chain, S_arr);
}

template <typename T, int S, int CPS, int DPL, bool EXT>
__global__ void __launch_bounds__(kGridWaves * kWave, 1) sampler_grid_kernel(SamplerArgs A, int groups,
                                                                            int resident, double* partials,
                                                                            double* result, GridSync* sync)
{
    static_assert(LdsBlock<T, CPS, S>::kBytes == lds_block_bytes(sizeof(T) == 8 ? NUTS_F64 : NUTS_F32, S, CPS),
                  "the host sizes resident blocks as the kernel lays them out");
    extern __shared__ double lds[];
    __shared__ GridShared<DPL, kGridWaves> sh;
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
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    if (wave == 0) {
        // published by the first collective's barrier
        if (lane() == 0) __hip_atomic_store(&sh.stop, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        GridEval<T, S, CPS, DPL, kGridWaves> ev;
        ev.c = c;
        ev.sh = &sh;
        ev.inv_s2 = 1.0 / (A.prior_scale * A.prior_scale);
        ev.prior_const = (double)A.data.D * (log(A.prior_scale) + kHalfLog2Pi);
        ev.step = 0;
        ev.gen = 0;
        ev.abort = false;
        run_chain<DPL, EXT>(A, ev, 0, lds);
        ev.finish();
    } else {
        unsigned long long step = 0;
        double q[DPL], r[DPL + 1];
#pragma unroll
        for (int m = 0; m < DPL; ++m) q[m] = 0.0;
        // kGridPrefetch: the first block of the wave's share does not depend
        // on the position, so its loads are issued while the wave waits for
        // the next command (they land during the exchange and the
        // controller's step) and every collective starts on a block already
        // in registers.
        constexpr int R = BlockShape<T, S>::R;
        using LB = LdsBlock<T, CPS, S>;
        char* res_base = reinterpret_cast<char*>(lds) + grid_resident_offset(c.D, A.max_depth, A.sub_merge) +
                         (size_t)(wave - 1) * resident * LB::kBytes;
        const WaveShare share = grid_wave_share(c.nb, groups, wave, resident, res_base);
        // the resident blocks, loaded once
#pragma unroll 1
        for (int r = 0; r < share.res.count; ++r) {
            const int64_t b = share.res.first_block + r * share.stride;
            LB::store(res_base + (size_t)r * LB::kBytes,
                      load_block<T, CPS, S, kGridPipe<T>>((const T*)c.X + b * c.D * R, c.y + b * R, c.D));
        }
        const int64_t fb = share.first < c.nb ? share.first : 0;  // a valid block either way
        const T* Xf = (const T*)c.X + fb * c.D * R;
        const uint8_t* yf = c.y + fb * R;
        for (;;) {
            bool ab;
            int gen = 0;
            int cmd;
            if constexpr (kGridPrefetch<T>) {
                const BlockRegs<T, CPS, S> pre = load_block<T, CPS, S, kGridPipe<T>>(Xf, yf, c.D);
                cmd = grid_begin<T, S, CPS, DPL, kGridWaves, true>(c, sh, q, 0, 0, &gen, &share, &pre);
            } else {
                cmd = grid_begin<T, S, CPS, DPL, kGridWaves, true>(c, sh, q, 0, 0, &gen, &share);
            }
            if (cmd == kCmdExit) break;
            if (grid_end<T, S, CPS, DPL, kGridWaves, true>(c, sh, step, gen, false, r, &ab)) step++;
        }
    }
}

// Kernel for a data shape (S, CPS, DPL as pass_shape gives them).
template <typename T, bool EXT>
const void* grid_kernel_for(const DataView& dv)
{
    const int D = dv.D;
    if (D <= 8) return (const void*)sampler_grid_kernel<T, 1, 8, 1, EXT>;
    if (D <= 16) return (const void*)sampler_grid_kernel<T, 1, 16, 1, EXT>;
    if (D <= 32) return (const void*)sampler_grid_kernel<T, 4, 8, 1, EXT>;
    if (D <= 64) return (const void*)sampler_grid_kernel<T, 8, 8, 1, EXT>;
    if (D <= 128) return (const void*)sampler_grid_kernel<T, 16, 8, 2, EXT>;
    if (D <= 192) return (const void*)sampler_grid_kernel<T, 32, 8, 3, EXT>;
    if (D <= 256) return (const void*)sampler_grid_kernel<T, 32, 8, 4, EXT>;
    return (const void*)sampler_grid_kernel<T, 32, 10, 5, EXT>;
}

// Chains per group of the LDS-resident variant (the most of 4 .. 1 whose
// data sets fit), or 0 if not even one chain's data fits.
template <typename T, int S, int CPS>
int resident_chains_per_group(const SamplerArgs& a)
{
    using G = WaveLds<T, S, CPS>;
    for (int cpg = kWaveChainsPerGroup; cpg >= 1; --cpg) {
        if (cpg > a.num_chains && cpg > 1) continue;
        if (G::bytes(a.data.D, a.data.nb, a.max_depth, a.sub_merge, true, cpg) <= kMaxGroupLds) return cpg;
    }
    return 0;
}

template <typename T, int S, int CPS, bool EXT>
hipError_t wave_launch(const SamplerArgs& a, hipStream_t stream)
{
    using G = WaveLds<T, S, CPS>;
    const int cpg = resident_chains_per_group<T, S, CPS>(a);
    if (cpg > 0) {
        const size_t lds = G::bytes(a.data.D, a.data.nb, a.max_depth, a.sub_merge, true, cpg);
        const void* k = (const void*)sampler_wave_kernel<T, S, CPS, true, EXT>;
        hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        const unsigned grid = (unsigned)((a.num_chains + cpg - 1) / cpg);
        hipLaunchKernelGGL((sampler_wave_kernel<T, S, CPS, true, EXT>), dim3(grid),
                           dim3(kWaveChainsPerGroup * kWave), lds, stream, a, cpg);
    } else {
        // chains per group whose tree state fits (four unless the merge
        // stacks of a deep tree take more)
        int c4 = kWaveChainsPerGroup;
        while (c4 > 1 && G::bytes(a.data.D, a.data.nb, a.max_depth, a.sub_merge, false, c4) > kMaxGroupLds) --c4;
        const size_t lds = G::bytes(a.data.D, a.data.nb, a.max_depth, a.sub_merge, false, c4);
        if (lds > kMaxGroupLds) return hipErrorInvalidValue;
        const void* k = (const void*)sampler_wave_kernel<T, S, CPS, false, EXT>;
        hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        const unsigned grid = (unsigned)((a.num_chains + c4 - 1) / c4);
        hipLaunchKernelGGL((sampler_wave_kernel<T, S, CPS, false, EXT>), dim3(grid),
                           dim3(kWaveChainsPerGroup * kWave), lds, stream, a, c4);
    }
    return hipGetLastError();
}

// Whether the resident variant takes this shape.
template <typename T>
bool wave_resident_split(const SamplerArgs& a)
{
    if (a.data.split == 1) {
        if (a.data.cols == 16) return resident_chains_per_group<T, 1, 16>(a) > 0;
        return resident_chains_per_group<T, 1, 8>(a) > 0;
    }
    if (a.data.split == 4) return resident_chains_per_group<T, 4, 8>(a) > 0;
    return resident_chains_per_group<T, 8, 8>(a) > 0;
}

template <typename T, bool EXT>
hipError_t wave_launch_split(const SamplerArgs& a, hipStream_t stream)
{
    if (a.data.split == 1) {
        if (a.data.cols == 16) return wave_launch<T, 1, 16, EXT>(a, stream);
        return wave_launch<T, 1, 8, EXT>(a, stream);
    }
    if (a.data.split == 4) return wave_launch<T, 4, 8, EXT>(a, stream);
    return wave_launch<T, 8, 8, EXT>(a, stream);
}

}  // namespace sampler
}  // namespace nuts
