// The data pass of the logistic potential on gfx950.
//
// Layout: X is stored in blocks of R = RPL * 64 / S rows; inside a block,
// column c is R consecutive elements (one per row).  A wavefront processes one
// block per step: lane L works on rows RPL * (L / S) .. + RPL - 1 (RPL = 2 for
// fp32, 1 for fp64) and on the columns c = k * S + L % S, k < CPS, so that S
// lanes share a row and each holds at most CPS columns in registers.  For a
// fixed k the 64 lanes read columns k*S .. k*S + S - 1 of all R rows: one
// contiguous 512-byte segment per load instruction.
//
// Per row: the S partial dot products are combined with xor shuffles (every
// lane of the row ends with the same eta), the loss and residual follow from
// one exp (evaluated in fp32 for fp32 data), and residual * x is added into
// CPS fp64 per-lane accumulators.
// At the end of a pass the accumulators are reduced over the rows of the
// wave; the interleaved column order makes column c land in lane c when
// CPS == R, and in a fixed lane computed by column_source_lane otherwise.
#pragma once

#include <type_traits>

#include "device.h"

namespace nuts {

// Lanes per row for a column count D with at most CPS columns per lane.
__host__ __device__ constexpr int lanes_per_row(int D, int CPS)
{
    return D <= CPS ? 1 : D <= 2 * CPS ? 2 : D <= 4 * CPS ? 4 : D <= 8 * CPS ? 8 : D <= 16 * CPS ? 16 : 32;
}

// Rows per lane: fp32 blocks give each lane two consecutive rows so that a
// load instruction moves 512 bytes, as for fp64; with one lane per row (S =
// 1) fp64 lanes take two rows as well (16-byte loads, and two independent
// rows of per-row arithmetic per lane).
template <typename T, int S>
struct RowsPerLane {
    static constexpr int value = (sizeof(T) == 4 || S == 1) ? 2 : 1;
};

template <typename T, int N>
struct VecOf;
template <>
struct VecOf<float, 2> {
    using type = float2;
};
template <>
struct VecOf<double, 1> {
    using type = double;
};
template <>
struct VecOf<double, 2> {
    using type = double2;
};

template <typename T, int S>
struct BlockShape {
    static constexpr int RPL = RowsPerLane<T, S>::value;
    static constexpr int R = RPL * kWave / S;  // rows per block
};

// Raw registers of one block for one lane: CPS column slots of RPL rows,
// and the RPL labels as loaded (one byte each, row i in bits 8 i .. 8 i + 7;
// they are taken apart where they are used, so a loaded block needs no work
// before its computation starts).
template <typename T, int CPS, int S>
struct BlockRegs {
    using V = typename VecOf<T, BlockShape<T, S>::RPL>::type;
    using Y = typename std::conditional<BlockShape<T, S>::RPL == 2, uint16_t, uint8_t>::type;
    V x[CPS];
    Y y;
};

// An empty instruction that reads and rewrites a loaded block's registers:
// the compiler waits for the block's loads right there and cannot move work
// that uses them above it.  The stream loop below places it after the
// computation of the other block, so that the loads stay in flight across
// that computation whatever the scheduler would otherwise choose (left to
// itself it has converted a block right after issuing its loads, waiting for
// them at once, when the kernel around the loop changed).
template <typename V>
__device__ __forceinline__ void hold_value(V& v)
{
    if constexpr (sizeof(V) == 8) {
        uint64_t u = __builtin_bit_cast(uint64_t, v);
        asm volatile("" : "+v"(u));
        v = __builtin_bit_cast(V, u);
    } else {
        static_assert(sizeof(V) == 16, "8- or 16-byte column slots");
        struct U2 { uint64_t a, b; };
        U2 u = __builtin_bit_cast(U2, v);
        asm volatile("" : "+v"(u.a), "+v"(u.b));
        v = __builtin_bit_cast(V, u);
    }
}

__device__ __forceinline__ void set_zero(float2& v) { v = make_float2(0.0f, 0.0f); }
__device__ __forceinline__ void set_zero(double2& v) { v = make_double2(0.0, 0.0); }
__device__ __forceinline__ void set_zero(double& v) { v = 0.0; }

template <typename T, int CPS, int S>
__device__ __forceinline__ void hold_block(BlockRegs<T, CPS, S>& b)
{
#pragma unroll
    for (int k = 0; k < CPS; ++k) hold_value(b.x[k]);
    uint32_t y = b.y;
    asm volatile("" : "+v"(y));
    b.y = (typename BlockRegs<T, CPS, S>::Y)y;
}

// Issue the loads of one block.  By default the loads are unconditional: a
// slot past column D - 1 reads the next block's memory (or the zeroed tail of
// the allocation, at least kTailElems long), a finite value that meets a zero
// position component in eta and only feeds an accumulator slot that is never
// output.  For rows of at most 8 lanes those bytes are a small share of a
// block and mostly L2 hits.  For rows of 16 or 32 lanes they can be a quarter
// to a half of the block (D = 257 in 320 slots, D = 129 in 256), and part of
// them came from HBM a second time (8 % over the algorithmic bytes at
// D = 257); with MASK such rows skip every slot whose column is past D - 1
// (it holds zero; slots whose columns are all used load without a lane
// test), at the cost of registers, so the callers with registers to spare
// ask for it.
template <typename T, int CPS, int S, bool MASK>
__device__ __forceinline__ BlockRegs<T, CPS, S> load_block(const T* __restrict__ blk,
                                                           const uint8_t* __restrict__ yb, int D)
{
    using B = BlockRegs<T, CPS, S>;
    constexpr int RPL = BlockShape<T, S>::RPL;
    constexpr int R = BlockShape<T, S>::R;
    const int L = lane();
    const int p = L & (S - 1);
    const int row0 = (L / S) * RPL;
    const T* base = blk + p * R + row0;
    B out;
#pragma unroll
    for (int k = 0; k < CPS; ++k) {
        const typename B::V* src = reinterpret_cast<const typename B::V*>(base + k * S * R);
        if constexpr (MASK && S >= 16) {
            if ((k + 1) * S <= D) {  // wave-uniform: every lane's column is used
                out.x[k] = *src;
            } else {
                typename B::V v;
                set_zero(v);
                if (k * S + p < D) v = *src;
                out.x[k] = v;
            }
        } else {
            out.x[k] = *src;
        }
    }
    out.y = *reinterpret_cast<const typename B::Y*>(yb + row0);  // row0 is a multiple of RPL
    return out;
}

// A block kept in LDS from one pass to the next, as the registers a lane
// loads for it: slot k of lane L at element k * 64 + L, then the lanes'
// label words (one or two bytes a lane).  Writing a loaded block and reading
// it back gives the same registers, so a pass computes the same rows from
// either copy.
template <typename T, int CPS, int S>
struct LdsBlock {
    using B = BlockRegs<T, CPS, S>;
    using V = typename B::V;
    using Y = typename B::Y;
    static constexpr int kSlotBytes = CPS * kWave * (int)sizeof(V);
    static constexpr int kBytes = kSlotBytes + kWave * (int)sizeof(Y);  // a multiple of 16

    __device__ static void store(char* base, const B& b)
    {
        const int L = lane();
        V* slots = reinterpret_cast<V*>(base);
#pragma unroll
        for (int k = 0; k < CPS; ++k) slots[k * kWave + L] = b.x[k];
        reinterpret_cast<Y*>(base + kSlotBytes)[L] = b.y;
    }
    __device__ static B load(const char* base)
    {
        const int L = lane();
        const V* slots = reinterpret_cast<const V*>(base);
        B b;
#pragma unroll
        for (int k = 0; k < CPS; ++k) b.x[k] = slots[k * kWave + L];
        b.y = reinterpret_cast<const Y*>(base + kSlotBytes)[L];
        return b;
    }
};

// The blocks of a wave's share that sit in LDS: `count` of them from `base`,
// LdsBlock::kBytes apart, holding blocks first_block, first_block + stride, ...
struct ResidentBlocks {
    const char* base = nullptr;
    int count = 0;
    int64_t first_block = 0;
};

// Rows of one loaded block.  qv[k] must hold q[k * S + L % S] (zero for
// columns c >= D).  Rows at or past rows_left add nothing.
template <typename T, int CPS, int S>
__device__ __forceinline__ void compute_block(const BlockRegs<T, CPS, S>& in, int64_t rows_left,
                                              const double (&qv)[CPS], double (&acc)[CPS], double& loss)
{
    constexpr int RPL = BlockShape<T, S>::RPL;
    const int L = lane();
    const int p = L & (S - 1);
    const int row0 = (L / S) * RPL;
    double x[RPL][CPS];
#pragma unroll
    for (int k = 0; k < CPS; ++k) {
        if constexpr (RPL == 2) {
            x[0][k] = (double)in.x[k].x;
            x[1][k] = (double)in.x[k].y;
        } else {
            x[0][k] = (double)in.x[k];
        }
    }
    double r[RPL];
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
        double eta = 0.0;
#pragma unroll
        for (int k = 0; k < CPS; ++k) eta = fma(x[i][k], qv[k], eta);
        if constexpr (S >= 2) eta += pair_move<1>(eta);
        if constexpr (S >= 4) eta += pair_move<2>(eta);
        if constexpr (S >= 8) eta += pair_move<4>(eta);
        if constexpr (S >= 16) eta += pair_move<8>(eta);
        if constexpr (S >= 32) eta += pair_move<16>(eta);
        const RowTerms rt = logistic_row_t<T>(eta, ((in.y >> (8 * i)) & 0xff) != 0);
        const bool valid = row0 + i < rows_left;
        r[i] = valid ? rt.resid : 0.0;
        loss += (valid && p == 0) ? rt.loss : 0.0;
    }
#pragma unroll
    for (int k = 0; k < CPS; ++k) {
#pragma unroll
        for (int i = 0; i < RPL; ++i) acc[k] = fma(r[i], x[i][k], acc[k]);
    }
}

// The blocks first, first + stride, ... < nb of one data set.
//
// PIPE (the grid-wide and standalone passes, where each wave streams many
// blocks from HBM): the next block's loads are in flight while the current
// block is computed.  Two register sets take turns (the loop body handles
// two blocks), so no loaded block is copied from one set to the other: such
// a copy waits for the loads to land and would leave the wave with no loads
// in flight at the end of each block.  The loop runs a known count, so no
// path out of the body leaves a prefetched block unused (with an exit test
// after the computation the compiler moves the loads behind it, onto the
// path that uses them).
//
// Without PIPE (where the extra register set would not fit beside the rest of
// the kernel's state): one register set; the next block's loads are issued
// while the current block's gradient terms are added.  MASK as for
// load_block.
//
// ABORT: the pass may be called off while it runs (its result is then not
// used): the LDS word *stop is read before each block (PIPE: each pair of
// blocks) is loaded, and once it holds `token` the wave finishes the block it
// holds and stops.  The block in hand is always computed, so no loaded
// registers are dead on that path and the loads keep their place ahead of
// the computation.
//
// RES: besides the blocks first, first + stride, ... < nb from memory, the
// wave computes the LDS-resident blocks `res`: one after each block from
// memory whose successor's loads are in flight (its registers are free
// then), the rest after the last one.
template <bool ABORT>
__device__ __forceinline__ bool stop_requested(const int* stop, int token)
{
    if constexpr (ABORT) return __hip_atomic_load(stop, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) == token;
    return false;
}

//
// stream_blocks_from takes block `first` already loaded (its loads may still
// be in flight), so that a caller can issue them before the position is
// known; stream_blocks loads it itself.
template <typename T, int CPS, int S, bool PIPE, bool MASK, bool ABORT = false, bool RES = false>
__device__ __forceinline__ void stream_blocks_from(BlockRegs<T, CPS, S> a, const T* __restrict__ X,
                                                   const uint8_t* __restrict__ y, int D, int64_t N, int64_t nb,
                                                   int64_t first, int64_t stride, const double (&qv)[CPS],
                                                   double (&acc)[CPS], double& loss, const int* stop = nullptr,
                                                   int token = 0, const ResidentBlocks& res = ResidentBlocks())
{
    constexpr int R = BlockShape<T, S>::R;
    using LB = LdsBlock<T, CPS, S>;
    if (first >= nb) return;
    int64_t b = first;
    int r = 0;            // resident blocks done
    bool called_off = false;
    // one resident block into the free register set `dst`, if any is left
    const auto resident_step = [&](BlockRegs<T, CPS, S>& dst) {
        if constexpr (RES) {
            if (uni(r < res.count)) {
                dst = LB::load(res.base + r * LB::kBytes);
                compute_block<T, CPS, S>(dst, N - (res.first_block + r * stride) * R, qv, acc, loss);
                ++r;
            }
        }
    };
    if constexpr (PIPE) {
        const int64_t count = (nb - 1 - first) / stride + 1;  // blocks of this wave
        int64_t count_left = count;
        int64_t i = 1;                                         // blocks loaded so far
#pragma unroll 1
        for (; i + 1 < count_left; i += 2) {
            if (stop_requested<ABORT>(stop, token)) {
                count_left = i;  // no more loads: the tail computes the block in hand
                called_off = true;
                break;
            }
            const int64_t b1 = b + stride, b2 = b1 + stride;
            BlockRegs<T, CPS, S> c = load_block<T, CPS, S, MASK>(X + b1 * D * R, y + b1 * R, D);
            __builtin_amdgcn_sched_barrier(0);  // the loads are issued before the computation
            compute_block<T, CPS, S>(a, N - b * R, qv, acc, loss);
            __builtin_amdgcn_sched_barrier(0);  // and it is done before the wait for the loads
            resident_step(a);
            __builtin_amdgcn_sched_barrier(0);
            hold_block(c);
            a = load_block<T, CPS, S, MASK>(X + b2 * D * R, y + b2 * R, D);
            __builtin_amdgcn_sched_barrier(0);
            compute_block<T, CPS, S>(c, N - b1 * R, qv, acc, loss);
            __builtin_amdgcn_sched_barrier(0);
            hold_block(a);
            b = b2;
        }
        if (i < count_left) {
            const int64_t b1 = b + stride;
            BlockRegs<T, CPS, S> c = load_block<T, CPS, S, MASK>(X + b1 * D * R, y + b1 * R, D);
            __builtin_amdgcn_sched_barrier(0);
            compute_block<T, CPS, S>(a, N - b * R, qv, acc, loss);
            __builtin_amdgcn_sched_barrier(0);
            resident_step(a);
            __builtin_amdgcn_sched_barrier(0);
            hold_block(c);
            compute_block<T, CPS, S>(c, N - b1 * R, qv, acc, loss);
        } else {
            compute_block<T, CPS, S>(a, N - b * R, qv, acc, loss);
        }
    } else {
#pragma unroll 1
        for (;;) {
            const int64_t nx = b + stride;
            const bool stopped = stop_requested<ABORT>(stop, token);
            const bool more = nx < nb && !stopped;
            const int64_t lb = more ? nx : b;  // a valid block either way
            const BlockRegs<T, CPS, S> nxt = load_block<T, CPS, S, MASK>(X + lb * D * R, y + lb * R, D);
            compute_block<T, CPS, S>(a, N - b * R, qv, acc, loss);
            if (!more) {
                called_off = stopped;
                break;
            }
            resident_step(a);
            a = nxt;
            b = nx;
        }
    }
    if constexpr (RES) {
#pragma unroll 1
        while (uni(!called_off && r < res.count)) resident_step(a);
    }
}

template <typename T, int CPS, int S, bool PIPE, bool MASK, bool ABORT = false, bool RES = false>
__device__ __forceinline__ void stream_blocks(const T* __restrict__ X, const uint8_t* __restrict__ y, int D,
                                              int64_t N, int64_t nb, int64_t first, int64_t stride,
                                              const double (&qv)[CPS], double (&acc)[CPS], double& loss,
                                              const int* stop = nullptr, int token = 0,
                                              const ResidentBlocks& res = ResidentBlocks())
{
    constexpr int R = BlockShape<T, S>::R;
    if (first >= nb) return;
    const BlockRegs<T, CPS, S> a = load_block<T, CPS, S, MASK>(X + first * D * R, y + first * R, D);
    stream_blocks_from<T, CPS, S, PIPE, MASK, ABORT, RES>(a, X, y, D, N, nb, first, stride, qv, acc, loss, stop,
                                                          token, res);
}

// Lane that holds column c after reduce_rows<CPS, S>.
template <int CPS, int S>
__device__ __forceinline__ int column_source_lane(int c)
{
    constexpr int LANES_PER_PART = kWave / S;
    static_assert(CPS <= LANES_PER_PART, "one slot per row lane at least");
    const int sigma = c / S, p = c & (S - 1);
    const int rho = sigma * (LANES_PER_PART / CPS);
    return (rho * S) | p;
}

// Sum the CPS per-lane accumulators over the rows of the wave (lane bits
// from 32 down to S).  The first log2(CPS) steps halve the live slots (the
// lane whose partner bit is set keeps the upper half); the rest add.
template <int BIT, int H, int N>
__device__ __forceinline__ void halve(double (&a)[N], int L)
{
    const bool upper = (L & BIT) != 0;
#pragma unroll
    for (int i = 0; i < H; ++i) {
        const double send = upper ? a[i] : a[i + H];
        const double keep = upper ? a[i + H] : a[i];
        a[i] = keep + xor_move<BIT>(send);
    }
}

template <int BIT, int H, int S, int N>
__device__ __forceinline__ void reduce_step(double (&a)[N], double& v, int L)
{
    if constexpr (BIT >= S) {
        if constexpr (H >= 1) {
            halve<BIT, H>(a, L);
            if constexpr (H == 1) v = a[0];
        } else {
            v += xor_move<BIT>(v);
        }
        reduce_step<BIT / 2, H / 2, S>(a, v, L);
    }
}

template <int CPS, int S>
__device__ __forceinline__ double reduce_rows(double (&a)[CPS])
{
    static_assert(CPS >= 1 && (CPS & (CPS - 1)) == 0, "CPS is a power of two");
    double v = a[0];
    reduce_step<kWave / 2, CPS / 2, S>(a, v, lane());
    return v;
}

// Sum the per-lane accumulators over the rows of the wave (lane bits from 32
// down to S) with plain xor butterflies, then store column k * S + p's
// total from the lanes of row 0 into row[] (columns < D only) and the loss
// total into row[loss_slot].  For wide rows, where the transposing
// reduction has too few row lanes per slot.
template <int BIT, int S, int CPS>
__device__ __forceinline__ void add_over_rows(double (&a)[CPS])
{
    if constexpr (BIT >= S) {
#pragma unroll
        for (int k = 0; k < CPS; ++k) a[k] += xor_move<BIT>(a[k]);
        add_over_rows<BIT / 2, S>(a);
    }
}

template <int CPS, int S>
__device__ __forceinline__ void finish_pass_to_row(double (&acc)[CPS], double loss, double* row, int D,
                                                   int loss_slot)
{
    add_over_rows<kWave / 2, S>(acc);
    loss = wave_sum(loss);
    const int L = lane();
    if (L < S) {
#pragma unroll
        for (int k = 0; k < CPS; ++k) {
            const int c = k * S + L;
            if (c < D) row[c] = acc[k];
        }
    }
    if (L == 0) row[loss_slot] = loss;
}

// Finish a wave's pass: column c's wave total in lane c (c < CPS * S, zero
// elsewhere), and the wave's total loss in every lane.
template <int CPS, int S>
__device__ __forceinline__ double finish_pass(double (&acc)[CPS], double& loss)
{
    const double v = reduce_rows<CPS, S>(acc);
    loss = wave_sum(loss);
    const int L = lane();
    const double col = __shfl(v, column_source_lane<CPS, S>(L < CPS * S ? L : 0));
    return L < CPS * S ? col : 0.0;
}

// Load q (lane-per-dimension, zero past D) into the per-lane column order.
template <int CPS, int S>
__device__ __forceinline__ void spread_position(double q, double (&qv)[CPS])
{
    const int p = lane() & (S - 1);
#pragma unroll
    for (int k = 0; k < CPS; ++k) qv[k] = __shfl(q, (k * S + p) & (kWave - 1));
}

// The same from a position vector in LDS (zero past D).
template <int CPS, int S>
__device__ __forceinline__ void spread_position_lds(const double* q, int D, double (&qv)[CPS])
{
    const int p = lane() & (S - 1);
#pragma unroll
    for (int k = 0; k < CPS; ++k) {
        const int c = k * S + p;
        qv[k] = c < D ? q[c] : 0.0;
    }
}

}  // namespace nuts
