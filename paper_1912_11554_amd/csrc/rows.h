// The data pass of the logistic potential on gfx950.
//
// Layout: X is stored in blocks of R = 64 / S rows; inside a block, column c
// is R consecutive elements (one per row).  A wavefront processes one block
// per step: lane L works on row L / S and on the columns c = k * S + L % S,
// k < CPS, so that S lanes share a row and each holds at most CPS columns in
// registers.  For a fixed k the 64 lanes read columns k*S .. k*S + S - 1 of
// all R rows: one contiguous 64-element segment per load instruction.
//
// Per row: the S partial dot products are combined with xor shuffles (every
// lane of the row ends with the same eta), the loss and residual follow from
// one exp (evaluated in fp32 for fp32 data), and residual * x is added into
// CPS fp64 per-lane accumulators.
// At the end of a pass the accumulators are reduced over the rows of the
// wave; the interleaved column order makes column c land in lane c when
// CPS == R, and in a fixed lane computed by column_source_lane otherwise.
#pragma once

#include "device.h"

namespace nuts {

// Lanes per row for a column count D with at most CPS columns per lane.
__host__ __device__ constexpr int lanes_per_row(int D, int CPS)
{
    return D <= CPS ? 1 : D <= 2 * CPS ? 2 : D <= 4 * CPS ? 4 : D <= 8 * CPS ? 8 : D <= 16 * CPS ? 16 : 32;
}

template <int S>
struct RowSplit {
    static_assert(S >= 1 && S <= 32 && (S & (S - 1)) == 0, "S is a power of two");
    static constexpr int R = kWave / S;  // rows per block
    static constexpr int LOG_S = S == 1 ? 0 : S == 2 ? 1 : S == 4 ? 2 : S == 8 ? 3 : S == 16 ? 4 : 5;
};

// qv[k] must hold q[k * S + L % S], which is zero for columns c >= D.  The
// loads are unconditional: a slot past column D - 1 reads the next block's
// memory (or the zeroed tail of the allocation, at least kTailElems long), a
// finite value that meets a zero position in eta and only feeds an
// accumulator slot that is never output.
template <typename T, int CPS, int S>
__device__ __forceinline__ void accumulate_block(const T* __restrict__ blk,
                                                 const uint8_t* __restrict__ yb, int D,
                                                 int64_t rows_left, const double (&qv)[CPS],
                                                 double (&acc)[CPS], double& loss)
{
    constexpr int R = RowSplit<S>::R;
    const int L = lane();
    const int p = L & (S - 1);
    const int row = L / S;
    const T* base = blk + p * R + row;
    (void)D;
    double x[CPS];
#pragma unroll
    for (int k = 0; k < CPS; ++k) x[k] = (double)base[k * S * R];
    double eta = 0.0;
#pragma unroll
    for (int k = 0; k < CPS; ++k) eta = fma(x[k], qv[k], eta);
    if constexpr (S >= 2) eta += pair_move<1>(eta);
    if constexpr (S >= 4) eta += pair_move<2>(eta);
    if constexpr (S >= 8) eta += pair_move<4>(eta);
    if constexpr (S >= 16) eta += pair_move<8>(eta);
    if constexpr (S >= 32) eta += pair_move<16>(eta);
    const RowTerms rt = logistic_row_t<T>(eta, yb[row] != 0);
    const bool valid = row < rows_left;
    const double r = valid ? rt.resid : 0.0;
    loss += (valid && p == 0) ? rt.loss : 0.0;
#pragma unroll
    for (int k = 0; k < CPS; ++k) acc[k] = fma(r, x[k], acc[k]);
}

// Lane that holds column c after reduce_rows<CPS, S>.
template <int CPS, int S>
__device__ __forceinline__ int column_source_lane(int c)
{
    constexpr int R = RowSplit<S>::R;
    static_assert(CPS <= R, "one slot per row lane at least");
    const int sigma = c / S, p = c & (S - 1);
    const int rho = sigma * (R / CPS);
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

}  // namespace nuts
