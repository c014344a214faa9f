// The data pass of the logistic potential: one 64-row column block per wave,
// one row per lane.  Each lane forms eta = x . q for its row from the block's
// columns (coalesced: a column of a block is 64 consecutive elements), then
// the row's loss and residual, and adds residual * x into per-column fp64
// partial sums that stay in registers until the pass ends.
#pragma once

#include "device.h"

namespace nuts {

// MAXD: compile-time column capacity (power of two, >= D).  Columns c >= D
// are neither loaded nor accumulated (x and q are zero there).
template <typename T, int MAXD>
__device__ __forceinline__ void accumulate_block(const T* __restrict__ xb,
                                                 const uint8_t* __restrict__ yb, int D,
                                                 int64_t rows_left, const double (&qv)[MAXD],
                                                 double (&acc)[MAXD], double& loss)
{
    const int l = lane();
    double x[MAXD];
#pragma unroll
    for (int c = 0; c < MAXD; ++c) x[c] = (c < D) ? (double)xb[c * kBlockRows + l] : 0.0;
    double eta = 0.0;
#pragma unroll
    for (int c = 0; c < MAXD; ++c) eta = fma(x[c], qv[c], eta);
    const RowTerms rt = logistic_row(eta, yb[l] != 0);
    const bool valid = l < rows_left;
    const double r = valid ? rt.resid : 0.0;
    loss += valid ? rt.loss : 0.0;
#pragma unroll
    for (int c = 0; c < MAXD; ++c) acc[c] = fma(r, x[c], acc[c]);
}

// Finish a wave's pass: returns column c's wave total in lane c (c < MAXD)
// and sets `loss` to the wave total of the row losses in every lane.
template <int MAXD>
__device__ __forceinline__ double finish_wave(double (&acc)[MAXD], double& loss)
{
    const double red = transpose_reduce<MAXD>(acc);
    loss = wave_sum(loss);
    return __shfl(red, (lane() * (kWave / MAXD)) & (kWave - 1));
}

}  // namespace nuts
