// Host-side launchers of the gfx950 kernels and the plain structs they share
// with the C-ABI layer.  Every launcher enqueues on `stream` and returns the
// HIP status of the launch; shapes are validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/nuts.h"

namespace nuts {

// Device layout of one or more data sets: X as column blocks of R rows
// (R = 64 / S for fp64, 128 / S for fp32; S lanes of a wavefront share a row,
// each lane takes one fp64 or two fp32 rows), block b of data set s at element
// offset (s * nb + b) * D * R, column c of the block at + c * R, row r of the
// block at + r; rows past N are zero.  y as bytes at (s * nb + b) * R + r,
// zero past N.
struct DataView {
    const void* X;
    const uint8_t* y;
    int64_t N;
    int D;
    int dtype;        // NUTS_F64 or NUTS_F32
    int split;        // S: lanes per row, 64 / rows per block
    int64_t nb;       // ceil(N / R)
    int64_t nds;      // number of data sets
};

// Columns one lane holds in registers during the data pass.
constexpr int kColsPerLane = 8;

// Zeroed elements after the last block of an X allocation: the data pass
// reads up to kColsPerLane * 128 elements from a block's start.
constexpr int64_t kTailElems = (int64_t)kColsPerLane * 128;

inline int rows_per_block(const DataView& dv) { return (dv.dtype == NUTS_F32 ? 128 : 64) / dv.split; }

// Largest D the lane-per-dimension kernels accept: dimension d lives in lane d
// and lane 63 carries the potential through the reductions.
constexpr int kMaxDim = 63;

hipError_t launch_to_blocks(const void* X_rowmajor, const uint8_t* y_in, DataView dst,
                            void* X_out, uint8_t* y_out, unsigned int* bad_label,
                            hipStream_t stream);

// Workspace of the batched potential/gradient: partial sums [K][G][64].
struct PotentialPlan {
    int groups_per_item;  // G
    int waves_per_group;
};
PotentialPlan plan_potential(const DataView& dv, int64_t K, int num_cu);
hipError_t launch_potential_grad(const DataView& dv, double prior_scale, const double* W, int64_t K,
                                 const PotentialPlan& plan, double* partials, double* out_U,
                                 double* out_grad, hipStream_t stream);

// Sampler arguments common to both paths (device pointers).
struct SamplerArgs {
    DataView data;
    int per_chain_data;
    double prior_scale;
    double step_size;
    const double* inv_mass;   // [D] or null
    int max_depth;
    int64_t num_warmup, num_samples;
    int64_t num_chains;
    int64_t chain_offset;     // first chain index this launch runs
    uint64_t seed;
    int64_t first_iter;
    int adapt_diag;
    const double* init_q;     // [C][D] or null
    double* out_samples;      // [C][S][D] or null
    nuts_stats* out_stats;    // [C][S] or null
    double* out_final_q;      // [C][D] or null
    double* out_inv_mass;     // [C][D] or null
    unsigned long long* grad_evals;  // [C]
};

// One wavefront per chain: launches ceil(C / 4) groups of four waves.
hipError_t launch_sampler_wave(const SamplerArgs& a, hipStream_t stream);

// One chain over the whole device.  `sync` holds the arrival counter and the
// error flag, zeroed by this call; `partials` holds [2][groups][64] doubles,
// `result` [2][64] (marked empty by this call).
struct GridSync {
    unsigned long long counter;          // completed group slots, (step + 1) * min(groups, 8) after step
    unsigned long long pad0[15];
    unsigned int error;                  // a wait timed out
    unsigned int pad1[31];
    unsigned long long slot[8][16];      // group arrivals per slot (group index mod 8)
};
hipError_t launch_sampler_grid(const SamplerArgs& a, int groups, double* partials, double* result,
                               GridSync* sync, hipStream_t stream);
int grid_sampler_groups(const DataView& dv, int max_depth, int num_cu);

}  // namespace nuts
