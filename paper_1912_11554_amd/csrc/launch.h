// Host-side launchers of the gfx950 kernels and the plain structs they share
// with the C-ABI layer.  Every launcher enqueues on `stream` and returns the
// HIP status of the launch; shapes are validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/nuts.h"

namespace nuts {

// Device layout of one or more data sets: X as column blocks of 64 rows,
// block b of data set s at element offset (s * nb + b) * D * 64, column c of
// the block at + c * 64, row r of the block at + r; rows past N are zero.
// y as bytes at (s * nb + b) * 64 + r, zero past N.
struct DataView {
    const void* X;
    const uint8_t* y;
    int64_t N;
    int D;
    int dtype;        // NUTS_F64 or NUTS_F32
    int64_t nb;       // ceil(N / 64)
    int64_t nds;      // number of data sets
};

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

// One chain over the whole device.  `sync` holds the grid-barrier counters,
// zeroed by this call; `partials` holds [2][groups][64] doubles, `result`
// [2][64].  Returns the group count used through *groups_used.
struct GridSync {
    unsigned long long counter;
    unsigned long long flag;
    unsigned int error;
    unsigned int pad;
};
hipError_t launch_sampler_grid(const SamplerArgs& a, int groups, double* partials, double* result,
                               GridSync* sync, hipStream_t stream);
int grid_sampler_groups(const DataView& dv, int max_depth, int num_cu);

}  // namespace nuts
