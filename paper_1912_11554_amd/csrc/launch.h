// Host-side launchers of the gfx950 kernels and the plain structs they share
// with the C-ABI layer.  Every launcher enqueues on `stream` and returns the
// HIP status of the launch; shapes are validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/nuts.h"

namespace nuts {

// Largest D the kernels accept: lanes hold up to 5 dimensions each.
constexpr int kMaxDim = 320;

// Shape of the data pass for D columns: S lanes of a wavefront share a row
// and each lane holds `cols` column slots of it (slot k of lane part p is
// column k * S + p); `dims` = ceil(D / 64) dimensions per lane in the tree
// state (dimension d in lane d % 64, component d / 64).
struct PassShape {
    int split;  // S
    int cols;   // CPS
    int dims;   // DPL
};

inline PassShape pass_shape(int D)
{
    const int dims = (D + 63) / 64;
    if (D <= 8) return {1, 8, dims};
    if (D <= 16) return {1, 16, dims};
    if (D <= 32) return {4, 8, dims};
    if (D <= 64) return {8, 8, dims};
    if (D <= 128) return {16, 8, dims};
    if (D <= 256) return {32, 8, dims};
    return {32, 10, dims};
}

// Device layout of one or more data sets: X as column blocks of R rows
// (R = RPL * 64 / S; each lane takes RPL rows: two for fp32 or S = 1, one
// otherwise), block b of data set s at element offset (s * nb + b) * D * R,
// column c of the block at + c * R, row r of the block at + r; rows past N
// are zero.  y as bytes at (s * nb + b) * R + r, zero past N.
struct DataView {
    const void* X;
    const uint8_t* y;
    int64_t N;
    int D;
    int dtype;        // NUTS_F64 or NUTS_F32
    int split;        // S
    int cols;         // CPS
    int64_t nb;       // ceil(N / R)
    int64_t nds;      // number of data sets
};

// Zeroed elements after the last block of an X allocation: the data pass
// reads up to cols * S * R <= 16 * 128 elements from a block's start.
constexpr int64_t kTailElems = 2048;

inline int rows_per_block(const DataView& dv)
{
    const int rpl = (dv.dtype == NUTS_F32 || dv.split == 1) ? 2 : 1;
    return rpl * 64 / dv.split;
}

// Width of one partial-sum row: the D columns padded to whole lanes, then
// one more lane-row whose slot 0 is the loss sum.
inline int partial_width(int D) { return 64 * ((D + 63) / 64 + 1); }

hipError_t launch_to_blocks(const void* X_rowmajor, const uint8_t* y_in, DataView dst,
                            void* X_out, uint8_t* y_out, unsigned int* bad_label,
                            hipStream_t stream);

// Workspace of the batched potential/gradient: K * G * width doubles of
// partial-sum slots (item k's used columns c = 0..D, the loss last, as rows
// of G group slots at k * G * width + c * G), every slot marked empty
// (mark_partials_empty) before the first launch; each launch leaves every
// slot it used empty again.
struct PotentialPlan {
    int groups_per_item;  // G
    int width;            // partial_width(D)
    bool own_cu;          // G * K groups fit the device once: one group a CU
    bool items;           // many items with few blocks each: one wave an item, no partial rows
};
constexpr int kMaxPotentialItems = 65535;
constexpr int kMaxPotentialGroups = 256;  // groups per item
PotentialPlan plan_potential(const DataView& dv, int64_t K, int num_cu);
hipError_t launch_potential_grad(const DataView& dv, double prior_scale, const double* W, int64_t K,
                                 const PotentialPlan& plan, double* partials, double* out_U, double* out_grad,
                                 hipStream_t stream);
// Mark n partial-sum slots empty (a kernel on `stream`).
hipError_t mark_partials_empty(double* p, int64_t n, hipStream_t stream);

// The allocation-free form of launch_potential_grad keeps its partial-sum
// slots in a fixed device array of kStaticScratchBytes.
// static_workspace_setup, called once per device with that device current
// (nuts_init does), finds this device's copy of the array and marks its slots
// empty; it returns the array's device address.  Calls that overlap on one
// device race on the array.
constexpr size_t kStaticScratchBytes = (size_t)8 << 20;
constexpr int64_t kStaticMaxItems = 16384;
hipError_t static_workspace_setup(int device, hipStream_t stream, void** out);

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
    int adapt_step;           // dual-averaging step size during warmup
    double target_accept;     // its target acceptance
    int uturn_gen;            // the generalised (momentum-sum) U-turn criterion
    int sub_merge;            // subtree proposals chosen at the merges of halves
    const double* init_q;     // [C][D] or null
    double* out_samples;      // [C][S][D] or null
    nuts_stats* out_stats;    // [C][S] or null
    double* out_final_q;      // [C][D] or null
    double* out_inv_mass;     // [C][D] or null
    double* out_step_size;    // [C] or null
    unsigned long long* grad_evals;  // [C]
};

// One wavefront per chain (D <= 64): ceil(C / 4) groups of four waves.
hipError_t launch_sampler_wave(const SamplerArgs& a, hipStream_t stream);
bool wave_path_supports(const DataView& dv);
// The chains' data sets fit in LDS (the resident variant of the wave path).
bool wave_path_resident(const SamplerArgs& a);

// One chain over the whole device.  `sync` holds the error flag, zeroed by
// this call; `partials` holds grid_partial_elems(D, groups) doubles and
// `result` grid_result_elems(D) doubles, both marked empty by this call.
// The result row of each phase is kept in kGridReplicas copies, kReplicaStride
// doubles apart (4 KiB + 256 B, so that the copies fall in different memory
// channels): every controller polls its row once per round trip, and 256 of
// them on one row queue at the channel that holds it.
constexpr int kGridPhases = 3;
constexpr int kGridReplicas = 16;
constexpr int kReplicaStride = 544;  // >= partial_width(D) for D <= 448
inline int64_t grid_partial_elems(int D, int groups) { return (int64_t)kGridPhases * (D + 1) * groups; }
inline int64_t grid_result_elems(int) { return (int64_t)kGridPhases * kGridReplicas * kReplicaStride; }
struct GridSync {
    unsigned int error;  // a wait timed out
    unsigned int pad[63];
};
// `at_launch` (optional): an event recorded right before the sampler kernel,
// after the set-up kernel.
hipError_t launch_sampler_grid(const SamplerArgs& a, int groups, double* partials, double* result,
                               GridSync* sync, hipStream_t stream, hipEvent_t at_launch = nullptr);
int grid_sampler_groups(const DataView& dv, int max_depth, int sub_merge, int num_cu);

// ---------------------------------------------------------------------------
// Batched chains on shared fp32 data: the potential and gradient of K
// positions as one contraction E = X Q (N x D by D x K) on the matrix cores,
// the row terms on E, then G = X^T R (D x N by N x K).
//
// Layout: stages of 64 rows; a stage is 64 rows of `stride` floats, row r of
// stage s at (s * 64 + r) * stride.  The first 16 kp floats of a row
// (kp = kt rounded up to a multiple of 4) hold the columns that feed the
// matrix cores, permuted: slot g * kp + t holds column 16 t + g (g < 16,
// t < kp; zero for t >= kt), so that the 16-column chunks t of one column
// residue g are contiguous.  The last 4 floats hold the tail: up to four more
// columns (16 kt .. 16 kt + 3) handled on the vector ALUs.  Entries past N
// or past D are zero.  y is one byte per row, 0 past N (padding rows: zero X,
// label 0).
struct BatchView {
    const float* X;
    const uint8_t* y;
    int64_t N;
    int D;
    int kt;          // 16-column chunks on the matrix cores
    int tc;          // tail columns on the vector ALUs (0..4)
    int stride;      // 16 kp + 4 floats
    int64_t ns;      // stages: ceil(N / 64)
};
__host__ __device__ inline int batch_kp(int kt) { return (kt + 3) / 4 * 4; }
constexpr int kBatchStageRows = 64;
constexpr int kBatchMaxKT = 8;          // D <= 132
constexpr int kBatchTileChains = 128;   // chains (positions) per tile: 8 waves x 16
constexpr int kBatchMaxTiles = 2;       // tiles per sampler launch

// Chunk and tail counts for D columns; false if D is too wide.
inline bool batch_shape(int D, int* kt, int* tc)
{
    const int rem = D % 16;
    int k = D / 16, t = rem;
    if (rem > 4) {
        k += 1;
        t = 0;
    }
    if (k > kBatchMaxKT) return false;
    *kt = k;
    *tc = t;
    return true;
}

// Fill X/y of the batch layout from the column-block layout of `src` (fp32,
// one data set).
hipError_t launch_to_batch_layout(const DataView& src, const BatchView& dst, float* X, uint8_t* y,
                                  hipStream_t stream);

// Workspace of the batched potential: fp32 partial rows P[T][G][128][pw]
// and fp64 loss partials L[T][G][128], T = ceil(K / 128) tiles of G groups.
struct BatchPlan {
    int tiles;
    int groups;   // per tile
    int pw;       // 64 * ceil(D / 64)
};
BatchPlan plan_batch_potential(const BatchView& bv, int64_t K, int num_cu);
hipError_t launch_batch_potential(const BatchView& bv, double prior_scale, const double* W, int64_t K,
                                  const BatchPlan& plan, float* P, double* L, double* out_U, double* out_grad,
                                  hipStream_t stream);

// Log-likelihood of S draws over shared fp32 data on the matrix cores (the
// plan of plan_batch_potential for K = S): L holds tiles * groups * 128
// doubles; Pr tiles * ns * 64 floats when out_pred (mean of sigmoid(eta)
// over the draws, [N]) is wanted, else unused.  With out_y ([S][N] bytes)
// the pass writes the posterior predictive samples of the draws under
// `seed` instead, and nothing else.
hipError_t launch_batch_log_likelihood(const BatchView& bv, const double* W, int64_t S, const BatchPlan& plan,
                                       double* L, float* Pr, double* out_ll, double* out_pred, uint8_t* out_y,
                                       uint64_t seed, hipStream_t stream);
// ll[s] = -(U[s] - |w_s|^2 / 2 - D ln(2 pi) / 2) for potentials U taken with
// prior scale 1 (the streaming path's log-likelihood).
hipError_t launch_ll_from_potential(int D, const double* W, int64_t S, const double* U, double* out_ll,
                                    hipStream_t stream);
// log((1/S) sum_s exp(ll[s])) into *out.
hipError_t launch_expected_ll(const double* ll, int64_t S, double* out, hipStream_t stream);

// Batched sampler exchange state.  Zeroed per launch except done_at, which
// starts at all ones ("not finished").
struct BatchSync {
    unsigned int error;                                       // a wait timed out
    unsigned int pad0[31];
    unsigned long long tile_count[kBatchMaxTiles][16];        // groups done with step s: (s + 1) * G
    unsigned long long stamp[kBatchMaxTiles * kBatchTileChains];    // s + 1 once Q(s) of the chain is out
    unsigned long long done_at[kBatchMaxTiles * kBatchTileChains];  // first step with no iteration left
};
// Sampler on `tiles` tiles of `groups` groups (groups >= 128): chain slot i
// of tile t is run by group t * groups + i.  qbuf holds [2][tiles * 128][192]
// floats, P [2][tiles][groups][128][pw] floats, L [2][tiles][groups][128]
// doubles.  `at_launch` as for launch_sampler_grid.
hipError_t launch_sampler_batch(const SamplerArgs& a, const BatchView& bv, int tiles, int groups, float* qbuf,
                                float* P, double* L, BatchSync* sync, hipStream_t stream,
                                hipEvent_t at_launch = nullptr);
bool batch_sampler_supported(const BatchView& bv, int max_depth, int sub_merge, int num_cu);
constexpr int kBatchQWidth = 192;

// Per-dtype kernel entry points (sampler_f32.hip, sampler_f64.hip).
hipError_t launch_sampler_wave_f32(const SamplerArgs& a, hipStream_t stream);
hipError_t launch_sampler_wave_f64(const SamplerArgs& a, hipStream_t stream);
bool wave_resident_f32(const SamplerArgs& a);
bool wave_resident_f64(const SamplerArgs& a);
const void* grid_kernel_f32(const DataView& dv);
const void* grid_kernel_f64(const DataView& dv);
// The same with the optional features compiled in: warmup step-size
// adaptation, the generalised U-turn criterion (sampler_ext_*.hip).
hipError_t launch_sampler_wave_ext_f32(const SamplerArgs& a, hipStream_t stream);
hipError_t launch_sampler_wave_ext_f64(const SamplerArgs& a, hipStream_t stream);
const void* grid_kernel_ext_f32(const DataView& dv);
const void* grid_kernel_ext_f64(const DataView& dv);
// Whether a launch needs the kernels with the adaptation.
inline bool sampler_extended(const SamplerArgs& a)
{
    return (a.adapt_step && a.num_warmup > 0) || a.uturn_gen || a.sub_merge;
}
// Levels of waiting blocks a subtree of at most 2^(depth-1) leaves uses.
__host__ __device__ inline int merge_levels(int max_depth) { return max_depth > 1 ? max_depth - 1 : 1; }

// Doubles of one chain's tree state in LDS: the checkpoint array S
// [max(depth, 1)][2][D], then, with merge-structured subtree proposals, the
// waiting block of each level: its proposal [levels][3][D] (q, p, grad U)
// and [levels][3] scalars (log-weight, offset, U).
// LDS of one chain's tree state: the checkpoint array S, the waiting blocks
// of the merge-structured subtree proposals, and with edge_nodes the two
// trajectory edges and the two proposals (4 nodes of 3 * 64 * ceil(D / 64)
// + 1 doubles).
__host__ __device__ inline int64_t chain_lds_doubles(int D, int max_depth, int sub_merge, bool edge_nodes)
{
    const int slots = max_depth > 1 ? max_depth : 1;
    int64_t n = (int64_t)slots * 2 * D;
    if (sub_merge) n += (int64_t)merge_levels(max_depth) * (3 * D + 3);
    if (edge_nodes) n += 4 * (3 * 64 * (int64_t)((D + 63) / 64) + 1);
    return n;
}
// Whether the grid path's controller keeps its edge and proposal nodes in
// LDS (three or more components a lane), and the batch path's (the same,
// for the kernel without the extended features, whose LDS has the room).
__host__ __device__ inline bool grid_edge_nodes(int D) { return D > 128; }
__host__ __device__ inline bool batch_edge_nodes(int D, bool extended) { return D > 128 && !extended; }
constexpr int kGridWaves = 12;  // per group: 1 controller + 11 workers (3 waves per SIMD: 168 registers each)

// Grid path: every worker keeps the last blocks of its share in LDS for the
// whole launch (as many as the group's LDS beside the chain's state holds),
// so they are read from memory once per launch instead of once per
// evaluation.  A block takes lds_block_bytes: the registers one lane loads
// for it (cols slots of two rows for fp32 or one lane per row, else one
// row), 64 lanes, then the lanes' labels (one byte a row).  They start at
// byte grid_resident_offset of the group's dynamic LDS, after the chain's
// state.
__host__ __device__ constexpr int lds_block_bytes(int dtype, int split, int cols)
{
    const int rows_per_lane = (dtype == NUTS_F32 || split == 1) ? 2 : 1;
    return cols * 64 * rows_per_lane * (dtype == NUTS_F64 ? 8 : 4) + 64 * rows_per_lane;
}
__host__ __device__ inline size_t grid_resident_offset(int D, int max_depth, int sub_merge)
{
    const size_t b = (size_t)chain_lds_doubles(D, max_depth, sub_merge, grid_edge_nodes(D)) * sizeof(double);
    return (b + 15) & ~(size_t)15;
}

// Semi-supervised hidden Markov model (hmm.hip, hmm_ext.hip): symbols w [T]
// (< V), observed states z [Tsup] (< K), on the device.  Parameters: K (K-1)
// transition logits, then K (V-1) emission logits.
constexpr int kHmmSteps = 8;                     // unobserved steps per lane
constexpr int kHmmMaxUnobserved = kHmmSteps * 64;
struct HmmView {
    const uint8_t* w;
    const uint8_t* z;
    int T, Tsup, K, V;
};
inline int hmm_dim(int K, int V) { return K * (K - 1) + K * (V - 1); }
// Shapes the kernels take: 2 <= K <= 4, V >= 2, K*K + K*V <= 64 (one lane
// per simplex entry), T - Tsup <= kHmmMaxUnobserved.
inline bool hmm_supported(int K, int V, int64_t T, int64_t Tsup)
{
    return K >= 2 && K <= 4 && V >= 2 && K * K + K * V <= 64 && Tsup >= 0 && Tsup <= T && T >= 1 &&
           T - Tsup <= kHmmMaxUnobserved;
}
// One wave per chain; a.data.D = hmm_dim(K, V), the other data fields unused.
hipError_t launch_hmm_sampler(const SamplerArgs& a, const HmmView& hv, hipStream_t stream);
hipError_t launch_hmm_sampler_ext(const SamplerArgs& a, const HmmView& hv, hipStream_t stream);
// U and grad U at n positions Q [n][D]: out_U [n], out_grad [n][D].
hipError_t launch_hmm_potential(const HmmView& hv, const double* Q, int64_t n, double* out_U, double* out_grad,
                                hipStream_t stream);

}  // namespace nuts
