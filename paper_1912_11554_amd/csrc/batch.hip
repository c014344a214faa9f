// Batched chains on shared fp32 data (the many-chain case): the potential
// and gradient of up to 128 positions per tile as one fused pass of matrix
// products over X, and the persistent sampler that drives 128 chains per tile
// with it, one leapfrog step of every chain per pass.
#include "batch.h"
#include "sampler_impl.h"

namespace nuts {

// ---------------------------------------------------------------------------
// Layout conversion: column blocks (fp32, one data set) -> 64-row stages.

__global__ void __launch_bounds__(256) to_batch_kernel(const float* __restrict__ Xb, const uint8_t* __restrict__ yb,
                                                       int R, int64_t N, int D, int kt, float* __restrict__ X,
                                                       uint8_t* __restrict__ y, int stride, int64_t ns)
{
    const int kp = batch_kp(kt);
    const int64_t per_stage = (int64_t)kBatchStageRows * stride;
    const int64_t total = ns * per_stage;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int64_t st = o / per_stage;
        const int64_t rem = o - st * per_stage;
        const int r = (int)(rem / stride);
        const int c = (int)(rem - (int64_t)r * stride);
        const int64_t i = st * kBatchStageRows + r;
        // slot c: permuted matrix-core columns, then the tail
        int col;
        if (c < 16 * kp) {
            const int t = c % kp;
            col = t < kt ? 16 * t + c / kp : D;
        } else {
            col = 16 * kt + (c - 16 * kp);
        }
        float v = 0.0f;
        if (i < N && col < D) v = Xb[((i / R) * D + col) * R + (i % R)];
        X[o] = v;
        if (c == 0) y[i] = i < N ? yb[i] : (uint8_t)0;
    }
}

hipError_t launch_to_batch_layout(const DataView& src, const BatchView& dst, float* X, uint8_t* y,
                                  hipStream_t stream)
{
    const int64_t total = dst.ns * kBatchStageRows * dst.stride;
    if (total == 0) return hipSuccess;
    const int64_t want = (total + 255) / 256;
    const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(to_batch_kernel, dim3(grid), dim3(256), 0, stream, (const float*)src.X, src.y,
                       rows_per_block(src), src.N, src.D, dst.kt, X, y, dst.stride, dst.ns);
    return hipGetLastError();
}

namespace {

using batch::WaveAcc;
using batch::WaveQ;

// Store a wave's partial row for its 16 positions: G columns from the
// matrix-core accumulators, the tail columns and the loss from the lanes of
// the first row group.  ATOMIC selects agent-scope stores (read by other
// groups of the same launch).
// Buffer resource word 3 for raw dword access on gfx9-family devices, and the
// cache-policy operand of a buffer access at agent scope (the sc1 bit: the
// access is coherent across the device's L2 caches, as an agent-scope atomic
// load or store is).  Buffer accesses give 16-byte agent-scope transfers,
// which the atomic builtins (8 bytes at most) do not.
constexpr int kBufferWord3 = 0x00020000;
constexpr int kCachePolicyAgent = 16;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void* base)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff, kBufferWord3);
}

template <bool ATOMIC>
__device__ __forceinline__ void put_f(float* p, float v)
{
    if constexpr (ATOMIC) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else *p = v;
}
template <bool ATOMIC>
__device__ __forceinline__ void put_d(double* p, double v)
{
    if constexpr (ATOMIC) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else *p = v;
}
template <int KT, bool ATOMIC>
__device__ __forceinline__ void store_partials(const BatchView& bv, WaveAcc& acc, int widx, int pw, float* P,
                                               double* L)
{
    const int l = lane();
    const int m = l & 15;
    const int jj = l >> 4;
    batch::reduce_position(acc);
    const int slot = widx * 16 + m;
    float* row = P + (int64_t)slot * pw;
#pragma unroll
    for (int mt = 0; mt < KT; ++mt) {
        // 16-byte aligned: pw and 4 jj are multiples of 4
        if constexpr (ATOMIC)
            __builtin_amdgcn_raw_buffer_store_b128(acc.g[mt], buffer_of(row), (16 * mt + 4 * jj) * 4, 0,
                                                   kCachePolicyAgent);
        else
            *reinterpret_cast<batch::v4f*>(row + 16 * mt + 4 * jj) = acc.g[mt];
    }
    if (jj == 0) {
#pragma unroll
        for (int k = 0; k < batch::kTail; ++k)
            if (k < bv.tc) put_f<ATOMIC>(row + 16 * KT + k, acc.gt[k]);
        put_d<ATOMIC>(L + slot, acc.loss);
    }
}

// ---------------------------------------------------------------------------
// Stand-alone batched potential: pass 1 on a grid of (groups, tiles), pass 2
// adds the partial rows of each position in group order and the prior.

template <int KT>
__global__ void __launch_bounds__(batch::kWaves * kWave, 1) batch_pass_kernel(BatchView bv, const double* __restrict__ W,
                                                                              int64_t K, int groups, int pw,
                                                                              float* __restrict__ P,
                                                                              double* __restrict__ L)
{
    __shared__ __align__(16) float xs[2 * batch::kStageBuf];
    __shared__ __align__(16) float ys[2 * kBatchStageRows];
    const int l = lane();
    const int m = l & 15;
    const int jj = l >> 4;
    const int widx = threadIdx.x / kWave;
    const int g = blockIdx.x;
    const int t = blockIdx.y;
    const int D = bv.D;
    const int64_t pos = (int64_t)t * kBatchTileChains + widx * 16 + m;
    const bool live = pos < K;

    WaveQ Q;
    constexpr int KP = batch::Geo<KT>::KP;
#pragma unroll
    for (int t = 0; t < KP; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int col = batch::e_column<KT>(t, jj, i);
            const bool used = (col / 16) < KT && col < D;
            Q.q[4 * t + i] = (live && used) ? (float)W[pos * D + col] : 0.0f;
        }
#pragma unroll
    for (int k = 0; k < batch::kTail; ++k)
        Q.qt[k] = (live && k < bv.tc) ? (float)W[pos * D + 16 * KT + k] : 0.0f;

    WaveAcc acc;
    batch::zero(acc);
    int64_t h0, h1;
    batch::group_halves(bv.ns, g, groups, &h0, &h1);
    batch::stage_loop<KT, true>(bv, h0, h1, (int)threadIdx.x, xs, ys, Q, acc);
    const int64_t base = (int64_t)t * groups + g;
    store_partials<KT, false>(bv, acc, widx, pw, P + base * kBatchTileChains * pw, L + base * kBatchTileChains);
}

constexpr int kFinishWaves = 4;

__global__ void __launch_bounds__(kFinishWaves * kWave) batch_finish_kernel(int D, int groups, int pw, int npad,
                                                                           const double* __restrict__ W,
                                                                           const float* __restrict__ P,
                                                                           const double* __restrict__ L,
                                                                           double prior_scale,
                                                                           double* __restrict__ out_U,
                                                                           double* __restrict__ out_grad)
{
    extern __shared__ double red[];  // [kFinishWaves][pw + 64]
    const int l = lane();
    const int wave = threadIdx.x / kWave;
    const int64_t k = blockIdx.x;
    const int64_t t = k / kBatchTileChains;
    const int slot = (int)(k % kBatchTileChains);
    const int rw = pw + 64;
    const int64_t rstride = (int64_t)kBatchTileChains * pw;
    const float* src = P + t * groups * rstride + (int64_t)slot * pw;
    const double* lsrc = L + t * groups * kBatchTileChains + slot;
    for (int col = l; col < pw; col += 64) {
        double s = 0.0;
        if (col < D) {
            // eight groups' loads in flight at a time, added in group order
            constexpr int U = 8;
            int g = wave;
            for (; g + (U - 1) * kFinishWaves < groups; g += U * kFinishWaves) {
                float v[U];
#pragma unroll
                for (int u = 0; u < U; ++u) v[u] = src[(int64_t)(g + u * kFinishWaves) * rstride + col];
#pragma unroll
                for (int u = 0; u < U; ++u) s += (double)v[u];
            }
            for (; g < groups; g += kFinishWaves) s += (double)src[(int64_t)g * rstride + col];
        }
        red[wave * rw + col] = s;
    }
    // loss partials: lane l of wave w takes groups w + 4 l, w + 4 (l + 64), ...
    double ls = 0.0;
    for (int g = wave + kFinishWaves * l; g < groups; g += kFinishWaves * 64) ls += lsrc[(int64_t)g * kBatchTileChains];
    ls = wave_sum(ls);
    if (l == 0) red[wave * rw + pw] = ls;
    __syncthreads();
    if (wave != 0) return;
    const double inv_s2 = 1.0 / (prior_scale * prior_scale);
    double pr = 0.0;
    for (int col = l; col < D; col += 64) {
        double tot = 0.0;
#pragma unroll
        for (int w = 0; w < kFinishWaves; ++w) tot += red[w * rw + col];
        const double w = W[k * D + col];
        pr += 0.5 * w * w * inv_s2;
        out_grad[k * D + col] = tot + w * inv_s2;
    }
    const double prior = wave_sum(pr);
    if (l == 0) {
        double loss = 0.0;
        for (int w = 0; w < kFinishWaves; ++w) loss += red[w * rw + pw];
        loss -= (double)npad * (double)batch::kLn2f;  // padding rows of the last stage
        out_U[k] = loss + prior + (double)D * (log(prior_scale) + sampler::kHalfLog2Pi);
    }
}

}  // namespace

BatchPlan plan_batch_potential(const BatchView& bv, int64_t K, int num_cu)
{
    BatchPlan p;
    p.tiles = (int)((K + kBatchTileChains - 1) / kBatchTileChains);
    // one group per CU (a group's two LDS stages take most of a CU's LDS)
    int64_t g = (int64_t)num_cu / p.tiles;
    if (g > bv.ns) g = bv.ns;
    if (g < 1) g = 1;
    p.groups = (int)g;
    p.pw = 64 * ((bv.D + 63) / 64);
    return p;
}

namespace {

template <int KT>
void enqueue_batch_pass(const BatchView& bv, const double* W, int64_t K, const BatchPlan& plan, float* P, double* L,
                        hipStream_t stream)
{
    hipLaunchKernelGGL(batch_pass_kernel<KT>, dim3(plan.groups, plan.tiles), dim3(batch::kWaves * kWave), 0, stream,
                       bv, W, K, plan.groups, plan.pw, P, L);
}

}  // namespace

hipError_t launch_batch_potential(const BatchView& bv, double prior_scale, const double* W, int64_t K,
                                  const BatchPlan& plan, float* P, double* L, double* out_U, double* out_grad,
                                  hipStream_t stream)
{
    switch (bv.kt) {
    case 0: enqueue_batch_pass<0>(bv, W, K, plan, P, L, stream); break;
    case 1: enqueue_batch_pass<1>(bv, W, K, plan, P, L, stream); break;
    case 2: enqueue_batch_pass<2>(bv, W, K, plan, P, L, stream); break;
    case 3: enqueue_batch_pass<3>(bv, W, K, plan, P, L, stream); break;
    case 4: enqueue_batch_pass<4>(bv, W, K, plan, P, L, stream); break;
    case 5: enqueue_batch_pass<5>(bv, W, K, plan, P, L, stream); break;
    case 6: enqueue_batch_pass<6>(bv, W, K, plan, P, L, stream); break;
    case 7: enqueue_batch_pass<7>(bv, W, K, plan, P, L, stream); break;
    case 8: enqueue_batch_pass<8>(bv, W, K, plan, P, L, stream); break;
    default: return hipErrorInvalidValue;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(batch_finish_kernel, dim3((unsigned)K), dim3(kFinishWaves * kWave),
                       (size_t)kFinishWaves * (plan.pw + 64) * sizeof(double), stream, bv.D, plan.groups, plan.pw,
                       (int)(bv.ns * kBatchStageRows - bv.N), W, P, L, prior_scale, out_U, out_grad);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Log-likelihood over a batch of draws (fp32 matrix cores): one pass over X
// per tile of 128 draws computing E = X W^T, then per draw the negative log
// likelihood summed in fp64 (partial rows per group, added in group order by
// the finish kernel), and optionally per row the sum of sigmoid(eta) over
// the tile's live draws (one fp32 value per row and tile, added over tiles in
// fp64 in order).

namespace {

template <int KT, bool PRED, bool SAMPLE>
__global__ void __launch_bounds__(batch::kWaves * kWave, 1) batch_ll_kernel(BatchView bv, const double* __restrict__ W,
                                                                           int64_t S, int groups,
                                                                           double* __restrict__ L,
                                                                           float* __restrict__ Pr,
                                                                           uint8_t* __restrict__ Y, uint64_t seed)
{
    __shared__ __align__(16) float xs[2 * batch::kStageBuf];
    __shared__ __align__(16) float ys[2 * kBatchStageRows];
    __shared__ float rs[PRED ? 2 * batch::kWaves * kBatchStageRows : 1];
    const int l = lane();
    const int m = l & 15;
    const int jj = l >> 4;
    const int widx = threadIdx.x / kWave;
    const int g = blockIdx.x;
    const int t = blockIdx.y;
    const int D = bv.D;
    const int64_t pos = (int64_t)t * kBatchTileChains + widx * 16 + m;
    const bool live = pos < S;

    WaveQ Q;
    constexpr int KP = batch::Geo<KT>::KP;
#pragma unroll
    for (int c = 0; c < KP; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int col = batch::e_column<KT>(c, jj, i);
            const bool used = (col / 16) < KT && col < D;
            Q.q[4 * c + i] = (live && used) ? (float)W[pos * D + col] : 0.0f;
        }
#pragma unroll
    for (int k = 0; k < batch::kTail; ++k)
        Q.qt[k] = (live && k < bv.tc) ? (float)W[pos * D + 16 * KT + k] : 0.0f;

    double loss = 0.0;
    const int64_t st0 = (int64_t)g * bv.ns / groups;
    const int64_t st1 = (int64_t)(g + 1) * bv.ns / groups;
    batch::PredictOut po;
    po.y = (SAMPLE && live) ? Y + pos * bv.N : nullptr;
    po.seed = seed;
    po.s = (uint64_t)pos;
    po.N = bv.N;
    po.row0 = 0;
    batch::stage_loop_ll<KT, PRED, SAMPLE>(bv, st0, st1, (int)threadIdx.x, xs, ys, rs, Q, live ? 1.0f : 0.0f,
                                           loss, Pr + (int64_t)t * bv.ns * kBatchStageRows, po);
    // the four lanes of a position hold its four row groups
    loss += __shfl_xor(loss, 16);
    loss += __shfl_xor(loss, 32);
    if (jj == 0) L[((int64_t)t * groups + g) * kBatchTileChains + widx * 16 + m] = loss;
}

// ll[s] = -(sum over groups of the loss partials - the padding rows' ln 2).
__global__ void __launch_bounds__(64) batch_ll_finish_kernel(int64_t S, int groups, int npad,
                                                            const double* __restrict__ L,
                                                            double* __restrict__ out_ll)
{
    const int64_t s = (int64_t)blockIdx.x * 64 + threadIdx.x;
    if (s >= S) return;
    const int64_t t = s / kBatchTileChains;
    const double* src = L + t * groups * kBatchTileChains + s % kBatchTileChains;
    double tot = 0.0;
    for (int g = 0; g < groups; ++g) tot += src[(int64_t)g * kBatchTileChains];
    out_ll[s] = -(tot - (double)npad * (double)batch::kLn2f);
}

// pred_mean[i] = (sum over tiles of the row sums) / S.
__global__ void __launch_bounds__(256) batch_pred_kernel(int64_t N, int64_t rows, int tiles, int64_t S,
                                                        const float* __restrict__ Pr, double* __restrict__ out)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < N; i += (int64_t)gridDim.x * 256) {
        double tot = 0.0;
        for (int t = 0; t < tiles; ++t) tot += (double)Pr[(int64_t)t * rows + i];
        out[i] = tot / (double)S;
    }
}

template <int KT>
void enqueue_ll(const BatchView& bv, const double* W, int64_t S, int tiles, int groups, double* L, float* Pr,
                bool pred, uint8_t* Y, uint64_t seed, hipStream_t stream)
{
    const dim3 grid(groups, tiles), block(batch::kWaves * kWave);
    if (Y)
        hipLaunchKernelGGL((batch_ll_kernel<KT, false, true>), grid, block, 0, stream, bv, W, S, groups, L, Pr, Y,
                           seed);
    else if (pred)
        hipLaunchKernelGGL((batch_ll_kernel<KT, true, false>), grid, block, 0, stream, bv, W, S, groups, L, Pr, Y,
                           seed);
    else
        hipLaunchKernelGGL((batch_ll_kernel<KT, false, false>), grid, block, 0, stream, bv, W, S, groups, L, Pr, Y,
                           seed);
}

}  // namespace

hipError_t launch_batch_log_likelihood(const BatchView& bv, const double* W, int64_t S, const BatchPlan& plan,
                                       double* L, float* Pr, double* out_ll, double* out_pred, uint8_t* out_y,
                                       uint64_t seed, hipStream_t stream)
{
    const bool pred = out_pred != nullptr;
#define NUTS_LL_CASE(k)                                                                         \
    case k: enqueue_ll<k>(bv, W, S, plan.tiles, plan.groups, L, Pr, pred, out_y, seed, stream); break;
    switch (bv.kt) {
        NUTS_LL_CASE(0) NUTS_LL_CASE(1) NUTS_LL_CASE(2) NUTS_LL_CASE(3) NUTS_LL_CASE(4) NUTS_LL_CASE(5)
        NUTS_LL_CASE(6) NUTS_LL_CASE(7) NUTS_LL_CASE(8)
    default: return hipErrorInvalidValue;
    }
#undef NUTS_LL_CASE
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (out_y) return hipSuccess;  // the predictive samples only
    hipLaunchKernelGGL(batch_ll_finish_kernel, dim3((unsigned)((S + 63) / 64)), dim3(64), 0, stream, S, plan.groups,
                       (int)(bv.ns * kBatchStageRows - bv.N), L, out_ll);
    e = hipGetLastError();
    if (e != hipSuccess || !pred) return e;
    const int64_t want = (bv.N + 255) / 256;
    hipLaunchKernelGGL(batch_pred_kernel, dim3((unsigned)(want < 4096 ? want : 4096)), dim3(256), 0, stream, bv.N,
                       bv.ns * kBatchStageRows, plan.tiles, S, Pr, out_pred);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Persistent batched sampler.
//
// Tile t holds chain slots 0..127 and `groups` workgroups; group i of the
// tile runs the tree logic of slot i (if i < 128) in its wave 0 and the
// matrix-core pass over its stage range in waves 1..8.  A step s of the tile:
//   1. every slot's controller publishes its next position Q(s) (fp32) and
//      then stamp[slot] = s + 1; a slot with no iterations left first sets
//      done_at[slot] = s (once) and publishes zeros;
//   2. each group's wave 0 waits until all 128 stamps of the tile are > s;
//      if every done_at of the tile is <= s, the tile stops;
//   3. the workers compute the group's partial rows for all 128 positions
//      and store them; the group counts itself in at tile_count[t];
//   4. once the count reaches (s + 1) * groups, the group hosting slot i adds
//      the groups' partial rows of slot i in group order (all nine waves,
//      then in wave order) and hands U and grad U to its controller.
// Tiles never wait for each other.  Buffers alternate with the parity of s;
// a buffer of parity s & 1 is rewritten only at step s + 2, after every
// controller of the tile has consumed step s + 1 (stamps of s + 2 are out),
// hence after every reader of step s is done.  stamp only grows and done_at
// is written once, so every group reads the same stop decision at every step.

namespace {

constexpr int kGroupWaves = 1 + batch::kWaves;
constexpr int kCmdEval = 1, kCmdStop = 2, kCmdError = 3;

template <int DPL>
struct BatchShared {
    __align__(16) float xs[2 * batch::kStageBuf];
    __align__(16) float ys[2 * kBatchStageRows];
    double red[kGroupWaves][(DPL + 1) * 64];
    int cmd;
};

struct BatchCtx {
    BatchView bv;
    int tiles, groups;
    int t, i;  // this group's tile and index in the tile
    int64_t h0, h1;  // this group's halves of stages (group_halves)
    int pw;
    float* qbuf;
    float* P;
    double* L;
    BatchSync* sync;
};

__device__ __forceinline__ unsigned long long load_u64(const unsigned long long* p)
{
    return __hip_atomic_load(const_cast<unsigned long long*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_u64(unsigned long long* p, unsigned long long v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

constexpr uint64_t kWaitTicks = 1000000000ull;  // ~10 s of the 100 MHz real-time counter

__device__ __forceinline__ bool error_set(const BatchCtx& c)
{
    return __hip_atomic_load(&c.sync->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
}
__device__ __forceinline__ void raise_error(const BatchCtx& c)
{
    if (lane() == 0) __hip_atomic_store(&c.sync->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Slot of column `col` in a published position: the matrix-core operand
// order of the column contraction, lane group jj's 4 KP values contiguous
// (Q.q of load_q), so that a worker lane reads its share with 16-byte loads;
// the four tail columns after the 16 KP permuted ones.  Columns of chunks
// past KT have a slot and hold zero.
template <int KT>
__device__ __forceinline__ int q_slot(int col)
{
    constexpr int KP = batch::Geo<KT>::KP;
    const int c = col >> 4, g = col & 15;
    const int i = c & 3, h = c >> 2;
    const int f = KP == 8 ? 2 * g + h : g;
    return (f & 3) * 4 * KP + (f >> 2) * 4 + i;
}

template <int KT, int DPL>
__device__ void publish(const BatchCtx& c, unsigned long long step, const double (&q)[DPL], bool mark_done)
{
    constexpr int KP = batch::Geo<KT>::KP;
    const int l = lane();
    const int par = (int)(step & 1);
    const int64_t slot = (int64_t)c.t * kBatchTileChains + c.i;
    float* dst = c.qbuf + ((int64_t)par * c.tiles * kBatchTileChains + slot) * kBatchQWidth;
#pragma unroll
    for (int m = 0; m < kBatchQWidth / 64; ++m) {
        const int col = l + 64 * m;
        float v = 0.0f;
        if (m < DPL && col < c.bv.D) v = (float)q[m < DPL ? m : 0];
        if (col < 16 * KP)
            __hip_atomic_store(dst + q_slot<KT>(col), (col >> 4) < KT ? v : 0.0f, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        if (col >= 16 * KT && col < 16 * KT + batch::kTail)
            __hip_atomic_store(dst + 16 * KP + (col - 16 * KT), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    sampler::drain_memory_ops();
    if (mark_done) {
        if (l == 0) store_u64(&c.sync->done_at[slot], step);
        sampler::drain_memory_ops();
    }
    if (l == 0) store_u64(&c.sync->stamp[slot], step + 1);
}

// Wave 0: wait for the tile's positions of step s; returns the command.
__device__ int wait_positions(const BatchCtx& c, unsigned long long step)
{
    const int l = lane();
    const unsigned long long* st = c.sync->stamp + (int64_t)c.t * kBatchTileChains;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    bool a = false, b = false;
    for (;;) {
        if (!a) a = load_u64(st + l) > step;
        if (!b) b = load_u64(st + 64 + l) > step;
        if (__all(a && b)) break;
        if (error_set(c)) return kCmdError;
        if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) {
            raise_error(c);
            return kCmdError;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    const unsigned long long* da = c.sync->done_at + (int64_t)c.t * kBatchTileChains;
    const bool done = load_u64(da + l) <= step && load_u64(da + 64 + l) <= step;
    return __all(done) ? kCmdStop : kCmdEval;
}

// Wave 0: count the group in for step s and wait for the rest of the tile.
__device__ bool arrive_and_wait(const BatchCtx& c, unsigned long long step)
{
    unsigned long long* cnt = &c.sync->tile_count[c.t][0];
    if (lane() == 0) __hip_atomic_fetch_add(cnt, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned long long target = (step + 1) * (unsigned long long)c.groups;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    for (;;) {
        if (load_u64(cnt) >= target) return true;
        if (error_set(c)) return false;
        if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) {
            raise_error(c);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// One step of the tile for this group, executed by all nine waves with the
// same workgroup barriers.  LEADER is wave 0.  Returns the command; for the
// leader of a hosting group, `out` receives the sums for its slot: component
// m of lane l is column l + 64 m of X^T r, component DPL of lane 0 the loss.
template <int KT, int DPL, bool LEADER>
__device__ int batch_collective(const BatchCtx& c, BatchShared<DPL>& sh, unsigned long long step,
                                const double (&q)[DPL], bool publish_q, bool mark_done, double (&out)[DPL + 1])
{
    const int l = lane();
    const int wave = threadIdx.x / kWave;
    const int par = (int)(step & 1);
    const bool host = c.i < kBatchTileChains;
    if (LEADER) {
        if (publish_q && host) publish<KT, DPL>(c, step, q, mark_done);
        const int cmd = wait_positions(c, step);
        if (l == 0) sh.cmd = cmd;
    }
    __syncthreads();  // command out
    const int cmd = sh.cmd;
    if (cmd != kCmdEval) return cmd;

    const int64_t tile_base = ((int64_t)par * c.tiles + c.t) * c.groups;
    const int64_t rstride = (int64_t)kBatchTileChains * c.pw;
    if (LEADER) {
        WaveQ Q;
        WaveAcc acc;
        batch::stage_loop<KT, false>(c.bv, c.h0, c.h1, 0, sh.xs, sh.ys, Q, acc);
    } else {
        const int widx = wave - 1;
        const int m = l & 15;
        const int jj = l >> 4;
        const float* qsrc = c.qbuf + ((int64_t)par * c.tiles * kBatchTileChains +
                                      (int64_t)c.t * kBatchTileChains + widx * 16 + m) * kBatchQWidth;
        // the position in the order publish wrote it: this lane's 4 KP
        // operand values, then the tail, in 16-byte agent-scope loads
        WaveQ Q;
        constexpr int KP = batch::Geo<KT>::KP;
        const __amdgpu_buffer_rsrc_t qr = buffer_of(qsrc);
#pragma unroll
        for (int t = 0; t < KP; ++t) {
            const batch::v4f v = __builtin_amdgcn_raw_buffer_load_b128(qr, (jj * 4 * KP + 4 * t) * 4, 0,
                                                                       kCachePolicyAgent);
#pragma unroll
            for (int i = 0; i < 4; ++i) Q.q[4 * t + i] = v[i];
        }
        const batch::v4f tv = __builtin_amdgcn_raw_buffer_load_b128(qr, 16 * KP * 4, 0, kCachePolicyAgent);
#pragma unroll
        for (int k = 0; k < batch::kTail; ++k) Q.qt[k] = tv[k];
        WaveAcc acc;
        batch::zero(acc);
        batch::stage_loop<KT, true, true>(c.bv, c.h0, c.h1, (int)threadIdx.x - kWave, sh.xs, sh.ys, Q, acc);
        store_partials<KT, true>(c.bv, acc, widx, c.pw, c.P + (tile_base + c.i) * rstride,
                                 c.L + (tile_base + c.i) * kBatchTileChains);
        sampler::drain_memory_ops();
    }
    __syncthreads();  // the group's partial rows are out
    if (LEADER) {
        const bool ok = arrive_and_wait(c, step);
        if (l == 0) sh.cmd = ok ? kCmdEval : kCmdError;
    }
    __syncthreads();  // every group of the tile is in
    const int status = sh.cmd;
    if (LEADER && host) {
        // the leader keeps its registers for the tree state (sixteen loads in
        // flight would push it into scratch memory): its row of sums is zero
#pragma unroll
        for (int mm = 0; mm <= DPL; ++mm) sh.red[0][mm * 64 + l] = 0.0;
    } else if (host) {
        // this worker's share of the groups, in group order
        const float* src = c.P + tile_base * rstride + (int64_t)c.i * c.pw;
        const double* lsrc = c.L + tile_base * kBatchTileChains + c.i;
        // Lane l adds columns 4 l .. 4 l + 3 with 16-byte loads at agent
        // scope (buffer loads with the sc1 bit); every load of a wave's share
        // in flight at once: one round trip for up to 16 groups per wave (128
        // groups of the 8 workers); a group past the last re-reads the wave's
        // first group and is not added.  (4-byte loads of the same rows took three
        // times as long: the gather is bound by the count of uncached
        // requests, not by bytes.)
        const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float*>(src), (short)0, 0x7fffffff, kBufferWord3);
        const int nl = (c.bv.D + 3) / 4;
        const int lc = l < nl ? l : nl - 1;
        double s4[4] = {0.0, 0.0, 0.0, 0.0};
        double sl = 0.0;
        constexpr int B = 16;
        constexpr int NWK = kGroupWaves - 1;  // the workers
        for (int g0 = wave - 1; g0 < c.groups; g0 += B * NWK) {
            batch::v4f v[B];
            double lv[B];
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const int gg = g0 + b * NWK;
                const int gq = gg < c.groups ? gg : g0;
                v[b] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)((gq * rstride + 4 * lc) * 4), 0, kCachePolicyAgent);
                lv[b] = l == 0 ? sampler::load_shared(lsrc + (int64_t)gq * kBatchTileChains) : 0.0;
            }
#pragma unroll
            for (int b = 0; b < B; ++b) {
                if (g0 + b * NWK < c.groups) {
#pragma unroll
                    for (int k = 0; k < 4; ++k) s4[k] += (double)v[b][k];
                    sl += lv[b];
                }
            }
        }
        // column c at sh.red[wave][c] (component c / 64 of lane c % 64), the
        // loss at (DPL) * 64; columns from D on hold zero
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int col = 4 * l + k;
            if (l < nl) sh.red[wave][col] = col < c.bv.D ? s4[k] : 0.0;
        }
        for (int col = 4 * nl + l; col < DPL * 64; col += 64) sh.red[wave][col] = 0.0;
        sh.red[wave][DPL * 64 + l] = l == 0 ? sl : 0.0;
    }
    __syncthreads();  // per-wave sums in LDS
    if (LEADER && host) {
#pragma unroll
        for (int mm = 0; mm <= DPL; ++mm) {
            double tot = 0.0;
#pragma unroll
            for (int w = 0; w < kGroupWaves; ++w) tot += sh.red[w][mm * 64 + l];
            out[mm] = tot;
        }
        // padding rows of the last stage
        out[DPL] -= (double)(c.bv.ns * kBatchStageRows - c.bv.N) * (double)batch::kLn2f;
    }
    // a failed exchange ends the chain; the workers stay in step until the
    // leader's next call hands them the stop at the first barrier
    return LEADER ? status : kCmdEval;
}

template <int KT, int DPL, bool EXT>
struct BatchEval {
    static constexpr bool kSpeculative = false;
    // the edge and proposal nodes in LDS where the kernel without the
    // extended features has the room (see EdgeNodes and batch_edge_nodes)
    static constexpr bool kNodesInLds = DPL >= 3 && !EXT;
    BatchCtx c;
    BatchShared<DPL>* sh;
    double inv_s2, prior_const;
    unsigned long long step;
    bool abort;

    __device__ bool s_writer() const { return true; }
    __device__ bool out_writer() const { return true; }
    __device__ bool aborted() const { return abort; }

    __device__ void eval(const double (&q)[DPL], double& U, double (&g)[DPL])
    {
        double r[DPL + 1];
        const int cmd = batch_collective<KT, DPL, true>(c, *sh, step, q, true, false, r);
        step++;
        const int l = lane();
        if (cmd != kCmdEval) {
            abort = true;
            U = 0.0;
#pragma unroll
            for (int m = 0; m < DPL; ++m) g[m] = 0.0;
            return;
        }
        double pr = 0.0;
#pragma unroll
        for (int m = 0; m < DPL; ++m) pr += 0.5 * q[m] * q[m] * inv_s2;
        const double prior = wave_sum(pr);
        U = readlane_f64(r[DPL], 0) + prior + prior_const;
#pragma unroll
        for (int m = 0; m < DPL; ++m) g[m] = (l + 64 * m < c.bv.D) ? r[m] + q[m] * inv_s2 : 0.0;
    }

    // Keep the tile's steps going with zero positions until every slot of the
    // tile is finished (or an exchange failed).
    __device__ void finish(bool publish_q)
    {
        double q[DPL], r[DPL + 1];
#pragma unroll
        for (int m = 0; m < DPL; ++m) q[m] = 0.0;
        bool first = true;
        for (;;) {
            const int cmd = batch_collective<KT, DPL, true>(c, *sh, step, q, publish_q, first, r);
            first = false;
            step++;
            if (cmd != kCmdEval) break;
        }
    }
};

template <int KT, int DPL, bool EXT>
__global__ void __launch_bounds__(kGroupWaves * kWave, 1) sampler_batch_kernel(SamplerArgs A, BatchView bv,
                                                                              int tiles, int groups, float* qbuf,
                                                                              float* P, double* L,
                                                                              BatchSync* sync)
{
    extern __shared__ double lds[];  // the controller's checkpoint array
    __shared__ BatchShared<DPL> sh;
    BatchCtx c;
    c.bv = bv;
    c.tiles = tiles;
    c.groups = groups;
    c.t = (int)(blockIdx.x / groups);
    c.i = (int)(blockIdx.x % groups);
    batch::group_halves(bv.ns, c.i, groups, &c.h0, &c.h1);
    c.pw = 64 * DPL;
    c.qbuf = qbuf;
    c.P = P;
    c.L = L;
    c.sync = sync;
    const int wave = threadIdx.x / kWave;
    if (wave == 0) {
        BatchEval<KT, DPL, EXT> ev;
        ev.c = c;
        ev.sh = &sh;
        ev.inv_s2 = 1.0 / (A.prior_scale * A.prior_scale);
        ev.prior_const = (double)bv.D * (log(A.prior_scale) + sampler::kHalfLog2Pi);
        ev.step = 0;
        ev.abort = false;
        const int64_t chain = (int64_t)c.t * kBatchTileChains + c.i;
        const bool host = c.i < kBatchTileChains;
        if (host && chain < A.num_chains) sampler::run_chain<DPL, EXT>(A, ev, chain, lds);
        ev.finish(host);
    } else {
        double q[DPL], r[DPL + 1];
#pragma unroll
        for (int m = 0; m < DPL; ++m) q[m] = 0.0;
        for (unsigned long long step = 0;; ++step)
            if (batch_collective<KT, DPL, false>(c, sh, step, q, false, false, r) != kCmdEval) break;
    }
}

// Kernel for a shape: KT chunks (0..8) and DPL = ceil(D / 64) (1..3); the
// pairs that occur for D <= 132; EXT compiles the warmup step-size
// adaptation in.
template <bool EXT>
const void* batch_kernel_for_t(const BatchView& bv)
{
    const int dpl = (bv.D + 63) / 64;
    switch (bv.kt * 4 + dpl) {
    case 0 * 4 + 1: return (const void*)sampler_batch_kernel<0, 1, EXT>;
    case 1 * 4 + 1: return (const void*)sampler_batch_kernel<1, 1, EXT>;
    case 2 * 4 + 1: return (const void*)sampler_batch_kernel<2, 1, EXT>;
    case 3 * 4 + 1: return (const void*)sampler_batch_kernel<3, 1, EXT>;
    case 4 * 4 + 1: return (const void*)sampler_batch_kernel<4, 1, EXT>;
    case 4 * 4 + 2: return (const void*)sampler_batch_kernel<4, 2, EXT>;
    case 5 * 4 + 2: return (const void*)sampler_batch_kernel<5, 2, EXT>;
    case 6 * 4 + 2: return (const void*)sampler_batch_kernel<6, 2, EXT>;
    case 7 * 4 + 2: return (const void*)sampler_batch_kernel<7, 2, EXT>;
    case 8 * 4 + 2: return (const void*)sampler_batch_kernel<8, 2, EXT>;
    case 8 * 4 + 3: return (const void*)sampler_batch_kernel<8, 3, EXT>;
    default: return nullptr;
    }
}

const void* batch_kernel_for(const BatchView& bv, bool adapt)
{
    return adapt ? batch_kernel_for_t<true>(bv) : batch_kernel_for_t<false>(bv);
}

size_t batch_sampler_lds(const SamplerArgs& a)
{
    return (size_t)chain_lds_doubles(a.data.D, a.max_depth, a.sub_merge,
                                     batch_edge_nodes(a.data.D, sampler_extended(a))) *
           sizeof(double);
}

}  // namespace

bool batch_sampler_supported(const BatchView& bv, int max_depth, int sub_merge, int num_cu)
{
    if (bv.D > 64 * 3 || num_cu < kBatchTileChains) return false;
    int per_cu = 0;
    const size_t lds =
        (size_t)chain_lds_doubles(bv.D, max_depth, sub_merge, batch_edge_nodes(bv.D, sub_merge != 0)) * sizeof(double);
    const void* k = batch_kernel_for(bv, sub_merge != 0);
    if (!k) return false;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, kGroupWaves * kWave, lds) != hipSuccess) return false;
    return per_cu >= 1;
}

hipError_t launch_sampler_batch(const SamplerArgs& a, const BatchView& bv, int tiles, int groups, float* qbuf,
                                float* P, double* L, BatchSync* sync, hipStream_t stream, hipEvent_t at_launch)
{
    hipError_t e = hipMemsetAsync(sync, 0, sizeof(BatchSync), stream);
    if (e != hipSuccess) return e;
    e = hipMemsetAsync(sync->done_at, 0xFF, sizeof(sync->done_at), stream);
    if (e != hipSuccess) return e;
    SamplerArgs A = a;
    BatchView B = bv;
    void* args[] = {&A, &B, &tiles, &groups, &qbuf, &P, &L, &sync};
    const void* k = batch_kernel_for(bv, sampler_extended(a));
    if (!k) return hipErrorInvalidValue;
    e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)batch_sampler_lds(a));
    if (e != hipSuccess) return e;
    if (at_launch) {
        e = hipEventRecord(at_launch, stream);
        if (e != hipSuccess) return e;
    }
    return hipLaunchCooperativeKernel(k, dim3((unsigned)(tiles * groups)),
                                      dim3(kGroupWaves * kWave), args, (unsigned)batch_sampler_lds(a), stream);
}

}  // namespace nuts
