// Device side of the batched-chain contraction on the gfx950 matrix cores.
//
// One workgroup owns a range of 64-row stages and a tile of 128 positions
// (chains).  Eight waves each take 16 positions; the stage rows are staged in
// LDS once and read by all eight.  Per 16-row tile a wave computes
//   E[16 rows x 16 positions] = X_tile . Q          (v_mfma_f32_16x16x4f32,
//                                                     contraction over columns)
//   loss and residual of every (row, position) on E
//   G[D x 16] += X_tile^T . R                       (contraction over rows)
// with G held in registers across the whole row range.
//
// Operand layout of v_mfma_f32_16x16x4f32 (one 16x16 block): lane l gives
// A[l % 16][l / 16] and B[l / 16][l % 16]; result register r of lane l is
// C[4 (l / 16) + r][l % 16].  The contraction index of instruction (chunk t,
// sub-step i) is column 16 t + 4 (l / 16) + i, so that each lane reads four
// consecutive columns of its row with one 16-byte LDS load.  For G the
// contraction index of sub-step r is row 4 (l / 16) + r: exactly the rows whose
// residuals the lane already holds in register r of the E result, so R feeds
// the second product without any data movement.
//
// Precision: X and Q are fp32 and products accumulate in fp32 inside the
// matrix cores; the row terms use the fp32 hardware exp/log/rcp; the loss is
// accumulated in fp64 per lane and all partial rows are added in fp64 in a
// fixed order.
#pragma once

#include "device.h"
#include "launch.h"

namespace nuts {
namespace batch {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;                                   // matrix-core waves per group
constexpr int kTileRows = 16;
constexpr int kTiles = kBatchStageRows / kTileRows;         // MFMA tiles per stage
constexpr int kTail = 4;
constexpr int kMaxStride = 16 * kBatchMaxKT + kTail;        // 132 floats per row in HBM

// LDS geometry of a stage for KT chunks.  The HBM row (16 KP permuted
// matrix-core slots, then the tail) is spread out so that column residue g
// starts at g * GS: GS = 12 for KP = 8 (two 16-byte pieces per residue) and
// 4 for KP = 4, and the row stride RS = 16 GS + 4 is 4 mod 64 floats.  With
// these, a 16-lane phase of every 16-byte LDS read below (16 rows at one
// residue, or 16 residues of one row) touches 64 distinct banks.
template <int KT>
struct Geo {
    static constexpr int KP = (KT + 3) / 4 * 4;
    static constexpr int GS = KP == 8 ? 12 : 4;
    static constexpr int RS = 16 * GS + 4;
    static constexpr int HS = 16 * KP + 4;          // HBM row: floats
    static constexpr int HV = HS / 4;               // HBM row: 16-byte pieces
};
constexpr int kStageFloats = kBatchStageRows * Geo<kBatchMaxKT>::RS;  // largest LDS stage
constexpr int kStageBuf = kStageFloats + 4;                          // plus one junk 16-byte slot
constexpr int kStageVecs = (kBatchStageRows * kMaxStride / 4 + kWaves * kWave - 1) / (kWaves * kWave);

// Column of the matrix-core operand that lane group jj reads as component i
// of its 16-byte piece in chunk t of the column contraction (E = X Q):
// piece f = 4 t + jj of the row is residue g, half h of the permuted slots.
template <int KT>
__host__ __device__ constexpr int e_column(int t, int jj, int i)
{
    constexpr int KP = Geo<KT>::KP;
    const int f = 4 * t + jj;
    const int g = KP == 8 ? f >> 1 : f;
    const int h = KP == 8 ? f & 1 : 0;
    return 16 * (4 * h + i) + g;   // chunk 4 h + i (valid if < KT), residue g
}

__device__ __forceinline__ v4f mfma(float a, float b, v4f c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Negative log-likelihood and residual of one (row, position) from eta in
// fp32, with sgn = 1 - 2y: t = sgn eta, loss = softplus(t) = max(t, 0) +
// ln 2 log2(1 + e), residual = sgn sigmoid(t), e = exp(-|t|); three
// transcendentals (exp2, log2, reciprocal) on the fp32 hardware units.  The
// rounding of 1 + e costs at most 2^-24 absolute per term (log1p accuracy is
// not needed for a sum of softplus values that are O(1) each).  Padding rows
// (zero X, y = 0) have eta = 0 exactly and add exactly ln 2 (in fp32) to the
// loss and nothing to the gradient; the caller subtracts them.
constexpr float kLn2f = 0.69314718055994531f;

__device__ __forceinline__ void row_terms(float eta, float sgn, float& loss, float& resid)
{
    const float t = sgn * eta;
    const float e = __builtin_amdgcn_exp2f(-fabsf(t) * 1.4426950408889634f);
    const float u = 1.0f + e;
    const float inv = __builtin_amdgcn_rcpf(u);
    loss = __builtin_fmaf(kLn2f, __builtin_amdgcn_logf(u), fmaxf(t, 0.0f));
    resid = sgn * ((t >= 0.0f ? 1.0f : e) * inv);
}

// A wave's share of the positions: Q in the B-operand order of the column
// contraction (q[4 t + i] = Q[e_column(t, l / 16, i)][l % 16], zero where
// that chunk is >= KT) and the tail.
struct WaveQ {
    float q[4 * kBatchMaxKT];
    float qt[kTail];
};

struct WaveAcc {
    v4f g[kBatchMaxKT];  // G[16 mt + 4 (l / 16) + r][l % 16] in g[mt][r]
    float gt[kTail];     // tail columns, this lane's rows only
    double loss;         // this lane's (row, position) terms
};

__device__ __forceinline__ void zero(WaveAcc& a)
{
#pragma unroll
    for (int mt = 0; mt < kBatchMaxKT; ++mt) a.g[mt] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int k = 0; k < kTail; ++k) a.gt[k] = 0.0f;
    a.loss = 0.0;
}

// Registers of one stage on its way from HBM to LDS; thread `tid` of the
// kWaves * 64 loaders moves 16-byte pieces tid, tid + 512, ...
struct StageRegs {
    v4f v[kStageVecs];  // clang vector type: HIP's float4 class would pin the registers to scratch
    uint32_t y;
};

// RECOMPUTE (the sampler kernel, whose nine waves leave 168 registers a
// lane): the piece offsets are recomputed at every stage.  Hoisted out of the
// stage loop they were kept in scratch memory there, and each reload waited
// for every load issued before it, so the stage's loads went out one by one.
// Kernels with registers to spare keep them (recomputing cost them time).
template <bool RECOMPUTE>
__device__ __forceinline__ void load_stage(const BatchView& bv, int64_t st, int tid, StageRegs& r)
{
    if constexpr (RECOMPUTE) {
        int opaque_zero;
        asm volatile("v_mov_b32 %0, 0" : "=v"(opaque_zero));
        tid += opaque_zero;
    }
    const int last = kBatchStageRows * bv.stride / 4 - 1;
    const v4f* src = reinterpret_cast<const v4f*>(bv.X + st * kBatchStageRows * bv.stride);
    const uint32_t* ysrc = reinterpret_cast<const uint32_t*>(bv.y + st * kBatchStageRows);
    // with RECOMPUTE the labels first: whatever their address waits for (a
    // register reloaded from scratch waits for every load before it) is then
    // not the stage's pieces
    if (RECOMPUTE && tid < kBatchStageRows / 4) r.y = ysrc[tid];
    // unconditional loads (pieces past the stage re-read its last piece and
    // are not stored), so the loop unrolls into straight-line code
#pragma unroll
    for (int i = 0; i < kStageVecs; ++i) r.v[i] = src[min(tid + i * kWaves * kWave, last)];
    if (!RECOMPUTE && tid < kBatchStageRows / 4) r.y = ysrc[tid];
}

// Scatter a stage into the LDS geometry: HBM piece q of a row goes to
// residue q / (KP / 4), half q % (KP / 4); the last piece is the tail.
// RECOMPUTE as for load_stage: the destinations are recomputed at every
// stage (a few integer instructions) instead of reloaded from scratch.
template <int KT, bool RECOMPUTE>
__device__ __forceinline__ void store_stage(const StageRegs& r, int tid, float* xs, float* ys)
{
    using G = Geo<KT>;
    constexpr int last = kBatchStageRows * G::HV - 1;
    if constexpr (RECOMPUTE) {
        int opaque_zero;
        asm volatile("v_mov_b32 %0, 0" : "=v"(opaque_zero));
        tid += opaque_zero;
    }
#pragma unroll
    for (int i = 0; i < kStageVecs; ++i) {
        const int idx = tid + i * kWaves * kWave;
        const int row = idx / G::HV;
        const int q = idx - row * G::HV;
        int dst;
        if constexpr (G::KP == 8) dst = q < 32 ? (q >> 1) * 3 + (q & 1) : 4 * G::GS;
        else dst = q < 4 * G::KP ? q : 4 * G::GS;  // KP = 4: one piece per residue
        dst += row * (G::RS / 4);
        // pieces past the stage go to a junk slot after the buffer (never read)
        reinterpret_cast<v4f*>(xs)[idx <= last ? dst : kStageFloats / 4] = r.v[i];
    }
    if (tid < kBatchStageRows / 4) {
        // labels as signs 1 - 2y
        v4f sg;
#pragma unroll
        for (int k = 0; k < 4; ++k) sg[k] = ((r.y >> (8 * k)) & 1u) ? -1.0f : 1.0f;
        reinterpret_cast<v4f*>(ys)[tid] = sg;
    }
}

// All four 16-row tiles of one LDS stage for this wave's 16 positions, two
// tiles at a time so that two independent accumulation chains alternate on
// the matrix core.  KT is the chunk count; the four tail slots are always
// processed (slots past the tail hold zero columns and zero positions, so
// they add nothing).
//
// `flip` reverses the pair order: the two waves that share a SIMD (loader
// index w and w + 4) take the pairs in opposite orders.  Each wave raises its
// issue priority while it feeds the matrix core and lowers it for the row
// terms: left to the default (the older wave first), the younger wave of a
// SIMD fell a third behind within each stage and the older one waited for it
// at the stage barrier.
template <int KT>
__device__ __forceinline__ void compute_stage(const float* __restrict__ xs, const float* __restrict__ ys,
                                              const WaveQ& Q, WaveAcc& acc, bool flip, int pair_lo, int pair_hi)
{
    using G = Geo<KT>;
    const int l = lane();
    const int m = l & 15;
    const int jj = l >> 4;
    // this lane's piece of chunk 0 in its E row, and its G residue
    const int e_off = m * G::RS + (G::KP == 8 ? 12 * (jj >> 1) + 4 * (jj & 1) : 4 * jj);
    constexpr int e_step = G::KP == 8 ? 24 : 16;
    const int g_off = 4 * jj * G::RS + m * G::GS;
#pragma unroll 1
    for (int step = 0; step < kTiles; step += 2) {
        const int tp = flip ? kTiles - 2 - step : step;
        if (tp / 2 < pair_lo || tp / 2 >= pair_hi) continue;  // uniform: another group's rows
        const float* x0 = xs + tp * kTileRows * G::RS;
        const float* x1 = x0 + kTileRows * G::RS;
        v4f e0 = {0.0f, 0.0f, 0.0f, 0.0f};
        v4f e1 = {0.0f, 0.0f, 0.0f, 0.0f};
        __builtin_amdgcn_s_setprio(2);
#pragma unroll
        for (int t = 0; t < G::KP; ++t) {
            const v4f a0 = *reinterpret_cast<const v4f*>(x0 + e_off + e_step * t);
            const v4f a1 = *reinterpret_cast<const v4f*>(x1 + e_off + e_step * t);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                e0 = mfma(a0[i], Q.q[4 * t + i], e0);
                e1 = mfma(a1[i], Q.q[4 * t + i], e1);
            }
        }
        __builtin_amdgcn_s_setprio(0);
        // tail slots of this lane's four rows 4 jj + r of both tiles
        v4f xr0[4], xr1[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            xr0[r] = *reinterpret_cast<const v4f*>(x0 + (4 * jj + r) * G::RS + 16 * G::GS);
            xr1[r] = *reinterpret_cast<const v4f*>(x1 + (4 * jj + r) * G::RS + 16 * G::GS);
            e0[r] += ((xr0[r][0] * Q.qt[0] + xr0[r][1] * Q.qt[1]) + xr0[r][2] * Q.qt[2]) + xr0[r][3] * Q.qt[3];
            e1[r] += ((xr1[r][0] * Q.qt[0] + xr1[r][1] * Q.qt[1]) + xr1[r][2] * Q.qt[2]) + xr1[r][3] * Q.qt[3];
        }
        const v4f s0 = *reinterpret_cast<const v4f*>(ys + tp * kTileRows + 4 * jj);
        const v4f s1 = *reinterpret_cast<const v4f*>(ys + (tp + 1) * kTileRows + 4 * jj);
        float r0[4], r1[4];
        float lsum = 0.0f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float l0, l1;
            row_terms(e0[r], s0[r], l0, r0[r]);
            row_terms(e1[r], s1[r], l1, r1[r]);
            lsum += l0 + l1;
        }
        acc.loss += (double)lsum;
        __builtin_amdgcn_s_setprio(2);
        // G: residue m of row 4 jj + r holds chunks 4 h .. 4 h + 3 in piece h
#pragma unroll
        for (int r = 0; r < 4; ++r) {
#pragma unroll
            for (int h = 0; h < G::KP / 4; ++h) {
                const v4f b0 = *reinterpret_cast<const v4f*>(x0 + g_off + r * G::RS + 4 * h);
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (4 * h + i < KT) acc.g[4 * h + i] = mfma(b0[i], r0[r], acc.g[4 * h + i]);
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
#pragma unroll
            for (int h = 0; h < G::KP / 4; ++h) {
                const v4f b1 = *reinterpret_cast<const v4f*>(x1 + g_off + r * G::RS + 4 * h);
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (4 * h + i < KT) acc.g[4 * h + i] = mfma(b1[i], r1[r], acc.g[4 * h + i]);
            }
        }
        __builtin_amdgcn_s_setprio(0);
#pragma unroll
        for (int k = 0; k < kTail; ++k) {
            acc.gt[k] += ((xr0[0][k] * r0[0] + xr0[1][k] * r0[1]) + xr0[2][k] * r0[2]) + xr0[3][k] * r0[3];
            acc.gt[k] += ((xr1[0][k] * r1[0] + xr1[1][k] * r1[1]) + xr1[2][k] * r1[2]) + xr1[3][k] * r1[3];
        }
    }
}

// ---------------------------------------------------------------------------
// Log-likelihood over draws: the column contraction E = X Q alone, then per
// (row, position) the loss and, with PRED, sigma(eta) summed over the
// positions of each row.

// loss = softplus(t) as in row_terms; p1 = sigmoid(eta) (the probability of
// y = 1): sigma(t) when y = 0 (t = eta), sigma(-t) when y = 1 (t = -eta).
__device__ __forceinline__ void ll_terms(float eta, float sgn, float& loss, float& p1)
{
    const float t = sgn * eta;
    const float e = __builtin_amdgcn_exp2f(-fabsf(t) * 1.4426950408889634f);
    const float u = 1.0f + e;
    const float inv = __builtin_amdgcn_rcpf(u);
    loss = __builtin_fmaf(kLn2f, __builtin_amdgcn_logf(u), fmaxf(t, 0.0f));
    const float sig_t = t >= 0.0f ? inv : e * inv;
    const float sig_mt = t >= 0.0f ? e * inv : inv;
    p1 = sgn > 0.0f ? sig_t : sig_mt;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v)
{
    // every pattern used here reads a lane of the same row with all rows and
    // banks enabled
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

// Sum over the 16 positions of a wave (lanes 16 g .. 16 g + 15, one DPP row,
// share the row group g): pair butterflies inside the row on DPP moves, so no
// LDS instruction (as cross-lane shuffles these were over half of the kernel's
// LDS instructions); every lane of the 16 gets the same bits.
__device__ __forceinline__ float sum16(float v)
{
    v += dpp_f32<kDppXor1>(v);
    v += dpp_f32<kDppXor2>(v);
    v += dpp_f32<kDppHalfMirror>(v);
    v += dpp_f32<kDppMirror>(v);
    return v;
}

// Posterior predictive samples of one position (draw s): y[i] = 1 iff
// u_si < sigmoid(eta_i), the uniforms the words of the Philox block keyed
// (seed, s) at counter (0, kTagPredict << 32, i / 4, 0), word i % 4.
struct PredictOut {
    uint8_t* y;     // the position's row of the [S][N] output, or null (dead position)
    uint64_t seed;
    uint64_t s;
    int64_t N;
    int64_t row0;   // first row of the stage
};

// Draw and store the samples of four consecutive rows r0 .. r0 + 3 (r0 a
// multiple of 4) from their probabilities p.
__device__ __forceinline__ void predict_rows(const PredictOut& po, int64_t r0, const float (&p)[4])
{
    const Block4 b = philox4x64_10(0, kTagPredict << 32, (uint64_t)(r0 >> 2), 0, po.seed, po.s);
    const uint64_t w[4] = {b.w0, b.w1, b.w2, b.w3};
#pragma unroll
    for (int r = 0; r < 4; ++r)
        if (r0 + r < po.N) po.y[r0 + r] = unit53(w[r]) < (double)p[r] ? 1 : 0;
}

// One LDS stage for this wave's 16 positions: the loss of every live
// (row, position) into `loss`; with PRED, the wave's sums of sigma(eta) over
// its live positions for each of the 64 rows into rs[0..63]; with SAMPLE,
// the position's predictive samples of the stage's rows.
template <int KT, bool PRED, bool SAMPLE>
__device__ __forceinline__ void compute_stage_ll(const float* __restrict__ xs, const float* __restrict__ ys,
                                                 const WaveQ& Q, float live, double& loss, float* rs,
                                                 const PredictOut& po, bool tail)
{
    using G = Geo<KT>;
    const int l = lane();
    const int m = l & 15;
    const int jj = l >> 4;
    const int e_off = m * G::RS + (G::KP == 8 ? 12 * (jj >> 1) + 4 * (jj & 1) : 4 * jj);
    constexpr int e_step = G::KP == 8 ? 24 : 16;
#pragma unroll 1
    for (int tp = 0; tp < kTiles; tp += 2) {
        const float* x0 = xs + tp * kTileRows * G::RS;
        const float* x1 = x0 + kTileRows * G::RS;
        v4f e0 = {0.0f, 0.0f, 0.0f, 0.0f};
        v4f e1 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int t = 0; t < G::KP; ++t) {
            const v4f a0 = *reinterpret_cast<const v4f*>(x0 + e_off + e_step * t);
            const v4f a1 = *reinterpret_cast<const v4f*>(x1 + e_off + e_step * t);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                e0 = mfma(a0[i], Q.q[4 * t + i], e0);
                e1 = mfma(a1[i], Q.q[4 * t + i], e1);
            }
        }
        if (tail) {  // uniform: the data has tail columns
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const v4f xr0 = *reinterpret_cast<const v4f*>(x0 + (4 * jj + r) * G::RS + 16 * G::GS);
                const v4f xr1 = *reinterpret_cast<const v4f*>(x1 + (4 * jj + r) * G::RS + 16 * G::GS);
                e0[r] += ((xr0[0] * Q.qt[0] + xr0[1] * Q.qt[1]) + xr0[2] * Q.qt[2]) + xr0[3] * Q.qt[3];
                e1[r] += ((xr1[0] * Q.qt[0] + xr1[1] * Q.qt[1]) + xr1[2] * Q.qt[2]) + xr1[3] * Q.qt[3];
            }
        }
        const v4f s0 = *reinterpret_cast<const v4f*>(ys + tp * kTileRows + 4 * jj);
        const v4f s1 = *reinterpret_cast<const v4f*>(ys + (tp + 1) * kTileRows + 4 * jj);
        float lsum = 0.0f;
        float p0[4], p1[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float l0, l1;
            ll_terms(e0[r], s0[r], l0, p0[r]);
            ll_terms(e1[r], s1[r], l1, p1[r]);
            lsum += l0 + l1;
        }
        loss += (double)lsum;
        if constexpr (SAMPLE) {
            if (po.y) {
                predict_rows(po, po.row0 + tp * kTileRows + 4 * jj, p0);
                predict_rows(po, po.row0 + (tp + 1) * kTileRows + 4 * jj, p1);
            }
        }
        if constexpr (PRED) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float a = sum16(live * p0[r]);
                const float b = sum16(live * p1[r]);
                if (m == 0) {
                    rs[tp * kTileRows + 4 * jj + r] = a;
                    rs[(tp + 1) * kTileRows + 4 * jj + r] = b;
                }
            }
        }
    }
}

// Stage loop of the log-likelihood: as stage_loop, and with PRED the eight
// waves' row sums of each stage (rs[buffer][wave][64]) are added in wave
// order and stored to prow[stage * 64 + row] one stage later, after the
// barrier that ends it.
template <int KT, bool PRED, bool SAMPLE>
__device__ __forceinline__ void stage_loop_ll(const BatchView& bv, int64_t st0, int64_t st1, int tid, float* xs,
                                              float* ys, float* rs, const WaveQ& Q, float live, double& loss,
                                              float* prow, PredictOut po)
{
    const int widx = tid / kWave;
    auto flush = [&](int64_t st, int b) {
        if (PRED && tid < kBatchStageRows) {
            float s_ = 0.0f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) s_ += rs[(b * kWaves + w) * kBatchStageRows + tid];
            prow[st * kBatchStageRows + tid] = s_;
        }
    };
    if (st0 < st1) {
        StageRegs r;
        load_stage<false>(bv, st0, tid, r);
        store_stage<KT, false>(r, tid, xs, ys);
    }
    __syncthreads();
    for (int64_t st = st0; st < st1; ++st) {
        const int b = (int)((st - st0) & 1);
        const bool more = st + 1 < st1;
        StageRegs r;
        if (more) load_stage<false>(bv, st + 1, tid, r);
        if (st > st0) flush(st - 1, b ^ 1);
        po.row0 = st * kBatchStageRows;
        compute_stage_ll<KT, PRED, SAMPLE>(xs + b * kStageBuf, ys + b * kBatchStageRows, Q, live, loss,
                                           rs + (b * kWaves + widx) * kBatchStageRows, po, bv.tc > 0);
        if (more) store_stage<KT, false>(r, tid, xs + (b ^ 1) * kStageBuf, ys + (b ^ 1) * kBatchStageRows);
        __syncthreads();
    }
    if (st1 > st0) flush(st1 - 1, (int)((st1 - 1 - st0) & 1));
}

// A group's rows in halves of stages (pairs of 16-row tiles, 32 rows):
// the 2 ns halves split evenly over the groups, so that no group has more
// than one half more than another (whole stages left 53 of 128 groups a
// whole stage more).  A stage whose halves two groups share is loaded by
// both, each computing its own.
__host__ __device__ inline void group_halves(int64_t ns, int64_t i, int64_t groups, int64_t* h0, int64_t* h1)
{
    *h0 = i * 2 * ns / groups;
    *h1 = (i + 1) * 2 * ns / groups;
}

// The stage loop over the halves [h0, h1) (stages h0 / 2 .. (h1 - 1) / 2)
// with double-buffered LDS stages.  Workers (tid = loader index, 0 .. 511)
// load and compute; a non-worker wave of the same group passes the same
// workgroup barriers (one more than the stages) and does nothing else.
// RECOMPUTE as for load_stage.
template <int KT, bool WORKER, bool RECOMPUTE = false>
__device__ __forceinline__ void stage_loop(const BatchView& bv, int64_t h0, int64_t h1, int tid, float* xs,
                                           float* ys, const WaveQ& Q, WaveAcc& acc)
{
    const int64_t st0 = h0 / 2;
    const int64_t st1 = h1 > h0 ? (h1 + 1) / 2 : st0;
    if constexpr (!WORKER) {
        for (int64_t st = st0; st <= st1; ++st) __syncthreads();
    } else {
        if (st0 < st1) {
            StageRegs r;
            load_stage<RECOMPUTE>(bv, st0, tid, r);
            store_stage<KT, RECOMPUTE>(r, tid, xs, ys);
        }
        __syncthreads();
        for (int64_t st = st0; st < st1; ++st) {
            const int b = (int)((st - st0) & 1);
            const bool more = st + 1 < st1;
            StageRegs r;
            if (more) load_stage<RECOMPUTE>(bv, st + 1, tid, r);
            // the halves of this stage that are the group's
            const int lo = (int)(h0 > 2 * st ? h0 - 2 * st : 0);
            const int hi = (int)(h1 < 2 * st + 2 ? h1 - 2 * st : 2);
            compute_stage<KT>(xs + b * kStageBuf, ys + b * kBatchStageRows, Q, acc, tid >= 4 * kWave, lo, hi);
            if (more) store_stage<KT, RECOMPUTE>(r, tid, xs + (b ^ 1) * kStageBuf, ys + (b ^ 1) * kBatchStageRows);
            __syncthreads();
        }
    }
}

// Sum the tail and loss accumulators over the four lanes of a position
// (lanes m, m + 16, m + 32, m + 48); every one of them gets the same bits.
__device__ __forceinline__ void reduce_position(WaveAcc& acc)
{
#pragma unroll
    for (int k = 0; k < kTail; ++k) {
        acc.gt[k] += __shfl_xor(acc.gt[k], 16);
        acc.gt[k] += __shfl_xor(acc.gt[k], 32);
    }
    acc.loss += __shfl_xor(acc.loss, 16);
    acc.loss += __shfl_xor(acc.loss, 32);
}

}  // namespace batch
}  // namespace nuts
