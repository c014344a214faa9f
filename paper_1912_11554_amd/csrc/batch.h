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
constexpr int kMaxStride = 16 * kBatchMaxKT + kTail;        // 132 floats
constexpr int kStageFloats = kBatchStageRows * kMaxStride;  // one LDS stage buffer
constexpr int kStageBuf = kStageFloats + 4;                 // plus one junk 16-byte slot
constexpr int kStageVecs = (kStageFloats / 4 + kWaves * kWave - 1) / (kWaves * kWave);

__device__ __forceinline__ v4f mfma(float a, float b, v4f c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Negative log-likelihood and residual of one (row, position) from eta in
// fp32: with s = 1 - 2y and t = s eta, loss = softplus(t), residual =
// s sigmoid(t), both from one exp(-|t|); log1p(e) as log(u) e / (u - 1),
// u = 1 + e (Goldberg 1991, Thm. 4).  A label byte > 1 marks a padding row,
// which contributes nothing.
__device__ __forceinline__ void row_terms(float eta, uint32_t ybyte, float& loss, float& resid)
{
    const bool one = ybyte == 1u;
    const float t = one ? -eta : eta;
    const float a = fabsf(t);
    const float e = __builtin_amdgcn_exp2f(-a * 1.4426950408889634f);
    const float u = 1.0f + e;
    const float inv = __builtin_amdgcn_rcpf(u);
    const float um1 = u - 1.0f;
    const float lg = __builtin_amdgcn_logf(u) * 0.69314718055994531f;
    const float l1p = um1 == 0.0f ? e : lg * (e * __builtin_amdgcn_rcpf(um1));
    const float sig = t >= 0.0f ? inv : e * inv;
    const bool pad = ybyte > 1u;
    loss = pad ? 0.0f : fmaxf(t, 0.0f) + l1p;
    resid = pad ? 0.0f : (one ? -sig : sig);
}

// A wave's share of the positions: Q in the B-operand order of the column
// contraction (q[4 t + i] = Q[16 t + 4 (l / 16) + i][l % 16]) and the tail.
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

__device__ __forceinline__ void load_stage(const BatchView& bv, int64_t st, int tid, StageRegs& r)
{
    const int last = kBatchStageRows * bv.stride / 4 - 1;
    const v4f* src = reinterpret_cast<const v4f*>(bv.X + st * kBatchStageRows * bv.stride);
    // unconditional loads (pieces past the stage re-read its last piece and
    // are not stored), so the loop unrolls into straight-line code
#pragma unroll
    for (int i = 0; i < kStageVecs; ++i) r.v[i] = src[min(tid + i * kWaves * kWave, last)];
    if (tid < kBatchStageRows / 4) r.y = reinterpret_cast<const uint32_t*>(bv.y + st * kBatchStageRows)[tid];
}

__device__ __forceinline__ void store_stage(const BatchView& bv, const StageRegs& r, int tid, float* xs,
                                            uint32_t* ys)
{
    // pieces past the stage go to a junk slot after the buffer (never read)
    const int last = kBatchStageRows * bv.stride / 4 - 1;
#pragma unroll
    for (int i = 0; i < kStageVecs; ++i) {
        const int idx = tid + i * kWaves * kWave;
        reinterpret_cast<v4f*>(xs)[idx <= last ? idx : kStageFloats / 4] = r.v[i];
    }
    if (tid < kBatchStageRows / 4) ys[tid] = r.y;
}

// All four 16-row tiles of one LDS stage for this wave's 16 positions.  KT
// is the chunk count; the four tail slots are always processed (slots past
// the tail hold zero columns and zero positions, so they add nothing).
template <int KT>
__device__ __forceinline__ void compute_stage(const float* __restrict__ xs, const uint32_t* __restrict__ ys,
                                              int stride, const WaveQ& Q, WaveAcc& acc)
{
    const int l = lane();
    const int m = l & 15;
    const int jj = l >> 4;
#pragma unroll 1
    for (int ti = 0; ti < kTiles; ++ti) {
        const float* xt = xs + ti * kTileRows * stride;
        v4f e = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int t = 0; t < KT; ++t) {
            const v4f a = *reinterpret_cast<const v4f*>(xt + m * stride + 16 * t + 4 * jj);
            e = mfma(a[0], Q.q[4 * t + 0], e);
            e = mfma(a[1], Q.q[4 * t + 1], e);
            e = mfma(a[2], Q.q[4 * t + 2], e);
            e = mfma(a[3], Q.q[4 * t + 3], e);
        }
        // tail slots of this lane's four rows 4 jj + r
        v4f xr[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            xr[r] = *reinterpret_cast<const v4f*>(xt + (4 * jj + r) * stride + 16 * KT);
            e[r] += ((xr[r][0] * Q.qt[0] + xr[r][1] * Q.qt[1]) + xr[r][2] * Q.qt[2]) + xr[r][3] * Q.qt[3];
        }
        const uint32_t yw = ys[ti * 4 + jj];
        float rr[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float ls;
            row_terms(e[r], (yw >> (8 * r)) & 0xFFu, ls, rr[r]);
            acc.loss += (double)ls;
        }
#pragma unroll
        for (int mt = 0; mt < KT; ++mt) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
                acc.g[mt] = mfma(xt[(4 * jj + r) * stride + 16 * mt + m], rr[r], acc.g[mt]);
        }
#pragma unroll
        for (int k = 0; k < kTail; ++k)
            acc.gt[k] += ((xr[0][k] * rr[0] + xr[1][k] * rr[1]) + xr[2][k] * rr[2]) + xr[3][k] * rr[3];
    }
}

// The stage loop over [st0, st1) with double-buffered LDS stages.  Workers
// (tid = loader index, 0 .. 511) load and compute; a non-worker wave of the
// same group passes the same workgroup barriers (1 + st1 - st0 of them) and
// does nothing else.
template <int KT, bool WORKER>
__device__ __forceinline__ void stage_loop(const BatchView& bv, int64_t st0, int64_t st1, int tid, float* xs,
                                           uint32_t* ys, const WaveQ& Q, WaveAcc& acc)
{
    if constexpr (!WORKER) {
        for (int64_t st = st0; st <= st1; ++st) __syncthreads();
    } else {
        if (st0 < st1) {
            StageRegs r;
            load_stage(bv, st0, tid, r);
            store_stage(bv, r, tid, xs, ys);
        }
        __syncthreads();
        for (int64_t st = st0; st < st1; ++st) {
            const int b = (int)((st - st0) & 1);
            const bool more = st + 1 < st1;
            StageRegs r;
            if (more) load_stage(bv, st + 1, tid, r);
            compute_stage<KT>(xs + b * kStageBuf, ys + b * (kBatchStageRows / 4), bv.stride, Q, acc);
            if (more) store_stage(bv, r, tid, xs + (b ^ 1) * kStageBuf, ys + (b ^ 1) * (kBatchStageRows / 4));
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
