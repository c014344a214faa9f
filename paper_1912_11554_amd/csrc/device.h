// Device helpers for the gfx950 NUTS kernels: counter-based Philox draws,
// wave64 reductions, numerically stable logistic terms.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nuts {

constexpr int kWave = 64;       // CDNA wavefront width
constexpr int kBlockRows = 64;  // rows per column block of the device layout (one per lane)

__device__ __forceinline__ int lane() { return __lane_id(); }

// Make a wave-uniform boolean an SGPR value so the branch on it is scalar.
__device__ __forceinline__ bool uni(bool b)
{
    return __builtin_amdgcn_readfirstlane((int)b) != 0;
}

// ---------------------------------------------------------------------------
// Philox4x64 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11).  Each round
// multiplies words 0 and 2 by fixed odd constants into 128-bit products; the
// high halves are xored with the other two words and the round key, and the
// words are permuted.  The two key words advance by the Weyl increments
// (golden ratio, sqrt(3) - 1) between rounds.
struct Block4 {
    uint64_t w0, w1, w2, w3;
};

__device__ __forceinline__ Block4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                uint64_t k0, uint64_t k1)
{
    constexpr uint64_t kMulA = 0xD2E7470EE14C6C93ull;
    constexpr uint64_t kMulB = 0xCA5A826395121157ull;
    constexpr uint64_t kWeylA = 0x9E3779B97F4A7C15ull;
    constexpr uint64_t kWeylB = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t hiA = __umul64hi(kMulA, c0), loA = kMulA * c0;
        const uint64_t hiB = __umul64hi(kMulB, c2), loB = kMulB * c2;
        const uint64_t n0 = hiB ^ c1 ^ k0;
        const uint64_t n2 = hiA ^ c3 ^ k1;
        c0 = n0;
        c1 = loB;
        c2 = n2;
        c3 = loA;
        k0 += kWeylA;
        k1 += kWeylB;
    }
    return Block4{c0, c1, c2, c3};
}

// Which quantity a block feeds; part of the counter.
enum : uint64_t { kTagMomentum = 1, kTagDirection = 2, kTagMerge = 3, kTagLeaf = 4 };

__device__ __forceinline__ Block4 draw(uint64_t seed, uint64_t chain, uint64_t iter, uint64_t tag,
                                       uint64_t doubling, uint64_t index)
{
    return philox4x64_10(iter, (tag << 32) | doubling, index, 0, seed, chain);
}

// Top 53 bits of a word as a double in [0, 1).
__device__ __forceinline__ double unit53(uint64_t w)
{
    return (double)(w >> 11) * 1.1102230246251565404236316680908203125e-16;  // 2^-53
}

// Standard normal number i of an iteration's momentum: block i/4 holds two
// Box-Muller pairs (u_a, u_b) giving (r cos th, r sin th), r = sqrt(-2 ln(1 -
// u_a)), th = 2 pi u_b.
__device__ __forceinline__ double momentum_normal(uint64_t seed, uint64_t chain, uint64_t iter, int i)
{
    const Block4 b = draw(seed, chain, iter, kTagMomentum, 0, (uint64_t)(i >> 2));
    const bool second_pair = (i & 2) != 0;
    const double ua = unit53(second_pair ? b.w2 : b.w0);
    const double ub = unit53(second_pair ? b.w3 : b.w1);
    const double r = sqrt(-2.0 * log(1.0 - ua));
    const double th = 6.283185307179586476925286766559 * ub;
    return (i & 1) ? r * sin(th) : r * cos(th);
}

// ---------------------------------------------------------------------------
// Wave reductions.  Butterflies over xor partners: every lane ends with the
// same total, summed in the same fixed tree order on every run.
__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int m = kWave / 2; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return v;
}

// Reduce SLOTS per-lane partial sums over the wave at once.  Each butterfly
// step halves the number of live slots: the lane whose partner bit is set
// keeps the upper half, the other the lower half, and each adds what its
// partner sends for the half it keeps.  After log2(SLOTS) steps lane L holds
// slot L / (64 / SLOTS); the remaining steps sum the lanes that share a slot.
// Cost is about SLOTS shuffles instead of 6 * SLOTS for slot-by-slot sums.
template <int SLOTS>
__device__ __forceinline__ double transpose_reduce(double (&a)[SLOTS])
{
    static_assert(SLOTS >= 1 && SLOTS <= kWave && (SLOTS & (SLOTS - 1)) == 0, "power of two");
    const int l = lane();
    int bit = kWave / 2;
#pragma unroll
    for (int h = SLOTS / 2; h >= 1; h /= 2) {
        const bool upper = (l & bit) != 0;
#pragma unroll
        for (int i = 0; i < h; ++i) {
            const double send = upper ? a[i] : a[i + h];
            const double keep = upper ? a[i + h] : a[i];
            a[i] = keep + __shfl_xor(send, bit);
        }
        bit >>= 1;
    }
    double v = a[0];
    for (; bit >= 1; bit >>= 1) v += __shfl_xor(v, bit);
    return v;
}

// ---------------------------------------------------------------------------
// Logistic row terms.  With s = 1 - 2y and t = s * eta, the row's negative
// log-likelihood is softplus(t) >= 0 and d/d eta of it is s * sigmoid(t); both
// come from one exp(-|t|).
struct RowTerms {
    double loss;
    double resid;
};

__device__ __forceinline__ RowTerms logistic_row(double eta, bool y_is_one)
{
    const double sgn = y_is_one ? -1.0 : 1.0;
    const double t = sgn * eta;
    const double e = exp(-fabs(t));
    const double inv = 1.0 / (1.0 + e);
    const double sig = t >= 0.0 ? inv : e * inv;
    return RowTerms{fmax(t, 0.0) + log1p(e), sgn * sig};
}

__device__ __forceinline__ double logaddexp(double a, double b)
{
    if (a == -INFINITY) return b;
    if (b == -INFINITY) return a;
    return fmax(a, b) + log1p(exp(-fabs(a - b)));
}

}  // namespace nuts
