// Device helpers for the gfx950 NUTS kernels: counter-based Philox draws,
// wave64 reductions, numerically stable logistic terms.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nuts {

constexpr int kWave = 64;       // CDNA wavefront width

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

// The 128-bit product of a 64-bit constant and x, from the four 32 x 32-bit
// partial products (each a 64-bit multiply-add on the vector ALU; no sum
// below overflows 64 bits): the high and low halves share them.
template <uint64_t A>
__device__ __forceinline__ void mul128(uint64_t x, uint64_t& hi, uint64_t& lo)
{
    constexpr uint32_t aL = (uint32_t)A, aH = (uint32_t)(A >> 32);
    const uint32_t xL = (uint32_t)x, xH = (uint32_t)(x >> 32);
    const uint64_t p00 = (uint64_t)aL * xL;
    const uint64_t t = (uint64_t)aL * xH + (p00 >> 32);
    const uint64_t u = (uint64_t)aH * xL + (uint32_t)t;
    hi = (uint64_t)aH * xH + (t >> 32) + (u >> 32);
    lo = (u << 32) | (uint32_t)p00;
}

__device__ __forceinline__ Block4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                uint64_t k0, uint64_t k1)
{
    constexpr uint64_t kMulA = 0xD2E7470EE14C6C93ull;
    constexpr uint64_t kMulB = 0xCA5A826395121157ull;
    constexpr uint64_t kWeylA = 0x9E3779B97F4A7C15ull;
    constexpr uint64_t kWeylB = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        uint64_t hiA, loA, hiB, loB;
        mul128<kMulA>(c0, hiA, loA);
        mul128<kMulB>(c2, hiB, loB);
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

// Which quantity a block feeds; part of the counter.  Block b of kTagTree
// (counter {iteration, kTagTree << 32, b, 0}) holds the direction of
// doubling b (word 0), the merge uniform of doubling b (word 1) and the
// uniforms of leaves 2b and 2b + 1 (words 2, 3), leaf n of doubling j being
// the iteration's leaf number 2^j - 1 + n.
enum : uint64_t { kTagMomentum = 1, kTagTree = 2, kTagStepSize = 5, kTagSubMerge = 6, kTagPredict = 7 };

// Kept out of line: it is called a few times per iteration, and inlining it
// would keep its temporaries and constants live across the tree loops.
__device__ __noinline__ Block4 draw(uint64_t seed, uint64_t chain, uint64_t iter, uint64_t tag,
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
__device__ __noinline__ double momentum_normal(uint64_t seed, uint64_t chain, uint64_t iter, int i,
                                               uint64_t tag = kTagMomentum)
{
    const Block4 b = draw(seed, chain, iter, tag, 0, (uint64_t)(i >> 2));
    const bool second_pair = (i & 2) != 0;
    const double ua = unit53(second_pair ? b.w2 : b.w0);
    const double ub = unit53(second_pair ? b.w3 : b.w1);
    const double r = sqrt(-2.0 * log(1.0 - ua));
    const double th = 6.283185307179586476925286766559 * ub;
    // both from one argument reduction (the lanes of a wave want either)
    double sn, cs;
    sincos(th, &sn, &cs);
    return (i & 1) ? r * sn : r * cs;
}

// ---------------------------------------------------------------------------
// Cross-lane moves.  DPP (data-parallel primitives) patterns act inside rows
// of 16 lanes at register-read cost; the rest go through ds_bpermute.
enum : int {
    kDppXor1 = 0xB1,        // quad_perm [1, 0, 3, 2]
    kDppXor2 = 0x4E,        // quad_perm [2, 3, 0, 1]
    kDppHalfMirror = 0x141, // lane i <-> 7 - i inside each 8 lanes
    kDppMirror = 0x140,     // lane i <-> 15 - i inside each 16 lanes
    kDppRor8 = 0x128        // lane i <-  (i + 8) mod 16, i.e. i ^ 8
};

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v)
{
    const int2 h = __builtin_bit_cast(int2, v);
    // every pattern here reads a lane of the same row with all rows and banks
    // enabled, so no lane keeps an old value and none needs setting up
    const int lo = __builtin_amdgcn_mov_dpp(h.x, CTRL, 0xF, 0xF, true);
    const int hi = __builtin_amdgcn_mov_dpp(h.y, CTRL, 0xF, 0xF, true);
    return __builtin_bit_cast(double, int2{lo, hi});
}

__device__ __forceinline__ double readlane_f64(double v, int src)
{
    const int2 h = __builtin_bit_cast(int2, v);
    return __builtin_bit_cast(double, int2{__builtin_amdgcn_readlane(h.x, src),
                                           __builtin_amdgcn_readlane(h.y, src)});
}

// The value of lane (this lane ^ M).
template <int M>
__device__ __forceinline__ double xor_move(double v)
{
    if constexpr (M == 1) return dpp_f64<kDppXor1>(v);
    else if constexpr (M == 2) return dpp_f64<kDppXor2>(v);
    else if constexpr (M == 8) return dpp_f64<kDppRor8>(v);
    else return __shfl_xor(v, M);
}

// For sums over aligned groups of 2M lanes: the value of a partner lane in
// the other half of this lane's group (an involution, not always i ^ M).
template <int M>
__device__ __forceinline__ double pair_move(double v)
{
    if constexpr (M == 4) return dpp_f64<kDppHalfMirror>(v);
    else if constexpr (M == 8) return dpp_f64<kDppMirror>(v);
    else return xor_move<M>(v);
}

// Sum over the whole wave; every lane gets the same bits.  Rows of 16 are
// summed by pair butterflies, then the four row sums are added in row order.
__device__ __forceinline__ double wave_sum(double v)
{
    v += pair_move<1>(v);
    v += pair_move<2>(v);
    v += pair_move<4>(v);
    v += pair_move<8>(v);
    return ((readlane_f64(v, 0) + readlane_f64(v, 16)) + readlane_f64(v, 32)) + readlane_f64(v, 48);
}

// wave_sum for values that are zero outside lanes 0..15 when `one_row` (a
// wave-uniform flag): then the first row's sum is the whole sum (adding the
// other rows' zeros changes at most the sign of a zero result).
__device__ __forceinline__ double wave_sum_rows(double v, bool one_row)
{
    v += pair_move<1>(v);
    v += pair_move<2>(v);
    v += pair_move<4>(v);
    v += pair_move<8>(v);
    if (one_row) return readlane_f64(v, 0);
    return ((readlane_f64(v, 0) + readlane_f64(v, 16)) + readlane_f64(v, 32)) + readlane_f64(v, 48);
}

// ---------------------------------------------------------------------------
// Logistic row terms.  With s = 1 - 2y and t = s * eta, the row's negative
// log-likelihood is softplus(t) >= 0 and d/d eta of it is s * sigmoid(t); both
// come from one exp(-|t|).  The fp64 versions below are written out (range
// reduction and series) for the arguments that occur here, at a few ulp,
// instead of the general library routines.
struct RowTerms {
    double loss;
    double resid;
};

// 1 / d to full fp64 precision: the hardware reciprocal refined by two
// Newton steps (each doubles the correct bits).
__device__ __forceinline__ double recip(double d)
{
    double r = __builtin_amdgcn_rcp(d);
    double err = fma(-d, r, 1.0);
    r = fma(r, err, r);
    err = fma(-d, r, 1.0);
    return fma(r, err, r);
}

// e^x for x <= 0: x = k ln 2 + r with |r| <= ln 2 / 2 (Cody-Waite: ln 2 split
// into its float rounding and the remainder, so k * hi is exact), e^r from
// its Taylor series to degree 13 (truncation below 5e-18 relative), scaled by
// 2^k (which underflows to 0 for very negative x).  NaN propagates.
__device__ __forceinline__ double exp_nonpos(double x)
{
    constexpr double kLog2e = 1.4426950408889634;
    constexpr double kLn2Hi = 0.693147182464599609375;  // ln 2 rounded to a float
    constexpr double kLn2Lo = -1.904654299957768e-09;   // ln 2 - kLn2Hi
    x = x < -1100.0 ? -1100.0 : x;                      // keeps NaN
    double k = rint(x * kLog2e);
    double r = fma(-k, kLn2Hi, x);
    r = fma(-k, kLn2Lo, r);
    // Horner over 1/n!, n = 13 .. 0
    double p = 1.6059043836821613e-10;
    p = fma(p, r, 2.08767569878681e-09);
    p = fma(p, r, 2.505210838544172e-08);
    p = fma(p, r, 2.755731922398589e-07);
    p = fma(p, r, 2.7557319223985893e-06);
    p = fma(p, r, 2.48015873015873e-05);
    p = fma(p, r, 0.0001984126984126984);
    p = fma(p, r, 0.001388888888888889);
    p = fma(p, r, 0.008333333333333333);
    p = fma(p, r, 0.041666666666666664);
    p = fma(p, r, 0.16666666666666666);
    p = fma(p, r, 0.5);
    p = fma(p, r, 1.0);
    p = fma(p, r, 1.0);
    k = k == k ? k : 0.0;
    return ldexp(p, (int)k);
}

// log(1 + e) for 0 <= e <= 1, given u = 1 + e rounded and inv = 1 / u.
// log u: m = u (or u / 2, adding ln 2) in [0.707, 1.415], s = (m - 1) /
// (m + 1) with |s| <= 3 - 2 sqrt 2, log m = 2 atanh s = 2 s sum_k s^2k /
// (2k + 1) to k = 11 (remainder below 2e-20); then the rounding of u is
// put back: log(1 + e) = log u + (e - (u - 1)) / u to first order.
__device__ __forceinline__ double log1p_unit(double e, double u, double inv)
{
    constexpr double kLn2 = 0.6931471805599453;
    const bool big = u > 1.4142135623730951;
    const double m = big ? 0.5 * u : u;
    const double s = (m - 1.0) * recip(m + 1.0);  // m - 1 is exact here
    const double w = s * s;
    double p = 0.043478260869565216;               // 1/23
    p = fma(p, w, 0.047619047619047616);           // 1/21
    p = fma(p, w, 0.05263157894736842);            // 1/19
    p = fma(p, w, 0.058823529411764705);           // 1/17
    p = fma(p, w, 0.06666666666666667);            // 1/15
    p = fma(p, w, 0.07692307692307693);            // 1/13
    p = fma(p, w, 0.09090909090909091);            // 1/11
    p = fma(p, w, 0.1111111111111111);             // 1/9
    p = fma(p, w, 0.14285714285714285);            // 1/7
    p = fma(p, w, 0.2);                            // 1/5
    p = fma(p, w, 0.3333333333333333);             // 1/3
    p = fma(p, w, 1.0);
    double lg = 2.0 * s * p;
    lg = big ? lg + kLn2 : lg;
    return lg + (e - (u - 1.0)) * inv;  // u - 1 is exact for u in [1, 2]
}

__device__ __forceinline__ RowTerms logistic_row(double eta, bool y_is_one)
{
    const double sgn = y_is_one ? -1.0 : 1.0;
    const double t = sgn * eta;
    const double e = exp_nonpos(-fabs(t));
    const double u = 1.0 + e;
    const double inv = recip(u);
    const double sig = t >= 0.0 ? inv : e * inv;
    return RowTerms{fmax(t, 0.0) + log1p_unit(e, u, inv), sgn * sig};
}

// The same terms for fp32 data: eta and t stay fp64; the exponential, log
// and reciprocal use the fp32 hardware instructions (v_exp_f32, v_log_f32,
// v_rcp_f32; a few ulp, i.e. ~1e-6 relative per row at worst) and return as
// fp64 for accumulation.  log1p(e) is formed as log(u) * e / (u - 1) with
// u = 1 + e, which cancels the rounding of u (Goldberg 1991, Thm. 4).
__device__ __forceinline__ RowTerms logistic_row_f32(double eta, bool y_is_one)
{
    const double sgn = y_is_one ? -1.0 : 1.0;
    const double t = sgn * eta;
    const float a = (float)fabs(t);
    const float e = __builtin_amdgcn_exp2f(-a * 1.4426950408889634f);
    const float u = 1.0f + e;
    const float inv = __builtin_amdgcn_rcpf(u);
    const float um1 = u - 1.0f;
    const float lg = __builtin_amdgcn_logf(u) * 0.69314718055994531f;
    const float l1p = um1 == 0.0f ? e : lg * (e * __builtin_amdgcn_rcpf(um1));
    const float sig = t >= 0.0 ? inv : e * inv;
    return RowTerms{fmax(t, 0.0) + (double)l1p, sgn * (double)sig};
}

template <typename T>
__device__ __forceinline__ RowTerms logistic_row_t(double eta, bool y_is_one);
template <>
__device__ __forceinline__ RowTerms logistic_row_t<double>(double eta, bool y_is_one)
{
    return logistic_row(eta, y_is_one);
}
template <>
__device__ __forceinline__ RowTerms logistic_row_t<float>(double eta, bool y_is_one)
{
    return logistic_row_f32(eta, y_is_one);
}

__device__ __forceinline__ double logaddexp(double a, double b)
{
    if (a == -INFINITY) return b;
    if (b == -INFINITY) return a;
    const double e = exp_nonpos(-fabs(a - b));
    const double u = 1.0 + e;
    return fmax(a, b) + log1p_unit(e, u, recip(u));
}

// logaddexp(a, b) and b's share e^b / (e^a + e^b) of the sum, both from the
// one exponential: with e = e^-|a - b| the share is 1 / (1 + e) when b >= a
// and e / (1 + e) otherwise (1 when a = -inf; b is finite).
__device__ __forceinline__ double logaddexp_share(double a, double b, double& share_b)
{
    if (a == -INFINITY) {
        share_b = 1.0;
        return b;
    }
    const double e = exp_nonpos(-fabs(a - b));
    const double u = 1.0 + e;
    const double inv = recip(u);
    share_b = b >= a ? inv : e * inv;
    return fmax(a, b) + log1p_unit(e, u, inv);
}

}  // namespace nuts
