// Batched potential and gradient of the logistic log-joint at K positions.
// Pass 1: a grid of (G groups) x (K items); each wave streams the column
// blocks b = g * waves + w, g * waves + w + G * waves, ... of its item's data
// set and each group writes one fp64 partial [64] (columns 0..D-1, the loss
// sum in slot 63).  Pass 2: one wave per item adds the G partials in group
// order and the Gaussian prior terms.  No floating-point atomics anywhere, so
// results are bitwise reproducible.
#include "launch.h"
#include "rows.h"

namespace nuts {

constexpr int kPotWaves = 8;

template <typename T, int MAXD>
__global__ void __launch_bounds__(kPotWaves * kWave) potential_pass_kernel(DataView dv,
                                                                           const double* __restrict__ W,
                                                                           int G,
                                                                           double* __restrict__ partials)
{
    const int l = lane();
    const int wave = threadIdx.x / kWave;
    const int64_t k = blockIdx.y;
    const int g = blockIdx.x;
    const int D = dv.D;
    const int64_t ds = dv.nds > 1 ? k : 0;
    const T* X = (const T*)dv.X + ds * dv.nb * (int64_t)D * kBlockRows;
    const uint8_t* y = dv.y + ds * dv.nb * kBlockRows;

    double qv[MAXD];
#pragma unroll
    for (int c = 0; c < MAXD; ++c) qv[c] = (c < D) ? W[k * D + c] : 0.0;
    double acc[MAXD];
#pragma unroll
    for (int c = 0; c < MAXD; ++c) acc[c] = 0.0;
    double loss = 0.0;

    const int64_t stride = (int64_t)G * kPotWaves;
    for (int64_t b = (int64_t)g * kPotWaves + wave; b < dv.nb; b += stride)
        accumulate_block<T, MAXD>(X + b * D * kBlockRows, y + b * kBlockRows, D,
                                  dv.N - b * kBlockRows, qv, acc, loss);

    const double col = finish_wave<MAXD>(acc, loss);
    __shared__ double part[kPotWaves][kWave];
    part[wave][l] = (l < D) ? col : (l == kWave - 1 ? loss : 0.0);
    __syncthreads();
    if (wave == 0) {
        double s = 0.0;
#pragma unroll
        for (int w = 0; w < kPotWaves; ++w) s += part[w][l];
        partials[(k * G + g) * kWave + l] = s;
    }
}

__global__ void __launch_bounds__(kWave) potential_finish_kernel(int D, const double* __restrict__ W,
                                                                 int G,
                                                                 const double* __restrict__ partials,
                                                                 double prior_scale,
                                                                 double* __restrict__ out_U,
                                                                 double* __restrict__ out_grad)
{
    const int l = lane();
    const int64_t k = blockIdx.x;
    double s = 0.0;
    for (int g = 0; g < G; ++g) s += partials[(k * G + g) * kWave + l];
    const double inv_s2 = 1.0 / (prior_scale * prior_scale);
    const double w = (l < D) ? W[k * D + l] : 0.0;
    const double prior = wave_sum(0.5 * w * w * inv_s2);
    const double loss = __shfl(s, kWave - 1);
    if (l < D) out_grad[k * D + l] = s + w * inv_s2;
    if (l == 0)
        out_U[k] = loss + prior + (double)D * (log(prior_scale) + 0.91893853320467274178032973640562);
}

PotentialPlan plan_potential(const DataView& dv, int64_t K, int num_cu)
{
    // enough groups to put ~4 per CU in total, but never more than there are
    // blocks for their waves
    int64_t want = ((int64_t)num_cu * 4 + K - 1) / K;
    int64_t most = (dv.nb + kPotWaves - 1) / kPotWaves;
    if (want > most) want = most;
    if (want < 1) want = 1;
    return PotentialPlan{(int)want, kPotWaves};
}

template <typename T, int MAXD>
static void enqueue_pass(const DataView& dv, const double* W, int64_t K, int G, double* partials,
                         hipStream_t stream)
{
    hipLaunchKernelGGL((potential_pass_kernel<T, MAXD>), dim3(G, (unsigned)K), dim3(kPotWaves * kWave),
                       0, stream, dv, W, G, partials);
}

hipError_t launch_potential_grad(const DataView& dv, double prior_scale, const double* W, int64_t K,
                                 const PotentialPlan& plan, double* partials, double* out_U,
                                 double* out_grad, hipStream_t stream)
{
    const int G = plan.groups_per_item;
    const bool f64 = dv.dtype == NUTS_F64;
    if (dv.D <= 16) {
        if (f64) enqueue_pass<double, 16>(dv, W, K, G, partials, stream);
        else enqueue_pass<float, 16>(dv, W, K, G, partials, stream);
    } else if (dv.D <= 32) {
        if (f64) enqueue_pass<double, 32>(dv, W, K, G, partials, stream);
        else enqueue_pass<float, 32>(dv, W, K, G, partials, stream);
    } else {
        if (f64) enqueue_pass<double, 64>(dv, W, K, G, partials, stream);
        else enqueue_pass<float, 64>(dv, W, K, G, partials, stream);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(potential_finish_kernel, dim3((unsigned)K), dim3(kWave), 0, stream, dv.D, W, G,
                       partials, prior_scale, out_U, out_grad);
    return hipGetLastError();
}

}  // namespace nuts
