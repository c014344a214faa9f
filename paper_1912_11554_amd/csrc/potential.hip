// Batched potential and gradient of the logistic log-joint at K positions.
// Pass 1: a grid of (G groups) x (K items); each wave streams the blocks
// b = g * waves + w, g * waves + w + G * waves, ... of its item's data set and
// each group writes one fp64 partial [64] (columns 0..D-1, the loss sum in
// slot 63).  Pass 2: four waves per item add the G partials in a fixed
// order, then the Gaussian prior terms.  No floating-point atomics anywhere,
// so results are bitwise reproducible.
#include "launch.h"
#include "rows.h"

namespace nuts {

constexpr int kPotWaves = 8;
constexpr int kFinishWaves = 4;

template <typename T, int CPS, int S>
__global__ void __launch_bounds__(kPotWaves * kWave, 4) potential_pass_kernel(DataView dv,
                                                                           const double* __restrict__ W,
                                                                           int G,
                                                                           double* __restrict__ partials)
{
    constexpr int R = BlockShape<T, S>::R;
    const int l = lane();
    const int wave = threadIdx.x / kWave;
    const int64_t k = blockIdx.y;
    const int g = blockIdx.x;
    const int D = dv.D;
    const int64_t ds = dv.nds > 1 ? k : 0;
    const T* X = (const T*)dv.X + ds * dv.nb * (int64_t)D * R;
    const uint8_t* y = dv.y + ds * dv.nb * R;

    const double q = (l < D) ? W[k * D + l] : 0.0;
    double qv[CPS];
    spread_position<CPS, S>(q, qv);
    double acc[CPS];
#pragma unroll
    for (int c = 0; c < CPS; ++c) acc[c] = 0.0;
    double loss = 0.0;

    stream_blocks<T, CPS, S>(X, y, D, dv.N, dv.nb, (int64_t)g * kPotWaves + wave, (int64_t)G * kPotWaves, qv,
                             acc, loss);

    const double col = finish_pass<CPS, S>(acc, loss);
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

__global__ void __launch_bounds__(kFinishWaves * kWave) potential_finish_kernel(
    int D, const double* __restrict__ W, int G, const double* __restrict__ partials, double prior_scale,
    double* __restrict__ out_U, double* __restrict__ out_grad)
{
    const int l = lane();
    const int wave = threadIdx.x / kWave;
    const int64_t k = blockIdx.x;
    // wave w adds groups w, w + 4, ... ; then wave order
    double s = 0.0;
#pragma unroll 8
    for (int g = wave; g < G; g += kFinishWaves) s += partials[(k * G + g) * kWave + l];
    __shared__ double red[kFinishWaves][kWave];
    red[wave][l] = s;
    __syncthreads();
    if (wave != 0) return;
    double tot = 0.0;
#pragma unroll
    for (int w = 0; w < kFinishWaves; ++w) tot += red[w][l];
    const double inv_s2 = 1.0 / (prior_scale * prior_scale);
    const double w = (l < D) ? W[k * D + l] : 0.0;
    const double prior = wave_sum(0.5 * w * w * inv_s2);
    const double loss = __shfl(tot, kWave - 1);
    if (l < D) out_grad[k * D + l] = tot + w * inv_s2;
    if (l == 0)
        out_U[k] = loss + prior + (double)D * (log(prior_scale) + 0.91893853320467274178032973640562);
}

PotentialPlan plan_potential(const DataView& dv, int64_t K, int num_cu)
{
    // about two groups per CU over all items, never more than the blocks
    // give their waves work
    int64_t want = ((int64_t)num_cu * 2 + K - 1) / K;
    int64_t most = (dv.nb + kPotWaves - 1) / kPotWaves;
    if (want > most) want = most;
    if (want < 1) want = 1;
    return PotentialPlan{(int)want, kPotWaves};
}

template <typename T, int S>
static void enqueue_pass(const DataView& dv, const double* W, int64_t K, int G, double* partials,
                         hipStream_t stream)
{
    hipLaunchKernelGGL((potential_pass_kernel<T, kColsPerLane, S>), dim3(G, (unsigned)K),
                       dim3(kPotWaves * kWave), 0, stream, dv, W, G, partials);
}

template <typename T>
static void enqueue_pass_split(const DataView& dv, const double* W, int64_t K, int G, double* partials,
                               hipStream_t stream)
{
    if (dv.split == 1) enqueue_pass<T, 1>(dv, W, K, G, partials, stream);
    else if (dv.split == 2) enqueue_pass<T, 2>(dv, W, K, G, partials, stream);
    else if (dv.split == 4) enqueue_pass<T, 4>(dv, W, K, G, partials, stream);
    else enqueue_pass<T, 8>(dv, W, K, G, partials, stream);
}

hipError_t launch_potential_grad(const DataView& dv, double prior_scale, const double* W, int64_t K,
                                 const PotentialPlan& plan, double* partials, double* out_U,
                                 double* out_grad, hipStream_t stream)
{
    const int G = plan.groups_per_item;
    if (dv.dtype == NUTS_F64) enqueue_pass_split<double>(dv, W, K, G, partials, stream);
    else enqueue_pass_split<float>(dv, W, K, G, partials, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(potential_finish_kernel, dim3((unsigned)K), dim3(kFinishWaves * kWave), 0, stream,
                       dv.D, W, G, partials, prior_scale, out_U, out_grad);
    return hipGetLastError();
}

}  // namespace nuts
