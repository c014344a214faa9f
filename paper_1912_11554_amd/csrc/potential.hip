// Batched potential and gradient of the logistic log-joint at K positions.
// Pass 1: a grid of (G groups) x (K items); each wave streams the blocks
// b = g * waves + w, g * waves + w + G * waves, ... of its item's data set and
// each group writes one fp64 partial row of width partial_width(D) (columns
// 0..D-1, the loss sum at 64 * ceil(D / 64)).  Pass 2: four waves per item
// add the G partials in a fixed order, then the Gaussian prior terms.  No
// floating-point atomics anywhere, so results are bitwise reproducible.
#include "launch.h"
#include "rows.h"

namespace nuts {

namespace {

constexpr int kPotWaves = 8;
constexpr int kFinishWaves = 4;
constexpr double kHalfLog2Pi = 0.91893853320467274178032973640562;

template <typename T, int S, int CPS>
__global__ void __launch_bounds__(kPotWaves * kWave, 4) potential_pass_kernel(DataView dv,
                                                                              const double* __restrict__ W,
                                                                              int G, int width,
                                                                              double* __restrict__ partials)
{
    constexpr int R = BlockShape<T, S>::R;
    extern __shared__ double part[];  // [kPotWaves][width]
    const int l = lane();
    const int wave = threadIdx.x / kWave;
    const int64_t k = blockIdx.y;
    const int g = blockIdx.x;
    const int D = dv.D;
    const int loss_slot = width - 64;
    const int64_t ds = dv.nds > 1 ? k : 0;
    const T* X = (const T*)dv.X + ds * dv.nb * (int64_t)D * R;
    const uint8_t* y = dv.y + ds * dv.nb * R;

    double qv[CPS];
    spread_position_lds<CPS, S>(W + k * D, D, qv);
    double acc[CPS];
#pragma unroll
    for (int c = 0; c < CPS; ++c) acc[c] = 0.0;
    double loss = 0.0;
    stream_blocks<T, CPS, S>(X, y, D, dv.N, dv.nb, (int64_t)g * kPotWaves + wave, (int64_t)G * kPotWaves, qv,
                             acc, loss);

    double* row = part + wave * width;
    if constexpr (S <= 8 && CPS == 8) {
        const double col = finish_pass<CPS, S>(acc, loss);
        if (l < D) row[l] = col;
        if (l == 0) row[loss_slot] = loss;
    } else {
        finish_pass_to_row<CPS, S>(acc, loss, row, D, loss_slot);
    }
    __syncthreads();
    if (wave == 0) {
        for (int col = l; col < width; col += 64) {
            const bool used = col < D || col == loss_slot;
            double s = 0.0;
            if (used) {
#pragma unroll
                for (int w = 0; w < kPotWaves; ++w) s += part[w * width + col];
            }
            partials[(k * G + g) * width + col] = s;
        }
    }
}

__global__ void __launch_bounds__(kFinishWaves * kWave) potential_finish_kernel(
    int D, int width, const double* __restrict__ W, int G, const double* __restrict__ partials,
    double prior_scale, double* __restrict__ out_U, double* __restrict__ out_grad)
{
    extern __shared__ double red[];  // [kFinishWaves][width]
    const int l = lane();
    const int wave = threadIdx.x / kWave;
    const int64_t k = blockIdx.x;
    // wave w adds groups w, w + 4, ... ; then wave order
    for (int col = l; col < width; col += 64) {
        double s = 0.0;
#pragma unroll 8
        for (int g = wave; g < G; g += kFinishWaves) s += partials[(k * G + g) * width + col];
        red[wave * width + col] = s;
    }
    __syncthreads();
    if (wave != 0) return;
    const double inv_s2 = 1.0 / (prior_scale * prior_scale);
    double pr = 0.0;
    double loss = 0.0;
    for (int col = l; col < width; col += 64) {
        double tot = 0.0;
#pragma unroll
        for (int w = 0; w < kFinishWaves; ++w) tot += red[w * width + col];
        if (col < D) {
            const double w = W[k * D + col];
            pr += 0.5 * w * w * inv_s2;
            out_grad[k * D + col] = tot + w * inv_s2;
        }
        if (col == width - 64) loss = tot;
    }
    const double prior = wave_sum(pr);
    loss = readlane_f64(loss, 0);  // the loss slot is column 64 * m of lane 0
    if (l == 0) out_U[k] = loss + prior + (double)D * (log(prior_scale) + kHalfLog2Pi);
}

template <typename T, int S, int CPS>
void enqueue_pass(const DataView& dv, const double* W, int64_t K, int G, int width, double* partials,
                  hipStream_t stream)
{
    hipLaunchKernelGGL((potential_pass_kernel<T, S, CPS>), dim3(G, (unsigned)K), dim3(kPotWaves * kWave),
                       (size_t)kPotWaves * width * sizeof(double), stream, dv, W, G, width, partials);
}

template <typename T>
void enqueue_pass_shape(const DataView& dv, const double* W, int64_t K, int G, int width, double* partials,
                        hipStream_t stream)
{
    const int D = dv.D;
    if (D <= 8) enqueue_pass<T, 1, 8>(dv, W, K, G, width, partials, stream);
    else if (D <= 16) enqueue_pass<T, 1, 16>(dv, W, K, G, width, partials, stream);
    else if (D <= 32) enqueue_pass<T, 4, 8>(dv, W, K, G, width, partials, stream);
    else if (D <= 64) enqueue_pass<T, 8, 8>(dv, W, K, G, width, partials, stream);
    else if (D <= 128) enqueue_pass<T, 16, 8>(dv, W, K, G, width, partials, stream);
    else if (D <= 256) enqueue_pass<T, 32, 8>(dv, W, K, G, width, partials, stream);
    else enqueue_pass<T, 32, 10>(dv, W, K, G, width, partials, stream);
}

}  // namespace

PotentialPlan plan_potential(const DataView& dv, int64_t K, int num_cu)
{
    // about two groups per CU over all items, never more than the blocks
    // give their waves work
    int64_t want = ((int64_t)num_cu * 2 + K - 1) / K;
    int64_t most = (dv.nb + kPotWaves - 1) / kPotWaves;
    if (want > most) want = most;
    if (want < 1) want = 1;
    return PotentialPlan{(int)want, partial_width(dv.D)};
}

hipError_t launch_potential_grad(const DataView& dv, double prior_scale, const double* W, int64_t K,
                                 const PotentialPlan& plan, double* partials, double* out_U,
                                 double* out_grad, hipStream_t stream)
{
    const int G = plan.groups_per_item;
    if (dv.dtype == NUTS_F64) enqueue_pass_shape<double>(dv, W, K, G, plan.width, partials, stream);
    else enqueue_pass_shape<float>(dv, W, K, G, plan.width, partials, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(potential_finish_kernel, dim3((unsigned)K), dim3(kFinishWaves * kWave),
                       (size_t)kFinishWaves * plan.width * sizeof(double), stream, dv.D, plan.width, W, G,
                       partials, prior_scale, out_U, out_grad);
    return hipGetLastError();
}

}  // namespace nuts
