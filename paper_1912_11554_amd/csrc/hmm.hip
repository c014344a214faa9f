// Semi-supervised HMM target: the sampler without the optional features, and
// the standalone potential.
#include "hmm_impl.h"

namespace nuts {

hipError_t launch_hmm_sampler(const SamplerArgs& a, const HmmView& hv, hipStream_t stream)
{
    if (sampler_extended(a)) return launch_hmm_sampler_ext(a, hv, stream);
    return hmm::hmm_sampler_dispatch<false>(a, hv, stream);
}

template <int K>
static hipError_t potential_launch(const HmmView& hv, const double* Q, int64_t n, double* out_U, double* out_grad,
                                   hipStream_t stream)
{
    const int D = hmm_dim(hv.K, hv.V);
    const hmm::HmmLds L = hmm::hmm_lds(K, hv.V, hv.T, hv.Tsup, D, 1, 0);
    const int cpg = hmm::hmm_chains_per_group(L, n);
    if (cpg == 0) return hipErrorInvalidValue;
    const size_t lds = (size_t)cpg * L.wave * sizeof(double);
    const void* k = (const void*)hmm::hmm_potential_kernel<K>;
    hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    const unsigned grid = (unsigned)((n + cpg - 1) / cpg);
    hipLaunchKernelGGL((hmm::hmm_potential_kernel<K>), dim3(grid), dim3(hmm::kHmmChainsPerGroup * kWave), lds,
                       stream, hv, D, Q, n, out_U, out_grad, cpg);
    return hipGetLastError();
}

hipError_t launch_hmm_potential(const HmmView& hv, const double* Q, int64_t n, double* out_U, double* out_grad,
                                hipStream_t stream)
{
    switch (hv.K) {
    case 2: return potential_launch<2>(hv, Q, n, out_U, out_grad, stream);
    case 3: return potential_launch<3>(hv, Q, n, out_U, out_grad, stream);
    case 4: return potential_launch<4>(hv, Q, n, out_U, out_grad, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace nuts
