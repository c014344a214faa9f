// Sampler kernels with the optional features compiled in (warmup step-size
// adaptation, the generalised U-turn criterion), for double data (their own
// translation unit keeps the build parallel).
#include "sampler_impl.h"

namespace nuts {

hipError_t launch_sampler_wave_ext_f64(const SamplerArgs& a, hipStream_t stream)
{
    return sampler::wave_launch_split<double, true>(a, stream);
}

const void* grid_kernel_ext_f64(const DataView& dv)
{
    return sampler::grid_kernel_for<double, true>(dv);
}

}  // namespace nuts
