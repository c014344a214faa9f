// Sampler kernels instantiated for double data (one translation unit per data
// type keeps the build parallel).
#include "sampler_impl.h"

namespace nuts {

hipError_t launch_sampler_wave_f64(const SamplerArgs& a, hipStream_t stream)
{
    return sampler::wave_launch_split<double, false>(a, stream);
}

bool wave_resident_f64(const SamplerArgs& a)
{
    return sampler::wave_resident_split<double>(a);
}

const void* grid_kernel_f64(const DataView& dv)
{
    return sampler::grid_kernel_for<double, false>(dv);
}

}  // namespace nuts
