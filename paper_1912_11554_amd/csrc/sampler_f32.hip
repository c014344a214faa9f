// Sampler kernels instantiated for float data (one translation unit per data
// type keeps the build parallel).
#include "sampler_impl.h"

namespace nuts {

hipError_t launch_sampler_wave_f32(const SamplerArgs& a, hipStream_t stream)
{
    return sampler::wave_launch_split<float, false>(a, stream);
}

bool wave_resident_f32(const SamplerArgs& a)
{
    return sampler::wave_resident_split<float>(a);
}

const void* grid_kernel_f32(const DataView& dv)
{
    return sampler::grid_kernel_for<float, false>(dv);
}

}  // namespace nuts
