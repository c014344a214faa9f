// Semi-supervised HMM sampler with the optional features compiled in (warmup
// step-size adaptation, the generalised U-turn criterion).
#include "hmm_impl.h"

namespace nuts {

hipError_t launch_hmm_sampler_ext(const SamplerArgs& a, const HmmView& hv, hipStream_t stream)
{
    return hmm::hmm_sampler_dispatch<true>(a, hv, stream);
}

}  // namespace nuts
