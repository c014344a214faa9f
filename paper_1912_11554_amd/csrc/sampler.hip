// Host-side dispatch of the sampler kernels (sampler_impl.h): path support,
// grid size, launches.
#include "sampler_impl.h"

namespace nuts {

namespace {

// Every exchange slot empty and the error flag clear, before a launch.
__global__ void fill_empty_slots(double* a, int64_t na, double* b, int64_t nb, GridSync* sync)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t first = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (first == 0) sync->error = 0u;
    for (int64_t i = first; i < na + nb; i += stride) {
        unsigned long long* p = reinterpret_cast<unsigned long long*>(i < na ? a + i : b + (i - na));
        *p = sampler::kEmptySlot;
    }
}

const void* pick_grid_kernel(const DataView& dv, bool adapt)
{
    if (adapt) return dv.dtype == NUTS_F64 ? grid_kernel_ext_f64(dv) : grid_kernel_ext_f32(dv);
    return dv.dtype == NUTS_F64 ? grid_kernel_f64(dv) : grid_kernel_f32(dv);
}

}  // namespace

bool wave_path_supports(const DataView& dv) { return dv.D <= 64; }

bool wave_path_resident(const SamplerArgs& a)
{
    return a.data.dtype == NUTS_F64 ? wave_resident_f64(a) : wave_resident_f32(a);
}

hipError_t launch_sampler_wave(const SamplerArgs& a, hipStream_t stream)
{
    if (sampler_extended(a))
        return a.data.dtype == NUTS_F64 ? launch_sampler_wave_ext_f64(a, stream)
                                        : launch_sampler_wave_ext_f32(a, stream);
    return a.data.dtype == NUTS_F64 ? launch_sampler_wave_f64(a, stream) : launch_sampler_wave_f32(a, stream);
}

int grid_sampler_groups(const DataView& dv, int max_depth, int sub_merge, int num_cu)
{
    const void* k = pick_grid_kernel(dv, sub_merge != 0);
    int per_cu = 0;
    const size_t lds = (size_t)chain_lds_doubles(dv.D, max_depth, sub_merge, grid_edge_nodes(dv.D)) * sizeof(double);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, kGridWaves * kWave, lds) != hipSuccess)
        per_cu = 1;
    else if (per_cu < 1)
        return 0;  // the group's LDS does not fit a CU
    if (per_cu > 1) per_cu = 1;
    int64_t groups = (int64_t)num_cu * per_cu;
    const int64_t most = (dv.nb + kGridWaves - 2) / (kGridWaves - 1);
    if (groups > most) groups = most;
    // a group gathers the partials of its used columns in one pass of its
    // worker lanes: ceil((D + 1) / groups) * groups <= D + groups slots
    const int64_t gather = (int64_t)(kGridWaves - 1) * kWave - dv.D;
    if (groups > gather) groups = gather;
    if (groups < 1) groups = 1;
    return (int)groups;
}

hipError_t launch_sampler_grid(const SamplerArgs& a, int groups, double* partials, double* result,
                               GridSync* sync, hipStream_t stream, hipEvent_t at_launch)
{
    hipLaunchKernelGGL(fill_empty_slots, dim3(64), dim3(256), 0, stream, partials,
                       grid_partial_elems(a.data.D, groups), result, grid_result_elems(a.data.D), sync);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const void* k = pick_grid_kernel(a.data, sampler_extended(a));
    // the chain's state, then as many resident blocks a worker as the rest
    // of the group's LDS holds (at most one fewer than the smallest share)
    hipFuncAttributes attr;
    e = hipFuncGetAttributes(&attr, k);
    if (e != hipSuccess) return e;
    const size_t chain = grid_resident_offset(a.data.D, a.max_depth, a.sub_merge);
    const size_t block = (size_t)lds_block_bytes(a.data.dtype, a.data.split, a.data.cols);
    const size_t used = attr.sharedSizeBytes + chain;
    int64_t resident = used < sampler::kMaxGroupLds ? (int64_t)((sampler::kMaxGroupLds - used) / ((kGridWaves - 1) * block)) : 0;
    const int64_t smallest_share = a.data.nb / ((int64_t)groups * (kGridWaves - 1));
    if (resident > smallest_share - 1) resident = smallest_share > 1 ? smallest_share - 1 : 0;
    int res = (int)resident;
    const size_t lds = chain + (size_t)res * (kGridWaves - 1) * block;
    e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    if (at_launch) {
        e = hipEventRecord(at_launch, stream);
        if (e != hipSuccess) return e;
    }
    SamplerArgs A = a;
    void* args[] = {&A, &groups, &res, &partials, &result, &sync};
    return hipLaunchCooperativeKernel(k, dim3(groups), dim3(kGridWaves * kWave), args, (unsigned)lds, stream);
}

}  // namespace nuts
