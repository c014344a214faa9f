// Row-major X [nds][N][D] -> column blocks of R rows, so that a wave reading
// one column slot of a block touches one contiguous segment.  Labels are
// copied to the same padded row order and checked to be 0 or 1.
#include "device.h"
#include "launch.h"

namespace nuts {

template <typename T>
__global__ void __launch_bounds__(256) to_blocks_kernel(const T* __restrict__ src,
                                                        const uint8_t* __restrict__ ysrc,
                                                        T* __restrict__ dst, uint8_t* __restrict__ ydst,
                                                        int64_t N, int D, int R, int64_t nb,
                                                        int64_t nds, unsigned int* bad_label)
{
    // one thread per destination element; consecutive threads write
    // consecutive rows of one block column
    const int64_t per_ds = nb * (int64_t)D * R;
    const int64_t total = per_ds * nds;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int64_t s = o / per_ds;
        const int64_t rem = o - s * per_ds;
        const int64_t b = rem / ((int64_t)D * R);
        const int64_t rem2 = rem - b * (int64_t)D * R;
        const int c = (int)(rem2 / R);
        const int r = (int)(rem2 - (int64_t)c * R);
        const int64_t row = b * R + r;
        T v = T(0);
        if (row < N) v = src[(s * N + row) * D + c];
        dst[o] = v;
        if (c == 0) {
            uint8_t yy = 0;
            if (row < N) {
                yy = ysrc[s * N + row];
                if (yy > 1) atomicOr(bad_label, 1u);
            }
            ydst[(s * nb + b) * R + r] = yy;
        }
    }
}

hipError_t launch_to_blocks(const void* X_rowmajor, const uint8_t* y_in, DataView dst, void* X_out,
                            uint8_t* y_out, unsigned int* bad_label, hipStream_t stream)
{
    const int R = rows_per_block(dst);
    const int64_t total = dst.nb * (int64_t)dst.D * R * dst.nds;
    if (total == 0) return hipSuccess;
    const int threads = 256;
    int64_t want = (total + threads - 1) / threads;
    const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
    if (dst.dtype == NUTS_F64)
        hipLaunchKernelGGL(to_blocks_kernel<double>, dim3(grid), dim3(threads), 0, stream,
                           (const double*)X_rowmajor, y_in, (double*)X_out, y_out, dst.N, dst.D, R,
                           dst.nb, dst.nds, bad_label);
    else
        hipLaunchKernelGGL(to_blocks_kernel<float>, dim3(grid), dim3(threads), 0, stream,
                           (const float*)X_rowmajor, y_in, (float*)X_out, y_out, dst.N, dst.D, R,
                           dst.nb, dst.nds, bad_label);
    return hipGetLastError();
}

}  // namespace nuts
