// Batched potential and gradient of the logistic log-joint at K positions,
// in one launch.  A grid of (G groups) x (K items); the NW waves of a group
// (8 for fp32 rows and wide fp64 rows, 16 for fp64 rows of at most 8 column
// slots) stream the blocks b = g * NW + w, g * NW + w + G * NW, ... of their
// item's data set, the group adds its waves' column sums in wave order and
// stores one fp64 partial row of width partial_width(D) (columns 0..D-1, the
// loss at 64 * ceil(D / 64)) into its slots, and every group but the item's
// first is done.  The first group, once its own rows are in, gathers the G
// partial rows: each slot holds a signalling-NaN pattern until it is written,
// so the gatherer waits on the values themselves (no counter, no ordering
// point between a group's stores and a count).  It adds them in a fixed
// order, adds the Gaussian prior terms, writes U and grad U, and marks every
// slot it read empty again for the next call.  No floating-point atomics
// anywhere, so results are bitwise reproducible.
#include <algorithm>
#include <mutex>

#include "launch.h"
#include "rows.h"

// Workspace of the allocation-free potential entry point: partial-row slots,
// marked empty when the library sets the device up.  Every device the
// library runs on holds its own copy until the process ends.  Host code
// never passes this name to a kernel or a copy (on the host it only stands
// for the symbol): it uses the address hipGetSymbolAddress gives for the
// current device.
static __device__ __align__(256) unsigned char scratch[nuts::kStaticScratchBytes];

namespace nuts {

namespace {

constexpr double kHalfLog2Pi = 0.91893853320467274178032973640562;

// waves per group: fp64 rows of at most 8 column slots take 16 waves (4 per
// SIMD, 128 registers a lane, one block register set); every other shape
// takes 8 waves, whose registers hold two block register sets (fp32 rows
// carry two rows a lane, converted to fp64 in registers, and wide rows carry
// 10 or 16 slots)
template <typename T, int S, int CPS>
constexpr int pot_waves() { return (sizeof(T) == 8 && CPS == 8) ? 16 : 8; }
// two block register sets in the stream for the 8-wave shapes and for fp64
// rows shared by several lanes (fp64 rows of one lane would spill with two);
// the lane-masked loads of the last column slots for wide rows
template <typename T, int S, int CPS>
constexpr bool pot_pipe() { return pot_waves<T, S, CPS>() == 8 || S > 1; }
template <int S, int CPS>
constexpr bool pot_mask() { return S >= 16; }
static_assert(kMaxDim + 1 <= 8 * kWave, "one thread per used column in the final sum");

// A slot not written yet: a signalling-NaN bit pattern that no arithmetic
// produces (sums of finite or non-finite values give quiet NaNs).
constexpr unsigned long long kEmptyPartial = 0x7FF4DEADBEEF0002ull;
// about 2 s of the 100 MHz constant clock: a slot that stays empty that long
// means another call overlapped this one on the device
constexpr uint64_t kGatherWaitTicks = 200000000ull;
// slots a gathering thread has in flight at once: enough for every slot of
// the covtype-sized shapes (G = 256 groups, D + 1 = 56 used columns) in one
// batch, 32 with 512 threads, 16 with 1024
template <int NW>
constexpr int gather_batch() { return NW == 16 ? 16 : 32; }

__device__ __forceinline__ void store_agent(double* p, double v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long load_bits(const double* p)
{
    return __hip_atomic_load(reinterpret_cast<unsigned long long*>(const_cast<double*>(p)), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void empty_slot(double* p)
{
    __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), kEmptyPartial, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

__global__ void __launch_bounds__(256) fill_empty_kernel(unsigned long long* __restrict__ p, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
        p[i] = kEmptyPartial;
}

template <typename T, int S, int CPS>
__global__ void __launch_bounds__((pot_waves<T, S, CPS>() * kWave)) potential_grad_kernel(
    DataView dv, const double* __restrict__ W, int G, int width, double* __restrict__ partials,
    double prior_scale, double* __restrict__ out_U, double* __restrict__ out_grad)
{
    constexpr int R = BlockShape<T, S>::R;
    constexpr int NW = pot_waves<T, S, CPS>();
    extern __shared__ double part[];  // [NW][width], later the per-set sums
    __shared__ int failed;
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
    stream_blocks<T, CPS, S, pot_pipe<T, S, CPS>(), pot_mask<S, CPS>()>(
        X, y, D, dv.N, dv.nb, (int64_t)g * NW + wave, (int64_t)G * NW, qv, acc, loss);

    double* row = part + wave * width;
    if constexpr (S <= 8 && CPS == 8) {
        const double col = finish_pass<CPS, S>(acc, loss);
        if (l < D) row[l] = col;
        if (l == 0) row[loss_slot] = loss;
    } else {
        finish_pass_to_row<CPS, S>(acc, loss, row, D, loss_slot);
    }
    if (threadIdx.x == 0) failed = 0;
    __syncthreads();  // per-wave sums in LDS
    double* item = partials + k * G * width;
    if (wave == 0) {
        double* mine = item + (int64_t)g * width;
        for (int col = l; col < width; col += 64) {
            if (col < D || col == loss_slot) {
                double s = 0.0;
#pragma unroll
                for (int w = 0; w < NW; ++w) s += part[w * width + col];
                store_agent(mine + col, s);
            }
        }
    }
    if (g != 0) return;

    // The item's first group gathers.  Thread t takes used column c = t mod
    // (D + 1) (column c < D, or the loss for c = D) of the groups j, j + J,
    // j + 2 J, ... (j = t div (D + 1), J sets) in increasing order, waiting on
    // each slot until it holds a value.
    const int used = D + 1;
    const int t = threadIdx.x;
    const int sets = (NW * kWave) / used;
    const int j = t / used;
    const int c = t - j * used;
    constexpr int kGatherBatch = gather_batch<NW>();
    double s = 0.0;
    bool ok = true;
    if (j < sets) {
        double* src = item + (c < D ? c : loss_slot);
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        for (int g0 = j; g0 < G; g0 += kGatherBatch * sets) {
            unsigned long long v[kGatherBatch];
#pragma unroll
            for (int i = 0; i < kGatherBatch; ++i) {
                const int gg = g0 + i * sets;
                v[i] = gg < G ? load_bits(src + (int64_t)gg * width) : 0ull;
            }
            for (;;) {
                bool pending = false;
#pragma unroll
                for (int i = 0; i < kGatherBatch; ++i) {
                    const int gg = g0 + i * sets;
                    if (gg < G && v[i] == kEmptyPartial) {
                        v[i] = load_bits(src + (int64_t)gg * width);
                        pending = true;
                    }
                }
                if (!pending) break;
                if (__builtin_amdgcn_s_memrealtime() - t0 > kGatherWaitTicks) {
                    ok = false;
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
            }
#pragma unroll
            for (int i = 0; i < kGatherBatch; ++i) {
                const int gg = g0 + i * sets;
                if (gg < G) {
                    s += __builtin_bit_cast(double, v[i]);
                    empty_slot(src + (int64_t)gg * width);  // for the next call
                }
            }
        }
    }
    if (!ok) __hip_atomic_store(&failed, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __syncthreads();  // no wave reads its LDS row any more
    if (j < sets) part[j * used + c] = s;
    __syncthreads();  // per-set sums in LDS
    if (wave != 0) return;
    // a slot that never filled: another call overlapped this one; the
    // results are NaN (every slot this group read is empty again)
    const double bad = failed ? __builtin_nan("") : 0.0;
    const double inv_s2 = 1.0 / (prior_scale * prior_scale);
    double pr = 0.0;
    double lossv = 0.0;
    for (int col = l; col < used; col += 64) {
        double tot = 0.0;
        for (int jj = 0; jj < sets; ++jj) tot += part[jj * used + col];
        if (col < D) {
            const double w = W[k * D + col];
            pr += 0.5 * w * w * inv_s2;
            out_grad[k * D + col] = tot + w * inv_s2 + bad;
        } else {
            lossv = tot;
        }
    }
    const double prior = wave_sum(pr);
    lossv = readlane_f64(lossv, D & 63);  // column D sits in lane D mod 64
    if (l == 0) out_U[k] = lossv + prior + (double)D * (log(prior_scale) + kHalfLog2Pi) + bad;
}

template <typename T, int S, int CPS>
void enqueue(const DataView& dv, double prior_scale, const double* W, int64_t K, int G, int width,
             double* partials, double* out_U, double* out_grad, hipStream_t stream)
{
    constexpr int NW = pot_waves<T, S, CPS>();
    hipLaunchKernelGGL((potential_grad_kernel<T, S, CPS>), dim3(G, (unsigned)K), dim3(NW * kWave),
                       (size_t)NW * width * sizeof(double), stream, dv, W, G, width, partials, prior_scale,
                       out_U, out_grad);
}

template <typename T>
void enqueue_shape(const DataView& dv, double prior_scale, const double* W, int64_t K, int G, int width,
                   double* partials, double* out_U, double* out_grad, hipStream_t stream)
{
    const int D = dv.D;
#define NUTS_POT(S_, C_) \
    enqueue<T, S_, C_>(dv, prior_scale, W, K, G, width, partials, out_U, out_grad, stream)
    if (D <= 8) NUTS_POT(1, 8);
    else if (D <= 16) NUTS_POT(1, 16);
    else if (D <= 32) NUTS_POT(4, 8);
    else if (D <= 64) NUTS_POT(8, 8);
    else if (D <= 128) NUTS_POT(16, 8);
    else if (D <= 256) NUTS_POT(32, 8);
    else NUTS_POT(32, 10);
#undef NUTS_POT
}

}  // namespace

namespace {

__global__ void __launch_bounds__(64) ll_from_potential_kernel(int D, const double* __restrict__ W, int64_t S,
                                                              const double* __restrict__ U,
                                                              double* __restrict__ out_ll)
{
    const int64_t s = (int64_t)blockIdx.x * 64 + threadIdx.x;
    if (s >= S) return;
    double pr = 0.0;
    for (int j = 0; j < D; ++j) pr += 0.5 * W[s * D + j] * W[s * D + j];
    out_ll[s] = -(U[s] - pr - (double)D * kHalfLog2Pi);
}

// One wave: the largest term factored out, then the exponentials summed by
// lane (draws l, l + 64, ... in order) and across lanes in a fixed order.
__global__ void __launch_bounds__(64) expected_ll_kernel(const double* __restrict__ ll, int64_t S,
                                                        double* __restrict__ out)
{
    const int l = lane();
    double mx = -INFINITY;
    for (int64_t s = l; s < S; s += 64) mx = fmax(mx, ll[s]);
#pragma unroll
    for (int b = 1; b < 64; b <<= 1) mx = fmax(mx, __shfl_xor(mx, b));
    double acc = 0.0;
    for (int64_t s = l; s < S; s += 64) acc += exp(ll[s] - mx);
    acc = wave_sum(acc);
    if (l == 0) *out = mx + log(acc) - log((double)S);
}

}  // namespace

hipError_t launch_ll_from_potential(int D, const double* W, int64_t S, const double* U, double* out_ll,
                                    hipStream_t stream)
{
    hipLaunchKernelGGL(ll_from_potential_kernel, dim3((unsigned)((S + 63) / 64)), dim3(64), 0, stream, D, W, S, U,
                       out_ll);
    return hipGetLastError();
}

hipError_t launch_expected_ll(const double* ll, int64_t S, double* out, hipStream_t stream)
{
    hipLaunchKernelGGL(expected_ll_kernel, dim3(1), dim3(64), 0, stream, ll, S, out);
    return hipGetLastError();
}

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_static_mutex;
void* g_static_ptr[kMaxDevices] = {};

}  // namespace

hipError_t mark_partials_empty(double* p, int64_t n, hipStream_t stream)
{
    if (n <= 0) return hipSuccess;
    const int64_t groups = std::min<int64_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(fill_empty_kernel, dim3((unsigned)groups), dim3(256), 0, stream,
                       reinterpret_cast<unsigned long long*>(p), n);
    return hipGetLastError();
}

hipError_t static_workspace_setup(int device, hipStream_t stream, void** out)
{
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_static_mutex);
    if (!g_static_ptr[device]) {
        // the caller has made `device` current: the symbol's address is this
        // device's copy of the array
        void* p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        // every slot starts empty (each call leaves the slots it used empty)
        e = mark_partials_empty((double*)p, (int64_t)(kStaticScratchBytes / sizeof(double)), stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) return e;
        g_static_ptr[device] = p;
    }
    *out = g_static_ptr[device];
    return hipSuccess;
}

PotentialPlan plan_potential(const DataView& dv, int64_t K, int num_cu)
{
    // one group per CU over all items, never more groups than the blocks give
    // their waves work
    int64_t want = ((int64_t)num_cu + K - 1) / K;
    int64_t most = (dv.nb + 15) / 16;
    if (want > most) want = most;
    if (want < 1) want = 1;
    return PotentialPlan{(int)want, partial_width(dv.D)};
}

hipError_t launch_potential_grad(const DataView& dv, double prior_scale, const double* W, int64_t K,
                                 const PotentialPlan& plan, double* partials, double* out_U, double* out_grad,
                                 hipStream_t stream)
{
    if (dv.dtype == NUTS_F64)
        enqueue_shape<double>(dv, prior_scale, W, K, plan.groups_per_item, plan.width, partials, out_U, out_grad,
                              stream);
    else
        enqueue_shape<float>(dv, prior_scale, W, K, plan.groups_per_item, plan.width, partials, out_U, out_grad,
                             stream);
    return hipGetLastError();
}

}  // namespace nuts
