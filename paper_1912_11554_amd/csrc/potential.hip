// Batched potential and gradient of the logistic log-joint at K positions,
// in one launch.  A grid of (G groups) x (K items); the NW waves of a group
// (8 for fp32 rows and wide fp64 rows, 16 for fp64 rows of at most 8 column
// slots) stream the blocks b = g * NW + w, g * NW + w + G * NW, ... of their
// item's data set, and the group adds its waves' column sums in wave order
// and stores its partial of each used column (the D gradient columns, then
// the loss) as one row of slots.  The used columns are cut into tiles of 16
// (one 128-byte line of each row); group g of the item owns the tiles g,
// g + G, ...: each slot holds a signalling-NaN pattern until it is written,
// so the owner's threads wait on the values themselves (no counter, no
// ordering point between a group's stores and a count).  The owner adds the
// G rows of each of its columns in a fixed order, adds the Gaussian prior
// term, writes its outputs (components of grad U, and U) and then marks the
// slots empty again for the next call.  One hop between groups per call;
// every transfer between groups moves whole lines; no floating-point atomics
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

// A slot not written yet: a signalling-NaN bit pattern that no arithmetic
// produces (sums of finite or non-finite values give quiet NaNs).
constexpr unsigned long long kEmptyPartial = 0x7FF4DEADBEEF0002ull;
// about 2 s of the 100 MHz constant clock: a slot that stays empty that long
// means another call overlapped this one on the device
constexpr uint64_t kGatherWaitTicks = 200000000ull;

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

// The 8-wave shapes run two waves per SIMD (one group per CU), so the
// compiler may give a lane up to 256 registers: left to aim at four waves
// per SIMD it squeezed the fp32 stream into 120 and the pass ran slower.
template <typename T, int S, int CPS>
__global__ void __launch_bounds__((pot_waves<T, S, CPS>() * kWave))
    __attribute__((amdgpu_waves_per_eu(1, pot_waves<T, S, CPS>() == 8 ? 2 : 4))) potential_grad_kernel(
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

    // the first block's loads go out before the position is read, so that
    // the two round trips overlap
    const int64_t first = (int64_t)g * NW + wave;
    BlockRegs<T, CPS, S> a;
    if (first < dv.nb) a = load_block<T, CPS, S, pot_mask<S, CPS>()>(X + first * D * R, y + first * R, D);
    double qv[CPS];
    spread_position_lds<CPS, S>(W + k * D, D, qv);
    double acc[CPS];
#pragma unroll
    for (int c = 0; c < CPS; ++c) acc[c] = 0.0;
    double loss = 0.0;
    if (first < dv.nb)
        stream_blocks_from<T, CPS, S, pot_pipe<T, S, CPS>(), pot_mask<S, CPS>()>(
            a, X, y, D, dv.N, dv.nb, first, (int64_t)G * NW, qv, acc, loss);

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
    // Row g of the item's slots (at item + g * width) holds the group's
    // partial of each used column: columns 0..D-1, the loss at D, then zeros
    // up to a whole number of 128-byte lines, so that every store and every
    // read between groups moves whole lines (a partial-line write to HBM is
    // a read-modify-write, and those slowed the other groups' streams).
    constexpr int kLine = 16;  // doubles in a 128-byte line
    const int used = D + 1;
    const int ntiles = (used + kLine - 1) / kLine;
    double* item = partials + k * G * width;
    if (wave == 0) {
        double* row = item + (int64_t)g * width;
        for (int col = l; col < ntiles * kLine; col += 64) {
            const int src = col < D ? col : (col == D ? loss_slot : -1);
            double s = 0.0;
            if (src >= 0) {
#pragma unroll
                for (int w = 0; w < NW; ++w) s += part[w * width + src];
            }
            store_agent(row + col, s);
        }
    }
    // Group g owns the tiles g, g + G, ... (tile j: used columns 16 j ..
    // 16 j + 15).  Its thread t takes column i = t mod 16 of the tile in rows
    // t / 16, t / 16 + RS, ... (RS = threads / 16), so that each load and
    // store of a wave covers whole lines, and waits for those slots; the
    // group adds the G rows of each column in a fixed order (each thread its
    // rows in order, then the four lanes of a wave that share the column,
    // then the waves in order) and writes the outputs, and only then marks
    // the slots empty again for the next call.
    constexpr int NT = NW * kWave;
    constexpr int RS = NT / kLine;
    constexpr int kMaxRows = (kMaxPotentialGroups + RS - 1) / RS;
    const int mine = g < ntiles ? (ntiles - 1 - g) / G + 1 : 0;
    if (mine == 0) return;  // uniform over the group
    const int t = threadIdx.x;
    const int ic = t & (kLine - 1);
    const int r0 = t / kLine;
    const double inv_s2 = 1.0 / (prior_scale * prior_scale);
    __syncthreads();  // the waves' rows are consumed: LDS is reused below
    for (int jt = 0; jt < mine; ++jt) {
        const int c0 = (g + jt * G) * kLine;
        const int col = c0 + ic;
        // what the outputs add besides the sums, read before the wait
        double extra = 0.0;
        if (col < D) extra = W[k * D + col] * inv_s2;
        if (wave == 0 && c0 <= D && D < c0 + kLine) {
            double pr = 0.0;
            for (int j = l; j < D; j += kWave) pr += 0.5 * W[k * D + j] * W[k * D + j] * inv_s2;
            const double prior = wave_sum(pr) + (double)D * (log(prior_scale) + kHalfLog2Pi);
            if (col == D) extra = prior;
        }
        // (one poll of the thread's slots at a time: more polls in flight, a
        // fraction of a round trip apart, made the slots arrive later)
        unsigned long long v[kMaxRows];
#pragma unroll
        for (int m = 0; m < kMaxRows; ++m) {
            const int r = r0 + m * RS;
            v[m] = r < G ? load_bits(item + (int64_t)r * width + col) : 0ull;  // 0: +0.0
        }
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        for (;;) {
            bool pending = false;
#pragma unroll
            for (int m = 0; m < kMaxRows; ++m) {
                const int r = r0 + m * RS;
                if (r < G && v[m] == kEmptyPartial) {
                    v[m] = load_bits(item + (int64_t)r * width + col);
                    pending = true;
                }
            }
            if (!pending) break;
            if (__builtin_amdgcn_s_memrealtime() - t0 > kGatherWaitTicks) {
                // another call overlapped this one: the results are NaN
                __hip_atomic_store(&failed, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
#pragma unroll
                for (int m = 0; m < kMaxRows; ++m) v[m] = v[m] == kEmptyPartial ? 0ull : v[m];
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        double s = 0.0;
#pragma unroll
        for (int m = 0; m < kMaxRows; ++m) s += __builtin_bit_cast(double, v[m]);
        s += xor_move<16>(s);
        s += xor_move<32>(s);
        if (l < kLine) part[wave * kLine + l] = s;
        __syncthreads();  // the waves' sums (and any failure) in LDS
        if (t < kLine && col <= D) {
            double tot = 0.0;
#pragma unroll
            for (int w = 0; w < NW; ++w) tot += part[w * kLine + t];
            const double bad = failed ? __builtin_nan("") : 0.0;
            if (col < D) out_grad[k * D + col] = tot + extra + bad;
            else out_U[k] = tot + extra + bad;
        }
#pragma unroll
        for (int m = 0; m < kMaxRows; ++m) {
            const int r = r0 + m * RS;
            if (r < G) empty_slot(item + (int64_t)r * width + col);  // for the next call
        }
        __syncthreads();  // part[] is reused by the next tile
    }
}

// Many items (K >= kItemMinK) of at most kItemMaxBlocks row blocks and
// D <= 64 (one lane a column): one wavefront an item, four a group.  The
// wave streams its item's blocks (the next block's loads in flight while the
// current one is computed), reduces the rows over the wave (column c in lane
// c) and writes U and grad U itself: no partial rows, no exchange.  With the
// multi-group kernel such an item took one group of 8 waves, most of them
// without a block, one group a CU.
constexpr int kItemWaves = 4;
constexpr int64_t kItemMaxBlocks = 32;
constexpr int64_t kItemMinK = 64;

template <typename T, int S, int CPS>
__global__ void __launch_bounds__(kItemWaves * kWave) potential_items_kernel(DataView dv,
                                                                             const double* __restrict__ W, int64_t K,
                                                                             double prior_scale,
                                                                             double* __restrict__ out_U,
                                                                             double* __restrict__ out_grad)
{
    constexpr int R = BlockShape<T, S>::R;
    constexpr bool kPipe = !(sizeof(T) == 8 && S == 1);  // fp64 rows of one lane: one register set
    const int l = lane();
    const int64_t k = (int64_t)blockIdx.x * kItemWaves + (int)(threadIdx.x / kWave);
    if (k >= K) return;  // uniform over the wave
    const int D = dv.D;
    const int64_t ds = dv.nds > 1 ? k : 0;
    const T* X = (const T*)dv.X + ds * dv.nb * (int64_t)D * R;
    const uint8_t* y = dv.y + ds * dv.nb * R;
    const double q = l < D ? W[k * D + l] : 0.0;
    double qv[CPS];
    spread_position<CPS, S>(q, qv);
    double acc[CPS];
#pragma unroll
    for (int c = 0; c < CPS; ++c) acc[c] = 0.0;
    double loss = 0.0;
    stream_blocks<T, CPS, S, kPipe, false>(X, y, D, dv.N, dv.nb, 0, 1, qv, acc, loss);
    const double col = finish_pass<CPS, S>(acc, loss);
    const double inv_s2 = 1.0 / (prior_scale * prior_scale);
    const double prior = wave_sum(0.5 * q * q * inv_s2);
    if (l < D) out_grad[k * D + l] = col + q * inv_s2;
    if (l == 0) out_U[k] = loss + prior + (double)D * (log(prior_scale) + kHalfLog2Pi);
}

template <typename T, int S, int CPS>
hipError_t enqueue_items(const DataView& dv, double prior_scale, const double* W, int64_t K, double* out_U,
                         double* out_grad, hipStream_t stream)
{
    hipLaunchKernelGGL((potential_items_kernel<T, S, CPS>), dim3((unsigned)((K + kItemWaves - 1) / kItemWaves)),
                       dim3(kItemWaves * kWave), 0, stream, dv, W, K, prior_scale, out_U, out_grad);
    return hipGetLastError();
}

template <typename T>
hipError_t enqueue_items_shape(const DataView& dv, double prior_scale, const double* W, int64_t K,
                               double* out_U, double* out_grad, hipStream_t stream)
{
    const int D = dv.D;
    if (D <= 8) return enqueue_items<T, 1, 8>(dv, prior_scale, W, K, out_U, out_grad, stream);
    if (D <= 16) return enqueue_items<T, 1, 16>(dv, prior_scale, W, K, out_U, out_grad, stream);
    if (D <= 32) return enqueue_items<T, 4, 8>(dv, prior_scale, W, K, out_U, out_grad, stream);
    return enqueue_items<T, 8, 8>(dv, prior_scale, W, K, out_U, out_grad, stream);
}

// The 8-wave shapes use at most 128 registers a lane, so two of their groups
// would fit in one CU, and the dispatcher does place two groups on one CU
// while another CU idles (the pass over the 581,012 x 55 fp32 set ran about
// 8 % slower that way).  Asking for more than half of a CU's 160 KiB of LDS
// gives every group a CU of its own, as the sizing of the grid assumes.
constexpr size_t kOwnCuLds = 96 * 1024;

template <typename T, int S, int CPS>
hipError_t enqueue(const DataView& dv, double prior_scale, const double* W, int64_t K, int G, int width,
                   bool own_cu, double* partials, double* out_U, double* out_grad, hipStream_t stream)
{
    constexpr int NW = pot_waves<T, S, CPS>();
    size_t lds = (size_t)NW * width * sizeof(double);
    // with more groups than CUs (many items) the groups share CUs instead
    if (NW == 8 && own_cu && lds < kOwnCuLds) lds = kOwnCuLds;
    const void* k = (const void*)potential_grad_kernel<T, S, CPS>;
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((potential_grad_kernel<T, S, CPS>), dim3(G, (unsigned)K), dim3(NW * kWave), lds, stream, dv,
                       W, G, width, partials, prior_scale, out_U, out_grad);
    return hipGetLastError();
}

template <typename T>
hipError_t enqueue_shape(const DataView& dv, double prior_scale, const double* W, int64_t K, int G, int width,
                         bool own_cu, double* partials, double* out_U, double* out_grad, hipStream_t stream)
{
    const int D = dv.D;
#define NUTS_POT(S_, C_) \
    return enqueue<T, S_, C_>(dv, prior_scale, W, K, G, width, own_cu, partials, out_U, out_grad, stream)
    if (D <= 8) NUTS_POT(1, 8);
    if (D <= 16) NUTS_POT(1, 16);
    if (D <= 32) NUTS_POT(4, 8);
    if (D <= 64) NUTS_POT(8, 8);
    if (D <= 128) NUTS_POT(16, 8);
    if (D <= 256) NUTS_POT(32, 8);
    NUTS_POT(32, 10);
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
    if (dv.D <= 64 && dv.nb <= kItemMaxBlocks && K >= kItemMinK)
        return PotentialPlan{1, partial_width(dv.D), false, true};
    // one group per CU over all items, never more groups than the blocks give
    // their waves work
    int64_t want = ((int64_t)num_cu + K - 1) / K;
    int64_t most = (dv.nb + 15) / 16;
    if (want > most) want = most;
    if (want > kMaxPotentialGroups) want = kMaxPotentialGroups;
    if (want < 1) want = 1;
    return PotentialPlan{(int)want, partial_width(dv.D), want * K <= num_cu, false};
}

hipError_t launch_potential_grad(const DataView& dv, double prior_scale, const double* W, int64_t K,
                                 const PotentialPlan& plan, double* partials, double* out_U, double* out_grad,
                                 hipStream_t stream)
{
    if (plan.items)
        return dv.dtype == NUTS_F64 ? enqueue_items_shape<double>(dv, prior_scale, W, K, out_U, out_grad, stream)
                                    : enqueue_items_shape<float>(dv, prior_scale, W, K, out_U, out_grad, stream);
    if (dv.dtype == NUTS_F64)
        return enqueue_shape<double>(dv, prior_scale, W, K, plan.groups_per_item, plan.width, plan.own_cu, partials, out_U,
                                     out_grad, stream);
    return enqueue_shape<float>(dv, prior_scale, W, K, plan.groups_per_item, plan.width, plan.own_cu, partials, out_U, out_grad,
                                stream);
}

}  // namespace nuts
