// C ABI of the NUTS library: argument validation, host/device pointer
// handling, device-layout data sets, path selection and launches.  No C++
// exception or abort crosses this boundary; every failure is a status code
// plus a message kept on the handle.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/nuts.h"
#include "launch.h"
#include "rows.h"

using namespace nuts;

struct nuts_data {
    DataView view;
    void* X = nullptr;
    uint8_t* y = nullptr;
    // row-stage copy for the batched (matrix-core) path, built on first use
    BatchView batch{};
    float* bX = nullptr;
    uint8_t* by = nullptr;
};

static void free_data_buffers(nuts_data* d)
{
    if (d->X) (void)hipFree(d->X);
    if (d->y) (void)hipFree(d->y);
    if (d->bX) (void)hipFree(d->bX);
    if (d->by) (void)hipFree(d->by);
}

struct nuts_handle {
    int device = 0;
    hipStream_t stream = nullptr;
    bool own_stream = false;
    int num_cu = 0;
    std::string err;
    // grow-only device scratch for partial sums and exchange buffers; a call
    // uses it between its launches and its final stream synchronisation
    void* scratch = nullptr;
    size_t scratch_bytes = 0;
    // partial-sum slots of the potential kernel, grow-only, marked empty on
    // allocation; every launch leaves the slots it used empty again
    double* pot_slots = nullptr;
    size_t pot_slot_bytes = 0;
    // this device's copy of the fixed workspace of the allocation-free entry
    // point (set up by nuts_init; never freed)
    void* static_ws = nullptr;
    // per-chain gradient-evaluation counts of a sampling call, grow-only, so
    // that a call on device-resident buffers allocates nothing before its
    // kernel starts
    unsigned long long* evals = nullptr;
    int64_t evals_cap = 0;
    // pinned host memory for the small read-backs that end a call (the
    // evaluation counts, a kernel's error flag), so that they are
    // asynchronous copies ahead of one stream synchronisation
    void* pinned = nullptr;
    size_t pinned_bytes = 0;
    // the events of nuts_sample_opts.out_kernel_ms, created on first use
    hipEvent_t kev[2] = {nullptr, nullptr};
};

// The handle's two timing events (created on first use).
static hipError_t handle_events(nuts_handle* h, hipEvent_t** out)
{
    for (int i = 0; i < 2; ++i) {
        if (!h->kev[i]) {
            hipError_t e = hipEventCreate(&h->kev[i]);
            if (e != hipSuccess) {
                h->kev[i] = nullptr;
                return e;
            }
        }
    }
    *out = h->kev;
    return hipSuccess;
}

static hipError_t handle_pinned(nuts_handle* h, size_t bytes, void** out)
{
    if (bytes > h->pinned_bytes) {
        if (h->pinned) {
            hipError_t e = hipStreamSynchronize(h->stream);
            if (e != hipSuccess) return e;
            (void)hipHostFree(h->pinned);
            h->pinned = nullptr;
            h->pinned_bytes = 0;
        }
        hipError_t e = hipHostMalloc(&h->pinned, bytes, hipHostMallocDefault);
        if (e != hipSuccess) {
            h->pinned = nullptr;
            return e;
        }
        h->pinned_bytes = bytes;
    }
    *out = h->pinned;
    return hipSuccess;
}

static hipError_t handle_evals(nuts_handle* h, int64_t C, unsigned long long** out)
{
    if (C > h->evals_cap) {
        if (h->evals) {
            hipError_t e = hipStreamSynchronize(h->stream);
            if (e != hipSuccess) return e;
            (void)hipFree(h->evals);
            h->evals = nullptr;
            h->evals_cap = 0;
        }
        hipError_t e = hipMalloc(&h->evals, (size_t)C * sizeof(unsigned long long));
        if (e != hipSuccess) return e;
        h->evals_cap = C;
    }
    *out = h->evals;
    return hipSuccess;
}

// Partial-sum slots of the potential kernel for `bytes`, all empty.
static hipError_t potential_slots(nuts_handle* h, size_t bytes, double** out)
{
    if (bytes > h->pot_slot_bytes) {
        if (h->pot_slots) {
            hipError_t e = hipStreamSynchronize(h->stream);
            if (e != hipSuccess) return e;
            (void)hipFree(h->pot_slots);
            h->pot_slots = nullptr;
            h->pot_slot_bytes = 0;
        }
        hipError_t e = hipMalloc(&h->pot_slots, bytes);
        if (e != hipSuccess) {
            h->pot_slots = nullptr;
            return e;
        }
        e = mark_partials_empty(h->pot_slots, (int64_t)(bytes / sizeof(double)), h->stream);
        if (e != hipSuccess) {
            (void)hipFree(h->pot_slots);
            h->pot_slots = nullptr;
            return e;
        }
        h->pot_slot_bytes = bytes;
    }
    *out = h->pot_slots;
    return hipSuccess;
}

// Scratch of at least `bytes`, 256-byte aligned, owned by the handle.
static hipError_t handle_scratch(nuts_handle* h, size_t bytes, void** out)
{
    if (bytes > h->scratch_bytes) {
        if (h->scratch) {
            hipError_t e = hipStreamSynchronize(h->stream);
            if (e != hipSuccess) return e;
            (void)hipFree(h->scratch);
            h->scratch = nullptr;
            h->scratch_bytes = 0;
        }
        hipError_t e = hipMalloc(&h->scratch, bytes);
        if (e != hipSuccess) return e;
        h->scratch_bytes = bytes;
    }
    *out = h->scratch;
    return hipSuccess;
}

static size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

static thread_local std::string g_init_error;

static int fail(nuts_handle* h, int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (h) h->err = buf;
    else g_init_error = buf;
    return code;
}

#define HIP_TRY(h, expr)                                                                         \
    do {                                                                                         \
        hipError_t e_ = (expr);                                                                  \
        if (e_ != hipSuccess)                                                                    \
            return fail((h), e_ == hipErrorOutOfMemory ? NUTS_ENOMEM : NUTS_EDEVICE, "%s: %s", \
                        #expr, hipGetErrorString(e_));                                           \
    } while (0)

namespace {

// Device memory owned for the duration of one call.
struct DevBuf {
    void* p = nullptr;
    DevBuf() = default;
    DevBuf(const DevBuf&) = delete;
    DevBuf& operator=(const DevBuf&) = delete;
    ~DevBuf()
    {
        if (p) (void)hipFree(p);
    }
    hipError_t alloc(size_t bytes)
    {
        return hipMalloc(&p, bytes ? bytes : 1);
    }
};

// True if `p` is device-accessible memory allocated by HIP (device or
// managed); plain or pinned host memory is copied explicitly instead.
bool is_device_ptr(const void* p)
{
    if (!p) return false;
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();  // clear the sticky "invalid value" of unknown host memory
        return false;
    }
    return attr.type == hipMemoryTypeDevice || attr.type == hipMemoryTypeManaged;
}

// Make a device copy of a host input (or pass a device input through).
hipError_t stage_in(const void* src, size_t bytes, DevBuf& tmp, const void** dev, hipStream_t s)
{
    if (!src || bytes == 0) {
        *dev = src;
        return hipSuccess;
    }
    if (is_device_ptr(src)) {
        *dev = src;
        return hipSuccess;
    }
    hipError_t e = tmp.alloc(bytes);
    if (e != hipSuccess) return e;
    e = hipMemcpyAsync(tmp.p, src, bytes, hipMemcpyHostToDevice, s);
    *dev = tmp.p;
    return e;
}

// A caller output: written in place if on the device, else through `tmp`
// and copied back by finish_out.
hipError_t stage_out(void* dst, size_t bytes, DevBuf& tmp, void** dev)
{
    if (!dst) {
        *dev = nullptr;
        return hipSuccess;
    }
    if (is_device_ptr(dst)) {
        *dev = dst;
        return hipSuccess;
    }
    hipError_t e = tmp.alloc(bytes);
    *dev = tmp.p;
    return e;
}

hipError_t finish_out(void* dst, size_t bytes, const DevBuf& tmp, hipStream_t s)
{
    if (!dst || !tmp.p || bytes == 0) return hipSuccess;
    return hipMemcpyAsync(dst, tmp.p, bytes, hipMemcpyDeviceToHost, s);
}

size_t elem_size(int dtype) { return dtype == NUTS_F64 ? 8 : 4; }

bool finite_pos(double x) { return std::isfinite(x) && x > 0.0; }

// hipSetDevice for the handle's device for the lifetime of a call.
struct DeviceScope {
    int prev = -1;
    explicit DeviceScope(int dev)
    {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        (void)hipSetDevice(dev);
    }
    ~DeviceScope()
    {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

// Arguments every sampling entry point shares.
int check_run(nuts_handle* h, uint32_t flags, uint32_t allowed, const nuts_sample_opts& o, double step_size,
              int max_tree_depth, int64_t num_warmup, int64_t num_samples, int64_t num_chains,
              double* target_accept)
{
    if (flags & ~allowed) return fail(h, NUTS_EINVAL, "unknown flag bits 0x%x", flags & ~allowed);
    *target_accept = o.target_accept == 0.0 ? 0.8 : o.target_accept;
    if (!(*target_accept > 0.0 && *target_accept < 1.0))
        return fail(h, NUTS_EINVAL, "target_accept must be in (0, 1) (got %g)", o.target_accept);
    if (!finite_pos(step_size)) return fail(h, NUTS_EINVAL, "step_size must be finite and > 0");
    if (max_tree_depth < 1 || max_tree_depth > 30)
        return fail(h, NUTS_EINVAL, "max_tree_depth must be in [1, 30] (got %d)", max_tree_depth);
    if (num_warmup < 0) return fail(h, NUTS_EINVAL, "num_warmup must be >= 0");
    if (num_samples < 1) return fail(h, NUTS_EINVAL, "num_samples must be >= 1");
    if (num_chains < 1) return fail(h, NUTS_EINVAL, "num_chains must be >= 1");
    if (o.first_iter < 0) return fail(h, NUTS_EINVAL, "first_iter must be >= 0");
    return NUTS_OK;
}

int check_inv_mass(nuts_handle* h, const double* inv_mass_diag, int D)
{
    if (!inv_mass_diag) return NUTS_OK;
    std::vector<double> im(D);
    if (is_device_ptr(inv_mass_diag)) {
        DeviceScope ds(h->device);
        HIP_TRY(h, hipMemcpy(im.data(), inv_mass_diag, (size_t)D * 8, hipMemcpyDeviceToHost));
    } else {
        std::memcpy(im.data(), inv_mass_diag, (size_t)D * 8);
    }
    for (int i = 0; i < D; ++i)
        if (!finite_pos(im[i])) return fail(h, NUTS_EINVAL, "inv_mass_diag[%d] must be finite and > 0", i);
    return NUTS_OK;
}

// Device copies of a sampling call's inputs and outputs, and the sampler
// arguments that point at them.
struct RunBuffers {
    DevBuf imb, iqb, smp, sts, fq, fim, fep;
    unsigned long long* gev = nullptr;  // the handle's counts
    int64_t C = 0, S = 0, D = 0;
    hipStream_t s = nullptr;

    // a.data and the model fields are the caller's; the rest is set here
    int stage(nuts_handle* h, SamplerArgs& a, uint32_t flags, const nuts_sample_opts& o, double target_accept,
              double step_size, const double* inv_mass_diag, int max_tree_depth, int64_t num_warmup,
              int64_t num_samples, int64_t num_chains, uint64_t seed, double* out_samples, nuts_stats* out_stats)
    {
        C = num_chains;
        S = num_samples;
        D = a.data.D;
        s = h->stream;
        const void *im_d = nullptr, *iq_d = nullptr;
        void *smp_d = nullptr, *sts_d = nullptr, *fq_d = nullptr, *fim_d = nullptr, *fep_d = nullptr;
        HIP_TRY(h, stage_in(inv_mass_diag, (size_t)D * 8, imb, &im_d, s));
        HIP_TRY(h, stage_in(o.init_q, (size_t)C * D * 8, iqb, &iq_d, s));
        HIP_TRY(h, stage_out(out_samples, (size_t)C * S * D * 8, smp, &smp_d));
        HIP_TRY(h, stage_out(out_stats, (size_t)C * S * sizeof(nuts_stats), sts, &sts_d));
        HIP_TRY(h, stage_out(o.out_final_q, (size_t)C * D * 8, fq, &fq_d));
        HIP_TRY(h, stage_out(o.out_inv_mass, (size_t)C * D * 8, fim, &fim_d));
        HIP_TRY(h, stage_out(o.out_step_size, (size_t)C * 8, fep, &fep_d));
        HIP_TRY(h, handle_evals(h, C, &gev));
        a.step_size = step_size;
        a.inv_mass = (const double*)im_d;
        a.max_depth = max_tree_depth;
        a.num_warmup = num_warmup;
        a.num_samples = num_samples;
        a.num_chains = C;
        a.chain_offset = 0;
        a.seed = seed;
        a.first_iter = o.first_iter;
        a.adapt_diag = (flags & NUTS_ADAPT_DIAG_MASS) ? 1 : 0;
        a.adapt_step = (flags & NUTS_ADAPT_STEP_SIZE) ? 1 : 0;
        a.uturn_gen = (flags & NUTS_UTURN_GENERALIZED) ? 1 : 0;
        a.sub_merge = (flags & NUTS_SUBTREE_MERGE) ? 1 : 0;
        a.target_accept = target_accept;
        a.init_q = (const double*)iq_d;
        a.out_samples = (double*)smp_d;
        a.out_stats = (nuts_stats*)sts_d;
        a.out_final_q = (double*)fq_d;
        a.out_inv_mass = (double*)fim_d;
        a.out_step_size = (double*)fep_d;
        a.grad_evals = gev;
        return NUTS_OK;
    }

    // copy host outputs back, sum the gradient evaluations, synchronise.
    // With `flag` (a kernel's device error word), also read it back and
    // fail with `flag_msg` if it is set.
    int finish(nuts_handle* h, const nuts_sample_opts& o, double* out_samples, nuts_stats* out_stats,
               const unsigned int* flag = nullptr, const char* flag_msg = nullptr)
    {
        HIP_TRY(h, finish_out(out_samples, (size_t)C * S * D * 8, smp, s));
        HIP_TRY(h, finish_out(out_stats, (size_t)C * S * sizeof(nuts_stats), sts, s));
        HIP_TRY(h, finish_out(o.out_final_q, (size_t)C * D * 8, fq, s));
        HIP_TRY(h, finish_out(o.out_inv_mass, (size_t)C * D * 8, fim, s));
        HIP_TRY(h, finish_out(o.out_step_size, (size_t)C * 8, fep, s));
        void* pin = nullptr;
        const size_t eb = (size_t)C * sizeof(unsigned long long);
        HIP_TRY(h, handle_pinned(h, eb + 8, &pin));
        unsigned long long* ev = (unsigned long long*)pin;
        unsigned int* fl = (unsigned int*)((char*)pin + eb);
        *fl = 0u;
        HIP_TRY(h, hipMemcpyAsync(ev, gev, eb, hipMemcpyDeviceToHost, s));
        if (flag) HIP_TRY(h, hipMemcpyAsync(fl, flag, sizeof(unsigned int), hipMemcpyDeviceToHost, s));
        HIP_TRY(h, hipStreamSynchronize(s));
        if (flag && *fl) return fail(h, NUTS_EDEVICE, "%s", flag_msg);
        if (o.out_kernel_ms) {
            float ms = 0.0f;
            HIP_TRY(h, hipEventElapsedTime(&ms, h->kev[0], h->kev[1]));
            *o.out_kernel_ms = ms;
        }
        if (o.out_grad_evals) {
            unsigned long long tot = 0;
            for (int64_t c = 0; c < C; ++c) tot += ev[c];
            *o.out_grad_evals = (int64_t)tot;
        }
        return NUTS_OK;
    }
};


// Check an HMM sequence on the host and put it on the device.
int hmm_stage(nuts_handle* h, const uint8_t* w, int64_t T, const uint8_t* z, int64_t Tsup, int K, int V,
              DevBuf& wb, DevBuf& zb, HmmView* hv)
{
    if (!w) return fail(h, NUTS_EINVAL, "w is NULL");
    if (Tsup > 0 && !z) return fail(h, NUTS_EINVAL, "z is NULL with Tsup = %lld", (long long)Tsup);
    if (T < 1 || Tsup < 0 || Tsup > T || T > ((int64_t)1 << 30))
        return fail(h, NUTS_EINVAL, "need 1 <= T <= 2^30 and 0 <= Tsup <= T (T = %lld, Tsup = %lld)",
                    (long long)T, (long long)Tsup);
    if (!hmm_supported(K, V, T, Tsup))
        return fail(h, NUTS_EUNSUPPORTED,
                    "the HMM kernels take 2 <= K <= 4, V >= 2, K*K + K*V <= 64 and T - Tsup <= %d "
                    "(K = %d, V = %d, T - Tsup = %lld)",
                    kHmmMaxUnobserved, K, V, (long long)(T - Tsup));
    std::vector<uint8_t> hw((size_t)T), hz((size_t)Tsup);
    DeviceScope ds(h->device);
    if (is_device_ptr(w)) HIP_TRY(h, hipMemcpy(hw.data(), w, (size_t)T, hipMemcpyDeviceToHost));
    else std::memcpy(hw.data(), w, (size_t)T);
    if (Tsup > 0) {
        if (is_device_ptr(z)) HIP_TRY(h, hipMemcpy(hz.data(), z, (size_t)Tsup, hipMemcpyDeviceToHost));
        else std::memcpy(hz.data(), z, (size_t)Tsup);
    }
    for (int64_t t = 0; t < T; ++t)
        if (hw[t] >= V) return fail(h, NUTS_EINVAL, "w[%lld] = %d is not below V = %d", (long long)t, hw[t], V);
    for (int64_t t = 0; t < Tsup; ++t)
        if (hz[t] >= K) return fail(h, NUTS_EINVAL, "z[%lld] = %d is not below K = %d", (long long)t, hz[t], K);
    HIP_TRY(h, wb.alloc((size_t)T));
    HIP_TRY(h, zb.alloc((size_t)Tsup));
    HIP_TRY(h, hipMemcpyAsync(wb.p, hw.data(), (size_t)T, hipMemcpyHostToDevice, h->stream));
    if (Tsup > 0) HIP_TRY(h, hipMemcpyAsync(zb.p, hz.data(), (size_t)Tsup, hipMemcpyHostToDevice, h->stream));
    // the host copies must outlive the copies
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    hv->w = (const uint8_t*)wb.p;
    hv->z = (const uint8_t*)zb.p;
    hv->T = (int)T;
    hv->Tsup = (int)Tsup;
    hv->K = K;
    hv->V = V;
    return NUTS_OK;
}

}  // namespace

extern "C" {

int nuts_init(nuts_handle** out, int device_ordinal, void* hip_stream)
{
    if (!out) return fail(nullptr, NUTS_EINVAL, "nuts_init: out is NULL");
    *out = nullptr;
    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e != hipSuccess || count == 0)
        return fail(nullptr, NUTS_EDEVICE, "nuts_init: no HIP device (%s)", hipGetErrorString(e));
    if (device_ordinal < 0 || device_ordinal >= count)
        return fail(nullptr, NUTS_EINVAL, "nuts_init: device %d out of range [0, %d)", device_ordinal, count);
    DeviceScope ds(device_ordinal);
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, device_ordinal);
    if (e != hipSuccess) return fail(nullptr, NUTS_EDEVICE, "nuts_init: %s", hipGetErrorString(e));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(nullptr, NUTS_EUNSUPPORTED, "nuts_init: built for gfx950, device is %s", prop.gcnArchName);
    nuts_handle* h = new (std::nothrow) nuts_handle();
    if (!h) return fail(nullptr, NUTS_ENOMEM, "nuts_init: out of host memory");
    h->device = device_ordinal;
    h->num_cu = prop.multiProcessorCount;
    if (hip_stream) {
        h->stream = (hipStream_t)hip_stream;
    } else {
        e = hipStreamCreate(&h->stream);
        if (e != hipSuccess) {
            delete h;
            return fail(nullptr, NUTS_EDEVICE, "nuts_init: hipStreamCreate: %s", hipGetErrorString(e));
        }
        h->own_stream = true;
    }
    e = static_workspace_setup(device_ordinal, h->stream, &h->static_ws);
    if (e != hipSuccess) {
        if (h->own_stream) (void)hipStreamDestroy(h->stream);
        delete h;
        return fail(nullptr, NUTS_EDEVICE, "nuts_init: fixed workspace: %s", hipGetErrorString(e));
    }
    *out = h;
    return NUTS_OK;
}

void nuts_free(nuts_handle* h)
{
    if (!h) return;
    DeviceScope ds(h->device);
    (void)hipStreamSynchronize(h->stream);
    if (h->scratch) (void)hipFree(h->scratch);
    if (h->pot_slots) (void)hipFree(h->pot_slots);
    if (h->evals) (void)hipFree(h->evals);
    if (h->pinned) (void)hipHostFree(h->pinned);
    for (hipEvent_t ev : h->kev)
        if (ev) (void)hipEventDestroy(ev);
    if (h->own_stream) (void)hipStreamDestroy(h->stream);
    delete h;
}

const char* nuts_last_error(const nuts_handle* h)
{
    return h ? h->err.c_str() : g_init_error.c_str();
}

int nuts_data_create(nuts_handle* h, const void* X, const uint8_t* y, int64_t N, int64_t D, int dtype,
                     int64_t num_datasets, nuts_data** out)
{
    if (!h) return NUTS_EINVAL;
    h->err.clear();
    if (!out) return fail(h, NUTS_EINVAL, "nuts_data_create: out is NULL");
    *out = nullptr;
    if (dtype != NUTS_F64 && dtype != NUTS_F32) return fail(h, NUTS_EINVAL, "dtype must be NUTS_F64 or NUTS_F32");
    if (N < 0) return fail(h, NUTS_EINVAL, "N must be >= 0 (got %lld)", (long long)N);
    if (D < 1) return fail(h, NUTS_EINVAL, "D must be >= 1 (got %lld)", (long long)D);
    if (D > kMaxDim)
        return fail(h, NUTS_EUNSUPPORTED, "D = %lld exceeds the %d columns the kernels support", (long long)D, kMaxDim);
    if (num_datasets < 1) return fail(h, NUTS_EINVAL, "num_datasets must be >= 1");
    if (N > 0 && (!X || !y)) return fail(h, NUTS_EINVAL, "X and y must be non-NULL when N > 0");

    DeviceScope ds(h->device);
    nuts_data* d = new (std::nothrow) nuts_data();
    if (!d) return fail(h, NUTS_ENOMEM, "out of host memory");
    d->view.N = N;
    d->view.D = (int)D;
    d->view.dtype = dtype;
    const PassShape shape = pass_shape((int)D);
    d->view.split = shape.split;
    d->view.cols = shape.cols;
    const int R = rows_per_block(d->view);
    d->view.nb = (N + R - 1) / R;
    d->view.nds = num_datasets;
    const size_t es = elem_size(dtype);
    const size_t xblk = ((size_t)d->view.nb * D * R * num_datasets + (size_t)kTailElems) * es;
    const size_t yblk = (size_t)d->view.nb * R * num_datasets;
    auto cleanup = [&](int code) {
        free_data_buffers(d);
        delete d;
        return code;
    };
    hipError_t e;
    if (xblk) {
        e = hipMalloc(&d->X, xblk);
        if (e != hipSuccess) return cleanup(fail(h, NUTS_ENOMEM, "hipMalloc(%zu) for X: %s", xblk, hipGetErrorString(e)));
        e = hipMalloc((void**)&d->y, yblk);
        if (e != hipSuccess) return cleanup(fail(h, NUTS_ENOMEM, "hipMalloc(%zu) for y: %s", yblk, hipGetErrorString(e)));
        DevBuf xs, ys, flag;
        const void* Xd = nullptr;
        const void* yd = nullptr;
        e = stage_in(X, (size_t)N * D * num_datasets * es, xs, &Xd, h->stream);
        if (e == hipSuccess) e = stage_in(y, (size_t)N * num_datasets, ys, &yd, h->stream);
        if (e == hipSuccess) e = hipMemsetAsync(d->X, 0, xblk, h->stream);
        if (e == hipSuccess) e = flag.alloc(sizeof(unsigned int));
        if (e == hipSuccess) e = hipMemsetAsync(flag.p, 0, sizeof(unsigned int), h->stream);
        if (e == hipSuccess)
            e = launch_to_blocks(Xd, (const uint8_t*)yd, d->view, d->X, d->y, (unsigned int*)flag.p, h->stream);
        unsigned int bad = 0;
        if (e == hipSuccess) e = hipMemcpyAsync(&bad, flag.p, sizeof bad, hipMemcpyDeviceToHost, h->stream);
        if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
        if (e != hipSuccess)
            return cleanup(fail(h, e == hipErrorOutOfMemory ? NUTS_ENOMEM : NUTS_EDEVICE, "data layout: %s",
                                hipGetErrorString(e)));
        if (bad) return cleanup(fail(h, NUTS_EINVAL, "y holds a value other than 0 or 1"));
    }
    d->view.X = d->X;
    d->view.y = d->y;
    *out = d;
    return NUTS_OK;
}

void nuts_data_free(nuts_handle* h, nuts_data* d)
{
    if (!d) return;
    if (h) {
        DeviceScope ds(h->device);
        (void)hipStreamSynchronize(h->stream);
        free_data_buffers(d);
    } else {
        free_data_buffers(d);
    }
    delete d;
}

int nuts_data_potential_grad(nuts_handle* h, const nuts_data* d, double prior_scale, const double* W,
                             int64_t K, double* out_U, double* out_grad)
{
    if (!h) return NUTS_EINVAL;
    h->err.clear();
    if (!d) return fail(h, NUTS_EINVAL, "data is NULL");
    if (!W || !out_U || !out_grad) return fail(h, NUTS_EINVAL, "W, out_U and out_grad must be non-NULL");
    if (K < 1 || K > kMaxPotentialItems)
        return fail(h, NUTS_EINVAL, "K must be in [1, %d] (got %lld)", kMaxPotentialItems, (long long)K);
    if (d->view.nds > 1 && K != d->view.nds)
        return fail(h, NUTS_EINVAL, "per-chain data: K (%lld) must equal the number of data sets (%lld)",
                    (long long)K, (long long)d->view.nds);
    if (!finite_pos(prior_scale)) return fail(h, NUTS_EINVAL, "prior_scale must be finite and > 0");
    DeviceScope ds(h->device);
    const int D = d->view.D;
    DevBuf wt, ut, gt;
    const void* Wd = nullptr;
    void *Ud = nullptr, *Gd = nullptr;
    HIP_TRY(h, stage_in(W, (size_t)K * D * 8, wt, &Wd, h->stream));
    HIP_TRY(h, stage_out(out_U, (size_t)K * 8, ut, &Ud));
    HIP_TRY(h, stage_out(out_grad, (size_t)K * D * 8, gt, &Gd));
    const PotentialPlan plan = plan_potential(d->view, K, h->num_cu);
    double* part = nullptr;
    HIP_TRY(h, potential_slots(h, (size_t)K * plan.groups_per_item * plan.width * sizeof(double), &part));
    HIP_TRY(h, launch_potential_grad(d->view, prior_scale, (const double*)Wd, K, plan, part, (double*)Ud,
                                     (double*)Gd, h->stream));
    HIP_TRY(h, finish_out(out_U, (size_t)K * 8, ut, h->stream));
    HIP_TRY(h, finish_out(out_grad, (size_t)K * D * 8, gt, h->stream));
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    return NUTS_OK;
}

int nuts_data_potential_grad_noalloc(nuts_handle* h, const nuts_data* d, double prior_scale, const double* W,
                                     int64_t K, double* out_U, double* out_grad)
{
    if (!h) return NUTS_EINVAL;
    h->err.clear();
    if (!d) return fail(h, NUTS_EINVAL, "data is NULL");
    if (!W || !out_U || !out_grad) return fail(h, NUTS_EINVAL, "W, out_U and out_grad must be non-NULL");
    if (K < 1 || K > kStaticMaxItems)
        return fail(h, NUTS_EINVAL, "K must be in [1, %lld] (got %lld)", (long long)kStaticMaxItems, (long long)K);
    if (d->view.nds > 1 && K != d->view.nds)
        return fail(h, NUTS_EINVAL, "per-chain data: K (%lld) must equal the number of data sets (%lld)",
                    (long long)K, (long long)d->view.nds);
    if (!finite_pos(prior_scale)) return fail(h, NUTS_EINVAL, "prior_scale must be finite and > 0");
    if (!is_device_ptr(W) || !is_device_ptr(out_U) || !is_device_ptr(out_grad))
        return fail(h, NUTS_EINVAL, "W, out_U and out_grad must be device memory (this entry point copies nothing)");
    const PotentialPlan plan = plan_potential(d->view, K, h->num_cu);
    const size_t need = plan.items ? 0 : (size_t)K * plan.groups_per_item * plan.width * sizeof(double);
    if (need > kStaticScratchBytes)
        return fail(h, NUTS_EINVAL,
                    "K = %lld positions need %zu bytes of partial sums (%d groups of %d doubles each), more than "
                    "the %zu bytes of the fixed workspace",
                    (long long)K, need, plan.groups_per_item, plan.width, kStaticScratchBytes);
    DeviceScope ds(h->device);
    HIP_TRY(h, launch_potential_grad(d->view, prior_scale, W, K, plan, (double*)h->static_ws, out_U, out_grad,
                                     h->stream));
    return NUTS_OK;
}

// The row-stage layout of a shared fp32 data set (built on first use).
static int ensure_batch_layout(nuts_handle* h, const nuts_data* dc)
{
    nuts_data* d = const_cast<nuts_data*>(dc);
    if (d->bX) return NUTS_OK;
    if (d->view.dtype != NUTS_F32)
        return fail(h, NUTS_EUNSUPPORTED, "the batched path takes fp32 data");
    if (d->view.nds != 1) return fail(h, NUTS_EUNSUPPORTED, "the batched path takes one shared data set");
    int kt = 0, tc = 0;
    if (!batch_shape(d->view.D, &kt, &tc))
        return fail(h, NUTS_EUNSUPPORTED, "the batched path takes D <= %d (got %d)", 16 * kBatchMaxKT + 4,
                    d->view.D);
    BatchView b;
    b.N = d->view.N;
    b.D = d->view.D;
    b.kt = kt;
    b.tc = tc;
    b.stride = 16 * batch_kp(kt) + 4;
    b.ns = (b.N + kBatchStageRows - 1) / kBatchStageRows;
    const size_t xb = (size_t)b.ns * kBatchStageRows * b.stride * sizeof(float);
    const size_t yb = (size_t)b.ns * kBatchStageRows;
    float* X = nullptr;
    uint8_t* y = nullptr;
    if (xb) {
        hipError_t e = hipMalloc(&X, xb);
        if (e == hipSuccess) e = hipMalloc(&y, yb);
        if (e == hipSuccess) e = launch_to_batch_layout(d->view, b, X, y, h->stream);
        if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
        if (e != hipSuccess) {
            if (X) (void)hipFree(X);
            if (y) (void)hipFree(y);
            return fail(h, e == hipErrorOutOfMemory ? NUTS_ENOMEM : NUTS_EDEVICE, "batched layout: %s",
                        hipGetErrorString(e));
        }
    }
    b.X = X;
    b.y = y;
    d->batch = b;
    d->bX = X;
    d->by = y;
    return NUTS_OK;
}

int nuts_data_potential_grad_batched(nuts_handle* h, const nuts_data* d, double prior_scale, const double* W,
                                     int64_t K, double* out_U, double* out_grad)
{
    if (!h) return NUTS_EINVAL;
    h->err.clear();
    if (!d) return fail(h, NUTS_EINVAL, "data is NULL");
    if (!W || !out_U || !out_grad) return fail(h, NUTS_EINVAL, "W, out_U and out_grad must be non-NULL");
    if (K < 1 || K > 65535) return fail(h, NUTS_EINVAL, "K must be in [1, 65535] (got %lld)", (long long)K);
    if (!finite_pos(prior_scale)) return fail(h, NUTS_EINVAL, "prior_scale must be finite and > 0");
    if (d->view.N < 1) return fail(h, NUTS_EINVAL, "the batched path needs N >= 1");
    DeviceScope ds(h->device);
    const int rc = ensure_batch_layout(h, d);
    if (rc != NUTS_OK) return rc;
    const int D = d->view.D;
    DevBuf wt, ut, gt;
    const void* Wd = nullptr;
    void *Ud = nullptr, *Gd = nullptr;
    HIP_TRY(h, stage_in(W, (size_t)K * D * 8, wt, &Wd, h->stream));
    HIP_TRY(h, stage_out(out_U, (size_t)K * 8, ut, &Ud));
    HIP_TRY(h, stage_out(out_grad, (size_t)K * D * 8, gt, &Gd));
    const BatchPlan plan = plan_batch_potential(d->batch, K, h->num_cu);
    const size_t rows = (size_t)plan.tiles * plan.groups * kBatchTileChains;
    const size_t pbytes = align256(rows * plan.pw * sizeof(float));
    void* scratch = nullptr;
    HIP_TRY(h, handle_scratch(h, pbytes + rows * sizeof(double), &scratch));
    HIP_TRY(h, launch_batch_potential(d->batch, prior_scale, (const double*)Wd, K, plan, (float*)scratch,
                                      (double*)((char*)scratch + pbytes), (double*)Ud, (double*)Gd, h->stream));
    HIP_TRY(h, finish_out(out_U, (size_t)K * 8, ut, h->stream));
    HIP_TRY(h, finish_out(out_grad, (size_t)K * D * 8, gt, h->stream));
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    return NUTS_OK;
}

int nuts_data_log_likelihood(nuts_handle* h, const nuts_data* d, const double* W, int64_t S, double* out_ll,
                             double* out_elpd, double* out_pred_mean)
{
    if (!h) return NUTS_EINVAL;
    h->err.clear();
    if (!d) return fail(h, NUTS_EINVAL, "data is NULL");
    if (!W || !out_ll) return fail(h, NUTS_EINVAL, "W and out_ll must be non-NULL");
    if (S < 1 || S > kMaxPotentialItems)
        return fail(h, NUTS_EINVAL, "S must be in [1, %d] (got %lld)", kMaxPotentialItems, (long long)S);
    if (d->view.nds != 1) return fail(h, NUTS_EINVAL, "the log-likelihood takes one shared data set");
    if (d->view.N < 1) return fail(h, NUTS_EINVAL, "the log-likelihood needs N >= 1");
    DeviceScope ds(h->device);
    const int D = d->view.D;
    const int64_t N = d->view.N;
    int kt = 0, tc = 0;
    const bool mfma = d->view.dtype == NUTS_F32 && batch_shape(D, &kt, &tc);
    if (!mfma && out_pred_mean)
        return fail(h, NUTS_EUNSUPPORTED, "the predictive mean takes fp32 data with D <= %d", 16 * kBatchMaxKT + 4);
    DevBuf wt, lt, et, pt;
    const void* Wd = nullptr;
    void *Ld = nullptr, *Ed = nullptr, *Pd = nullptr;
    HIP_TRY(h, stage_in(W, (size_t)S * D * 8, wt, &Wd, h->stream));
    HIP_TRY(h, stage_out(out_ll, (size_t)S * 8, lt, &Ld));
    HIP_TRY(h, stage_out(out_elpd, 8, et, &Ed));
    HIP_TRY(h, stage_out(out_pred_mean, (size_t)N * 8, pt, &Pd));
    if (mfma) {
        const int rc = ensure_batch_layout(h, d);
        if (rc != NUTS_OK) return rc;
        const BatchPlan plan = plan_batch_potential(d->batch, S, h->num_cu);
        const size_t lbytes = align256((size_t)plan.tiles * plan.groups * kBatchTileChains * sizeof(double));
        const size_t rbytes = out_pred_mean ? (size_t)plan.tiles * d->batch.ns * kBatchStageRows * sizeof(float) : 0;
        void* scratch = nullptr;
        HIP_TRY(h, handle_scratch(h, lbytes + rbytes, &scratch));
        HIP_TRY(h, launch_batch_log_likelihood(d->batch, (const double*)Wd, S, plan, (double*)scratch,
                                               (float*)((char*)scratch + lbytes), (double*)Ld, (double*)Pd,
                                               nullptr, 0, h->stream));
    } else {
        // the potential at prior scale 1 per draw, then the prior taken off
        const PotentialPlan plan = plan_potential(d->view, S, h->num_cu);
        const size_t ubytes = align256((size_t)S * sizeof(double));
        void* scratch = nullptr;
        HIP_TRY(h, handle_scratch(h, ubytes + (size_t)S * D * sizeof(double), &scratch));
        double* U = (double*)scratch;
        double* G = (double*)((char*)scratch + ubytes);
        double* part = nullptr;
        HIP_TRY(h, potential_slots(h, (size_t)S * plan.groups_per_item * plan.width * sizeof(double), &part));
        HIP_TRY(h, launch_potential_grad(d->view, 1.0, (const double*)Wd, S, plan, part, U, G, h->stream));
        HIP_TRY(h, launch_ll_from_potential(D, (const double*)Wd, S, U, (double*)Ld, h->stream));
    }
    if (out_elpd) HIP_TRY(h, launch_expected_ll((const double*)Ld, S, (double*)Ed, h->stream));
    HIP_TRY(h, finish_out(out_ll, (size_t)S * 8, lt, h->stream));
    HIP_TRY(h, finish_out(out_elpd, 8, et, h->stream));
    HIP_TRY(h, finish_out(out_pred_mean, (size_t)N * 8, pt, h->stream));
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    return NUTS_OK;
}

int nuts_data_posterior_predictive(nuts_handle* h, const nuts_data* d, const double* W, int64_t S, uint64_t seed,
                                   uint8_t* out_y)
{
    if (!h) return NUTS_EINVAL;
    h->err.clear();
    if (!d) return fail(h, NUTS_EINVAL, "data is NULL");
    if (!W || !out_y) return fail(h, NUTS_EINVAL, "W and out_y must be non-NULL");
    if (S < 1 || S > kMaxPotentialItems)
        return fail(h, NUTS_EINVAL, "S must be in [1, %d] (got %lld)", kMaxPotentialItems, (long long)S);
    if (d->view.nds != 1) return fail(h, NUTS_EINVAL, "the predictive takes one shared data set");
    if (d->view.N < 1) return fail(h, NUTS_EINVAL, "the predictive needs N >= 1");
    const int D = d->view.D;
    const int64_t N = d->view.N;
    int kt = 0, tc = 0;
    if (d->view.dtype != NUTS_F32 || !batch_shape(D, &kt, &tc))
        return fail(h, NUTS_EUNSUPPORTED, "the predictive samples take fp32 data with D <= %d", 16 * kBatchMaxKT + 4);
    DeviceScope ds(h->device);
    DevBuf wt, yt;
    const void* Wd = nullptr;
    void* Yd = nullptr;
    HIP_TRY(h, stage_in(W, (size_t)S * D * 8, wt, &Wd, h->stream));
    HIP_TRY(h, stage_out(out_y, (size_t)S * N, yt, &Yd));
    const int rc = ensure_batch_layout(h, d);
    if (rc != NUTS_OK) return rc;
    const BatchPlan plan = plan_batch_potential(d->batch, S, h->num_cu);
    const size_t lbytes = align256((size_t)plan.tiles * plan.groups * kBatchTileChains * sizeof(double));
    void* scratch = nullptr;
    HIP_TRY(h, handle_scratch(h, lbytes, &scratch));
    HIP_TRY(h, launch_batch_log_likelihood(d->batch, (const double*)Wd, S, plan, (double*)scratch, nullptr, nullptr,
                                           nullptr, (uint8_t*)Yd, seed, h->stream));
    HIP_TRY(h, finish_out(out_y, (size_t)S * N, yt, h->stream));
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    return NUTS_OK;
}

int nuts_potential_grad(nuts_handle* h, const void* X, const uint8_t* y, int64_t N, int64_t D, int dtype,
                        double prior_scale, const double* w, double* out_U, double* out_grad)
{
    nuts_data* d = nullptr;
    int rc = nuts_data_create(h, X, y, N, D, dtype, 1, &d);
    if (rc != NUTS_OK) return rc;
    rc = nuts_data_potential_grad(h, d, prior_scale, w, 1, out_U, out_grad);
    nuts_data_free(h, d);
    return rc;
}

int nuts_sample_data(nuts_handle* h, const nuts_data* d, uint32_t flags, double prior_scale, double step_size,
                     const double* inv_mass_diag, int max_tree_depth, int64_t num_warmup, int64_t num_samples,
                     int64_t num_chains, uint64_t seed, double* out_samples, nuts_stats* out_stats,
                     const nuts_sample_opts* opts)
{
    if (!h) return NUTS_EINVAL;
    h->err.clear();
    nuts_sample_opts o;
    std::memset(&o, 0, sizeof o);
    if (opts) o = *opts;
    if (!d) return fail(h, NUTS_EINVAL, "data is NULL");
    double target_accept = 0.0;
    int rc = check_run(h, flags, NUTS_DATA_PER_CHAIN | NUTS_ADAPT_DIAG_MASS | NUTS_ADAPT_STEP_SIZE |
                                     NUTS_UTURN_GENERALIZED | NUTS_SUBTREE_MERGE,
                       o, step_size, max_tree_depth, num_warmup, num_samples, num_chains, &target_accept);
    if (rc != NUTS_OK) return rc;
    if (!finite_pos(prior_scale)) return fail(h, NUTS_EINVAL, "prior_scale must be finite and > 0");
    if (d->view.N < 1) return fail(h, NUTS_EINVAL, "sampling needs N >= 1");
    const bool per_chain = (flags & NUTS_DATA_PER_CHAIN) != 0;
    const int sub_merge = (flags & NUTS_SUBTREE_MERGE) ? 1 : 0;
    if (per_chain && d->view.nds != num_chains)
        return fail(h, NUTS_EINVAL, "NUTS_DATA_PER_CHAIN: data holds %lld sets for %lld chains",
                    (long long)d->view.nds, (long long)num_chains);
    if (!per_chain && d->view.nds != 1)
        return fail(h, NUTS_EINVAL, "data holds %lld sets; pass NUTS_DATA_PER_CHAIN", (long long)d->view.nds);
    const int D = d->view.D;
    rc = check_inv_mass(h, inv_mass_diag, D);
    if (rc != NUTS_OK) return rc;

    DeviceScope ds(h->device);
    int path = o.path;
    if (path == NUTS_PATH_AUTO) {
        // many chains on a large shared fp32 data set: the matrix-core batch;
        // one wave per chain when there are many chains or the data is small;
        // the whole device on one chain when the data is large
        int kt = 0, tc = 0;
        const bool batchable = !per_chain && d->view.dtype == NUTS_F32 && num_chains >= 16 &&
                               (double)d->view.N * d->view.D >= 262144.0 && batch_shape(d->view.D, &kt, &tc);
        const bool small = d->view.nb <= 6;  // a few blocks: one wave beats a grid-wide exchange
        // a lone chain whose data set fits in one group's LDS is faster on
        // one wave than on a grid-wide exchange per step
        SamplerArgs probe;
        std::memset(&probe, 0, sizeof probe);
        probe.data = d->view;
        probe.max_depth = max_tree_depth;
        probe.num_chains = num_chains;
        probe.sub_merge = sub_merge;
        const bool resident = wave_path_supports(d->view) && wave_path_resident(probe);
        if (batchable && ensure_batch_layout(h, d) == NUTS_OK &&
            batch_sampler_supported(d->batch, max_tree_depth, sub_merge, h->num_cu))
            path = NUTS_PATH_BATCH;
        else
            path = ((per_chain || small || resident || num_chains > 1) && wave_path_supports(d->view))
                       ? NUTS_PATH_WAVE
                       : NUTS_PATH_GRID;
        h->err.clear();
    }
    if (path != NUTS_PATH_WAVE && path != NUTS_PATH_GRID && path != NUTS_PATH_BATCH)
        return fail(h, NUTS_EINVAL, "unknown path %d", path);
    if ((path == NUTS_PATH_GRID || path == NUTS_PATH_BATCH) && per_chain)
        return fail(h, NUTS_EUNSUPPORTED, "the grid and batch paths run chains on shared data only");
    if (path == NUTS_PATH_WAVE && !wave_path_supports(d->view))
        return fail(h, NUTS_EUNSUPPORTED, "the one-wave-per-chain path takes D <= 64 (got %d)", d->view.D);
    if (path == NUTS_PATH_BATCH) {
        const int rc = ensure_batch_layout(h, d);
        if (rc != NUTS_OK) return rc;
        if (!batch_sampler_supported(d->batch, max_tree_depth, sub_merge, h->num_cu))
            return fail(h, NUTS_EUNSUPPORTED, "the batch path needs >= %d compute units and D <= 132",
                        kBatchTileChains);
    }

    hipStream_t s = h->stream;
    const int64_t C = num_chains;
    RunBuffers rb;
    SamplerArgs a;
    std::memset(&a, 0, sizeof a);
    a.data = d->view;
    a.per_chain_data = per_chain ? 1 : 0;
    a.prior_scale = prior_scale;
    rc = rb.stage(h, a, flags, o, target_accept, step_size, inv_mass_diag, max_tree_depth, num_warmup, num_samples,
                  num_chains, seed, out_samples, out_stats);
    if (rc != NUTS_OK) return rc;

    hipEvent_t* kev = nullptr;
    if (o.out_kernel_ms) HIP_TRY(h, handle_events(h, &kev));
    if (path == NUTS_PATH_WAVE) {
        if (kev) HIP_TRY(h, hipEventRecord(kev[0], s));
        HIP_TRY(h, launch_sampler_wave(a, s));
        if (kev) HIP_TRY(h, hipEventRecord(kev[1], s));
    } else if (path == NUTS_PATH_BATCH) {
        // launches of up to kBatchMaxTiles tiles of 128 chains, the groups of
        // the device split evenly between the tiles of a launch
        const int max_tiles = std::min(kBatchMaxTiles, h->num_cu / kBatchTileChains);
        const int64_t per_launch = (int64_t)max_tiles * kBatchTileChains;
        const int pw = 64 * ((D + 63) / 64);
        const int max_groups = h->num_cu;  // one tile: every group
        const size_t qbytes = align256((size_t)2 * max_tiles * kBatchTileChains * kBatchQWidth * sizeof(float));
        const size_t rows = (size_t)2 * max_groups * kBatchTileChains;  // [2][tiles][groups][128]
        const size_t pbytes = align256(rows * pw * sizeof(float));
        const size_t lbytes = align256(rows * sizeof(double));
        void* scratch = nullptr;
        HIP_TRY(h, handle_scratch(h, qbytes + pbytes + lbytes + sizeof(BatchSync), &scratch));
        float* qbuf = (float*)scratch;
        float* P = (float*)((char*)scratch + qbytes);
        double* L = (double*)((char*)scratch + qbytes + pbytes);
        BatchSync* sync = (BatchSync*)((char*)scratch + qbytes + pbytes + lbytes);
        for (int64_t c0 = 0; c0 < C; c0 += per_launch) {
            SamplerArgs ac = a;
            ac.num_chains = std::min(per_launch, C - c0);
            ac.chain_offset = c0;
            const int tiles = (int)((ac.num_chains + kBatchTileChains - 1) / kBatchTileChains);
            const int groups = h->num_cu / tiles;
            HIP_TRY(h, launch_sampler_batch(ac, d->batch, tiles, groups, qbuf, P, L, sync, s,
                                            kev && c0 == 0 ? kev[0] : nullptr));
            if (kev) HIP_TRY(h, hipEventRecord(kev[1], s));
            unsigned int err = 0;
            HIP_TRY(h, hipMemcpyAsync(&err, &sync->error, sizeof err, hipMemcpyDeviceToHost, s));
            HIP_TRY(h, hipStreamSynchronize(s));
            if (err)
                return fail(h, NUTS_EDEVICE, "batch exchange timed out in chains %lld.. (a group stopped responding)",
                            (long long)c0);
        }
    } else {
        const int groups = grid_sampler_groups(d->view, max_tree_depth, sub_merge, h->num_cu);
        if (groups == 0)
            return fail(h, NUTS_EUNSUPPORTED, "the grid path's tree state (D = %d, depth %d) does not fit a CU's LDS",
                        D, max_tree_depth);
        const size_t part_bytes = align256((size_t)grid_partial_elems(D, groups) * sizeof(double));
        const size_t res_bytes = align256((size_t)grid_result_elems(D) * sizeof(double));
        void* scratch = nullptr;
        HIP_TRY(h, handle_scratch(h, part_bytes + res_bytes + sizeof(GridSync), &scratch));
        double* part = (double*)scratch;
        double* res = (double*)((char*)scratch + part_bytes);
        GridSync* sync = (GridSync*)((char*)scratch + part_bytes + res_bytes);
        for (int64_t c = 0; c < C; ++c) {
            SamplerArgs ac = a;
            ac.num_chains = 1;
            ac.chain_offset = c;
            HIP_TRY(h, launch_sampler_grid(ac, groups, part, res, sync, s, kev && c == 0 ? kev[0] : nullptr));
            if (kev) HIP_TRY(h, hipEventRecord(kev[1], s));
            if (c + 1 < C) {
                // the next chain's launch clears the flag: check this one's first
                GridSync hs;
                HIP_TRY(h, hipMemcpyAsync(&hs, sync, sizeof hs, hipMemcpyDeviceToHost, s));
                HIP_TRY(h, hipStreamSynchronize(s));
                if (hs.error)
                    return fail(h, NUTS_EDEVICE, "grid barrier timed out in chain %lld (a group stopped responding)",
                                (long long)c);
            }
        }
        // the last chain's flag is read with the outputs
        return rb.finish(h, o, out_samples, out_stats, &sync->error,
                         "grid barrier timed out in the last chain (a group stopped responding)");
    }
    return rb.finish(h, o, out_samples, out_stats);
}

int nuts_hmm_potential_grad(nuts_handle* h, const uint8_t* w, int64_t T, const uint8_t* z, int64_t Tsup, int K,
                            int V, const double* Q, int64_t num_points, double* out_U, double* out_grad)
{
    if (!h) return NUTS_EINVAL;
    h->err.clear();
    if (!Q || !out_U || !out_grad) return fail(h, NUTS_EINVAL, "Q, out_U and out_grad must not be NULL");
    if (num_points < 1 || num_points > ((int64_t)1 << 31))
        return fail(h, NUTS_EINVAL, "num_points must be in [1, 2^31] (got %lld)", (long long)num_points);
    DevBuf wb, zb;
    HmmView hv;
    int rc = hmm_stage(h, w, T, z, Tsup, K, V, wb, zb, &hv);
    if (rc != NUTS_OK) return rc;
    DeviceScope ds(h->device);
    hipStream_t s = h->stream;
    const int D = hmm_dim(K, V);
    DevBuf qb, ub, gb;
    const void* q_d = nullptr;
    void *u_d = nullptr, *g_d = nullptr;
    HIP_TRY(h, stage_in(Q, (size_t)num_points * D * 8, qb, &q_d, s));
    HIP_TRY(h, stage_out(out_U, (size_t)num_points * 8, ub, &u_d));
    HIP_TRY(h, stage_out(out_grad, (size_t)num_points * D * 8, gb, &g_d));
    HIP_TRY(h, launch_hmm_potential(hv, (const double*)q_d, num_points, (double*)u_d, (double*)g_d, s));
    HIP_TRY(h, finish_out(out_U, (size_t)num_points * 8, ub, s));
    HIP_TRY(h, finish_out(out_grad, (size_t)num_points * D * 8, gb, s));
    HIP_TRY(h, hipStreamSynchronize(s));
    return NUTS_OK;
}

int nuts_hmm_sample(nuts_handle* h, const uint8_t* w, int64_t T, const uint8_t* z, int64_t Tsup, int K, int V,
                    uint32_t flags, double step_size, const double* inv_mass_diag, int max_tree_depth,
                    int64_t num_warmup, int64_t num_samples, int64_t num_chains, uint64_t seed, double* out_samples,
                    nuts_stats* out_stats, const nuts_sample_opts* opts)
{
    if (!h) return NUTS_EINVAL;
    h->err.clear();
    nuts_sample_opts o;
    std::memset(&o, 0, sizeof o);
    if (opts) o = *opts;
    double target_accept = 0.0;
    int rc = check_run(h, flags,
                       NUTS_ADAPT_DIAG_MASS | NUTS_ADAPT_STEP_SIZE | NUTS_UTURN_GENERALIZED | NUTS_SUBTREE_MERGE, o,
                       step_size,
                       max_tree_depth, num_warmup, num_samples, num_chains, &target_accept);
    if (rc != NUTS_OK) return rc;
    if (o.path != NUTS_PATH_AUTO && o.path != NUTS_PATH_WAVE)
        return fail(h, NUTS_EUNSUPPORTED, "the HMM runs on the one-wave-per-chain path only");
    DevBuf wb, zb;
    HmmView hv;
    rc = hmm_stage(h, w, T, z, Tsup, K, V, wb, zb, &hv);
    if (rc != NUTS_OK) return rc;
    const int D = hmm_dim(K, V);
    rc = check_inv_mass(h, inv_mass_diag, D);
    if (rc != NUTS_OK) return rc;
    DeviceScope ds(h->device);
    RunBuffers rb;
    SamplerArgs a;
    std::memset(&a, 0, sizeof a);
    a.data.D = D;
    a.data.N = T;
    a.data.nds = 1;
    a.prior_scale = 1.0;
    rc = rb.stage(h, a, flags, o, target_accept, step_size, inv_mass_diag, max_tree_depth, num_warmup, num_samples,
                  num_chains, seed, out_samples, out_stats);
    if (rc != NUTS_OK) return rc;
    hipEvent_t* kev = nullptr;
    if (o.out_kernel_ms) HIP_TRY(h, handle_events(h, &kev));
    if (kev) HIP_TRY(h, hipEventRecord(kev[0], h->stream));
    const hipError_t e = launch_hmm_sampler(a, hv, h->stream);
    if (kev && e == hipSuccess) HIP_TRY(h, hipEventRecord(kev[1], h->stream));
    if (e == hipErrorInvalidValue)
        return fail(h, NUTS_EUNSUPPORTED, "max_tree_depth %d: the HMM chain's LDS does not fit", max_tree_depth);
    HIP_TRY(h, e);
    return rb.finish(h, o, out_samples, out_stats);
}

int nuts_sample(nuts_handle* h, const void* X, const uint8_t* y, int64_t N, int64_t D, int dtype, uint32_t flags,
                double prior_scale, double step_size, const double* inv_mass_diag, int max_tree_depth,
                int64_t num_warmup, int64_t num_samples, int64_t num_chains, uint64_t seed, double* out_samples,
                nuts_stats* out_stats)
{
    if (!h) return NUTS_EINVAL;
    if (num_chains < 1) return fail(h, NUTS_EINVAL, "num_chains must be >= 1");
    const int64_t nds = (flags & NUTS_DATA_PER_CHAIN) ? num_chains : 1;
    nuts_data* d = nullptr;
    int rc = nuts_data_create(h, X, y, N, D, dtype, nds, &d);
    if (rc != NUTS_OK) return rc;
    rc = nuts_sample_data(h, d, flags, prior_scale, step_size, inv_mass_diag, max_tree_depth, num_warmup,
                          num_samples, num_chains, seed, out_samples, out_stats, nullptr);
    nuts_data_free(h, d);
    return rc;
}

}  // extern "C"
