// C ABI of liblh (declared in include/lh.h): argument validation, launch
// planning and dispatch.  Every check runs on the host before anything is
// enqueued; a failing call touches no buffer.
#include "lh.h"

#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "lh_internal.hpp"
#include "prefill_fft.hpp"
#include "companion.hpp"

namespace {

thread_local char g_last_error[512] = "";

lh_status fail(lh_status s, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return s;
}

struct Buf {
    const char* name;
    uintptr_t lo;
    uintptr_t hi;  // exclusive
};

bool overlaps(const Buf& a, const Buf& b)
{
    if (a.lo == a.hi || b.lo == b.hi) return false;  // empty ranges
    return a.lo < b.hi && b.lo < a.hi;
}

Buf buf(const char* name, const void* p, size_t bytes)
{
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Buf{name, lo, lo + bytes};
}

bool mul_ok(int64_t a, int64_t b, int64_t* out)
{
    return !__builtin_mul_overflow(a, b, out) && *out <= (INT64_C(1) << 60);
}

lh_status check_sizes(int64_t B, int64_t D, int64_t d, int64_t T)
{
    if (B < 1) return fail(LH_ERR_INVALID_ARG, "B = %lld must be >= 1", (long long)B);
    if (D < 1) return fail(LH_ERR_INVALID_ARG, "D = %lld must be >= 1", (long long)D);
    if (d < 1 || d > LH_MAX_MODES)
        return fail(LH_ERR_INVALID_ARG, "d = %lld must be in [1, %d]", (long long)d, LH_MAX_MODES);
    if (T < 0) return fail(LH_ERR_INVALID_ARG, "T = %lld must be >= 0", (long long)T);
    int64_t bd, bdd, btd;
    if (!mul_ok(B, D, &bd) || !mul_ok(bd, d, &bdd) || !mul_ok(bdd, 8, &bdd) ||
        !mul_ok(bd, T > 0 ? T : 1, &btd) || !mul_ok(btd, d, &btd) || !mul_ok(btd, 8, &btd))
        return fail(LH_ERR_INVALID_ARG, "sizes overflow (B=%lld D=%lld d=%lld T=%lld)",
                    (long long)B, (long long)D, (long long)d, (long long)T);
    return LH_OK;
}

lh_status check_dtype(lh_dtype t)
{
    if (t != LH_F32 && t != LH_BF16)
        return fail(LH_ERR_UNSUPPORTED_DTYPE, "io_dtype %d is neither LH_F32 nor LH_BF16", (int)t);
    return LH_OK;
}

lh_status check_align(const Buf& b, uintptr_t a)
{
    if (b.lo % a != 0)
        return fail(LH_ERR_INVALID_ARG, "%s is not %u-byte aligned", b.name, (unsigned)a);
    return LH_OK;
}

lh_status check_device(int* dev)
{
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || n < 1) {
        (void)hipGetLastError();
        return fail(LH_ERR_NO_DEVICE, "no HIP device is visible");
    }
    if (hipGetDevice(dev) != hipSuccess) {
        (void)hipGetLastError();
        return fail(LH_ERR_NO_DEVICE, "hipGetDevice failed");
    }
    return LH_OK;
}

// The range [lo, hi) must be memory the current device can access: device
// memory of this device, or pinned / managed host memory, and it must lie
// inside one allocation.
lh_status check_accessible(const Buf& b, int dev)
{
    if (b.lo == b.hi) return LH_OK;
    void* p = reinterpret_cast<void*>(b.lo);
    hipPointerAttribute_t a;
    memset(&a, 0, sizeof(a));
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();
        return fail(LH_ERR_INVALID_ARG, "%s (%p) is not memory known to HIP", b.name, p);
    }
    if (a.type == hipMemoryTypeUnregistered)
        return fail(LH_ERR_INVALID_ARG, "%s (%p) is unregistered host memory", b.name, p);
    if (a.type == hipMemoryTypeDevice && a.device != dev)
        return fail(LH_ERR_INVALID_ARG, "%s lives on device %d, the current device is %d", b.name,
                    a.device, dev);
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, p) == hipSuccess && base != nullptr) {
        // compared as offsets from the base so that a reported size near
        // SIZE_MAX cannot wrap the allocation's end around
        const uintptr_t blo = reinterpret_cast<uintptr_t>(base);
        if (b.lo < blo || b.hi - blo > size)
            return fail(LH_ERR_INVALID_ARG,
                        "%s [%p, +%zu) extends past its allocation [%p, +%zu)", b.name, p,
                        (size_t)(b.hi - b.lo), base, size);
    } else {
        (void)hipGetLastError();
    }
    return LH_OK;
}

lh_status from_hip(hipError_t e, const char* what)
{
    if (e == hipSuccess) return LH_OK;
    return fail(LH_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Buffer checks shared by both prefill entry points: alignment, workspace
// size, overlaps, and that every buffer is accessible from the current device.
lh_status check_prefill_buffers(const lh_c32* lambda, const lh_c32* R, const float* h0,
                                const void* u, int64_t B, int64_t D, int64_t d, int64_t T,
                                lh_dtype io_dtype, lh_c32* state, void* y, void* workspace,
                                size_t ws_needed, size_t workspace_bytes)
{
    lh_status s;
    const size_t es = io_dtype == LH_BF16 ? 2 : 4;
    const size_t n_io = static_cast<size_t>(B) * T * D;
    const Buf b_lam = buf("lambda", lambda, sizeof(lh_c32) * D * d);
    const Buf b_R = buf("R", R, sizeof(lh_c32) * D * d);
    const Buf b_h0 = buf("h0", h0, sizeof(float) * D);
    const Buf b_u = buf("u", u, T > 0 ? es * n_io : 0);
    const Buf b_state = buf("state", state, sizeof(lh_c32) * B * D * d);
    const Buf b_y = buf("y", y, T > 0 ? es * n_io : 0);
    // workspace == nullptr with ws_needed > 0 is reported below; the
    // library's own scratch is passed as nullptr, 0, 0 and not checked here
    const Buf b_ws = buf("workspace", workspace, workspace ? ws_needed : 0);

    if ((s = check_align(b_lam, 8)) || (s = check_align(b_R, 8)) || (s = check_align(b_h0, 4)) ||
        (s = check_align(b_state, 8)) || (s = check_align(b_u, es)) || (s = check_align(b_y, es)))
        return s;
    if (ws_needed > 0) {
        if (!workspace)
            return fail(LH_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", ws_needed);
        if (workspace_bytes < ws_needed)
            return fail(LH_ERR_WORKSPACE, "workspace has %zu bytes, %zu are needed",
                        workspace_bytes, ws_needed);
        if ((s = check_align(b_ws, 256))) return s;
    }
    const Buf* ins[] = {&b_lam, &b_R, &b_h0, &b_u};
    const Buf* outs[] = {&b_state, &b_y, &b_ws};
    for (const Buf* o : outs) {
        for (const Buf* i : ins)
            if (overlaps(*o, *i))
                return fail(LH_ERR_OVERLAP, "%s overlaps %s", o->name, i->name);
        for (const Buf* o2 : outs)
            if (o != o2 && overlaps(*o, *o2))
                return fail(LH_ERR_OVERLAP, "%s overlaps %s", o->name, o2->name);
    }

    int dev = 0;
    if ((s = check_device(&dev)) != LH_OK) return s;
    const Buf* all[] = {&b_lam, &b_R, &b_h0, &b_u, &b_state, &b_y, &b_ws};
    for (const Buf* b : all)
        if ((s = check_accessible(*b, dev)) != LH_OK) return s;
    return LH_OK;
}

// ---- static scratch of lh_prefill_noalloc
//
// Device memory that the library itself holds: one array per GPU the
// library runs on, from the code object's load until the process ends.  In
// host code `scratch` names a host-side stand-in, not the device array, so
// it is never passed to a kernel or a copy: the device address comes from
// hipGetSymbolAddress, resolved once per device (with that device current)
// and kept in g_scratch_ptr.
constexpr size_t kScratchBytes = size_t(LH_NOALLOC_SCRATCH_BYTES);
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of this device's scratch array (resolved on first use).
lh_status scratch_of(int dev, void** out)
{
    if (dev < 0 || dev >= kMaxDevices)
        return fail(LH_ERR_NO_DEVICE, "device %d is beyond the %d devices the static scratch serves",
                    dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || ptr == nullptr) {
            (void)hipGetLastError();
            return fail(LH_ERR_HIP, "hipGetSymbolAddress of the static scratch: %s",
                        hipGetErrorString(e));
        }
        if (reinterpret_cast<uintptr_t>(ptr) % 256 != 0)
            return fail(LH_ERR_HIP, "the static scratch is not 256-byte aligned");
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return LH_OK;
}

}  // namespace

extern "C" {

int lh_abi_version(void) { return LH_ABI_VERSION; }

const char* lh_status_string(lh_status s)
{
    switch (s) {
        case LH_OK: return "LH_OK";
        case LH_ERR_INVALID_ARG: return "LH_ERR_INVALID_ARG: invalid argument";
        case LH_ERR_OVERLAP: return "LH_ERR_OVERLAP: an output overlaps another buffer";
        case LH_ERR_UNSUPPORTED_DTYPE: return "LH_ERR_UNSUPPORTED_DTYPE: unsupported io dtype";
        case LH_ERR_NO_DEVICE: return "LH_ERR_NO_DEVICE: no HIP device";
        case LH_ERR_WORKSPACE: return "LH_ERR_WORKSPACE: workspace missing or too small";
        case LH_ERR_HIP: return "LH_ERR_HIP: HIP runtime error";
    }
    return "unknown lh_status";
}

const char* lh_last_error(void) { return g_last_error; }

size_t lh_prefill_with_plan_workspace_bytes(int64_t B, int64_t D, int64_t d, int64_t T,
                                            int64_t plan)
{
    if (check_sizes(B, D, d, T) != LH_OK || plan < LH_PREFILL_MFMA_SEG) return (size_t)-1;
    lh::PrefillPlan p;
    if (!lh::make_prefill_plan(B, D, d, T, plan, -1, &p)) return (size_t)-1;
    return p.ws_bytes;
}

size_t lh_prefill_workspace_bytes(int64_t B, int64_t D, int64_t d, int64_t T)
{
    return lh_prefill_with_plan_workspace_bytes(B, D, d, T, LH_PREFILL_AUTO);
}

int lh_prefill_plan(int64_t B, int64_t D, int64_t d, int64_t T, int64_t plan, lh_dtype io_dtype)
{
    if (check_sizes(B, D, d, T) != LH_OK || plan < LH_PREFILL_MFMA_SEG ||
        (io_dtype != LH_F32 && io_dtype != LH_BF16))
        return -1;
    lh::PrefillPlan p;
    if (!lh::make_prefill_plan(B, D, d, T, plan, io_dtype == LH_BF16 ? 1 : 0, &p)) return -1;
    return p.mfma_seg ? LH_PLAN_MFMA_SEG : p.mfma ? LH_PLAN_MFMA : LH_PLAN_SCAN;
}

lh_status lh_prefill_with_plan(const lh_c32* lambda, const lh_c32* R, const float* h0,
                               const void* u, int64_t B, int64_t D, int64_t d, int64_t T,
                               lh_dtype io_dtype, lh_c32* state, void* y, int64_t plan,
                               void* workspace, size_t workspace_bytes, void* stream)
{
    g_last_error[0] = '\0';
    lh_status s;
    if (!lambda || !R || !h0 || !state)
        return fail(LH_ERR_INVALID_ARG, "lambda, R, h0 and state must not be NULL");
    if ((s = check_sizes(B, D, d, T)) != LH_OK) return s;
    if (T > 0 && (!u || !y)) return fail(LH_ERR_INVALID_ARG, "u and y must not be NULL when T > 0");
    if (plan < LH_PREFILL_MFMA_SEG)
        return fail(LH_ERR_INVALID_ARG,
                    "plan must be >= 0, LH_PREFILL_MFMA or LH_PREFILL_MFMA_SEG");
    if ((s = check_dtype(io_dtype)) != LH_OK) return s;
    lh::PrefillPlan pl;
    if (!lh::make_prefill_plan(B, D, d, T, plan, io_dtype == LH_BF16 ? 1 : 0, &pl))
        return fail(LH_ERR_INVALID_ARG, "no prefill plan for these sizes%s",
                    plan == LH_PREFILL_MFMA
                        ? " (the matrix-core plan needs T >= 1 and d = 16 or 32 with D % 8 == 0, "
                          "or d = 64 with float32 u/y and D % 4 == 0)"
                    : plan == LH_PREFILL_MFMA_SEG
                        ? " (the segmented matrix-core plan also needs T = s * 2^k * 32 "
                          "steps, k >= 1, segments of at least 256 steps)"
                        : "");
    if (pl.mfma_forced && (reinterpret_cast<uintptr_t>(u) % 16 != 0 ||
                           reinterpret_cast<uintptr_t>(y) % 16 != 0))
        return fail(LH_ERR_INVALID_ARG, "the matrix-core plan needs 16-byte aligned u and y");

    if ((s = check_prefill_buffers(lambda, R, h0, u, B, D, d, T, io_dtype, state, y, workspace,
                                   pl.ws_bytes, workspace_bytes)) != LH_OK)
        return s;

    return from_hip(
        lh::launch_prefill(reinterpret_cast<const float2*>(lambda),
                           reinterpret_cast<const float2*>(R), h0, u, io_dtype == LH_BF16, B, D,
                           d, T, reinterpret_cast<float2*>(state), y, pl, workspace,
                           static_cast<hipStream_t>(stream)),
        "prefill launch");
}

lh_status lh_prefill(const lh_c32* lambda, const lh_c32* R, const float* h0, const void* u,
                     int64_t B, int64_t D, int64_t d, int64_t T, lh_dtype io_dtype,
                     lh_c32* state, void* y, void* workspace, size_t workspace_bytes,
                     void* stream)
{
    return lh_prefill_with_plan(lambda, R, h0, u, B, D, d, T, io_dtype, state, y,
                                LH_PREFILL_AUTO, workspace, workspace_bytes, stream);
}

lh_status lh_prefill_noalloc(const lh_c32* lambda, const lh_c32* R, const float* h0,
                             const void* u, int64_t B, int64_t D, int64_t d, int64_t T,
                             lh_dtype io_dtype, lh_c32* state, void* y, void* stream)
{
    g_last_error[0] = '\0';
    lh_status s;
    if (!lambda || !R || !h0 || !state)
        return fail(LH_ERR_INVALID_ARG, "lambda, R, h0 and state must not be NULL");
    if ((s = check_sizes(B, D, d, T)) != LH_OK) return s;
    if (T > 0 && (!u || !y)) return fail(LH_ERR_INVALID_ARG, "u and y must not be NULL when T > 0");
    if ((s = check_dtype(io_dtype)) != LH_OK) return s;
    lh::PrefillPlan pl;
    if (!lh::make_prefill_plan(B, D, d, T, LH_PREFILL_AUTO, io_dtype == LH_BF16 ? 1 : 0, &pl))
        return fail(LH_ERR_INVALID_ARG, "no prefill plan for these sizes");
    if (pl.ws_bytes > kScratchBytes)
        return fail(LH_ERR_WORKSPACE,
                    "these sizes need %zu bytes of scratch; the static scratch of "
                    "lh_prefill_noalloc holds %zu (call lh_prefill with a workspace)",
                    pl.ws_bytes, kScratchBytes);
    if ((s = check_prefill_buffers(lambda, R, h0, u, B, D, d, T, io_dtype, state, y, nullptr, 0,
                                   0)) != LH_OK)
        return s;
    int dev = 0;
    if ((s = check_device(&dev)) != LH_OK) return s;
    void* ws = nullptr;
    if (pl.ws_bytes > 0 && (s = scratch_of(dev, &ws)) != LH_OK) return s;
    return from_hip(
        lh::launch_prefill(reinterpret_cast<const float2*>(lambda),
                           reinterpret_cast<const float2*>(R), h0, u, io_dtype == LH_BF16, B, D,
                           d, T, reinterpret_cast<float2*>(state), y, pl, ws,
                           static_cast<hipStream_t>(stream)),
        "prefill launch");
}

size_t lh_prefill_fft_workspace_bytes(int64_t B, int64_t D, int64_t d, int64_t T)
{
    if (check_sizes(B, D, d, T) != LH_OK) return (size_t)-1;
    lh::FftPlan p;
    if (!lh::make_fft_plan(B, D, d, T, &p)) return (size_t)-1;
    return p.ws_bytes;
}

lh_status lh_prefill_fft(const lh_c32* lambda, const lh_c32* R, const float* h0, const void* u,
                         int64_t B, int64_t D, int64_t d, int64_t T, lh_dtype io_dtype,
                         lh_c32* state, void* y, void* workspace, size_t workspace_bytes,
                         void* stream)
{
    g_last_error[0] = '\0';
    lh_status s;
    if (!lambda || !R || !h0 || !state)
        return fail(LH_ERR_INVALID_ARG, "lambda, R, h0 and state must not be NULL");
    if ((s = check_sizes(B, D, d, T)) != LH_OK) return s;
    if (T > LH_FFT_MAX_T)
        return fail(LH_ERR_INVALID_ARG, "T = %lld exceeds LH_FFT_MAX_T = %lld", (long long)T,
                    (long long)LH_FFT_MAX_T);
    if (T > 0 && (!u || !y)) return fail(LH_ERR_INVALID_ARG, "u and y must not be NULL when T > 0");
    if ((s = check_dtype(io_dtype)) != LH_OK) return s;
    lh::FftPlan plan;
    if (!lh::make_fft_plan(B, D, d, T, &plan))
        return fail(LH_ERR_INVALID_ARG, "no FFT prefill plan for B=%lld D=%lld d=%lld T=%lld",
                    (long long)B, (long long)D, (long long)d, (long long)T);
    if ((s = check_prefill_buffers(lambda, R, h0, u, B, D, d, T, io_dtype, state, y, workspace,
                                   plan.ws_bytes, workspace_bytes)) != LH_OK)
        return s;
    return from_hip(
        lh::launch_prefill_fft(reinterpret_cast<const float2*>(lambda),
                               reinterpret_cast<const float2*>(R), h0, u, io_dtype == LH_BF16, B,
                               D, d, T, reinterpret_cast<float2*>(state), y, plan, workspace,
                               static_cast<hipStream_t>(stream)),
        "FFT prefill launch");
}

lh_status lh_companion_coeffs(const lh_c32* lambda, const lh_c32* R, int64_t D, int64_t d,
                              double* a, double* beta, void* stream)
{
    g_last_error[0] = '\0';
    lh_status s;
    if (!lambda || !R || !a || !beta)
        return fail(LH_ERR_INVALID_ARG, "lambda, R, a and beta must not be NULL");
    if (d < 1 || d > LH_COMPANION_MAX_MODES)
        return fail(LH_ERR_INVALID_ARG, "d = %lld must be in [1, %d]", (long long)d,
                    LH_COMPANION_MAX_MODES);
    if ((s = check_sizes(1, D, d, 0)) != LH_OK) return s;
    const Buf b_lam = buf("lambda", lambda, sizeof(lh_c32) * D * d);
    const Buf b_R = buf("R", R, sizeof(lh_c32) * D * d);
    const Buf b_a = buf("a", a, sizeof(double) * D * 2 * d);
    const Buf b_beta = buf("beta", beta, sizeof(double) * D * 2 * d);
    if ((s = check_align(b_lam, 8)) || (s = check_align(b_R, 8)) || (s = check_align(b_a, 8)) ||
        (s = check_align(b_beta, 8)))
        return s;
    const Buf* ins[] = {&b_lam, &b_R};
    const Buf* outs[] = {&b_a, &b_beta};
    for (const Buf* o : outs)
        for (const Buf* i : ins)
            if (overlaps(*o, *i)) return fail(LH_ERR_OVERLAP, "%s overlaps %s", o->name, i->name);
    if (overlaps(b_a, b_beta)) return fail(LH_ERR_OVERLAP, "a overlaps beta");
    int dev = 0;
    if ((s = check_device(&dev)) != LH_OK) return s;
    for (const Buf* b : {&b_lam, &b_R, &b_a, &b_beta})
        if ((s = check_accessible(*b, dev)) != LH_OK) return s;
    return from_hip(lh::launch_companion_coeffs(reinterpret_cast<const float2*>(lambda),
                                                reinterpret_cast<const float2*>(R), D, d, a, beta,
                                                static_cast<hipStream_t>(stream)),
                    "companion coefficients launch");
}

lh_status lh_companion_step(const double* a, const double* beta, const float* h0, double* state,
                            const void* u_t, void* y_t, int64_t B, int64_t D, int64_t d,
                            lh_dtype io_dtype, void* stream)
{
    g_last_error[0] = '\0';
    lh_status s;
    if (!a || !beta || !h0 || !state || !u_t || !y_t)
        return fail(LH_ERR_INVALID_ARG, "a, beta, h0, state, u_t and y_t must not be NULL");
    if (d < 1 || d > LH_COMPANION_MAX_MODES)
        return fail(LH_ERR_INVALID_ARG, "d = %lld must be in [1, %d]", (long long)d,
                    LH_COMPANION_MAX_MODES);
    if ((s = check_sizes(B, D, d, 0)) != LH_OK) return s;
    if ((s = check_dtype(io_dtype)) != LH_OK) return s;
    const size_t es = io_dtype == LH_BF16 ? 2 : 4;
    const Buf b_a = buf("a", a, sizeof(double) * D * 2 * d);
    const Buf b_beta = buf("beta", beta, sizeof(double) * D * 2 * d);
    const Buf b_h0 = buf("h0", h0, sizeof(float) * D);
    const Buf b_state = buf("state", state, sizeof(double) * B * D * 2 * d);
    const Buf b_u = buf("u_t", u_t, es * B * D);
    const Buf b_y = buf("y_t", y_t, es * B * D);
    if ((s = check_align(b_a, 16)) || (s = check_align(b_beta, 16)) || (s = check_align(b_h0, 4)) ||
        (s = check_align(b_state, 16)) || (s = check_align(b_u, es)) || (s = check_align(b_y, es)))
        return s;
    const Buf* all[] = {&b_a, &b_beta, &b_h0, &b_state, &b_u, &b_y};
    for (const Buf* o : {&b_state, &b_y})
        for (const Buf* i : all)
            if (o != i && overlaps(*o, *i))
                return fail(LH_ERR_OVERLAP, "%s overlaps %s", o->name, i->name);
    int dev = 0;
    if ((s = check_device(&dev)) != LH_OK) return s;
    for (const Buf* b : all)
        if ((s = check_accessible(*b, dev)) != LH_OK) return s;
    return from_hip(lh::launch_companion_step(a, beta, h0, state, u_t, y_t, io_dtype == LH_BF16,
                                              B, D, d, static_cast<hipStream_t>(stream)),
                    "companion step launch");
}

size_t lh_companion_init_workspace_bytes(int64_t D, int64_t d, int64_t T)
{
    if (d < 1 || d > LH_COMPANION_MAX_MODES || check_sizes(1, D, d, T) != LH_OK) return (size_t)-1;
    return lh::companion_init_workspace_bytes(D, T);
}

lh_status lh_companion_init(const double* a, const void* u, int64_t B, int64_t D, int64_t d,
                            int64_t T, lh_dtype io_dtype, double* state, void* workspace,
                            size_t workspace_bytes, void* stream)
{
    g_last_error[0] = '\0';
    lh_status s;
    if (!a || !state) return fail(LH_ERR_INVALID_ARG, "a and state must not be NULL");
    if (d < 1 || d > LH_COMPANION_MAX_MODES)
        return fail(LH_ERR_INVALID_ARG, "d = %lld must be in [1, %d]", (long long)d,
                    LH_COMPANION_MAX_MODES);
    if ((s = check_sizes(B, D, d, T)) != LH_OK) return s;
    if (T > 0 && !u) return fail(LH_ERR_INVALID_ARG, "u must not be NULL when T > 0");
    if ((s = check_dtype(io_dtype)) != LH_OK) return s;
    const size_t need = lh::companion_init_workspace_bytes(D, T);
    const size_t es = io_dtype == LH_BF16 ? 2 : 4;
    const Buf b_a = buf("a", a, sizeof(double) * D * 2 * d);
    const Buf b_u = buf("u", u, T > 0 ? es * B * T * D : 0);
    const Buf b_state = buf("state", state, sizeof(double) * B * D * 2 * d);
    const Buf b_ws = buf("workspace", workspace, need);
    if ((s = check_align(b_a, 8)) || (s = check_align(b_u, es)) || (s = check_align(b_state, 16)))
        return s;
    if (need > 0) {
        if (!workspace)
            return fail(LH_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", need);
        if (workspace_bytes < need)
            return fail(LH_ERR_WORKSPACE, "workspace has %zu bytes, %zu are needed",
                        workspace_bytes, need);
        if ((s = check_align(b_ws, 256))) return s;
    }
    const Buf* ins[] = {&b_a, &b_u};
    for (const Buf* o : {&b_state, &b_ws})
        for (const Buf* i : ins)
            if (overlaps(*o, *i)) return fail(LH_ERR_OVERLAP, "%s overlaps %s", o->name, i->name);
    if (overlaps(b_state, b_ws)) return fail(LH_ERR_OVERLAP, "state overlaps workspace");
    int dev = 0;
    if ((s = check_device(&dev)) != LH_OK) return s;
    for (const Buf* b : {&b_a, &b_u, &b_state, &b_ws})
        if ((s = check_accessible(*b, dev)) != LH_OK) return s;
    return from_hip(lh::launch_companion_init(a, u, io_dtype == LH_BF16, B, D, d, T, state,
                                              workspace, static_cast<hipStream_t>(stream)),
                    "companion initialisation launch");
}

lh_status lh_step(const lh_c32* lambda, const lh_c32* R, const float* h0, lh_c32* state,
                  const void* u_t, void* y_t, int64_t B, int64_t D, int64_t d,
                  lh_dtype io_dtype, void* stream)
{
    g_last_error[0] = '\0';
    lh_status s;
    if (!lambda || !R || !h0 || !state || !u_t || !y_t)
        return fail(LH_ERR_INVALID_ARG, "lambda, R, h0, state, u_t and y_t must not be NULL");
    if ((s = check_sizes(B, D, d, 0)) != LH_OK) return s;
    if ((s = check_dtype(io_dtype)) != LH_OK) return s;

    const size_t es = io_dtype == LH_BF16 ? 2 : 4;
    const Buf b_lam = buf("lambda", lambda, sizeof(lh_c32) * D * d);
    const Buf b_R = buf("R", R, sizeof(lh_c32) * D * d);
    const Buf b_h0 = buf("h0", h0, sizeof(float) * D);
    const Buf b_u = buf("u_t", u_t, es * B * D);
    const Buf b_state = buf("state", state, sizeof(lh_c32) * B * D * d);
    const Buf b_y = buf("y_t", y_t, es * B * D);
    // the 16-byte path of the step kernel needs 16-byte aligned complex arrays
    if ((s = check_align(b_lam, 8)) || (s = check_align(b_R, 8)) || (s = check_align(b_h0, 4)) ||
        (s = check_align(b_state, 8)) || (s = check_align(b_u, es)) || (s = check_align(b_y, es)))
        return s;
    const Buf* ins[] = {&b_lam, &b_R, &b_h0, &b_u};
    for (const Buf* i : ins) {
        if (overlaps(b_state, *i)) return fail(LH_ERR_OVERLAP, "state overlaps %s", i->name);
        if (overlaps(b_y, *i)) return fail(LH_ERR_OVERLAP, "y_t overlaps %s", i->name);
    }
    if (overlaps(b_y, b_state)) return fail(LH_ERR_OVERLAP, "y_t overlaps state");

    int dev = 0;
    if ((s = check_device(&dev)) != LH_OK) return s;
    const Buf* all[] = {&b_lam, &b_R, &b_h0, &b_u, &b_state, &b_y};
    for (const Buf* b : all)
        if ((s = check_accessible(*b, dev)) != LH_OK) return s;

    const bool aligned16 = b_lam.lo % 16 == 0 && b_R.lo % 16 == 0 && b_state.lo % 16 == 0;
    return from_hip(lh::launch_step(reinterpret_cast<const float2*>(lambda),
                                    reinterpret_cast<const float2*>(R), h0,
                                    reinterpret_cast<float2*>(state), u_t, y_t,
                                    io_dtype == LH_BF16, B, D, d, aligned16,
                                    static_cast<hipStream_t>(stream)),
                    "step launch");
}

lh_status lh_mh_step(const lh_c32* lambda, const lh_c32* R, const float* h0, lh_c32* state,
                      const void* q, const void* k, const void* v, void* y, int64_t B,
                      int64_t M, int64_t N, int64_t d, lh_dtype io_dtype, void* stream)
{
    g_last_error[0] = '\0';
    lh_status s;
    if (!lambda || !R || !h0 || !state || !q || !k || !v || !y)
        return fail(LH_ERR_INVALID_ARG, "lambda, R, h0, state, q, k, v and y must not be NULL");
    if (M < 1) return fail(LH_ERR_INVALID_ARG, "M = %lld must be >= 1", (long long)M);
    if (N < 1) return fail(LH_ERR_INVALID_ARG, "N = %lld must be >= 1", (long long)N);
    int64_t D = 0, rows = 0;
    if (!mul_ok(M, N, &D)) return fail(LH_ERR_INVALID_ARG, "M * N overflows");
    if ((s = check_sizes(B, D, d, 0)) != LH_OK) return s;
    int64_t cells = 0;  // complex entries of the state
    if (!mul_ok(B, D, &rows) || !mul_ok(rows, N, &cells) || !mul_ok(cells, d, &cells) ||
        !mul_ok(cells, 8, &cells))
        return fail(LH_ERR_INVALID_ARG, "state size overflows (B=%lld M=%lld N=%lld d=%lld)",
                    (long long)B, (long long)M, (long long)N, (long long)d);
    if ((s = check_dtype(io_dtype)) != LH_OK) return s;

    const size_t es = io_dtype == LH_BF16 ? 2 : 4;
    const Buf b_lam = buf("lambda", lambda, sizeof(lh_c32) * M * d);
    const Buf b_R = buf("R", R, sizeof(lh_c32) * M * d);
    const Buf b_h0 = buf("h0", h0, sizeof(float) * M);
    const Buf b_q = buf("q", q, es * B * D);
    const Buf b_k = buf("k", k, es * B * D);
    const Buf b_v = buf("v", v, es * B * D);
    const Buf b_state = buf("state", state, size_t(cells));
    const Buf b_y = buf("y", y, es * B * D);
    if ((s = check_align(b_lam, 8)) || (s = check_align(b_R, 8)) || (s = check_align(b_h0, 4)) ||
        (s = check_align(b_state, 8)) || (s = check_align(b_q, es)) ||
        (s = check_align(b_k, es)) || (s = check_align(b_v, es)) || (s = check_align(b_y, es)))
        return s;
    const Buf* ins[] = {&b_lam, &b_R, &b_h0, &b_q, &b_k, &b_v};
    for (const Buf* i : ins) {
        if (overlaps(b_state, *i)) return fail(LH_ERR_OVERLAP, "state overlaps %s", i->name);
        if (overlaps(b_y, *i)) return fail(LH_ERR_OVERLAP, "y overlaps %s", i->name);
    }
    if (overlaps(b_y, b_state)) return fail(LH_ERR_OVERLAP, "y overlaps state");

    int dev = 0;
    if ((s = check_device(&dev)) != LH_OK) return s;
    const Buf* all[] = {&b_lam, &b_R, &b_h0, &b_q, &b_k, &b_v, &b_state, &b_y};
    for (const Buf* b : all)
        if ((s = check_accessible(*b, dev)) != LH_OK) return s;

    const bool aligned16 = b_lam.lo % 16 == 0 && b_R.lo % 16 == 0 && b_state.lo % 16 == 0;
    return from_hip(lh::launch_mh_step(reinterpret_cast<const float2*>(lambda),
                                       reinterpret_cast<const float2*>(R), h0,
                                       reinterpret_cast<float2*>(state), q, k, v, y,
                                       io_dtype == LH_BF16, B, M, N, d, aligned16,
                                       static_cast<hipStream_t>(stream)),
                    "multi-head step launch");
}

lh_status lh_distill(const float* A, const float* theta, const lh_c32* R, const float* target,
                     int64_t D, int64_t d, int64_t L, float* loss, float* dA, float* dtheta,
                     lh_c32* dR, float* hhat, void* stream)
{
    g_last_error[0] = '\0';
    lh_status s;
    if (!A || !theta || !R || !target || !loss || !dA || !dtheta || !dR)
        return fail(LH_ERR_INVALID_ARG,
                    "A, theta, R, target, loss, dA, dtheta and dR must not be NULL");
    if (L < 1) return fail(LH_ERR_INVALID_ARG, "L = %lld must be >= 1", (long long)L);
    if ((s = check_sizes(1, D, d, L)) != LH_OK) return s;
    const Buf b_A = buf("A", A, sizeof(float) * D * d);
    const Buf b_th = buf("theta", theta, sizeof(float) * D * d);
    const Buf b_R = buf("R", R, sizeof(lh_c32) * D * d);
    const Buf b_tg = buf("target", target, sizeof(float) * D * L);
    const Buf b_loss = buf("loss", loss, sizeof(float) * D);
    const Buf b_dA = buf("dA", dA, sizeof(float) * D * d);
    const Buf b_dth = buf("dtheta", dtheta, sizeof(float) * D * d);
    const Buf b_dR = buf("dR", dR, sizeof(lh_c32) * D * d);
    const Buf b_h = buf("hhat", hhat, hhat ? sizeof(float) * D * L : 0);
    if ((s = check_align(b_A, 4)) || (s = check_align(b_th, 4)) || (s = check_align(b_R, 8)) ||
        (s = check_align(b_tg, 4)) || (s = check_align(b_loss, 4)) || (s = check_align(b_dA, 4)) ||
        (s = check_align(b_dth, 4)) || (s = check_align(b_dR, 8)) || (s = check_align(b_h, 4)))
        return s;
    const Buf* ins[] = {&b_A, &b_th, &b_R, &b_tg};
    const Buf* outs[] = {&b_loss, &b_dA, &b_dth, &b_dR, &b_h};
    for (const Buf* o : outs) {
        for (const Buf* i : ins)
            if (overlaps(*o, *i)) return fail(LH_ERR_OVERLAP, "%s overlaps %s", o->name, i->name);
        for (const Buf* o2 : outs)
            if (o2 != o && overlaps(*o, *o2))
                return fail(LH_ERR_OVERLAP, "%s overlaps %s", o->name, o2->name);
    }
    int dev = 0;
    if ((s = check_device(&dev)) != LH_OK) return s;
    const Buf* all[] = {&b_A, &b_th, &b_R, &b_tg, &b_loss, &b_dA, &b_dth, &b_dR, &b_h};
    for (const Buf* b : all)
        if ((s = check_accessible(*b, dev)) != LH_OK) return s;
    return from_hip(lh::launch_distill(A, theta, reinterpret_cast<const float2*>(R), target, D,
                                       d, L, loss, dA, dtheta, reinterpret_cast<float2*>(dR),
                                       hhat, static_cast<hipStream_t>(stream)),
                    "distillation launch");
}

}  // extern "C"
