// Decode step of the distilled modal recurrence (Proposition
// "modal_realization", Sec. 3.4; real output as in App. B.1):
//
//   y[b,c]       = Re(sum_n R[c,n] x[b,c,n]) + h0[c] u[b,c]
//   x[b,c,n]    <- lambda[c,n] x[b,c,n] + u[b,c]          (in place)
//
// One pass over the [B, D, d] complex64 state: read once, written once, so the
// kernel is bound by HBM bandwidth (about 16 bytes of state traffic per mode
// against 12 flops).  The d modes of a (b, c) row are spread over LPR
// consecutive lanes (VEC = 2: pairs of adjacent modes per access), so that a wave
// reads and writes one contiguous span of the state with 8- or 16-byte
// accesses; the per-row sum is a butterfly over those lanes.
//
// Blocks are mapped XCD-aware: hardware workgroup i runs on XCD (i mod 8), so
// the logical block index is permuted to give each XCD a contiguous range of
// channel tiles.  A tile's lambda/R (shared by all batch rows) then stays in
// that XCD's L2 instead of being fetched by all eight.
#include "lh_internal.hpp"

namespace lh {
namespace {

constexpr int kBlock = 256;
constexpr int kXcds = 8;

__device__ __forceinline__ int64_t xcd_logical_block(int64_t hw, int64_t nblocks) {
    // hardware block hw -> XCD (hw % 8), k-th block of that XCD; XCD x owns
    // logical blocks [x * per, (x + 1) * per).
    const int64_t per = (nblocks + kXcds - 1) / kXcds;
    const int64_t x = hw % kXcds;
    const int64_t k = hw / kXcds;
    return x * per + k;
}

// VEC = 2: each lane owns NI pairs of modes (16-byte accesses); requires
// d % (2 * LPR) == 0.  VEC = 1: each lane owns modes j, j + LPR, ... (8-byte
// accesses), any d.
template <typename IO, int LPR, int VEC>
__global__ __launch_bounds__(kBlock) void step_kernel(
    const float2* __restrict__ lam, const float2* __restrict__ R, const float* __restrict__ h0,
    float2* __restrict__ state, const IO* __restrict__ u, IO* __restrict__ y,
    int64_t B, int64_t D, int64_t d, int64_t nblocks)
{
    constexpr int kRows = kBlock / LPR;  // rows (channels) per block
    const int64_t lb = xcd_logical_block(blockIdx.x, nblocks);
    if (lb >= nblocks) return;
    const int64_t ct = lb / B;  // channel tile
    const int64_t b = lb - ct * B;
    const int j = threadIdx.x % LPR;
    const int64_t c = ct * kRows + threadIdx.x / LPR;
    const bool valid = c < D;
    const int64_t cc = valid ? c : D - 1;  // keep every address in bounds

    const float uv = io_load(u + b * D + cc);
    const float2* lrow = lam + cc * d;
    const float2* rrow = R + cc * d;
    float2* xrow = state + (b * D + cc) * d;

    float acc = 0.f;
    if constexpr (VEC == 2) {
        const int64_t ni = d / (2 * LPR);
        for (int64_t i = 0; i < ni; ++i) {
            const int64_t m = 2 * (j + i * LPR);
            const float4 l4 = *reinterpret_cast<const float4*>(lrow + m);
            const float4 r4 = *reinterpret_cast<const float4*>(rrow + m);
            const float4 x4 = valid ? *reinterpret_cast<const float4*>(xrow + m)
                                    : make_float4(0.f, 0.f, 0.f, 0.f);
            acc = fmaf(r4.x, x4.x, acc);
            acc = fmaf(-r4.y, x4.y, acc);
            acc = fmaf(r4.z, x4.z, acc);
            acc = fmaf(-r4.w, x4.w, acc);
            float4 n4;
            n4.x = fmaf(l4.x, x4.x, fmaf(-l4.y, x4.y, uv));
            n4.y = fmaf(l4.x, x4.y, l4.y * x4.x);
            n4.z = fmaf(l4.z, x4.z, fmaf(-l4.w, x4.w, uv));
            n4.w = fmaf(l4.z, x4.w, l4.w * x4.z);
            if (valid) *reinterpret_cast<float4*>(xrow + m) = n4;
        }
    } else {
        for (int64_t m = j; m < d; m += LPR) {
            const float2 l2 = lrow[m];
            const float2 r2 = rrow[m];
            const float2 x2 = valid ? xrow[m] : make_float2(0.f, 0.f);
            acc = fmaf(r2.x, x2.x, acc);
            acc = fmaf(-r2.y, x2.y, acc);
            float2 n2;
            n2.x = fmaf(l2.x, x2.x, fmaf(-l2.y, x2.y, uv));
            n2.y = fmaf(l2.x, x2.y, l2.y * x2.x);
            if (valid) xrow[m] = n2;
        }
    }
#pragma unroll
    for (int off = 1; off < LPR; off <<= 1) acc += __shfl_xor(acc, off, LPR);
    if (valid && j == 0) io_store(y + b * D + c, fmaf(h0[c], uv, acc));
}

template <typename IO, int VEC>
hipError_t launch_lpr(int lpr, const float2* lam, const float2* R, const float* h0,
                      float2* state, const void* u, void* y, int64_t B, int64_t D, int64_t d,
                      hipStream_t stream)
{
    const int64_t rows_per_block = kBlock / lpr;
    const int64_t ntiles = (D + rows_per_block - 1) / rows_per_block;
    const int64_t nblocks = ntiles * B;
    const int64_t grid = ((nblocks + kXcds - 1) / kXcds) * kXcds;  // every XCD gets `per` slots
    if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
    const IO* uu = static_cast<const IO*>(u);
    IO* yy = static_cast<IO*>(y);
#define LH_STEP_CASE(L)                                                                   \
    case L:                                                                               \
        hipLaunchKernelGGL((step_kernel<IO, L, VEC>), dim3(static_cast<uint32_t>(grid)), \
                           dim3(kBlock), 0, stream, lam, R, h0, state, uu, yy, B, D, d,   \
                           nblocks);                                                      \
        break;
    switch (lpr) {
        LH_STEP_CASE(1)
        LH_STEP_CASE(2)
        LH_STEP_CASE(4)
        LH_STEP_CASE(8)
        LH_STEP_CASE(16)
        LH_STEP_CASE(32)
        LH_STEP_CASE(64)
        default:
            return hipErrorInvalidValue;
    }
#undef LH_STEP_CASE
    return hipGetLastError();
}

}  // namespace

hipError_t launch_step(const float2* lam, const float2* R, const float* h0, float2* state,
                       const void* u_t, void* y_t, bool bf16_io, int64_t B, int64_t D,
                       int64_t d, bool aligned16, hipStream_t stream)
{
    // Lane layout: with d even (and 16-byte aligned arrays), lanes take pairs
    // of modes (16-byte accesses) and LPR is the largest power of two dividing
    // d / 2, capped at 32; otherwise LPR is the next power of two >= d, capped
    // at 64, and lanes take single modes.
    int lpr = 1;
    const bool vec2 = (d % 2) == 0 && aligned16;
    if (vec2) {
        const int64_t pairs = d / 2;
        while (lpr < 32 && pairs % (2 * lpr) == 0) lpr *= 2;
    } else {
        while (lpr < 64 && lpr < d) lpr *= 2;
    }
    (void)hipGetLastError();  // clear a stale error so the status below is this launch's
    if (vec2) {
        return bf16_io ? launch_lpr<bf16, 2>(lpr, lam, R, h0, state, u_t, y_t, B, D, d, stream)
                       : launch_lpr<float, 2>(lpr, lam, R, h0, state, u_t, y_t, B, D, d, stream);
    }
    return bf16_io ? launch_lpr<bf16, 1>(lpr, lam, R, h0, state, u_t, y_t, B, D, d, stream)
                   : launch_lpr<float, 1>(lpr, lam, R, h0, state, u_t, y_t, B, D, d, stream);
}

}  // namespace lh
