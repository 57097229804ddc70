// Decode step of the distilled modal recurrence (Proposition
// "modal_realization", Sec. 3.4; real output as in App. B.1):
//
//   y[b,c]       = Re(sum_n R[c,n] x[b,c,n]) + h0[c] u[b,c]
//   x[b,c,n]    <- lambda[c,n] x[b,c,n] + u[b,c]          (in place)
//
// One pass over the [B, D, d] complex64 state: read once, written once, so the
// kernel is bound by memory bandwidth (16 bytes of state traffic per mode
// against 12 flops).
//
// Fast path (d even, d/2 a power of two <= 64, 16-byte aligned arrays): the
// d/2 mode pairs of a (b, c) row sit on LPR = d/2 consecutive lanes, one
// 16-byte access each, so a wavefront reads and writes one contiguous span
// of the state; the row sum is a butterfly over those lanes (DPP within 16
// lanes).  Each thread serves NB batch rows of the same (c, mode pair):
// lambda and R are loaded once for the NB rows, and every thread has NB
// independent 16-byte state loads in flight before it computes.  NB = 8
// where that still gives 2048 wavefronts (two per SIMD), else 4 where that
// does, else 2: small states are latency-bound, and more wavefronts with
// fewer rows each finish sooner (B = 16, D = 768, d = 16: 1.95 us per step
// with NB = 2 against 2.51 us with NB = 8; B = 64, D = 2048: 6.0 us with
// NB = 8 against 6.3 us with NB = 4).  A workgroup is one wavefront
// (64 / LPR channels x NB batch rows) up to LPR = 16; with LPR >= 32 (d >=
// 64, two channels or fewer per wavefront) it is four wavefronts, so that
// a workgroup covers 8 channels (B = 256, D = 2048, d = 64: 71 us per step
// against 76 us with one-wavefront workgroups).
//
// Cache policy: the state is written with the non-temporal hint, and read
// with it when the whole state fits the L2s with room to spare (at most
// kStreamStateBytes, 16 MiB: half of the 8 XCDs' 4 MB L2s).  An in-place
// pass that reads its lines with ordinary loads leaves them in the caches to
// be written back later; a state streaming from HBM (as the states of a
// model's layers together do) then runs about a quarter slower than a copy
// of the same bytes, and with non-temporal loads at the copy's rate.  A
// state that fits the L2s and is stepped again right away stays there either
// way (16 MiB: within 1%).  A larger state stepped again right away keeps
// part of itself in the 256 MB Infinity Cache only when read with ordinary
// loads (32 MiB: 11.0 us per step against 11.8 us; 256 MiB: 76 us against
// 87 us), so those take ordinary loads.  y_t is stored with ordinary stores:
// its 16-byte pieces per wavefront and batch row are merged into whole lines
// in the L2 before they reach HBM.
//
// Workgroups are ordered so that XCD x (workgroup i runs on XCD i mod 8)
// owns one contiguous range of channel tiles: its lambda / R rows, its slice
// of every batch row of the state, and whole 128-byte lines of u_t and y_t
// stay with one L2.
//
// Generic path (any other d): lanes take single modes j, j + LPR, ...
// (LPR = next power of two >= d, <= 64) or pairs, one batch row per thread.
#include "lh_internal.hpp"

namespace lh {
namespace {

constexpr int kBlock = 256;  // generic path

// fast path: threads per workgroup for LPR lanes per row
constexpr int pairs_block(int lpr) { return lpr >= 32 ? 256 : 64; }
constexpr int kXcds = 8;
constexpr int kMaxRowsPerThread = 8;
constexpr int64_t kMinWaves = 2048;  // wavefronts the row count per thread is chosen for
constexpr int64_t kStreamStateBytes = INT64_C(16) << 20;  // non-temporal state loads up to this size

typedef float f4v __attribute__((ext_vector_type(4)));

// 16-byte accesses.  NT is a template argument, not a run-time flag: with a
// flag, both branches would store the same value to the same address and the
// compiler merges them into one plain access before the flag is known,
// dropping the non-temporal hint.
template <bool NT>
__device__ __forceinline__ float4 load4(const float2* p)
{
    const f4v* q = reinterpret_cast<const f4v*>(p);
    f4v v;
    if constexpr (NT)
        v = __builtin_nontemporal_load(q);
    else
        v = *q;
    return make_float4(v.x, v.y, v.z, v.w);
}

template <bool NT>
__device__ __forceinline__ void store4(float2* p, float4 a)
{
    f4v* q = reinterpret_cast<f4v*>(p);
    const f4v v = {a.x, a.y, a.z, a.w};
    if constexpr (NT)
        __builtin_nontemporal_store(v, q);
    else
        *q = v;
}

// Butterfly step of a row sum over LPR lanes: after the steps for offsets
// 1 .. off/2 every aligned group of `off` lanes holds one partial sum, so any
// lane permutation that pairs each group with its neighbour group completes
// the step.  Within a row of 16 lanes this is DPP on the VALU (quad_perm for
// 1 and 2, half-row mirror for 4, row mirror for 8); wider steps use a shuffle.
template <int OFF>
__device__ __forceinline__ float butterfly(float v)
{
    const int x = __builtin_bit_cast(int, v);
    int p;
    if constexpr (OFF == 1)
        p = __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
    else if constexpr (OFF == 2)
        p = __builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
    else if constexpr (OFF == 4)
        p = __builtin_amdgcn_mov_dpp(x, 0x141, 0xF, 0xF, false);  // row_half_mirror
    else if constexpr (OFF == 8)
        p = __builtin_amdgcn_mov_dpp(x, 0x140, 0xF, 0xF, false);  // row_mirror
    else
        return v + __shfl_xor(v, OFF, 64);
    return v + __builtin_bit_cast(float, p);
}

template <int LPR>
__device__ __forceinline__ float row_sum(float v)
{
    if constexpr (LPR >= 2) v = butterfly<1>(v);
    if constexpr (LPR >= 4) v = butterfly<2>(v);
    if constexpr (LPR >= 8) v = butterfly<4>(v);
    if constexpr (LPR >= 16) v = butterfly<8>(v);
    if constexpr (LPR >= 32) v = butterfly<16>(v);
    if constexpr (LPR >= 64) v = butterfly<32>(v);
    return v;
}

// complex multiply-add of two modes held as (re0, im0, re1, im1)
__device__ __forceinline__ float4 step_pair(float4 l, float4 x, float uv)
{
    float4 n;
    n.x = fmaf(l.x, x.x, fmaf(-l.y, x.y, uv));
    n.y = fmaf(l.x, x.y, l.y * x.x);
    n.z = fmaf(l.z, x.z, fmaf(-l.w, x.w, uv));
    n.w = fmaf(l.z, x.w, l.w * x.z);
    return n;
}

__device__ __forceinline__ float re_dot_pair(float4 r, float4 x)
{
    return fmaf(r.x, x.x, fmaf(-r.y, x.y, fmaf(r.z, x.z, -r.w * x.w)));
}

// Fast path: LPR = d / 2 lanes per row, NB rows per thread, 2-D grid of
// (channel tile, batch group) workgroups.  gridDim.x is the tile count padded
// to a multiple of 8; workgroup x runs on XCD x % 8, which owns tiles
// [(x % 8) T8, (x % 8 + 1) T8) with T8 = gridDim.x / 8.  NTL: non-temporal
// state loads.
template <typename IO, int LPR, bool NTL, int NB>
__global__ __launch_bounds__(pairs_block(LPR)) void step_pairs_kernel(
    const float2* __restrict__ lam, const float2* __restrict__ R, const float* __restrict__ h0,
    float2* __restrict__ state, const IO* __restrict__ u, IO* __restrict__ y, int B, int D,
    int ntiles)
{
    constexpr int kRows = pairs_block(LPR) / LPR;  // channels per workgroup
    constexpr int d = 2 * LPR;
    const int ct = int(blockIdx.x % kXcds) * int(gridDim.x / kXcds) + int(blockIdx.x / kXcds);
    const int b0 = blockIdx.y * NB;
    if (ct >= ntiles) return;  // padding tiles
    const int j = threadIdx.x % LPR;
    const int c = ct * kRows + threadIdx.x / LPR;
    const bool cvalid = c < D;
    const int cc = cvalid ? c : D - 1;  // every address stays in bounds

    const float4 l4 = load4<false>(lam + int64_t(cc) * d + 2 * j);
    const float4 r4 = load4<false>(R + int64_t(cc) * d + 2 * j);
    float4 x[NB];
    float uv[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        const int b = (b0 + i < B) ? b0 + i : B - 1;
        const int64_t row = int64_t(b) * D + cc;
        x[i] = load4<NTL>(state + row * d + 2 * j);
        uv[i] = io_load(u + row);
    }
    const float hz = h0[cc];
    // a use of every u value here keeps all the loads above issued together:
    // left alone, the compiler sinks the first row's u load into its
    // conditional store block, where it is issued only after the first wait
#pragma unroll
    for (int i = 0; i < NB; ++i) asm volatile("" ::"v"(uv[i]));
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        const int b = b0 + i;
        const float acc = row_sum<LPR>(re_dot_pair(r4, x[i]));
        const float4 n4 = step_pair(l4, x[i], uv[i]);
        if (cvalid && b < B) {
            const int64_t row = int64_t(b) * D + c;
            store4<true>(state + row * d + 2 * j, n4);
            if (j == 0) io_store(y + row, fmaf(hz, uv[i], acc));
        }
    }
}

// Generic path.  VEC = 2: each lane owns pairs m = 2 (j + i LPR), requires
// d % (2 LPR) == 0 and 16-byte alignment; VEC = 1: modes j, j + LPR, ...
template <typename IO, int LPR, int VEC>
__global__ __launch_bounds__(kBlock) void step_generic_kernel(
    const float2* __restrict__ lam, const float2* __restrict__ R, const float* __restrict__ h0,
    float2* __restrict__ state, const IO* __restrict__ u, IO* __restrict__ y, int64_t B,
    int64_t D, int64_t d, int64_t nblocks)
{
    constexpr int kRows = kBlock / LPR;
    const int64_t lb = blockIdx.x;
    if (lb >= nblocks) return;
    const int64_t ct = lb / B;
    const int64_t b = lb - ct * B;
    const int j = threadIdx.x % LPR;
    const int64_t c = ct * kRows + threadIdx.x / LPR;
    const bool valid = c < D;
    const int64_t cc = valid ? c : D - 1;

    const float uv = io_load(u + b * D + cc);
    const float2* lrow = lam + cc * d;
    const float2* rrow = R + cc * d;
    float2* xrow = state + (b * D + cc) * d;
    float acc = 0.f;
    if constexpr (VEC == 2) {
        const int64_t ni = d / (2 * LPR);
        for (int64_t i = 0; i < ni; ++i) {
            const int64_t m = 2 * (j + i * LPR);
            const float4 x4 = load4<false>(xrow + m);
            acc += re_dot_pair(load4<false>(rrow + m), x4);
            const float4 n4 = step_pair(load4<false>(lrow + m), x4, uv);
            if (valid) store4<false>(xrow + m, n4);
        }
    } else {
        for (int64_t m = j; m < d; m += LPR) {
            const float2 l2 = lrow[m];
            const float2 r2 = rrow[m];
            const float2 x2 = xrow[m];
            acc = fmaf(r2.x, x2.x, acc);
            acc = fmaf(-r2.y, x2.y, acc);
            float2 n2;
            n2.x = fmaf(l2.x, x2.x, fmaf(-l2.y, x2.y, uv));
            n2.y = fmaf(l2.x, x2.y, l2.y * x2.x);
            if (valid) xrow[m] = n2;
        }
    }
    acc = row_sum<LPR>(acc);
    if (valid && j == 0) io_store(y + b * D + c, fmaf(h0[c], uv, acc));
}

// Batch rows per thread of the fast path (see the file comment).
int pairs_rows_per_thread(int lpr, int64_t B, int64_t D)
{
    const int64_t waves_per_group = (D * lpr + 63) / 64;
    for (int nb = kMaxRowsPerThread; nb > 2; nb /= 2)
        if ((B + nb - 1) / nb * waves_per_group >= kMinWaves) return nb;
    return 2;
}

// 2-D grid of the fast path; false when it does not fit the grid limits
bool pairs_grid(int lpr, int nb, int64_t B, int64_t D, dim3* g, int* ntiles)
{
    const int64_t rows_per_block = pairs_block(lpr) / lpr;
    const int64_t nt = (D + rows_per_block - 1) / rows_per_block;
    const int64_t nbg = (B + nb - 1) / nb;
    const int64_t ntp = (nt + kXcds - 1) / kXcds * kXcds;
    if (ntp > 0x7fffffff || nbg > 65535) return false;
    *g = dim3(uint32_t(ntp), uint32_t(nbg));
    *ntiles = int(nt);
    return true;
}

template <typename IO, bool NTL, int NB>
hipError_t launch_pairs(int lpr, dim3 grid, int ntiles, const float2* lam, const float2* R,
                        const float* h0, float2* state, const void* u, void* y, int64_t B,
                        int64_t D, hipStream_t stream)
{
    const IO* uu = static_cast<const IO*>(u);
    IO* yy = static_cast<IO*>(y);
    const int b = int(B), dd = int(D);
#define LH_PAIRS(L)                                                                          \
    case L:                                                                                  \
        hipLaunchKernelGGL((step_pairs_kernel<IO, L, NTL, NB>), grid, dim3(pairs_block(L)), 0, \
                           stream, lam, R, h0, state, uu, yy, b, dd, ntiles);                \
        break;
    switch (lpr) {
        LH_PAIRS(1)
        LH_PAIRS(2)
        LH_PAIRS(4)
        LH_PAIRS(8)
        LH_PAIRS(16)
        LH_PAIRS(32)
        LH_PAIRS(64)
        default:
            return hipErrorInvalidValue;
    }
#undef LH_PAIRS
    return hipGetLastError();
}

template <typename IO, bool NTL>
hipError_t launch_pairs_nb(int nb, int lpr, dim3 grid, int ntiles, const float2* lam,
                           const float2* R, const float* h0, float2* state, const void* u, void* y,
                           int64_t B, int64_t D, hipStream_t stream)
{
    switch (nb) {
        case 8:
            return launch_pairs<IO, NTL, 8>(lpr, grid, ntiles, lam, R, h0, state, u, y, B, D, stream);
        case 4:
            return launch_pairs<IO, NTL, 4>(lpr, grid, ntiles, lam, R, h0, state, u, y, B, D, stream);
        case 2:
            return launch_pairs<IO, NTL, 2>(lpr, grid, ntiles, lam, R, h0, state, u, y, B, D, stream);
        default:
            return hipErrorInvalidValue;
    }
}

template <typename IO, int VEC>
hipError_t launch_generic(int lpr, const float2* lam, const float2* R, const float* h0,
                          float2* state, const void* u, void* y, int64_t B, int64_t D, int64_t d,
                          hipStream_t stream)
{
    const int64_t rows_per_block = kBlock / lpr;
    const int64_t nblocks = (D + rows_per_block - 1) / rows_per_block * B;
    if (nblocks > 0x7fffffff) return hipErrorInvalidConfiguration;
    const IO* uu = static_cast<const IO*>(u);
    IO* yy = static_cast<IO*>(y);
#define LH_GEN(L)                                                                            \
    case L:                                                                                  \
        hipLaunchKernelGGL((step_generic_kernel<IO, L, VEC>), dim3(uint32_t(nblocks)),       \
                           dim3(kBlock), 0, stream, lam, R, h0, state, uu, yy, B, D, d,      \
                           nblocks);                                                         \
        break;
    switch (lpr) {
        LH_GEN(1)
        LH_GEN(2)
        LH_GEN(4)
        LH_GEN(8)
        LH_GEN(16)
        LH_GEN(32)
        LH_GEN(64)
        default:
            return hipErrorInvalidValue;
    }
#undef LH_GEN
    return hipGetLastError();
}

}  // namespace

hipError_t launch_step(const float2* lam, const float2* R, const float* h0, float2* state,
                       const void* u_t, void* y_t, bool bf16_io, int64_t B, int64_t D,
                       int64_t d, bool aligned16, hipStream_t stream)
{
    (void)hipGetLastError();  // clear a stale error so the status below is this launch's
    const int64_t pairs = d / 2;
    const bool pow2_pairs = d % 2 == 0 && pairs >= 1 && pairs <= 64 && (pairs & (pairs - 1)) == 0;
    dim3 grid;
    int ntiles = 0;
    const int fast_lpr = static_cast<int>(pairs);
    const int nb = pow2_pairs ? pairs_rows_per_thread(fast_lpr, B, D) : 2;
    if (pow2_pairs && aligned16 && B < (INT64_C(1) << 31) && D < (INT64_C(1) << 31) &&
        pairs_grid(fast_lpr, nb, B, D, &grid, &ntiles)) {
        const bool ntl = 8 * B * D * d <= kStreamStateBytes;
        if (bf16_io)
            return ntl ? launch_pairs_nb<bf16, true>(nb, fast_lpr, grid, ntiles, lam, R, h0,
                                                     state, u_t, y_t, B, D, stream)
                       : launch_pairs_nb<bf16, false>(nb, fast_lpr, grid, ntiles, lam, R, h0,
                                                      state, u_t, y_t, B, D, stream);
        return ntl ? launch_pairs_nb<float, true>(nb, fast_lpr, grid, ntiles, lam, R, h0, state,
                                                  u_t, y_t, B, D, stream)
                   : launch_pairs_nb<float, false>(nb, fast_lpr, grid, ntiles, lam, R, h0, state,
                                                   u_t, y_t, B, D, stream);
    }
    // generic layouts
    int lpr = 1;
    const bool vec2 = d % 2 == 0 && aligned16;
    if (vec2) {
        while (lpr < 32 && pairs % (2 * lpr) == 0) lpr *= 2;
        return bf16_io ? launch_generic<bf16, 2>(lpr, lam, R, h0, state, u_t, y_t, B, D, d, stream)
                       : launch_generic<float, 2>(lpr, lam, R, h0, state, u_t, y_t, B, D, d,
                                                  stream);
    }
    while (lpr < 64 && lpr < d) lpr *= 2;
    return bf16_io ? launch_generic<bf16, 1>(lpr, lam, R, h0, state, u_t, y_t, B, D, d, stream)
                   : launch_generic<float, 1>(lpr, lam, R, h0, state, u_t, y_t, B, D, d, stream);
}

}  // namespace lh
