// Decode step of the multi-head (head-tied) long convolution with distilled
// filters (Sec. 5, "Multi-head Long Convolutions"; the state of every entry
// follows Proposition "modal_realization", Sec. 3.4).
//
// Per batch row b, head m (channels m N .. m N + N - 1 of q, k, v, y) and
// output channel i:
//
//   z[i,j]        = k[b, mN+i] v[b, mN+j]
//   w[i,j]        = Re(sum_n R[m,n] x[b,m,i,j,n]) + h0[m] z[i,j]   (reads x)
//   y[b, mN+i]    = sum_j w[i,j] q[b, mN+j]
//   x[b,m,i,j,n] <- lambda[m,n] x[b,m,i,j,n] + z[i,j]               (in place)
//
// One pass over the [B, M, N, N, d] complex64 state, read once and written
// once: bound by memory bandwidth like the per-channel step, with the head's
// lambda and R shared by its N x N entries.
//
// Fast path (d even, d/2 a power of two <= 64, 16-byte aligned arrays): a
// wavefront owns one output row (b, m, i) and streams its N x d state, which
// is contiguous; LPR = d/2 lanes hold the d modes of one entry (two modes and
// one 16-byte access per lane), so a wave covers 64 / LPR entries per access
// and one contiguous kilobyte.  The entry loop is unrolled four times so that
// every lane has four state loads in flight.  Each lane accumulates q_j times
// its share of w[i,j] over all its entries; one reduction over the wave gives
// y.  A workgroup is four waves = four consecutive rows i of one (b, m), which
// share their q and v loads through the cache.  (Measured on the 256 MiB
// bench state: non-temporal state stores, 2 or 8 rows per workgroup and
// unrolling by 2 or 8 were all within 2%, none faster.)
//
// Generic path (any other d or alignment): a wavefront per row as well, one
// entry per lane and a loop over the modes.
#include "lh_internal.hpp"

namespace lh {
namespace {

constexpr int kWaves = 4;  // rows per workgroup
constexpr int kUnroll = 4;

typedef float f4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4 ld4(const float2* p)
{
    const f4v v = *reinterpret_cast<const f4v*>(p);
    return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void st4(float2* p, float4 a)
{
    const f4v v = {a.x, a.y, a.z, a.w};
    *reinterpret_cast<f4v*>(p) = v;
}

// sum over the 64 lanes of a wave, returned in every lane: DPP within rows of
// 16 lanes (after the steps for offsets below 2^k every aligned group of 2^k
// lanes holds one partial sum, so any pairing of neighbour groups completes
// the next step), then the four row sums
__device__ __forceinline__ float wave_sum(float v)
{
    int x = __builtin_bit_cast(int, v);
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false));  // quad_perm [1,0,3,2]
    x = __builtin_bit_cast(int, v);
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false));  // quad_perm [2,3,0,1]
    x = __builtin_bit_cast(int, v);
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(x, 0x141, 0xF, 0xF, false));  // row_half_mirror
    x = __builtin_bit_cast(int, v);
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(x, 0x140, 0xF, 0xF, false));  // row_mirror
    x = __builtin_bit_cast(int, v);
    const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(x, 0));
    const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(x, 16));
    const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(x, 32));
    const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(x, 48));
    return (r0 + r1) + (r2 + r3);
}

template <typename IO, int LPR>
__global__ __launch_bounds__(64 * kWaves) void mh_step_pairs_kernel(
    const float2* __restrict__ lam, const float2* __restrict__ R, const float* __restrict__ h0,
    float2* __restrict__ state, const IO* __restrict__ q, const IO* __restrict__ k,
    const IO* __restrict__ v, IO* __restrict__ y, int M, int N, int64_t nrowblk)
{
    constexpr int d = 2 * LPR;
    constexpr int G = 64 / LPR;  // entries per access of the wave
    const int64_t blk = blockIdx.x;
    if (blk >= nrowblk) return;
    const int nib = (N + kWaves - 1) / kWaves;  // row blocks per (b, m)
    const int64_t bm = blk / nib;                // b * M + m
    const int i = int(blk - bm * nib) * kWaves + int(threadIdx.x) / 64;
    if (i >= N) return;  // whole wave
    const int m = int(bm % M);
    const int lane = threadIdx.x % 64;
    const int p = lane % LPR;   // mode pair of this lane
    const int e = lane / LPR;   // entry offset within an access

    const float4 l4 = ld4(lam + int64_t(m) * d + 2 * p);
    const float4 r4 = ld4(R + int64_t(m) * d + 2 * p);
    const float hz = p == 0 ? h0[m] : 0.f;  // the pass-through term once per entry
    const int64_t io0 = bm * N;               // first channel of head m in row b
    const float ki = io_load(k + io0 + i);
    float2* xrow = state + (bm * N + i) * int64_t(N) * d;

    float acc = 0.f;
    for (int j0 = 0; j0 < N; j0 += kUnroll * G) {
        float4 x[kUnroll];
        float vj[kUnroll], qj[kUnroll];
#pragma unroll
        for (int s = 0; s < kUnroll; ++s) {
            const int j = min(j0 + s * G + e, N - 1);  // clamped: every address in range
            x[s] = ld4(xrow + int64_t(j) * d + 2 * p);
            vj[s] = io_load(v + io0 + j);
            qj[s] = io_load(q + io0 + j);
        }
#pragma unroll
        for (int s = 0; s < kUnroll; ++s) {
            const int j = j0 + s * G + e;
            const float z = ki * vj[s];
            const float w = fmaf(r4.x, x[s].x, fmaf(-r4.y, x[s].y, fmaf(r4.z, x[s].z,
                                 fmaf(-r4.w, x[s].w, hz * z))));
            float4 n4;
            n4.x = fmaf(l4.x, x[s].x, fmaf(-l4.y, x[s].y, z));
            n4.y = fmaf(l4.x, x[s].y, l4.y * x[s].x);
            n4.z = fmaf(l4.z, x[s].z, fmaf(-l4.w, x[s].w, z));
            n4.w = fmaf(l4.z, x[s].w, l4.w * x[s].z);
            if (j < N) {
                acc = fmaf(qj[s], w, acc);
                st4(xrow + int64_t(j) * d + 2 * p, n4);
            }
        }
    }
    const float yi = wave_sum(acc);
    if (lane == 0) io_store(y + io0 + i, yi);
}

// generic path: one entry per lane, modes in a loop
template <typename IO>
__global__ __launch_bounds__(64 * kWaves) void mh_step_generic_kernel(
    const float2* __restrict__ lam, const float2* __restrict__ R, const float* __restrict__ h0,
    float2* __restrict__ state, const IO* __restrict__ q, const IO* __restrict__ k,
    const IO* __restrict__ v, IO* __restrict__ y, int M, int N, int d, int64_t nrowblk)
{
    const int64_t blk = blockIdx.x;
    if (blk >= nrowblk) return;
    const int nib = (N + kWaves - 1) / kWaves;
    const int64_t bm = blk / nib;
    const int i = int(blk - bm * nib) * kWaves + int(threadIdx.x) / 64;
    if (i >= N) return;
    const int m = int(bm % M);
    const int lane = threadIdx.x % 64;
    const int64_t io0 = bm * N;
    const float ki = io_load(k + io0 + i);
    const float hm = h0[m];
    const float2* lm = lam + int64_t(m) * d;
    const float2* rm = R + int64_t(m) * d;
    float2* xrow = state + (bm * N + i) * int64_t(N) * d;
    float acc = 0.f;
    for (int j = lane; j < N; j += 64) {
        const float z = ki * io_load(v + io0 + j);
        float w = hm * z;
        float2* xe = xrow + int64_t(j) * d;
        for (int n = 0; n < d; ++n) {
            const float2 x = xe[n], l = lm[n], r = rm[n];
            w = fmaf(r.x, x.x, fmaf(-r.y, x.y, w));
            xe[n] = make_float2(fmaf(l.x, x.x, fmaf(-l.y, x.y, z)), fmaf(l.x, x.y, l.y * x.x));
        }
        acc = fmaf(io_load(q + io0 + j), w, acc);
    }
    const float yi = wave_sum(acc);
    if (lane == 0) io_store(y + io0 + i, yi);
}

template <typename IO>
hipError_t launch(const float2* lam, const float2* R, const float* h0, float2* state,
                  const void* q, const void* k, const void* v, void* y, int64_t B, int64_t M,
                  int64_t N, int64_t d, bool aligned16, hipStream_t stream)
{
    const int64_t nrowblk = B * M * ((N + kWaves - 1) / kWaves);
    if (nrowblk > 0x7fffffff || N > 0x7fffffff || M > 0x7fffffff || d > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    const IO* qq = static_cast<const IO*>(q);
    const IO* kk = static_cast<const IO*>(k);
    const IO* vv = static_cast<const IO*>(v);
    IO* yy = static_cast<IO*>(y);
    const dim3 grid(static_cast<uint32_t>(nrowblk));
    const dim3 block(64 * kWaves);
    const int64_t pairs = d / 2;
    const bool pow2 = d % 2 == 0 && pairs >= 1 && pairs <= 64 && (pairs & (pairs - 1)) == 0;
    if (pow2 && aligned16) {
        switch (pairs) {
#define LH_MH(L)                                                                              \
    case L:                                                                                   \
        hipLaunchKernelGGL((mh_step_pairs_kernel<IO, L>), grid, block, 0, stream, lam, R, h0, \
                           state, qq, kk, vv, yy, int(M), int(N), nrowblk);                  \
        return hipGetLastError();
            LH_MH(1)
            LH_MH(2)
            LH_MH(4)
            LH_MH(8)
            LH_MH(16)
            LH_MH(32)
            LH_MH(64)
#undef LH_MH
            default:
                break;
        }
    }
    hipLaunchKernelGGL((mh_step_generic_kernel<IO>), grid, block, 0, stream, lam, R, h0, state,
                       qq, kk, vv, yy, int(M), int(N), int(d), nrowblk);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_mh_step(const float2* lam, const float2* R, const float* h0, float2* state,
                          const void* q, const void* k, const void* v, void* y, bool bf16_io,
                          int64_t B, int64_t M, int64_t N, int64_t d, bool aligned16,
                          hipStream_t stream)
{
    (void)hipGetLastError();
    return bf16_io ? launch<bf16>(lam, R, h0, state, q, k, v, y, B, M, N, d, aligned16, stream)
                   : launch<float>(lam, R, h0, state, q, k, v, y, B, M, N, d, aligned16, stream);
}

}  // namespace lh
