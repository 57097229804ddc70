// Prefill of the distilled modal recurrence: all prompt outputs and the
// post-prompt state (Sec. 3.4, "fast pre-filling").
//
// The prompt of each (b, c) row is cut into nchunks chunks of C steps that run
// in parallel (the blocked form of the parallel-scan prefill of Sec. 3.4):
//
//   1. pow    : lambda^C per (c, n), computed in float64 and rounded once;
//   2. state  : each chunk but the last runs x <- lambda x + u from x = 0 and
//               writes its end state s_k (no outputs);
//   3. carry  : per (b, c, n), x_in[0] = 0, x_in[k+1] = lambda^C x_in[k] + s_k,
//               written over s_k (a sequential scan over <= a few dozen chunks);
//   4. output : each chunk restarts from x_in[k] and runs the full step of
//               Proposition "modal_realization" (y_t = Re(R x_t) + h0 u_t, then
//               x_{t+1} = lambda x_t + u_t), writing y; the last chunk writes
//               x_T to the state.
//
// When the plan has one chunk (enough (b, c) rows to fill the GPU), only the
// output pass runs, from x = 0: a single sequential pass per row.
//
// Lane layout of the state/output passes: a wavefront covers CW = 64 / LPR
// consecutive channels of one (b, chunk); lane l handles channel
// cblk * CW + (l % CW) and modes [(l / CW) * MPL, (l / CW + 1) * MPL).  Every
// time step a wave therefore reads (and writes) one contiguous run of CW
// channels of u (y), and the LPR mode groups of a row are combined with a
// butterfly over lanes CW apart.  Inputs are prefetched kPf steps ahead; the
// main loop carries no bounds checks (the channel index is clamped for lanes
// past D, whose results are discarded), a short tail loop finishes the chunk.
#include "lh_internal.hpp"

namespace lh {
namespace {

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / 64;
constexpr int kPf = 16;  // prefetch depth (time steps)

// ---------------------------------------------------------------- pow kernel
__global__ __launch_bounds__(kBlock) void pow_kernel(const float2* __restrict__ lam,
                                                     float2* __restrict__ lamC, int64_t n,
                                                     int64_t C)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i >= n) return;
    // binary exponentiation in float64: lambda^C with a relative error of a
    // few float64 ulps, rounded once to complex64
    double br = lam[i].x, bi = lam[i].y;
    double pr = 1.0, pi = 0.0;
    for (int64_t e = C; e > 0; e >>= 1) {
        if (e & 1) {
            const double tr = pr * br - pi * bi;
            pi = pr * bi + pi * br;
            pr = tr;
        }
        const double sr = br * br - bi * bi;
        bi = 2.0 * br * bi;
        br = sr;
    }
    lamC[i] = make_float2(static_cast<float>(pr), static_cast<float>(pi));
}

// ------------------------------------------------------------ carry kernel
// One thread per (b, c, n); xs is [B, nchunks, D, d]: on entry slot k < nchunks-1
// holds s_k, on exit slot k holds x_in[k].
__global__ __launch_bounds__(kBlock) void carry_kernel(const float2* __restrict__ lamC,
                                                       float2* __restrict__ xs, int64_t B,
                                                       int64_t Dd, int64_t nchunks)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i >= B * Dd) return;
    const int64_t b = i / Dd;
    const int64_t e = i - b * Dd;  // c * d + n
    const float2 lc = lamC[e];
    float2* p = xs + b * nchunks * Dd + e;
    float xr = 0.f, xi = 0.f;
    for (int64_t k = 0; k < nchunks; ++k) {
        const float2 s = (k + 1 < nchunks) ? p[k * Dd] : make_float2(0.f, 0.f);
        p[k * Dd] = make_float2(xr, xi);
        const float nr = fmaf(lc.x, xr, fmaf(-lc.y, xi, s.x));
        const float ni = fmaf(lc.x, xi, fmaf(lc.y, xr, s.y));
        xr = nr;
        xi = ni;
    }
}

// ---------------------------------------------------------- zero-fill kernel
__global__ __launch_bounds__(kBlock) void zero_kernel(float2* __restrict__ p, int64_t n)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i < n) p[i] = make_float2(0.f, 0.f);
}

// ------------------------------------------------------- chunk scan kernel
// OUTPUT = false: state pass over chunks 0 .. nk-1 (nk = nchunks - 1), from 0,
//                 end state written to xs slot k.
// OUTPUT = true : output pass over chunks 0 .. nchunks-1, from xs slot k (or 0
//                 when nchunks == 1), writes y; the last chunk writes state.
template <int MPL, bool OUTPUT>
struct Modes {
    float lr[MPL], li[MPL], rr[MPL], ri[MPL], xr[MPL], xi[MPL];

    // Re(sum_n R_n x_n) over this lane's modes (two chains for ILP)
    __device__ __forceinline__ float re_rx() const {
        float a0 = 0.f, a1 = 0.f;
#pragma unroll
        for (int m = 0; m < MPL; ++m) {
            a0 = fmaf(rr[m], xr[m], a0);
            a1 = fmaf(ri[m], xi[m], a1);
        }
        return a0 - a1;
    }
    // x <- lambda x + u
    __device__ __forceinline__ void advance(float uv) {
#pragma unroll
        for (int m = 0; m < MPL; ++m) {
            const float nr = fmaf(lr[m], xr[m], fmaf(-li[m], xi[m], uv));
            const float ni = fmaf(lr[m], xi[m], li[m] * xr[m]);
            xr[m] = nr;
            xi[m] = ni;
        }
    }
};

template <typename IO, int LPR, int MPL, bool OUTPUT>
__global__ __launch_bounds__(kBlock) void chunk_scan_kernel(
    const float2* __restrict__ lam, const float2* __restrict__ R, const float* __restrict__ h0,
    const IO* __restrict__ u, IO* __restrict__ y, float2* __restrict__ state,
    float2* __restrict__ xs, int64_t B, int64_t D, int64_t d, int64_t T, int64_t C,
    int64_t nchunks, int64_t nk)
{
    constexpr int CW = 64 / LPR;  // channels per wave
    const int lane = threadIdx.x % 64;
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + threadIdx.x / 64;
    const int64_t ncblk = (D + CW - 1) / CW;
    const int64_t nwaves = nk * B * ncblk;
    if (wave >= nwaves) return;  // whole wave exits together
    const int64_t cblk = wave % ncblk;
    const int64_t bk = wave / ncblk;
    const int64_t b = bk % B;
    const int64_t k = bk / B;

    const int64_t c = cblk * CW + (lane % CW);
    const bool valid = c < D;
    const int64_t cc = valid ? c : D - 1;  // all loads stay in bounds
    const int grp = lane / CW;
    const int64_t n0 = static_cast<int64_t>(grp) * MPL;
    const int64_t Dd = D * d;

    Modes<MPL, OUTPUT> md;
#pragma unroll
    for (int m = 0; m < MPL; ++m) {
        const int64_t n = n0 + m;
        const bool mv = n < d;
        const float2 l2 = mv ? lam[cc * d + n] : make_float2(0.f, 0.f);
        md.lr[m] = l2.x;
        md.li[m] = l2.y;
        md.rr[m] = md.ri[m] = md.xr[m] = md.xi[m] = 0.f;
        if constexpr (OUTPUT) {
            const float2 r2 = mv ? R[cc * d + n] : make_float2(0.f, 0.f);
            md.rr[m] = r2.x;
            md.ri[m] = r2.y;
            if (mv && nchunks > 1) {
                const float2 x2 = xs[(b * nchunks + k) * Dd + cc * d + n];
                md.xr[m] = x2.x;
                md.xi[m] = x2.y;
            }
        }
    }
    const float hz = OUTPUT ? h0[cc] : 0.f;

    const int64_t t0 = k * C;
    const int64_t n = ((t0 + C < T) ? t0 + C : T) - t0;  // steps of this chunk, wave-uniform
    const IO* up = u + (b * T + t0) * D + cc;
    IO* yp = y + (b * T + t0) * D + cc;

    auto one_step = [&](float uv, IO* yt) {
        if constexpr (OUTPUT) {
            float acc = md.re_rx();
#pragma unroll
            for (int off = CW; off < 64; off <<= 1) acc += __shfl_xor(acc, off, 64);
            // Every lane stores: lanes of one row hold bit-identical sums (the
            // butterfly adds commute at each level) and lanes past D repeat
            // channel D-1 exactly, so duplicate stores write the same value.
            io_store(yt, fmaf(hz, uv, acc));
        }
        md.advance(uv);
    };

    int64_t t = 0;
    if (n >= 2 * kPf) {
        // main loop: block t computed while block t + kPf is in flight
        float ub[kPf];
#pragma unroll
        for (int s = 0; s < kPf; ++s) ub[s] = io_load(up + s * D);
        for (; t + 2 * kPf <= n; t += kPf) {
            float un[kPf];
#pragma unroll
            for (int s = 0; s < kPf; ++s) un[s] = io_load(up + (kPf + s) * D);
#pragma unroll
            for (int s = 0; s < kPf; ++s) one_step(ub[s], yp + s * D);
#pragma unroll
            for (int s = 0; s < kPf; ++s) ub[s] = un[s];
            up += kPf * D;
            yp += kPf * D;
        }
        // block t is loaded (t + kPf <= n)
#pragma unroll
        for (int s = 0; s < kPf; ++s) one_step(ub[s], yp + s * D);
        t += kPf;
        up += kPf * D;
        yp += kPf * D;
    }
    for (; t < n; ++t) {  // tail (< 2 kPf steps)
        one_step(io_load(up), yp);
        up += D;
        yp += D;
    }

    // end state: s_k (state pass) or x_T (last chunk of the output pass)
    float2* dst = nullptr;
    if constexpr (OUTPUT) {
        if (k == nchunks - 1) dst = state + (b * D + cc) * d;
    } else {
        dst = xs + (b * nchunks + k) * Dd + cc * d;
    }
    if (dst != nullptr && valid) {
#pragma unroll
        for (int m = 0; m < MPL; ++m) {
            const int64_t nn = n0 + m;
            if (nn < d) dst[nn] = make_float2(md.xr[m], md.xi[m]);
        }
    }
}

template <typename IO, int LPR, int MPL, bool OUTPUT>
hipError_t launch_scan(const float2* lam, const float2* R, const float* h0, const void* u,
                       void* y, float2* state, float2* xs, int64_t B, int64_t D, int64_t d,
                       int64_t T, int64_t C, int64_t nchunks, int64_t nk, hipStream_t stream)
{
    constexpr int CW = 64 / LPR;
    const int64_t ncblk = (D + CW - 1) / CW;
    const int64_t nwaves = nk * B * ncblk;
    const int64_t grid = (nwaves + kWavesPerBlock - 1) / kWavesPerBlock;
    if (grid == 0) return hipSuccess;
    if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((chunk_scan_kernel<IO, LPR, MPL, OUTPUT>),
                       dim3(static_cast<uint32_t>(grid)), dim3(kBlock), 0, stream, lam, R, h0,
                       static_cast<const IO*>(u), static_cast<IO*>(y), state, xs, B, D, d, T, C,
                       nchunks, nk);
    return hipGetLastError();
}

template <typename IO, bool OUTPUT>
hipError_t dispatch_scan(int lpr, int mpl, const float2* lam, const float2* R, const float* h0,
                         const void* u, void* y, float2* state, float2* xs, int64_t B,
                         int64_t D, int64_t d, int64_t T, int64_t C, int64_t nchunks,
                         int64_t nk, hipStream_t stream)
{
#define LH_SCAN(L, M)                                                                       \
    if (lpr == L && mpl == M)                                                               \
        return launch_scan<IO, L, M, OUTPUT>(lam, R, h0, u, y, state, xs, B, D, d, T, C,    \
                                             nchunks, nk, stream);
    // d <= 16: one lane per row, mpl = next power of two >= d
    LH_SCAN(1, 1)
    LH_SCAN(1, 2)
    LH_SCAN(1, 4)
    LH_SCAN(1, 8)
    LH_SCAN(1, 16)
    // d > 16: 16 modes per lane over lpr = ceil(d / 16) (power of two) lanes
    LH_SCAN(2, 16)
    LH_SCAN(4, 16)
    LH_SCAN(8, 16)
    LH_SCAN(16, 16)
    LH_SCAN(32, 16)
    LH_SCAN(64, 16)
#undef LH_SCAN
    return hipErrorInvalidValue;
}

// 1-D grid for n threads; false when it would exceed the grid limit
inline bool grid_for(int64_t n, dim3* g)
{
    const int64_t blocks = (n + kBlock - 1) / kBlock;
    if (blocks > 0x7fffffff) return false;
    *g = dim3(static_cast<uint32_t>(blocks));
    return true;
}

}  // namespace

bool make_prefill_plan(int64_t B, int64_t D, int64_t d, int64_t T, int64_t request, int io,
                       PrefillPlan* plan)
{
    if (io < 0) {  // workspace for either input type
        // (a type with no plan for these sizes, such as bfloat16 under the
        // forced matrix-core plan at d = 64, adds nothing)
        PrefillPlan pf, pb;
        const bool f = make_prefill_plan(B, D, d, T, request, 0, &pf);
        const bool b = make_prefill_plan(B, D, d, T, request, 1, &pb);
        if (!f && !b) return false;
        *plan = f ? pf : pb;
        if (f && b && pb.ws_bytes > plan->ws_bytes) plan->ws_bytes = pb.ws_bytes;
        return true;
    }
    if (B < 1 || D < 1 || d < 1 || d > 1024 || T < 0 || request < -2) return false;
    // element counts must fit comfortably in int64 (and the byte sizes too)
    const int64_t lim = INT64_C(1) << 58;
    if (B > lim / D || B * D > lim / (T > d ? (T > 0 ? T : 1) : d)) return false;

    PrefillPlan p{};
    if (d <= 16) {
        p.lpr = 1;
        p.mpl = 1;
        while (p.mpl < d) p.mpl *= 2;
    } else {
        p.mpl = 16;
        p.lpr = 1;
        while (p.lpr * 16 < d) p.lpr *= 2;
    }
    if (T == 0) {
        p.C = 0;
        p.nchunks = 0;
    } else if (request > 0) {
        p.C = request < T ? request : T;
        p.nchunks = (T + p.C - 1) / p.C;
    } else {
        // Automatic: keep one sequential pass when the (b, c) rows alone give
        // at least 2 waves per SIMD (1024 SIMDs); otherwise cut time into
        // chunks so that about 4 waves per SIMD run, with chunks >= 64 steps.
        const int64_t cw = 64 / p.lpr;
        const int64_t waves = B * ((D + cw - 1) / cw);
        const int64_t kFull = 2048, kTarget = 4096;
        if (waves >= kFull) {
            p.C = T;
        } else {
            const int64_t want = (kTarget + waves - 1) / waves;
            int64_t C = (T + want - 1) / want;
            if (C < 64) C = 64;
            C = (C + 7) / 8 * 8;
            p.C = C < T ? C : T;
        }
        p.nchunks = (T + p.C - 1) / p.C;
    }
    p.ws_bytes = 0;
    p.off_pow = 0;
    p.off_xin = 0;
    if (p.nchunks > 1) {
        const size_t pow_bytes = static_cast<size_t>(D) * d * sizeof(float2);
        p.off_xin = (pow_bytes + 255) / 256 * 256;
        p.ws_bytes = p.off_xin + static_cast<size_t>(B) * p.nchunks * D * d * sizeof(float2);
    }
    // The automatic plan runs on the matrix cores where supported; the
    // workspace also covers the VALU plan above, taken when u or y is not
    // 16-byte aligned.
    p.mfma_forced = request == -1 || request == -2;
    if (p.mfma_forced && !mfma_supported(B, D, d, T, io == 1)) return false;
    const int choice = request == 0 && mfma_supported(B, D, d, T, io == 1)
                           ? mfma_auto_plan(B, D, d, T, io == 1)
                           : 0;
    p.mfma = request == -1 || choice == 1;
    p.mfma_seg = false;
    p.off_mfma = 0;
    if (p.mfma) {
        const size_t mb = mfma_workspace_bytes(D, d);
        if (p.mfma_forced || mb > p.ws_bytes) p.ws_bytes = mb;  // a forced plan has no fallback
    } else if (request == -2 || choice == 2) {
        // too few (batch row, channel group) tiles for the whole-prompt matrix-core
        // plan: cut the prompt into segments that run in parallel, on the matrix
        // cores, with the chunked scan's carry in between
        const int64_t nseg = mfma_segments(B, D, d, T);
        if (nseg >= 2) {
            p.mfma_seg = true;
            p.C = T / nseg;
            p.nchunks = nseg;
            const size_t pow_bytes = static_cast<size_t>(D) * d * sizeof(float2);
            p.off_pow = 0;
            p.off_xin = (pow_bytes + 255) / 256 * 256;
            const size_t xin_bytes = static_cast<size_t>(B) * nseg * D * d * sizeof(float2);
            p.off_mfma = (p.off_xin + xin_bytes + 255) / 256 * 256;
            p.ws_bytes = p.off_mfma + mfma_workspace_bytes(D, d);
        } else if (request == -2) {
            return false;
        }
    }
    *plan = p;
    return true;
}

hipError_t launch_prefill(const float2* lam, const float2* R, const float* h0, const void* u,
                          bool bf16_io, int64_t B, int64_t D, int64_t d, int64_t T,
                          float2* state, void* y, const PrefillPlan& p, void* workspace,
                          hipStream_t stream)
{
    (void)hipGetLastError();  // clear a stale error so the status below is ours
    dim3 g_state, g_pow;
    if (!grid_for(B * D * d, &g_state) || !grid_for(D * d, &g_pow))
        return hipErrorInvalidConfiguration;
    if (T == 0) {
        hipLaunchKernelGGL(zero_kernel, g_state, dim3(kBlock), 0, stream, state, B * D * d);
        return hipGetLastError();
    }
    const bool aligned16 = reinterpret_cast<uintptr_t>(u) % 16 == 0 &&
                           reinterpret_cast<uintptr_t>(y) % 16 == 0;
    if (p.mfma && aligned16)
        return launch_prefill_mfma(lam, R, h0, u, bf16_io, B, D, d, T, state, y, workspace,
                                   stream);
    if (p.mfma_seg && aligned16) {
        char* ws = static_cast<char*>(workspace);
        float2* lamC = reinterpret_cast<float2*>(ws + p.off_pow);
        float2* xs = reinterpret_cast<float2*>(ws + p.off_xin);
        void* mws = ws + p.off_mfma;
        hipError_t e;
        hipLaunchKernelGGL(pow_kernel, g_pow, dim3(kBlock), 0, stream, lam, lamC, D * d, p.C);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = launch_mfma_setup(lam, R, h0, D, d, bf16_io, mws, stream)) != hipSuccess) return e;
        if ((e = launch_mfma_segment_pass(false, lam, u, bf16_io, B, D, d, T, int(p.nchunks), p.C,
                                          xs, state, y, mws, stream)) != hipSuccess)
            return e;
        hipLaunchKernelGGL(carry_kernel, g_state, dim3(kBlock), 0, stream, lamC, xs, B, D * d,
                           p.nchunks);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        return launch_mfma_segment_pass(true, lam, u, bf16_io, B, D, d, T, int(p.nchunks), p.C,
                                        xs, state, y, mws, stream);
    }
    float2* lamC = nullptr;
    float2* xs = nullptr;
    hipError_t e;
    if (p.nchunks > 1) {
        lamC = reinterpret_cast<float2*>(static_cast<char*>(workspace) + p.off_pow);
        xs = reinterpret_cast<float2*>(static_cast<char*>(workspace) + p.off_xin);
        hipLaunchKernelGGL(pow_kernel, g_pow, dim3(kBlock), 0, stream, lam, lamC, D * d, p.C);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        e = bf16_io ? dispatch_scan<bf16, false>(p.lpr, p.mpl, lam, R, h0, u, y, state, xs, B, D,
                                                 d, T, p.C, p.nchunks, p.nchunks - 1, stream)
                    : dispatch_scan<float, false>(p.lpr, p.mpl, lam, R, h0, u, y, state, xs, B,
                                                  D, d, T, p.C, p.nchunks, p.nchunks - 1, stream);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(carry_kernel, g_state, dim3(kBlock), 0, stream, lamC, xs, B, D * d,
                           p.nchunks);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return bf16_io ? dispatch_scan<bf16, true>(p.lpr, p.mpl, lam, R, h0, u, y, state, xs, B, D, d,
                                               T, p.C, p.nchunks, p.nchunks, stream)
                   : dispatch_scan<float, true>(p.lpr, p.mpl, lam, R, h0, u, y, state, xs, B, D,
                                                d, T, p.C, p.nchunks, p.nchunks, stream);
}

}  // namespace lh
