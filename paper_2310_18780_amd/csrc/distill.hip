// Distillation objective of the modal form (Sec. 3.2, "Modal canonical form"):
// per channel c, poles in polar form lambda_n = A_n e^{i theta_n}, residues
// R_n, and a real target filter h_1 .. h_L,
//
//   hhat_t = Re sum_n R_n lambda_n^(t-1)          (eq. "modal_impulse", t = 1..L)
//   e_t    = hhat_t - h_t,   loss = sum_t e_t^2
//   d loss / dR_n     = 2 conj(sum_t e_t lambda_n^(t-1))          (as d/dRe R + i d/dIm R)
//   d loss / dA_n     = 2 Re(R_n e^{i theta_n} S_n)
//   d loss / dtheta_n = 2 Re(i R_n lambda_n S_n),   S_n = sum_t e_t (t-1) lambda_n^(t-2)
//
// and, optionally, the materialised filter hhat (the O(dL) evaluation of
// Lemma "ssmd_impulse").
//
// One workgroup of 256 threads per channel.  The time axis is cut into
// segments of 256 x 16 steps; in a segment thread k owns 16 consecutive steps.
// Pass 1 sums the filter over the modes (in chunks of 8, so any d fits the
// registers) for the thread's steps, from start powers lambda^(t0-1) evaluated
// in polar form (the logarithm of A and the angle reduction in float64, then
// float32 exp and sincos) followed by float32 running products over the 16
// steps; it forms e_t, the loss and, if asked, writes hhat.  Pass 2 walks the
// same powers again and accumulates e_t lambda^(t-1) and e_t (t-1)
// lambda^(t-2) per mode; each chunk's sums are reduced over the wave with DPP
// row permutations and the four row sums, then over the four waves in LDS.
// Per-mode constants (lambda in float32, ln A and theta in float64) are formed
// once per workgroup in LDS.  The gradients are finalised without dividing by
// lambda, so A = 0 is exact.  The work is about 20 flops per (t, n) on the
// VALU; the traffic is the target read once.
#include "lh_internal.hpp"

namespace lh {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesD = kThreads / 64;
constexpr int kTB = 16;                    // steps per thread in a segment
constexpr int kSeg = kThreads * kTB;       // steps per segment
constexpr int kMC = 8;                     // modes per chunk

__device__ __forceinline__ float wave_sum64(float v)
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
    return (__builtin_bit_cast(float, __builtin_amdgcn_readlane(x, 0)) +
            __builtin_bit_cast(float, __builtin_amdgcn_readlane(x, 16))) +
           (__builtin_bit_cast(float, __builtin_amdgcn_readlane(x, 32)) +
            __builtin_bit_cast(float, __builtin_amdgcn_readlane(x, 48)));
}

// lambda^e in polar form: A^e = exp(e ln A) (ln A in float64), the angle
// e theta reduced modulo 2 pi in float64, then float32 exp and sincos; A = 0
// gives 0^0 = 1 and 0 otherwise
__device__ __forceinline__ float2 polar_pow(double lnA, bool zero, double theta, int64_t e)
{
    if (e < 0) return make_float2(0.f, 0.f);
    if (zero) return e == 0 ? make_float2(1.f, 0.f) : make_float2(0.f, 0.f);
    const float mag = __expf(float(double(e) * lnA));
    const double kTwoPi = 6.283185307179586476925286766559;
    const double kInvTwoPi = 0.15915494309189533576888376337251;
    double ang = double(e) * theta;
    ang = fma(-kTwoPi, floor(ang * kInvTwoPi), ang);
    float sn, cs;
    __sincosf(float(ang), &sn, &cs);
    return make_float2(mag * cs, mag * sn);
}

__device__ __forceinline__ float2 cmul(float2 a, float2 b)
{
    return make_float2(fmaf(a.x, b.x, -a.y * b.y), fmaf(a.x, b.y, a.y * b.x));
}

__global__ __launch_bounds__(kThreads) void distill_kernel(
    const float* __restrict__ A, const float* __restrict__ theta, const float2* __restrict__ R,
    const float* __restrict__ target, int d, int64_t L, float* __restrict__ loss,
    float* __restrict__ dA, float* __restrict__ dtheta, float2* __restrict__ dR,
    float* __restrict__ hhat)
{
    const int c = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % 64, wv = tid / 64;
    __shared__ float red[kWavesD][kMC][4];  // per-wave chunk sums: Re/Im of g and S
    __shared__ float acc_s[kWavesD];
    // dynamic LDS: gs [d][4] (sum_t e lambda^(t-1), sum_t e (t-1) lambda^(t-2)),
    // then per mode lambda (float2), ln A and theta (double)
    extern __shared__ __attribute__((aligned(16))) double dyn[];
    double* lnA_s = dyn;
    double* th_s = dyn + d;
    float2* lam_s = reinterpret_cast<float2*>(dyn + 2 * d);
    float* gs = reinterpret_cast<float*>(lam_s + d);
    const float* Ac = A + int64_t(c) * d;
    const float* Tc = theta + int64_t(c) * d;
    const float2* Rc = R + int64_t(c) * d;
    const float* hc = target + int64_t(c) * L;
    for (int i = tid; i < 4 * d; i += kThreads) gs[i] = 0.f;
    for (int n = tid; n < d; n += kThreads) {
        const double a = Ac[n], th = Tc[n];
        lnA_s[n] = a > 0.0 ? log(a) : 0.0;
        th_s[n] = th;
        lam_s[n] = make_float2(float(a * cos(th)), float(a * sin(th)));
    }
    float lacc = 0.f;
    __syncthreads();

    for (int64_t seg0 = 0; seg0 < L; seg0 += kSeg) {
        const int64_t s0 = seg0 + int64_t(tid) * kTB;  // index of t - 1 of the first step
        float hh[kTB];
#pragma unroll
        for (int s = 0; s < kTB; ++s) hh[s] = 0.f;
        // pass 1: hhat over the thread's steps
        for (int n0 = 0; n0 < d; n0 += kMC) {
#pragma unroll
            for (int q = 0; q < kMC; ++q) {
                const int n = n0 + q;
                if (n >= d) break;
                const float2 lam = lam_s[n];
                float2 p = polar_pow(lnA_s[n], Ac[n] == 0.f, th_s[n], s0);
                const float2 r = Rc[n];
#pragma unroll
                for (int s = 0; s < kTB; ++s) {
                    hh[s] = fmaf(r.x, p.x, fmaf(-r.y, p.y, hh[s]));
                    p = cmul(p, lam);
                }
            }
        }
        float e[kTB];
#pragma unroll
        for (int s = 0; s < kTB; ++s) {
            const int64_t t = s0 + s;
            const bool in = t < L;
            e[s] = in ? hh[s] - hc[in ? t : 0] : 0.f;
            lacc = fmaf(e[s], e[s], lacc);
            if (hhat && in) hhat[int64_t(c) * L + t] = hh[s];
        }
        // pass 2: gradient sums, one chunk of modes at a time
        for (int n0 = 0; n0 < d; n0 += kMC) {
            float sums[kMC][4];
#pragma unroll
            for (int q = 0; q < kMC; ++q) {
                const int n = n0 + q;
                sums[q][0] = sums[q][1] = sums[q][2] = sums[q][3] = 0.f;
                if (n >= d) continue;
                const float2 lam = lam_s[n];
                // lambda^(t-2) (0 at t = 1) and lambda^(t-1)
                float2 pm = polar_pow(lnA_s[n], Ac[n] == 0.f, th_s[n], s0 - 1);
                float2 p = s0 == 0 ? make_float2(1.f, 0.f) : cmul(pm, lam);
#pragma unroll
                for (int s = 0; s < kTB; ++s) {
                    const float w = e[s] * float(s0 + s);  // e_t (t - 1)
                    sums[q][0] = fmaf(e[s], p.x, sums[q][0]);
                    sums[q][1] = fmaf(e[s], p.y, sums[q][1]);
                    sums[q][2] = fmaf(w, pm.x, sums[q][2]);
                    sums[q][3] = fmaf(w, pm.y, sums[q][3]);
                    pm = p;
                    p = cmul(p, lam);
                }
            }
#pragma unroll
            for (int q = 0; q < kMC; ++q)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float v = wave_sum64(sums[q][j]);
                    if (lane == 0) red[wv][q][j] = v;
                }
            __syncthreads();
            if (tid < kMC * 4) {
                const int q = tid / 4, j = tid % 4;
                if (n0 + q < d) {
                    float v = 0.f;
#pragma unroll
                    for (int w2 = 0; w2 < kWavesD; ++w2) v += red[w2][q][j];
                    gs[(n0 + q) * 4 + j] += v;
                }
            }
            __syncthreads();
        }
    }
    const float lw = wave_sum64(lacc);
    if (lane == 0) acc_s[wv] = lw;
    __syncthreads();
    if (tid == 0) {
        float v = 0.f;
        for (int w2 = 0; w2 < kWavesD; ++w2) v += acc_s[w2];
        loss[c] = v;
    }
    for (int n = tid; n < d; n += kThreads) {
        const float2 g = make_float2(gs[4 * n], gs[4 * n + 1]);
        const float2 S = make_float2(gs[4 * n + 2], gs[4 * n + 3]);
        const float2 r = Rc[n];
        const double th = th_s[n];
        const float2 unit = make_float2(float(cos(th)), float(sin(th)));
        const float2 lam = lam_s[n];
        const float2 rs = cmul(r, S);
        dR[int64_t(c) * d + n] = make_float2(2.f * g.x, -2.f * g.y);
        dA[int64_t(c) * d + n] = 2.f * cmul(rs, unit).x;
        dtheta[int64_t(c) * d + n] = -2.f * cmul(rs, lam).y;  // Re(i z) = -Im(z)
    }
}

}  // namespace

hipError_t launch_distill(const float* A, const float* theta, const float2* R,
                          const float* target, int64_t D, int64_t d, int64_t L, float* loss,
                          float* dA, float* dtheta, float2* dR, float* hhat, hipStream_t stream)
{
    (void)hipGetLastError();
    if (D > 0x7fffffff || d > 0x7fffffff) return hipErrorInvalidConfiguration;
    const size_t shm = size_t(d) * (2 * sizeof(double) + sizeof(float2) + 4 * sizeof(float));
    hipLaunchKernelGGL(distill_kernel, dim3(uint32_t(D)), dim3(kThreads), shm, stream, A, theta,
                       R, target, int(d), L, loss, dA, dtheta, dR, hhat);
    return hipGetLastError();
}

}  // namespace lh
