// Prefill "via convolutions" (Sec. 3.4, fast pre-filling; the prefill of the
// paper's throughput benchmark), the alternative to the chunked scan:
//
//   1. the filter is materialised from its modal form (Lemma "ssmd_impulse",
//      O(dT)):  hhat_0 = h0,  hhat_t = Re sum_n R_n lambda_n^(t-1), t < T;
//   2. y[b, t] = sum_{j <= t} hhat_{t-j} u[b, j]  (eq. "cnn") for t < T, by
//      N-point FFTs, N the smallest power of two >= 2T - 1, so that the
//      circular wrap-around of the product of spectra misses every output
//      kept;
//   3. the state by the Vandermonde contraction x_T,n = sum_k lambda_n^(T-1-k) u_k
//      (the value at T-1 of the input filtered by the mode's geometric series).
//
// Transforms.  Two real batch rows travel as one complex sequence
// z = u[2p] + i u[2p+1]: the filter is real, so hhat * z = hhat * u[2p] +
// i hhat * u[2p+1] and the real and imaginary parts of the inverse transform
// are the two rows' outputs.  N = N1 N2 with n = n1 + N1 n2 and f = f2 + N2 f1
// (the four-step factorisation):
//
//   pass A (columns): for each n1, Z[f2][n1] = omega_N^(n1 f2) DFT_N2(z[n1 + N1 .])[f2]
//   pass B (rows):    for each f2, X[f2 + N2 f1] = DFT_N1(Z[f2][.])[f1]; times the
//                     filter spectrum H; inverse DFT_N1; times omega_N^(-n1 f2)
//   pass C (columns): for each n1, y[n1 + N1 n2] = IDFT_N2(Z[.][n1])[n2] / N
//
// The filter spectrum comes from the same passes A and B (forward only).
// Every pass keeps the channel index fastest in memory, as u and y have it:
// a workgroup transforms CW adjacent channels, so each global access is a
// contiguous run of CW values, and the transform itself runs in LDS
// (in-place radix-2 stages fused in pairs into 4-point butterflies;
// decimation in time from bit-reversed rows, decimation in frequency into
// bit-reversed rows, so no reordering pass is needed).  Twiddles come from
// one N-point table computed in float64 and rounded once.
//
// The filter is evaluated per thread over 64 consecutive steps from a start
// power in polar form (log2 |lambda| and the angle reduction in float64, then
// float32 exp2 and sincos) followed by running float32 products; the state
// contraction does the same over 256-step ranges, walking time backwards so
// that the powers grow by multiplication by lambda.
#include "prefill_fft.hpp"

namespace lh {
namespace {

constexpr int kThreads = 256;
constexpr int kLdsElems = 8192;   // LDS transform buffer: L x CW complex64 = 64 KiB
constexpr int kHSeg = 64;         // filter steps per thread
constexpr int kSSeg = 256;        // state contraction: steps between polar restarts
constexpr int kSM = 8;            // state contraction: modes per lane
constexpr int kSR = 4;            // state contraction: batch rows per lane
constexpr int kStateWaves = 8192; // state contraction: waves to aim for (8 per SIMD)

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cmul(float2 a, float2 b)
{
    return make_float2(fmaf(a.x, b.x, -a.y * b.y), fmaf(a.x, b.y, a.y * b.x));
}

// omega_N^k (conjugate for the inverse transform)
template <bool INV>
__device__ __forceinline__ float2 twiddle(const float2* __restrict__ tw, int64_t k)
{
    const float2 w = tw[k];
    return INV ? make_float2(w.x, -w.y) : w;
}

// times omega_4 = -i (forward) or +i (inverse)
template <bool INV>
__device__ __forceinline__ float2 quarter(float2 t)
{
    return INV ? make_float2(-t.y, t.x) : make_float2(t.y, -t.x);
}

__device__ __forceinline__ int brev(int x, int bits)
{
    return bits == 0 ? 0 : static_cast<int>(__builtin_bitreverse32(static_cast<uint32_t>(x)) >> (32 - bits));
}

// In-place FFT of L = 2^logL points of CW interleaved sequences in LDS
// (x[row * CW + ch]): decimation in time, rows in bit-reversed order on entry
// and in natural order on exit.  Radix-2 stages of sizes m1 and 2 m1 are
// fused into one 4-point butterfly (a single radix-2 stage first when logL is
// odd); every fused pass ends with a barrier.  tw is the N-point table
// (N = 2^logN >= L).
template <int CW, bool INV>
__device__ void fft_dit(float2* x, int logL, const float2* __restrict__ tw, int logN)
{
    const int L = 1 << logL;
    int s = 1;
    if (logL & 1) {
        for (int q = threadIdx.x; q < (L >> 1) * CW; q += kThreads) {
            const int ch = q % CW, k = q / CW;
            float2* p = x + 2 * k * CW + ch;
            const float2 a = p[0], b = p[CW];
            p[0] = cadd(a, b);
            p[CW] = csub(a, b);
        }
        __syncthreads();
        s = 2;
    }
    for (; s < logL; s += 2) {
        const int m1 = 1 << s, h1 = m1 >> 1;
        for (int q = threadIdx.x; q < (L >> 2) * CW; q += kThreads) {
            const int ch = q % CW, tq = q / CW;
            const int g = tq >> (s - 1), j = tq & (h1 - 1);
            float2* p = x + (2 * g * m1 + j) * CW + ch;
            float2 x0 = p[0], x1 = p[h1 * CW], x2 = p[m1 * CW], x3 = p[(m1 + h1) * CW];
            const float2 w1 = twiddle<INV>(tw, int64_t(j) << (logN - s));      // omega_m1^j
            const float2 w2 = twiddle<INV>(tw, int64_t(j) << (logN - s - 1));  // omega_2m1^j
            float2 t = cmul(w1, x1);
            x1 = csub(x0, t);
            x0 = cadd(x0, t);
            t = cmul(w1, x3);
            x3 = csub(x2, t);
            x2 = cadd(x2, t);
            t = cmul(w2, x2);
            x2 = csub(x0, t);
            x0 = cadd(x0, t);
            t = quarter<INV>(cmul(w2, x3));  // omega_2m1^(j + m1/2)
            x3 = csub(x1, t);
            x1 = cadd(x1, t);
            p[0] = x0;
            p[h1 * CW] = x1;
            p[m1 * CW] = x2;
            p[(m1 + h1) * CW] = x3;
        }
        __syncthreads();
    }
}

// The same transform by decimation in frequency: rows in natural order on
// entry, bit-reversed on exit.  The caller has synchronised the buffer.
template <int CW, bool INV>
__device__ void fft_dif(float2* x, int logL, const float2* __restrict__ tw, int logN)
{
    const int L = 1 << logL;
    int s = logL;
    for (; s >= 2; s -= 2) {
        const int m1 = 1 << (s - 1), h1 = m1 >> 1;
        for (int q = threadIdx.x; q < (L >> 2) * CW; q += kThreads) {
            const int ch = q % CW, tq = q / CW;
            const int g = tq >> (s - 2), j = tq & (h1 - 1);
            float2* p = x + (2 * g * m1 + j) * CW + ch;
            float2 x0 = p[0], x1 = p[h1 * CW], x2 = p[m1 * CW], x3 = p[(m1 + h1) * CW];
            const float2 w2 = twiddle<INV>(tw, int64_t(j) << (logN - s));      // omega_2m1^j
            const float2 w1 = twiddle<INV>(tw, int64_t(j) << (logN - s + 1));  // omega_m1^j
            float2 a = cadd(x0, x2), b = cmul(csub(x0, x2), w2);
            x0 = a;
            x2 = b;
            a = cadd(x1, x3);
            b = quarter<INV>(cmul(csub(x1, x3), w2));
            x1 = a;
            x3 = b;
            a = cadd(x0, x1);
            b = cmul(csub(x0, x1), w1);
            x0 = a;
            x1 = b;
            a = cadd(x2, x3);
            b = cmul(csub(x2, x3), w1);
            x2 = a;
            x3 = b;
            p[0] = x0;
            p[h1 * CW] = x1;
            p[m1 * CW] = x2;
            p[(m1 + h1) * CW] = x3;
        }
        __syncthreads();
    }
    if (s == 1) {
        for (int q = threadIdx.x; q < (L >> 1) * CW; q += kThreads) {
            const int ch = q % CW, k = q / CW;
            float2* p = x + 2 * k * CW + ch;
            const float2 a = p[0], b = p[CW];
            p[0] = cadd(a, b);
            p[CW] = csub(a, b);
        }
        __syncthreads();
    }
}

// lambda^e from (log2 |lambda|, arg lambda): float64 exponent and angle
// reduction, float32 exp2 and sincos; lambda^0 = 1 (also for lambda = 0,
// whose log2 is -inf and gives 0 for e > 0)
__device__ __forceinline__ float2 polar_pow(double2 pol, int64_t e)
{
    if (e == 0) return make_float2(1.f, 0.f);
    const float mag = exp2f(static_cast<float>(static_cast<double>(e) * pol.x));
    const double kTwoPi = 6.283185307179586476925286766559;
    const double kInvTwoPi = 0.15915494309189533576888376337251;
    double ang = static_cast<double>(e) * pol.y;
    ang = fma(-kTwoPi, floor(ang * kInvTwoPi), ang);
    float sn, cs;
    sincosf(static_cast<float>(ang), &sn, &cs);
    return make_float2(mag * cs, mag * sn);
}

// ------------------------------------------------------------ tables
__global__ __launch_bounds__(kThreads) void fft_table_kernel(float2* __restrict__ tw, int logN)
{
    const int64_t k = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (k >= (int64_t(1) << logN)) return;
    double s, c;
    sincospi(2.0 * static_cast<double>(k) / static_cast<double>(int64_t(1) << logN), &s, &c);
    tw[k] = make_float2(static_cast<float>(c), static_cast<float>(-s));  // e^{-2 pi i k / N}
}

__global__ __launch_bounds__(kThreads) void fft_polar_kernel(const float2* __restrict__ lam,
                                                             int64_t n, double2* __restrict__ pol)
{
    const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= n) return;
    const double re = lam[i].x, im = lam[i].y;
    pol[i] = make_double2(log2(hypot(re, im)), atan2(im, re));
}

// ------------------------------------------------------------ filter
// hh[t][c] for t < T.  Lane = channel (64 per wave), wave = 64-step range.
__global__ __launch_bounds__(kThreads) void fft_filter_kernel(const float2* __restrict__ lam,
                                                              const float2* __restrict__ R,
                                                              const float* __restrict__ h0,
                                                              const double2* __restrict__ pol,
                                                              int64_t D, int d, int64_t T,
                                                              float* __restrict__ hh)
{
    const int64_t c = int64_t(blockIdx.x) * 64 + threadIdx.x % 64;
    const int64_t t0 = (int64_t(blockIdx.y) * (kThreads / 64) + threadIdx.x / 64) * kHSeg;
    if (c >= D || t0 >= T) return;
    float acc[kHSeg];
#pragma unroll
    for (int s = 0; s < kHSeg; ++s) acc[s] = 0.f;
    const int64_t base = c * d;
    for (int n = 0; n < d; ++n) {
        const float2 l = lam[base + n], r = R[base + n];
        // power lambda^(t-1) of the first step; t = 0 has no modal term
        float2 p = t0 == 0 ? make_float2(0.f, 0.f) : polar_pow(pol[base + n], t0 - 1);
#pragma unroll
        for (int s = 0; s < kHSeg; ++s) {
            acc[s] = fmaf(r.x, p.x, fmaf(-r.y, p.y, acc[s]));
            p = (s == 0 && t0 == 0) ? make_float2(1.f, 0.f) : cmul(p, l);
        }
    }
    if (t0 == 0) acc[0] += h0[c];
#pragma unroll
    for (int s = 0; s < kHSeg; ++s)
        if (t0 + s < T) hh[(t0 + s) * D + c] = acc[s];
}

// ------------------------------------------------------------ pass A
// Forward column transforms of the real input pairs (or of the filter, with
// B = 1): workgroup = (CW channels, column n1, pair p).
template <typename IO, int CW>
__global__ __launch_bounds__(kThreads) void fft_cols_fwd_kernel(const IO* __restrict__ u,
                                                                int64_t B, int64_t T, int64_t D,
                                                                int logN1, int logN2,
                                                                const float2* __restrict__ tw,
                                                                float2* __restrict__ Z)
{
    extern __shared__ float2 xs[];  // [N2][CW]
    const int logN = logN1 + logN2;
    const int64_t N1 = int64_t(1) << logN1;
    const int N2 = 1 << logN2;
    const int64_t c0 = int64_t(blockIdx.x) * CW;
    const int64_t n1 = blockIdx.y;
    const int64_t p = blockIdx.z;
    const IO* ua = u + 2 * p * T * D;
    const bool has_b = 2 * p + 1 < B;
    // rows n2 with n1 + N1 n2 < T hold inputs; the rest is zero padding
    const int rows = static_cast<int>((T - n1 + N1 - 1) / N1);
    for (int q = threadIdx.x; q < N2 * CW; q += kThreads) {
        const int ch = q % CW, n2 = q / CW;
        const int64_t c = c0 + ch;
        float2 v = make_float2(0.f, 0.f);
        if (n2 < rows && c < D) {
            const int64_t off = (n1 + N1 * n2) * D + c;
            v.x = io_load(ua + off);
            if (has_b) v.y = io_load(ua + T * D + off);
        }
        xs[brev(n2, logN2) * CW + ch] = v;
    }
    __syncthreads();
    fft_dit<CW, false>(xs, logN2, tw, logN);
    float2* zp = Z + (p << logN) * D;
    for (int q = threadIdx.x; q < N2 * CW; q += kThreads) {
        const int ch = q % CW, f2 = q / CW;
        const int64_t c = c0 + ch;
        if (c < D)
            zp[((int64_t(f2) << logN1) + n1) * D + c] =
                cmul(xs[f2 * CW + ch], twiddle<false>(tw, n1 * f2));
    }
}

// ------------------------------------------------------------ pass B
// Row transforms: workgroup = (CW channels, row f2, pair p).  CONV = false:
// forward only, the result is the filter spectrum (in place).  CONV = true:
// forward, times the filter spectrum, inverse, times omega_N^(-n1 f2).
template <int CW, bool CONV>
__global__ __launch_bounds__(kThreads) void fft_rows_kernel(float2* __restrict__ Z,
                                                            const float2* __restrict__ H,
                                                            int64_t D, int logN1, int logN2,
                                                            const float2* __restrict__ tw)
{
    extern __shared__ float2 xs[];  // [N1][CW]
    const int logN = logN1 + logN2;
    const int N1 = 1 << logN1;
    const int64_t c0 = int64_t(blockIdx.x) * CW;
    const int64_t f2 = blockIdx.y;
    const int64_t p = blockIdx.z;
    float2* zr = Z + ((p << logN) + (f2 << logN1)) * D;
    for (int q = threadIdx.x; q < N1 * CW; q += kThreads) {
        const int ch = q % CW, n1 = q / CW;
        const int64_t c = c0 + ch;
        xs[brev(n1, logN1) * CW + ch] = c < D ? zr[int64_t(n1) * D + c] : make_float2(0.f, 0.f);
    }
    __syncthreads();
    fft_dit<CW, false>(xs, logN1, tw, logN);
    if (!CONV) {
        for (int q = threadIdx.x; q < N1 * CW; q += kThreads) {
            const int ch = q % CW, f1 = q / CW;
            const int64_t c = c0 + ch;
            if (c < D) zr[int64_t(f1) * D + c] = xs[f1 * CW + ch];
        }
        return;
    }
    const float2* hr = H + (f2 << logN1) * D;
    for (int q = threadIdx.x; q < N1 * CW; q += kThreads) {
        const int ch = q % CW, f1 = q / CW;
        const int64_t c = c0 + ch;
        if (c < D) xs[f1 * CW + ch] = cmul(xs[f1 * CW + ch], hr[int64_t(f1) * D + c]);
    }
    __syncthreads();
    fft_dif<CW, true>(xs, logN1, tw, logN);
    for (int q = threadIdx.x; q < N1 * CW; q += kThreads) {
        const int ch = q % CW, n1 = q / CW;
        const int64_t c = c0 + ch;
        if (c < D)
            zr[int64_t(n1) * D + c] =
                cmul(xs[brev(n1, logN1) * CW + ch], twiddle<true>(tw, f2 * n1));
    }
}

// ------------------------------------------------------------ pass C
// Inverse column transforms: workgroup = (CW channels, column n1, pair p);
// the real part is row 2p's output, the imaginary part row 2p+1's.
template <typename IO, int CW>
__global__ __launch_bounds__(kThreads) void fft_cols_inv_kernel(const float2* __restrict__ Z,
                                                                int64_t B, int64_t T, int64_t D,
                                                                int logN1, int logN2,
                                                                const float2* __restrict__ tw,
                                                                IO* __restrict__ y)
{
    extern __shared__ float2 xs[];  // [N2][CW]
    const int logN = logN1 + logN2;
    const int64_t N1 = int64_t(1) << logN1;
    const int N2 = 1 << logN2;
    const int64_t c0 = int64_t(blockIdx.x) * CW;
    const int64_t n1 = blockIdx.y;
    const int64_t p = blockIdx.z;
    const float2* zp = Z + (p << logN) * D;
    for (int q = threadIdx.x; q < N2 * CW; q += kThreads) {
        const int ch = q % CW, f2 = q / CW;
        const int64_t c = c0 + ch;
        xs[brev(f2, logN2) * CW + ch] =
            c < D ? zp[((int64_t(f2) << logN1) + n1) * D + c] : make_float2(0.f, 0.f);
    }
    __syncthreads();
    fft_dit<CW, true>(xs, logN2, tw, logN);
    const float scale = 1.f / static_cast<float>(int64_t(1) << logN);  // exact power of two
    const int rows = static_cast<int>((T - n1 + N1 - 1) / N1);
    IO* ya = y + 2 * p * T * D;
    const bool has_b = 2 * p + 1 < B;
    for (int q = threadIdx.x; q < rows * CW; q += kThreads) {
        const int ch = q % CW, n2 = q / CW;
        const int64_t c = c0 + ch;
        if (c < D) {
            const float2 v = xs[n2 * CW + ch];
            const int64_t off = (n1 + N1 * n2) * D + c;
            io_store(ya + off, v.x * scale);
            if (has_b) io_store(ya + T * D + off, v.y * scale);
        }
    }
}

// ------------------------------------------------------------ state
// Partial Vandermonde sums over the time range [part * part_len, ...):
// out[part][b][c][n] = sum_k lambda_n^(T-1-k) u[b, k, c].  Lane = channel,
// wave = 8 modes x 4 batch rows; time runs backwards in 256-step ranges,
// each restarted from a polar power.
template <typename IO>
__global__ __launch_bounds__(kThreads) void fft_state_kernel(const IO* __restrict__ u,
                                                             const float2* __restrict__ lam,
                                                             const double2* __restrict__ pol,
                                                             int64_t B, int64_t D, int d,
                                                             int64_t T, int64_t part_len,
                                                             int nmcg, float2* __restrict__ out)
{
    const int64_t c = int64_t(blockIdx.x) * 64 + threadIdx.x % 64;
    const int mc = static_cast<int>(blockIdx.z % nmcg) * (kThreads / 64) + threadIdx.x / 64;
    const int64_t b0 = int64_t(blockIdx.z / nmcg) * kSR;
    const int64_t part = blockIdx.y;
    const int n0 = mc * kSM;
    if (n0 >= d) return;
    const int64_t cc = c < D ? c : D - 1;  // lanes past D repeat the last channel
    const IO* ur[kSR];
#pragma unroll
    for (int r = 0; r < kSR; ++r) ur[r] = u + (b0 + r < B ? b0 + r : B - 1) * T * D + cc;
    float2 l[kSM];
#pragma unroll
    for (int i = 0; i < kSM; ++i)
        l[i] = n0 + i < d ? lam[cc * d + n0 + i] : make_float2(0.f, 0.f);
    float2 acc[kSR][kSM];
#pragma unroll
    for (int r = 0; r < kSR; ++r)
#pragma unroll
        for (int i = 0; i < kSM; ++i) acc[r][i] = make_float2(0.f, 0.f);
    const int64_t k_lo = part * part_len;
    const int64_t k_hi = k_lo + part_len < T ? k_lo + part_len : T;
    for (int64_t hi = k_hi; hi > k_lo; hi -= kSSeg) {
        const int64_t lo = hi - kSSeg > k_lo ? hi - kSSeg : k_lo;
        float2 pw[kSM];  // lambda^(T-1-k) at k = hi - 1
#pragma unroll
        for (int i = 0; i < kSM; ++i)
            pw[i] = n0 + i < d ? polar_pow(pol[cc * d + n0 + i], T - hi) : make_float2(0.f, 0.f);
#pragma unroll 4
        for (int64_t k = hi - 1; k >= lo; --k) {
            float uv[kSR];
#pragma unroll
            for (int r = 0; r < kSR; ++r) uv[r] = io_load(ur[r] + k * D);
#pragma unroll
            for (int i = 0; i < kSM; ++i) {
#pragma unroll
                for (int r = 0; r < kSR; ++r) {
                    acc[r][i].x = fmaf(pw[i].x, uv[r], acc[r][i].x);
                    acc[r][i].y = fmaf(pw[i].y, uv[r], acc[r][i].y);
                }
                pw[i] = cmul(pw[i], l[i]);
            }
        }
    }
    if (c >= D) return;
#pragma unroll
    for (int r = 0; r < kSR; ++r) {
        if (b0 + r >= B) break;
        float2* o = out + ((part * B + b0 + r) * D + c) * d + n0;
#pragma unroll
        for (int i = 0; i < kSM; ++i)
            if (n0 + i < d) o[i] = acc[r][i];
    }
}

// state[i] = sum over the parts in order (deterministic)
__global__ __launch_bounds__(kThreads) void fft_state_sum_kernel(const float2* __restrict__ parts,
                                                                 int64_t nparts, int64_t n,
                                                                 float2* __restrict__ state)
{
    const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= n) return;
    float2 s = make_float2(0.f, 0.f);
    for (int64_t k = 0; k < nparts; ++k) s = cadd(s, parts[k * n + i]);
    state[i] = s;
}

__global__ __launch_bounds__(kThreads) void fft_zero_kernel(float2* __restrict__ p, int64_t n)
{
    const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i < n) p[i] = make_float2(0.f, 0.f);
}

// channels per workgroup of a transform of length 2^logL (64 KiB of LDS)
int cw_for(int logL) { return (1 << logL) * 32 <= kLdsElems ? 32 : (1 << logL) * 16 <= kLdsElems ? 16 : 8; }

bool blocks_for(int64_t n, int64_t per, uint32_t* g)
{
    const int64_t b = (n + per - 1) / per;
    if (b < 1 || b > 0x7fffffff) return false;
    *g = static_cast<uint32_t>(b);
    return true;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

template <typename IO, int CW>
hipError_t cols_fwd(const IO* u, int64_t B, int64_t T, int64_t D, int logN1, int logN2,
                    const float2* tw, float2* Z, int64_t npair, hipStream_t stream)
{
    uint32_t gx;
    if (!blocks_for(D, CW, &gx)) return hipErrorInvalidConfiguration;
    const dim3 grid(gx, 1u << logN1, static_cast<uint32_t>(npair));
    const size_t shm = sizeof(float2) * (size_t(1) << logN2) * CW;
    hipLaunchKernelGGL((fft_cols_fwd_kernel<IO, CW>), grid, dim3(kThreads), shm, stream, u, B, T, D,
                       logN1, logN2, tw, Z);
    return hipGetLastError();
}

template <typename IO>
hipError_t cols_fwd_any(const IO* u, int64_t B, int64_t T, int64_t D, int logN1, int logN2,
                        const float2* tw, float2* Z, int64_t npair, hipStream_t stream)
{
    switch (cw_for(logN2)) {
        case 32: return cols_fwd<IO, 32>(u, B, T, D, logN1, logN2, tw, Z, npair, stream);
        case 16: return cols_fwd<IO, 16>(u, B, T, D, logN1, logN2, tw, Z, npair, stream);
        default: return cols_fwd<IO, 8>(u, B, T, D, logN1, logN2, tw, Z, npair, stream);
    }
}

template <int CW, bool CONV>
hipError_t rows(float2* Z, const float2* H, int64_t D, int logN1, int logN2, const float2* tw,
                int64_t npair, hipStream_t stream)
{
    uint32_t gx;
    if (!blocks_for(D, CW, &gx)) return hipErrorInvalidConfiguration;
    const dim3 grid(gx, 1u << logN2, static_cast<uint32_t>(npair));
    const size_t shm = sizeof(float2) * (size_t(1) << logN1) * CW;
    hipLaunchKernelGGL((fft_rows_kernel<CW, CONV>), grid, dim3(kThreads), shm, stream, Z, H, D,
                       logN1, logN2, tw);
    return hipGetLastError();
}

template <bool CONV>
hipError_t rows_any(float2* Z, const float2* H, int64_t D, int logN1, int logN2,
                    const float2* tw, int64_t npair, hipStream_t stream)
{
    switch (cw_for(logN1)) {
        case 32: return rows<32, CONV>(Z, H, D, logN1, logN2, tw, npair, stream);
        case 16: return rows<16, CONV>(Z, H, D, logN1, logN2, tw, npair, stream);
        default: return rows<8, CONV>(Z, H, D, logN1, logN2, tw, npair, stream);
    }
}

template <typename IO, int CW>
hipError_t cols_inv(const float2* Z, int64_t B, int64_t T, int64_t D, int logN1, int logN2,
                    const float2* tw, IO* y, int64_t npair, hipStream_t stream)
{
    uint32_t gx;
    if (!blocks_for(D, CW, &gx)) return hipErrorInvalidConfiguration;
    const dim3 grid(gx, 1u << logN1, static_cast<uint32_t>(npair));
    const size_t shm = sizeof(float2) * (size_t(1) << logN2) * CW;
    hipLaunchKernelGGL((fft_cols_inv_kernel<IO, CW>), grid, dim3(kThreads), shm, stream, Z, B, T, D,
                       logN1, logN2, tw, y);
    return hipGetLastError();
}

template <typename IO>
hipError_t run(const float2* lam, const float2* R, const float* h0, const IO* u, int64_t B,
               int64_t D, int64_t d, int64_t T, float2* state, IO* y, const FftPlan& p,
               char* ws, hipStream_t stream)
{
    hipError_t e;
    const int logN = p.logN1 + p.logN2;
    float2* tw = reinterpret_cast<float2*>(ws + p.off_tw);
    double2* pol = reinterpret_cast<double2*>(ws + p.off_polar);
    float2* H = reinterpret_cast<float2*>(ws + p.off_H);
    float2* Z = reinterpret_cast<float2*>(ws + p.off_Z);
    float* hh = reinterpret_cast<float*>(ws + p.off_Z);
    uint32_t g;
    if (!blocks_for(int64_t(1) << logN, kThreads, &g)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(fft_table_kernel, dim3(g), dim3(kThreads), 0, stream, tw, logN);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (!blocks_for(D * d, kThreads, &g)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(fft_polar_kernel, dim3(g), dim3(kThreads), 0, stream, lam, D * d, pol);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    // filter and its spectrum
    uint32_t gc, gt;
    if (!blocks_for(D, 64, &gc) || !blocks_for(T, int64_t(kHSeg) * (kThreads / 64), &gt))
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(fft_filter_kernel, dim3(gc, gt), dim3(kThreads), 0, stream, lam, R, h0, pol,
                       D, static_cast<int>(d), T, hh);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = cols_fwd_any<float>(hh, 1, T, D, p.logN1, p.logN2, tw, H, 1, stream)) != hipSuccess)
        return e;
    if ((e = rows_any<false>(H, nullptr, D, p.logN1, p.logN2, tw, 1, stream)) != hipSuccess)
        return e;

    // outputs
    if ((e = cols_fwd_any<IO>(u, B, T, D, p.logN1, p.logN2, tw, Z, p.npair, stream)) != hipSuccess)
        return e;
    if ((e = rows_any<true>(Z, H, D, p.logN1, p.logN2, tw, p.npair, stream)) != hipSuccess)
        return e;
    switch (cw_for(p.logN2)) {
        case 32: e = cols_inv<IO, 32>(Z, B, T, D, p.logN1, p.logN2, tw, y, p.npair, stream); break;
        case 16: e = cols_inv<IO, 16>(Z, B, T, D, p.logN1, p.logN2, tw, y, p.npair, stream); break;
        default: e = cols_inv<IO, 8>(Z, B, T, D, p.logN1, p.logN2, tw, y, p.npair, stream); break;
    }
    if (e != hipSuccess) return e;

    // state
    const int nmc = static_cast<int>((d + kSM - 1) / kSM);
    const int nmcg = (nmc + kThreads / 64 - 1) / (kThreads / 64);
    const int64_t nrg = (B + kSR - 1) / kSR;
    if (nrg * nmcg > 0x7fffffff || p.nparts > 0xffff) return hipErrorInvalidConfiguration;
    float2* out = p.nparts > 1 ? reinterpret_cast<float2*>(ws + p.off_parts) : state;
    hipLaunchKernelGGL((fft_state_kernel<IO>),
                       dim3(gc, static_cast<uint32_t>(p.nparts), static_cast<uint32_t>(nrg * nmcg)),
                       dim3(kThreads), 0, stream, u, lam, pol, B, D, static_cast<int>(d), T,
                       p.part_len, nmcg, out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (p.nparts > 1) {
        if (!blocks_for(B * D * d, kThreads, &g)) return hipErrorInvalidConfiguration;
        hipLaunchKernelGGL(fft_state_sum_kernel, dim3(g), dim3(kThreads), 0, stream, out, p.nparts,
                           B * D * d, state);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

bool make_fft_plan(int64_t B, int64_t D, int64_t d, int64_t T, FftPlan* plan)
{
    if (B < 1 || D < 1 || d < 1 || d > 1024 || T < 0 || T > kFftMaxT) return false;
    FftPlan p{};
    p.npair = (B + 1) / 2;
    if (p.npair > 0xffff) return false;  // grid z of the transform passes
    if (T == 0) {
        *plan = p;
        return true;
    }
    int m = 0;
    while ((int64_t(1) << m) < 2 * T - 1) ++m;
    p.logN1 = (m + 1) / 2;
    p.logN2 = m / 2;
    const int64_t N = int64_t(1) << m;
    const int64_t lim = int64_t(1) << 58;
    if (D > lim / N || p.npair > lim / (N * D) || B > lim / D || B * D > lim / (d > 1 ? d : 1))
        return false;
    const int64_t nseg = (T + kSSeg - 1) / kSSeg;
    const int64_t waves = ((D + 63) / 64) * ((d + kSM - 1) / kSM) * ((B + kSR - 1) / kSR);
    int64_t want = (kStateWaves + waves - 1) / waves;
    if (want > nseg) want = nseg;
    const int64_t segs = (nseg + want - 1) / want;
    p.part_len = segs * kSSeg;
    p.nparts = (nseg + segs - 1) / segs;
    size_t off = 0;
    p.off_tw = off;
    off = align256(off + sizeof(float2) * N);
    p.off_polar = off;
    off = align256(off + sizeof(double) * 2 * D * d);
    p.off_H = off;
    off = align256(off + sizeof(float2) * N * D);
    p.off_Z = off;
    off = align256(off + sizeof(float2) * p.npair * N * D);
    p.off_parts = off;
    if (p.nparts > 1) off = align256(off + sizeof(float2) * p.nparts * B * D * d);
    p.ws_bytes = off;
    *plan = p;
    return true;
}

hipError_t launch_prefill_fft(const float2* lam, const float2* R, const float* h0,
                              const void* u, bool bf16_io, int64_t B, int64_t D, int64_t d,
                              int64_t T, float2* state, void* y, const FftPlan& plan,
                              void* workspace, hipStream_t stream)
{
    (void)hipGetLastError();
    if (T == 0) {
        uint32_t g;
        if (!blocks_for(B * D * d, kThreads, &g)) return hipErrorInvalidConfiguration;
        hipLaunchKernelGGL(fft_zero_kernel, dim3(g), dim3(kThreads), 0, stream, state, B * D * d);
        return hipGetLastError();
    }
    char* ws = static_cast<char*>(workspace);
    return bf16_io ? run<bf16>(lam, R, h0, static_cast<const bf16*>(u), B, D, d, T, state,
                               static_cast<bf16*>(y), plan, ws, stream)
                   : run<float>(lam, R, h0, static_cast<const float*>(u), B, D, d, T, state,
                                static_cast<float*>(y), plan, ws, stream);
}

}  // namespace lh
