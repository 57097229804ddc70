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
// contiguous run of CW values.  The transform runs on a tile in LDS as
// Stockham autosort stages (natural order in and out, so no reordering pass):
// radix-8 butterflies in registers, one radix-2 or radix-4 stage for the
// remaining factor, one barrier between the reads and the writes of a stage.
// Transform lengths are template parameters, so every loop over a thread's
// elements is unrolled and all of a tile's global loads are in flight
// together (the row pass also loads its slice of the filter spectrum up
// front).  Twiddles come from one N-point table computed in float64 and
// rounded once; a butterfly loads its base twiddle and forms the powers.
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
constexpr int kPf = 8;            // state contraction: steps per prefetched block
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

// Transform tile of L = 2^LOGL points for CW adjacent channels, in LDS as
// x[row * CW + ch] (64 KiB at most); every thread holds EPT elements.
template <int LOGL>
struct Tile {
    static constexpr int L = 1 << LOGL;
    static constexpr int CW = L * 32 <= kLdsElems ? 32 : L * 16 <= kLdsElems ? 16 : 8;
    static constexpr int E = L * CW;
    static constexpr int EPT = (E + kThreads - 1) / kThreads;
};

constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x / 2); }

// DFT of R = 2, 4 or 8 points in registers (forward: omega_R = e^{-2 pi i / R})
template <bool INV>
__device__ __forceinline__ void dft4(float2& a, float2& b, float2& c, float2& d)
{
    const float2 t0 = cadd(a, c), t1 = csub(a, c), t2 = cadd(b, d);
    const float2 t3 = quarter<INV>(csub(b, d));
    a = cadd(t0, t2);
    c = csub(t0, t2);
    b = cadd(t1, t3);
    d = csub(t1, t3);
}

template <int R, bool INV>
__device__ __forceinline__ void dft(float2 (&v)[R])
{
    if constexpr (R == 2) {
        const float2 a = v[0];
        v[0] = cadd(a, v[1]);
        v[1] = csub(a, v[1]);
    } else if constexpr (R == 4) {
        dft4<INV>(v[0], v[1], v[2], v[3]);
    } else {
        static_assert(R == 8, "radix 2, 4 or 8");
        float2 e0 = v[0], e1 = v[2], e2 = v[4], e3 = v[6];
        float2 o0 = v[1], o1 = v[3], o2 = v[5], o3 = v[7];
        dft4<INV>(e0, e1, e2, e3);
        dft4<INV>(o0, o1, o2, o3);
        const float h = 0.70710678118654752440f;  // omega_8 = (1 -+ i) / sqrt 2
        o1 = INV ? make_float2(h * (o1.x - o1.y), h * (o1.x + o1.y))
                 : make_float2(h * (o1.x + o1.y), h * (o1.y - o1.x));
        o2 = quarter<INV>(o2);
        o3 = INV ? make_float2(-h * (o3.x + o3.y), h * (o3.x - o3.y))
                 : make_float2(h * (o3.y - o3.x), -h * (o3.x + o3.y));
        v[0] = cadd(e0, o0);
        v[4] = csub(e0, o0);
        v[1] = cadd(e1, o1);
        v[5] = csub(e1, o1);
        v[2] = cadd(e2, o2);
        v[6] = csub(e2, o2);
        v[3] = cadd(e3, o3);
        v[7] = csub(e3, o3);
    }
}

// One Stockham autosort stage of radix R after NS points have been combined:
// butterfly j reads x[j + r L/R], multiplies by omega_(NS R)^((j mod NS) r),
// transforms, and writes x[(j / NS) NS R + (j mod NS) + r NS].  All reads
// happen before a barrier, all writes after it, so one buffer serves.
template <int LOGL, int R, int NS, bool INV>
__device__ __forceinline__ void stage(float2* xs, const float2* __restrict__ tw, int logN)
{
    constexpr int L = Tile<LOGL>::L, CW = Tile<LOGL>::CW;
    constexpr int NB = (L / R) * CW;
    constexpr int BPT = (NB + kThreads - 1) / kThreads;
    constexpr int kShift = ilog2(NS * R);
    float2 v[BPT][R];
    float2 w[BPT];
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
        const int q = threadIdx.x + b * kThreads;
        if (NB % kThreads == 0 || q < NB) {
            const int ch = q % CW, j = q / CW;
#pragma unroll
            for (int r = 0; r < R; ++r) v[b][r] = xs[(j + r * (L / R)) * CW + ch];
            if (NS > 1) w[b] = twiddle<INV>(tw, int64_t(j % NS) << (logN - kShift));
        }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
        const int q = threadIdx.x + b * kThreads;
        if (NB % kThreads == 0 || q < NB) {
            const int ch = q % CW, j = q / CW;
            if (NS > 1) {
                float2 wr = w[b];
#pragma unroll
                for (int r = 1; r < R; ++r) {
                    v[b][r] = cmul(v[b][r], wr);
                    if (r + 1 < R) wr = cmul(wr, w[b]);
                }
            }
            dft<R, INV>(v[b]);
            const int base = (j / NS) * NS * R + j % NS;
#pragma unroll
            for (int r = 0; r < R; ++r) xs[(base + r * NS) * CW + ch] = v[b][r];
        }
    }
    __syncthreads();
}

template <int LOGL, int NS, bool INV>
__device__ __forceinline__ void stages8(float2* xs, const float2* __restrict__ tw, int logN)
{
    if constexpr (NS < (1 << LOGL)) {
        stage<LOGL, 8, NS, INV>(xs, tw, logN);
        stages8<LOGL, NS * 8, INV>(xs, tw, logN);
    }
}

// In-place transform of the tile (natural order in and out): one stage of
// radix 2^(LOGL mod 3) (or 8) followed by radix-8 stages.  The caller has
// synchronised the buffer; it is synchronised on return.
template <int LOGL, bool INV>
__device__ __forceinline__ void fft_tile(float2* xs, const float2* __restrict__ tw, int logN)
{
    if constexpr (LOGL > 0) {
        constexpr int R0 = LOGL % 3 == 0 ? 8 : 1 << (LOGL % 3);
        stage<LOGL, R0, 1, INV>(xs, tw, logN);
        stages8<LOGL, R0, INV>(xs, tw, logN);
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
// B = 1): workgroup = (CW channels, column n1, pair p); N2 = 2^LOGL.
template <typename IO, int LOGL>
__global__ __launch_bounds__(kThreads) void fft_cols_fwd_kernel(const IO* __restrict__ u,
                                                                int64_t B, int64_t T, int64_t D,
                                                                int logN1,
                                                                const float2* __restrict__ tw,
                                                                float2* __restrict__ Z)
{
    using Tl = Tile<LOGL>;
    constexpr int CW = Tl::CW, E = Tl::E, EPT = Tl::EPT;
    __shared__ float2 xs[E];
    const int logN = logN1 + LOGL;
    const int64_t N1 = int64_t(1) << logN1;
    const int64_t c0 = int64_t(blockIdx.x) * CW;
    const int64_t n1 = blockIdx.y;
    const int64_t p = blockIdx.z;
    const IO* ua = u + 2 * p * T * D;
    const bool has_b = 2 * p + 1 < B;
    const IO* ub = has_b ? ua + T * D : ua;
    // rows n2 with n1 + N1 n2 < T hold inputs; the rest is zero padding.
    // Branch-free loads (padding reads element 0 and is discarded), so that
    // all of them are in flight together.
    const int rows = static_cast<int>((T - n1 + N1 - 1) / N1);
    float2 v[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        const int ch = q % CW, n2 = q / CW;
        const int64_t c = c0 + ch;
        const bool ok = (E % kThreads == 0 || q < E) && n2 < rows && c < D;
        const int64_t off = ok ? (n1 + N1 * n2) * D + c : 0;
        const float a = io_load(ua + off), b = io_load(ub + off);
        v[i] = make_float2(ok ? a : 0.f, ok && has_b ? b : 0.f);
    }
    float2 wv[EPT];  // omega_N^(n1 f2) of the outputs, loaded with the inputs
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        wv[i] = twiddle<false>(tw, E % kThreads == 0 || q < E ? n1 * (q / CW) : 0);
    }
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        if (E % kThreads == 0 || q < E) xs[q] = v[i];
    }
    __syncthreads();
    fft_tile<LOGL, false>(xs, tw, logN);
    float2* zp = Z + (p << logN) * D;
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        const int ch = q % CW, f2 = q / CW;
        const int64_t c = c0 + ch;
        if ((E % kThreads == 0 || q < E) && c < D)
            zp[((int64_t(f2) << logN1) + n1) * D + c] = cmul(xs[q], wv[i]);
    }
}

// ------------------------------------------------------------ pass B
// Row transforms: workgroup = (CW channels, row f2, pair p); N1 = 2^LOGL.
// CONV = false: forward only, the result is the filter spectrum (in place).
// CONV = true: forward, times the filter spectrum (loaded up front), inverse,
// times omega_N^(-n1 f2).  One-dimensional grid: workgroup i runs on XCD
// i mod 8, and the npair workgroups of a (channel group, row) tile are 8
// apart, so they run together on one XCD and read the tile's filter spectrum
// from HBM once (the rest from that XCD's L2).
template <int LOGL, bool CONV>
__global__ __launch_bounds__(kThreads) void fft_rows_kernel(float2* __restrict__ Z,
                                                            const float2* __restrict__ H,
                                                            int64_t D, int logN2, int64_t npair,
                                                            const float2* __restrict__ tw)
{
    using Tl = Tile<LOGL>;
    constexpr int CW = Tl::CW, E = Tl::E, EPT = Tl::EPT;
    __shared__ float2 xs[E];
    const int logN = LOGL + logN2;
    const int64_t gx = (D + CW - 1) / CW;
    const int64_t id = blockIdx.x;
    const int64_t tile = id / (8 * npair) * 8 + id % 8;
    if (tile >= (gx << logN2)) return;
    const int64_t p = id / 8 % npair;
    const int64_t c0 = tile % gx * CW;
    const int64_t f2 = tile / gx;
    float2* zr = Z + ((p << logN) + (f2 << LOGL)) * D;
    const float2* hr = H + (f2 << LOGL) * D;
    float2 v[EPT], hv[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        const int ch = q % CW, n = q / CW;
        const int64_t c = c0 + ch;
        const bool ok = (E % kThreads == 0 || q < E) && c < D;
        v[i] = ok ? zr[int64_t(n) * D + c] : make_float2(0.f, 0.f);
        if (CONV) hv[i] = ok ? hr[int64_t(n) * D + c] : make_float2(0.f, 0.f);
    }
    float2 wv[EPT];  // omega_N^(-n1 f2) of the outputs, loaded with the inputs
    if (CONV) {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const int q = threadIdx.x + i * kThreads;
            wv[i] = twiddle<true>(tw, E % kThreads == 0 || q < E ? f2 * (q / CW) : 0);
        }
    }
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        if (E % kThreads == 0 || q < E) xs[q] = v[i];
    }
    __syncthreads();
    fft_tile<LOGL, false>(xs, tw, logN);
    if (!CONV) {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const int q = threadIdx.x + i * kThreads;
            const int ch = q % CW, f1 = q / CW;
            const int64_t c = c0 + ch;
            if ((E % kThreads == 0 || q < E) && c < D) zr[int64_t(f1) * D + c] = xs[q];
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        if (E % kThreads == 0 || q < E) xs[q] = cmul(xs[q], hv[i]);
    }
    __syncthreads();
    fft_tile<LOGL, true>(xs, tw, logN);
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        const int ch = q % CW, n1 = q / CW;
        const int64_t c = c0 + ch;
        if ((E % kThreads == 0 || q < E) && c < D)
            zr[int64_t(n1) * D + c] = cmul(xs[q], wv[i]);
    }
}

// ------------------------------------------------------------ pass C
// Inverse column transforms: workgroup = (CW channels, column n1, pair p);
// the real part is row 2p's output, the imaginary part row 2p+1's.
template <typename IO, int LOGL>
__global__ __launch_bounds__(kThreads) void fft_cols_inv_kernel(const float2* __restrict__ Z,
                                                                int64_t B, int64_t T, int64_t D,
                                                                int logN1,
                                                                const float2* __restrict__ tw,
                                                                IO* __restrict__ y)
{
    using Tl = Tile<LOGL>;
    constexpr int CW = Tl::CW, E = Tl::E, EPT = Tl::EPT;
    __shared__ float2 xs[E];
    const int logN = logN1 + LOGL;
    const int64_t N1 = int64_t(1) << logN1;
    const int64_t c0 = int64_t(blockIdx.x) * CW;
    const int64_t n1 = blockIdx.y;
    const int64_t p = blockIdx.z;
    const float2* zp = Z + (p << logN) * D;
    float2 v[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        const int ch = q % CW, f2 = q / CW;
        const int64_t c = c0 + ch;
        v[i] = (E % kThreads == 0 || q < E) && c < D ? zp[((int64_t(f2) << logN1) + n1) * D + c]
                                                     : make_float2(0.f, 0.f);
    }
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        if (E % kThreads == 0 || q < E) xs[q] = v[i];
    }
    __syncthreads();
    fft_tile<LOGL, true>(xs, tw, logN);
    const float scale = 1.f / static_cast<float>(int64_t(1) << logN);  // exact power of two
    const int rows = static_cast<int>((T - n1 + N1 - 1) / N1);
    IO* ya = y + 2 * p * T * D;
    const bool has_b = 2 * p + 1 < B;
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int q = threadIdx.x + i * kThreads;
        const int ch = q % CW, n2 = q / CW;
        const int64_t c = c0 + ch;
        if ((E % kThreads == 0 || q < E) && n2 < rows && c < D) {
            const float2 r = xs[q];
            const int64_t off = (n1 + N1 * n2) * D + c;
            io_store(ya + off, r.x * scale);
            if (has_b) io_store(ya + T * D + off, r.y * scale);
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
    // one step k: acc += lambda^(T-1-k) u[., k], then the power advances
    auto step = [&](float2 (&pw)[kSM], const float (&uv)[kSR]) {
#pragma unroll
        for (int i = 0; i < kSM; ++i) {
#pragma unroll
            for (int r = 0; r < kSR; ++r) {
                acc[r][i].x = fmaf(pw[i].x, uv[r], acc[r][i].x);
                acc[r][i].y = fmaf(pw[i].y, uv[r], acc[r][i].y);
            }
            pw[i] = cmul(pw[i], l[i]);
        }
    };
    const int64_t k_lo = part * part_len;
    const int64_t k_hi = k_lo + part_len < T ? k_lo + part_len : T;
    for (int64_t hi = k_hi; hi > k_lo; hi -= kSSeg) {
        const int64_t lo = hi - kSSeg > k_lo ? hi - kSSeg : k_lo;
        float2 pw[kSM];  // lambda^(T-1-k) at k = hi - 1
#pragma unroll
        for (int i = 0; i < kSM; ++i)
            pw[i] = n0 + i < d ? polar_pow(pol[cc * d + n0 + i], T - hi) : make_float2(0.f, 0.f);
        // the top (hi - lo) mod 8 steps one by one, then blocks of 8 steps
        // with the next block's inputs loaded while the current one is used
        const int64_t nblk = (hi - lo) / kPf;
        int64_t k = hi - 1;
        for (; k >= lo + nblk * kPf; --k) {
            float uv[kSR];
#pragma unroll
            for (int r = 0; r < kSR; ++r) uv[r] = io_load(ur[r] + k * D);
            step(pw, uv);
        }
        if (nblk > 0) {
            // two buffers in turn: block i + 1 loads while block i is used
            float ba[kPf][kSR], bb[kPf][kSR];
            auto load = [&](float (&buf)[kPf][kSR], int64_t kk) {
#pragma unroll
                for (int s = 0; s < kPf; ++s)
#pragma unroll
                    for (int r = 0; r < kSR; ++r) buf[s][r] = io_load(ur[r] + (kk - s) * D);
                // keep the loads here, ahead of the arithmetic that follows
                asm volatile("" ::: "memory");
                __builtin_amdgcn_sched_barrier(0);
            };
            auto use = [&](const float (&buf)[kPf][kSR]) {
#pragma unroll
                for (int s = 0; s < kPf; ++s) step(pw, buf[s]);
            };
            load(ba, k);
            for (int64_t blk = 0; blk < nblk; blk += 2) {
                const bool more1 = blk + 1 < nblk, more2 = blk + 2 < nblk;
                load(bb, more1 ? k - kPf : k);  // past the last block: reload (unused)
                use(ba);
                k -= kPf;
                if (!more1) break;
                load(ba, more2 ? k - kPf : k);
                use(bb);
                k -= kPf;
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

bool blocks_for(int64_t n, int64_t per, uint32_t* g)
{
    const int64_t b = (n + per - 1) / per;
    if (b < 1 || b > 0x7fffffff) return false;
    *g = static_cast<uint32_t>(b);
    return true;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

#define LH_FFT_LENGTHS(X) X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10)

template <typename IO>
hipError_t cols_fwd(const IO* u, int64_t B, int64_t T, int64_t D, int logN1, int logN2,
                    const float2* tw, float2* Z, int64_t npair, hipStream_t stream)
{
    uint32_t gx;
    switch (logN2) {
#define LH_CASE(K)                                                                               \
    case K:                                                                                      \
        if (!blocks_for(D, Tile<K>::CW, &gx)) return hipErrorInvalidConfiguration;              \
        hipLaunchKernelGGL((fft_cols_fwd_kernel<IO, K>),                                         \
                           dim3(gx, 1u << logN1, static_cast<uint32_t>(npair)), dim3(kThreads),  \
                           0, stream, u, B, T, D, logN1, tw, Z);                                 \
        break;
        LH_FFT_LENGTHS(LH_CASE)
#undef LH_CASE
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <bool CONV>
hipError_t rows(float2* Z, const float2* H, int64_t D, int logN1, int logN2, const float2* tw,
                int64_t npair, hipStream_t stream)
{
    uint32_t gx;
    switch (logN1) {
#define LH_CASE(K)                                                                               \
    case K:                                                                                      \
        if (!blocks_for(((D + Tile<K>::CW - 1) / Tile<K>::CW << logN2) * npair, 8 * npair, &gx) \
            || int64_t(gx) * 8 * npair > 0x7fffffff)                                            \
            return hipErrorInvalidConfiguration;                                                 \
        hipLaunchKernelGGL((fft_rows_kernel<K, CONV>), dim3(gx * 8 * uint32_t(npair)),          \
                           dim3(kThreads), 0, stream, Z, H, D, logN2, npair, tw);                \
        break;
        LH_FFT_LENGTHS(LH_CASE)
#undef LH_CASE
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename IO>
hipError_t cols_inv(const float2* Z, int64_t B, int64_t T, int64_t D, int logN1, int logN2,
                    const float2* tw, IO* y, int64_t npair, hipStream_t stream)
{
    uint32_t gx;
    switch (logN2) {
#define LH_CASE(K)                                                                               \
    case K:                                                                                      \
        if (!blocks_for(D, Tile<K>::CW, &gx)) return hipErrorInvalidConfiguration;              \
        hipLaunchKernelGGL((fft_cols_inv_kernel<IO, K>),                                         \
                           dim3(gx, 1u << logN1, static_cast<uint32_t>(npair)), dim3(kThreads),  \
                           0, stream, Z, B, T, D, logN1, tw, y);                                 \
        break;
        LH_FFT_LENGTHS(LH_CASE)
#undef LH_CASE
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

#undef LH_FFT_LENGTHS

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
    if ((e = cols_fwd<float>(hh, 1, T, D, p.logN1, p.logN2, tw, H, 1, stream)) != hipSuccess)
        return e;
    if ((e = rows<false>(H, H, D, p.logN1, p.logN2, tw, 1, stream)) != hipSuccess) return e;

    // outputs
    if ((e = cols_fwd<IO>(u, B, T, D, p.logN1, p.logN2, tw, Z, p.npair, stream)) != hipSuccess)
        return e;
    if ((e = rows<true>(Z, H, D, p.logN1, p.logN2, tw, p.npair, stream)) != hipSuccess) return e;
    if ((e = cols_inv<IO>(Z, B, T, D, p.logN1, p.logN2, tw, y, p.npair, stream)) != hipSuccess)
        return e;

    // state
    const int nmc = static_cast<int>((d + kSM - 1) / kSM);
    const int nmcg = (nmc + kThreads / 64 - 1) / (kThreads / 64);
    const int64_t nrg = (B + kSR - 1) / kSR;
    if (nrg * nmcg > 0xffff || p.nparts > 0xffff) return hipErrorInvalidConfiguration;
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
    // grid z of the state contraction: batch groups x mode-chunk groups
    if ((B + kSR - 1) / kSR * ((d + 4 * kSM - 1) / (4 * kSM)) > 0xffff) return false;
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
