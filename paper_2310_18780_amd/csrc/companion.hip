// Companion (rational) form of a distilled filter (App. "From Transfer
// Function to State-Space", eq. "ssm_canon"; Lemma "efficient_recurrence";
// Proposition "fast_init").
//
// The real filter h_0 = h0, h_t = Re sum_n R_n lambda_n^(t-1) is the impulse
// response of a real system of order 2d: each pole comes with its conjugate
// and the residues are R_n / 2 and conj(R_n) / 2 (App. B.1).  In w = z^-1 its
// transfer function is h0 + beta(w) / p(w) with
//
//   p(w)    = prod_n q_n(w),   q_n(w) = 1 - 2 Re(lambda_n) w + |lambda_n|^2 w^2
//   beta(w) = sum_n w (Re R_n - Re(R_n conj(lambda_n)) w) prod_{m != n} q_m(w)
//
// (a conjugate pair of partial fractions brought over its real quadratic
// denominator, then over p), a_m and beta_m the coefficients of w^m, m =
// 1..2d.  The companion recurrence steps a real state of 2d entries:
//
//   y_t = beta . x_t + h0 u_t,   x_{t+1} = (u_t - a . x_t, x_t[0], ..., x_t[2d-2])
//
// and the fast initialisation gives the state after a prompt directly:
// x_T[j] = v_{T-1-j}, v = g * u, g the impulse response of 1 / p.
//
// Everything runs in float64.  The coefficients of p grow like binomial
// coefficients and the impulse response of 1 / p grows polynomially before
// its poles damp it, so the state becomes far larger than the outputs it
// combines: float32 loses the 1e-4 accuracy of the modal path from d = 4-8,
// float64 from d = 16 with poles near the unit circle (the paper flags the
// form as fragile there).  The modal path is the default; this form serves
// small orders.
#include "companion.hpp"

namespace lh {
namespace {

constexpr int kMaxOrd = 2 * kCompanionMaxModes;
constexpr int kThreads = 256;
constexpr int kBlk = 8;  // initialisation: steps per prefetched block
// initialisation: batch rows per thread (sharing the taps); one for the
// largest orders, whose accumulators would not fit twice in registers
__host__ __device__ constexpr int init_rows(int ord) { return ord <= 16 ? 2 : 1; }

// One 64-thread workgroup per channel; thread k owns the coefficient of w^k.
__global__ __launch_bounds__(64) void companion_coeffs_kernel(const float2* __restrict__ lam,
                                                             const float2* __restrict__ R,
                                                             int d, double* __restrict__ a,
                                                             double* __restrict__ beta)
{
    __shared__ double p[kMaxOrd + 1], q[kMaxOrd + 1], num[kMaxOrd + 1];
    const int64_t c = blockIdx.x;
    const int k = threadIdx.x;
    const int ord = 2 * d;
    const bool own = k <= ord;
    const float2* lc = lam + c * d;
    const float2* rc = R + c * d;
    // multiply the polynomial in buf by q_n (all threads take part in the barriers)
    auto times_q = [&](double* buf, int n) {
        const double lr = lc[n].x, li = lc[n].y;
        const double c1 = -2.0 * lr, c2 = lr * lr + li * li;
        double v = 0.0;
        if (own) {
            v = buf[k];
            if (k >= 1) v = fma(c1, buf[k - 1], v);
            if (k >= 2) v = fma(c2, buf[k - 2], v);
        }
        __syncthreads();
        if (own) buf[k] = v;
        __syncthreads();
    };
    if (own) {
        p[k] = k == 0 ? 1.0 : 0.0;
        num[k] = 0.0;
    }
    __syncthreads();
    for (int n = 0; n < d; ++n) times_q(p, n);
    for (int n = 0; n < d; ++n) {
        if (own) q[k] = k == 0 ? 1.0 : 0.0;
        __syncthreads();
        for (int m = 0; m < d; ++m)
            if (m != n) times_q(q, m);
        const double lr = lc[n].x, li = lc[n].y, rr = rc[n].x, ri = rc[n].y;
        const double e0 = rr, e1 = -(rr * lr + ri * li);  // Re R, -Re(R conj(lambda))
        if (own) {
            double v = num[k];
            if (k >= 1) v = fma(e0, q[k - 1], v);
            if (k >= 2) v = fma(e1, q[k - 2], v);
            num[k] = v;
        }
        __syncthreads();
    }
    if (own && k >= 1) {
        a[c * ord + k - 1] = p[k];
        beta[c * ord + k - 1] = num[k];
    }
}

// G = 2^k >= d lanes per (b, c) row, lane j holding the state pair
// (x[2j], x[2j+1]) (16 bytes: a wave moves contiguous kilobytes).  The two
// dot products are reduced over the row's lanes with DPP row permutations;
// the shift takes x[2j-1] from the lane below (DPP row shift).  Each thread serves kRows batch
// rows of one channel, so the channel's coefficient pair is loaded once for
// them; the grid is (channel tile, batch group).
constexpr int next_pow2(int x) { return x <= 1 ? 1 : 2 * next_pow2((x + 1) / 2); }
constexpr int kRows = 4;

// A float64 moved across lanes by a DPP row permutation (both 32-bit halves).
template <int CTRL>
__device__ __forceinline__ double dpp_move(double v)
{
    const unsigned long long bits = __builtin_bit_cast(unsigned long long, v);
    const int lo = __builtin_amdgcn_mov_dpp(static_cast<int>(bits & 0xffffffffu), CTRL, 0xF, 0xF,
                                            false);
    const int hi = __builtin_amdgcn_mov_dpp(static_cast<int>(bits >> 32), CTRL, 0xF, 0xF, false);
    return __builtin_bit_cast(double, static_cast<unsigned long long>(static_cast<unsigned>(lo)) |
                                         (static_cast<unsigned long long>(static_cast<unsigned>(hi))
                                          << 32));
}

// Sum over the G (a power of two <= 16) lanes of an aligned group: quad
// permutations, then the half-row and row mirrors; every lane gets the sum.
template <int G>
__device__ __forceinline__ double group_sum(double v)
{
    if constexpr (G >= 2) v += dpp_move<0xB1>(v);   // quad_perm [1,0,3,2]
    if constexpr (G >= 4) v += dpp_move<0x4E>(v);   // quad_perm [2,3,0,1]
    if constexpr (G >= 8) v += dpp_move<0x141>(v);  // row_half_mirror
    if constexpr (G >= 16) v += dpp_move<0x140>(v); // row_mirror
    return v;
}

template <typename IO, int ORD>
__global__ __launch_bounds__(kThreads) void companion_step_kernel(
    const double* __restrict__ a, const double* __restrict__ beta, const float* __restrict__ h0,
    double* __restrict__ state, const IO* __restrict__ u, IO* __restrict__ y, int64_t B,
    int64_t D)
{
    constexpr int P = ORD / 2;           // state pairs per row
    constexpr int G = next_pow2(P);      // lanes per row
    const int64_t c = int64_t(blockIdx.x) * (kThreads / G) + threadIdx.x / G;
    const int j = threadIdx.x % G;
    const int64_t b0 = int64_t(blockIdx.y) * kRows;
    // lanes past D or past the pairs compute on zeros and store nothing; no
    // exits before the shuffles
    const bool own = c < D && j < P;
    const int64_t cc = c < D ? c : D - 1;
    double2 av = make_double2(0.0, 0.0), bv = av;
    if (own) {
        av = reinterpret_cast<const double2*>(a + cc * ORD)[j];
        bv = reinterpret_cast<const double2*>(beta + cc * ORD)[j];
    }
    double2 x[kRows];
    double ut[kRows];
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int64_t b = b0 + i < B ? b0 + i : B - 1;
        const int64_t row = b * D + cc;
        x[i] = own ? reinterpret_cast<const double2*>(state + row * ORD)[j]
                   : make_double2(0.0, 0.0);
        ut[i] = io_load(u + row);
    }
    const double hz = h0[cc];
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        double out = fma(bv.x, x[i].x, bv.y * x[i].y);
        double fb = fma(av.x, x[i].x, av.y * x[i].y);
        out = group_sum<G>(out);
        fb = group_sum<G>(fb);
        const double below = dpp_move<0x111>(x[i].y);  // row_shr:1: x[2j-1] (unused at j = 0)
        const int64_t b = b0 + i;
        if (own && b < B) {
            const int64_t row = b * D + c;
            if (j == 0) io_store(y + row, static_cast<float>(fma(hz, ut[i], out)));
            reinterpret_cast<double2*>(state + row * ORD)[j] =
                make_double2(j == 0 ? ut[i] - fb : below, x[i].x);
        }
    }
}

// g_t for t < T per channel (one thread per channel): g_0 = 1,
// g_t = -sum_m a_m g_{t-m}.
template <int ORD>
__global__ __launch_bounds__(kThreads) void companion_g_kernel(const double* __restrict__ a,
                                                              int64_t D, int64_t T,
                                                              double* __restrict__ g)
{
    const int64_t c = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (c >= D) return;
    double am[ORD], w[ORD];  // w[m] = g_{t-1-m}
#pragma unroll
    for (int m = 0; m < ORD; ++m) {
        am[m] = a[c * ORD + m];
        w[m] = 0.0;
    }
    for (int64_t t = 0; t < T; ++t) {
        double acc = t == 0 ? 1.0 : 0.0;
#pragma unroll
        for (int m = 0; m < ORD; ++m) acc = fma(-am[m], w[m], acc);
        g[t * D + c] = acc;
#pragma unroll
        for (int m = ORD - 1; m > 0; --m) w[m] = w[m - 1];
        w[0] = acc;
    }
}

// state[b, c, j] = v_{T-1-j} = sum_{k <= T-1-j} g_{T-1-j-k} u_k: one thread
// per channel c and group of init_rows(2d) batch rows, which share the window of
// the 2d taps g_{T-1-j-k} sliding along k (one tap load per step for all the
// rows).
template <typename IO, int ORD>
__global__ __launch_bounds__(kThreads) void companion_init_kernel(const double* __restrict__ g,
                                                                 const IO* __restrict__ u,
                                                                 int64_t B, int64_t D, int64_t T,
                                                                 double* __restrict__ state)
{
    constexpr int NR = init_rows(ORD);
    const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    const int64_t nbg = (B + NR - 1) / NR;
    if (i >= nbg * D) return;
    const int64_t bg = i / D, c = i % D;
    const IO* ub[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int64_t b = bg * NR + r < B ? bg * NR + r : B - 1;  // loads stay in bounds
        ub[r] = u + b * T * D + c;
    }
    double win[ORD], acc[NR][ORD];
#pragma unroll
    for (int j = 0; j < ORD; ++j) {
        win[j] = T - 1 - j >= 0 ? g[(T - 1 - j) * D + c] : 0.0;
#pragma unroll
        for (int r = 0; r < NR; ++r) acc[r][j] = 0.0;
    }
    // one step k: accumulate, then slide the window (next tap g_{T-1-2d-k})
    auto step = [&](const double (&uk)[NR], double gnext) {
#pragma unroll
        for (int j = 0; j < ORD; ++j)
#pragma unroll
            for (int r = 0; r < NR; ++r) acc[r][j] = fma(win[j], uk[r], acc[r][j]);
#pragma unroll
        for (int j = 0; j < ORD - 1; ++j) win[j] = win[j + 1];
        win[ORD - 1] = gnext;
    };
    auto gtap = [&](int64_t k) { return T - 1 - ORD - k >= 0 ? g[(T - 1 - ORD - k) * D + c] : 0.0; };
    // blocks of kBlk steps, the next block's inputs loaded while the current
    // one is used (two buffers in turn), then the remaining steps
    const int64_t nblk = T / kBlk;
    double ua[kBlk][NR], ga[kBlk], ub2[kBlk][NR], gb[kBlk];
    auto load = [&](double (&uu)[kBlk][NR], double (&gg)[kBlk], int64_t k0) {
#pragma unroll
        for (int s2 = 0; s2 < kBlk; ++s2) {
#pragma unroll
            for (int r = 0; r < NR; ++r) uu[s2][r] = io_load(ub[r] + (k0 + s2) * D);
            gg[s2] = gtap(k0 + s2);
        }
        // keep the loads here, ahead of the arithmetic that follows
        asm volatile("" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
    };
    auto use = [&](const double (&uu)[kBlk][NR], const double (&gg)[kBlk]) {
#pragma unroll
        for (int s2 = 0; s2 < kBlk; ++s2) step(uu[s2], gg[s2]);
    };
    int64_t k = 0;
    if (nblk > 0) {
        load(ua, ga, 0);
        for (int64_t blk = 0; blk < nblk; blk += 2) {
            const bool more1 = blk + 1 < nblk, more2 = blk + 2 < nblk;
            load(ub2, gb, more1 ? k + kBlk : k);  // past the last block: reload (unused)
            use(ua, ga);
            k += kBlk;
            if (!more1) break;
            load(ua, ga, more2 ? k + kBlk : k);
            use(ub2, gb);
            k += kBlk;
        }
    }
    for (; k < T; ++k) {
        double uk[NR];
#pragma unroll
        for (int r = 0; r < NR; ++r) uk[r] = io_load(ub[r] + k * D);
        step(uk, gtap(k));
    }
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int64_t b = bg * NR + r;
        if (b >= B) break;
        double2* xs = reinterpret_cast<double2*>(state + (b * D + c) * ORD);
#pragma unroll
        for (int m = 0; m < ORD / 2; ++m) xs[m] = make_double2(acc[r][2 * m], acc[r][2 * m + 1]);
    }
}

__global__ __launch_bounds__(kThreads) void companion_zero_kernel(double* __restrict__ p,
                                                                 int64_t n)
{
    const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i < n) p[i] = 0.0;
}

bool blocks(int64_t n, uint32_t* g)
{
    const int64_t b = (n + kThreads - 1) / kThreads;
    if (b < 1 || b > 0x7fffffff) return false;
    *g = static_cast<uint32_t>(b);
    return true;
}

#define LH_COMPANION_ORDERS(X) \
    X(2) X(4) X(6) X(8) X(10) X(12) X(14) X(16) X(18) X(20) X(22) X(24) X(26) X(28) X(30) X(32)

template <typename IO>
hipError_t step_io(const double* a, const double* beta, const float* h0, double* state,
                   const void* u_t, void* y_t, int64_t B, int64_t D, int64_t d, hipStream_t s)
{
    const int64_t per_block = kThreads / next_pow2(static_cast<int>(d));  // channels per block
    const int64_t gx = (D + per_block - 1) / per_block;
    if (gx > 0x7fffffff) return hipErrorInvalidConfiguration;
    // batch rows in slices of at most 65535 row groups (the grid's y limit)
    constexpr int64_t kSlice = INT64_C(0xffff) * kRows;
    for (int64_t b0 = 0; b0 < B; b0 += kSlice) {
        const int64_t nb = B - b0 < kSlice ? B - b0 : kSlice;
        const dim3 g(static_cast<uint32_t>(gx), static_cast<uint32_t>((nb + kRows - 1) / kRows));
        double* st = state + b0 * D * 2 * d;
        const IO* uu = static_cast<const IO*>(u_t) + b0 * D;
        IO* yy = static_cast<IO*>(y_t) + b0 * D;
        switch (2 * d) {
#define LH_CASE(O)                                                                              \
    case O:                                                                                     \
        hipLaunchKernelGGL((companion_step_kernel<IO, O>), g, dim3(kThreads), 0, s, a, beta,    \
                           h0, st, uu, yy, nb, D);                                              \
        break;
            LH_COMPANION_ORDERS(LH_CASE)
#undef LH_CASE
            default: return hipErrorInvalidValue;
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <typename IO>
hipError_t init_io(const double* a, const void* u, int64_t B, int64_t D, int64_t d, int64_t T,
                   double* state, double* gbuf, hipStream_t s)
{
    uint32_t gc, gr;
    const int nr = init_rows(static_cast<int>(2 * d));
    if (!blocks(D, &gc) || !blocks((B + nr - 1) / nr * D, &gr)) return hipErrorInvalidConfiguration;
    hipError_t e;
    switch (2 * d) {
#define LH_CASE(O)                                                                               \
    case O:                                                                                      \
        hipLaunchKernelGGL((companion_g_kernel<O>), dim3(gc), dim3(kThreads), 0, s, a, D, T,     \
                           gbuf);                                                                \
        if ((e = hipGetLastError()) != hipSuccess) return e;                                     \
        hipLaunchKernelGGL((companion_init_kernel<IO, O>), dim3(gr), dim3(kThreads), 0, s, gbuf, \
                           static_cast<const IO*>(u), B, D, T, state);                           \
        break;
        LH_COMPANION_ORDERS(LH_CASE)
#undef LH_CASE
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

#undef LH_COMPANION_ORDERS

}  // namespace

hipError_t launch_companion_coeffs(const float2* lam, const float2* R, int64_t D, int64_t d,
                                   double* a, double* beta, hipStream_t stream)
{
    (void)hipGetLastError();
    if (D > 0x7fffffff || d < 1 || d > kCompanionMaxModes) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(companion_coeffs_kernel, dim3(static_cast<uint32_t>(D)), dim3(64), 0,
                       stream, lam, R, static_cast<int>(d), a, beta);
    return hipGetLastError();
}

hipError_t launch_companion_step(const double* a, const double* beta, const float* h0,
                                 double* state, const void* u_t, void* y_t, bool bf16_io,
                                 int64_t B, int64_t D, int64_t d, hipStream_t stream)
{
    (void)hipGetLastError();
    return bf16_io ? step_io<bf16>(a, beta, h0, state, u_t, y_t, B, D, d, stream)
                   : step_io<float>(a, beta, h0, state, u_t, y_t, B, D, d, stream);
}

hipError_t launch_companion_init(const double* a, const void* u, bool bf16_io, int64_t B,
                                 int64_t D, int64_t d, int64_t T, double* state,
                                 void* workspace, hipStream_t stream)
{
    (void)hipGetLastError();
    if (T == 0) {
        uint32_t g;
        if (!blocks(B * D * 2 * d, &g)) return hipErrorInvalidConfiguration;
        hipLaunchKernelGGL(companion_zero_kernel, dim3(g), dim3(kThreads), 0, stream, state,
                           B * D * 2 * d);
        return hipGetLastError();
    }
    double* gbuf = static_cast<double*>(workspace);
    return bf16_io ? init_io<bf16>(a, u, B, D, d, T, state, gbuf, stream)
                   : init_io<float>(a, u, B, D, d, T, state, gbuf, stream);
}

}  // namespace lh
