// Prefill of the distilled modal recurrence on the matrix cores (MFMA).
//
// The recurrence of Proposition "modal_realization" (Sec. 3.4), cut into
// chunks of C = 32 steps (the blocked form of the parallel-scan prefill of
// Sec. 3.4), is three dense contractions per channel c and chunk k, 16 batch
// rows at a time (the MFMA N dimension):
//
//   Y    = T U + W X_in            outputs of the chunk          [C x 16]
//   S    = P U                      chunk end state from zero     [2d x 16]
//   X_in <- lambda^C X_in + S       carry (complex, elementwise)  [2d x 16]
//
//   U[j][b] = u[b, kC + j, c]                        (inputs of the chunk)
//   T[t][j] = h_{t-j} for j <= t, else 0              (Toeplitz of the filter:
//             h_0 = h0, h_m = Re sum_n R_n lambda_n^(m-1), eq. "modal_impulse")
//   P[n][j] = Re / Im of lambda_n^(C-1-j)             (Vandermonde, 2d real rows)
//   W[t][n] = Re(R_n lambda_n^t) on the Re row of mode n and -Im(R_n lambda_n^t)
//             on its Im row, so that W X_in = Re sum_n R_n lambda_n^t x_in,n
//
// so that y_t = Re(R x_t) + h0 u_t at every step and the last carry is x_T.
//
// Arithmetic: v_mfma_f32_16x16x32_bf16 (float32 accumulation).  Every float32
// operand is split into three bfloat16 terms a = a1 + a2 + a3 (each the
// nearest bfloat16 of what the previous terms leave: 24 significant bits) and
// a product a b is accumulated as the six terms ai bj with i + j <= 4, which
// leaves an error of a few float32 ulps of |a b|; bfloat16 inputs are exact in
// one term, so their products take three MFMAs.  The carried state enters the
// output correction W X_in in two terms (four products; relative error near
// 2^-16 in that correction only, the carry itself stays float32).  The per-channel matrices and
// lambda^C come from float64 powers, rounded once to float32 and split by the
// setup kernel into the workspace, already in the lane order of the A operand.
//
// Work layout: a wavefront owns one channel and NBG groups of 16 batch rows
// and walks all chunks of the prompt, keeping its matrices (A operands) and
// the carried states in registers.  With the 16x16 accumulator layout (lane
// n + 16 g holds rows 4g..4g+3 of column n) and state rows ordered
// [Re modes | Im modes], the real and imaginary parts of a mode sit in the
// same lane, so the carry is lane-local, and X_in itself is the B operand of
// W X_in once W's columns are permuted to match (K index 8g + i <-> the
// lane's rows).  A workgroup is 8 waves = 8 consecutive channels.  The u tile
// of a chunk is staged through LDS (transposed to [channel][row][step]) from
// registers loaded one chunk ahead; the outputs go back through LDS so that
// every global access covers 8 channels.  Barriers order LDS only, so the
// prefetch stays in flight across them.
// Workgroups are ordered so that the 8 channel groups sharing 128-byte lines
// of u and y run on one XCD (workgroup i runs on XCD i mod 8).
//
// A last chunk shorter than C is computed with zero-padded inputs (causality
// keeps its outputs exact) and its end state by a VALU recurrence from its
// entry state over the staged inputs.
#include "lh_internal.hpp"

namespace lh {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kC = 32;     // chunk length = K of the MFMA
constexpr int kN = 16;     // batch rows per MFMA column block
constexpr int kW = 8;      // waves (channels) per workgroup
constexpr int kThreads = 64 * kW;
constexpr int kTerms = 3;  // bfloat16 terms of a split float32
constexpr int kYPad = 2;   // LDS padding (elements) of an output-stage row
constexpr int kMinWorkgroups = 256;  // automatic plan: at least one workgroup per CU

// A-operand fragments per channel: P (2d/16 tiles), T (2 tiles), W (2 tiles x d/16 K-steps)
__host__ __device__ constexpr int n_frag(int DM) { return 2 * DM + 2 + 2 * DM; }

__device__ __forceinline__ void split3(float v, __bf16& a, __bf16& b, __bf16& c)
{
    a = static_cast<__bf16>(v);
    const float r1 = v - static_cast<float>(a);
    b = static_cast<__bf16>(r1);
    const float r2 = r1 - static_cast<float>(b);
    c = static_cast<__bf16>(r2);
}

__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Workgroup barrier that orders LDS only: waits for this wave's LDS accesses
// (lgkmcnt(0); vmcnt and expcnt left at their maximum in the s_waitcnt
// encoding) and leaves global loads in flight, unlike __syncthreads(), whose
// fence also drains every outstanding global access.  The staging buffers
// live in LDS and the prefetched u rows in registers, so nothing else needs
// ordering across it.
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// ------------------------------------------------------------ setup kernel
// One workgroup per channel: float64 powers lambda_n^e (e = 0..C) and filter
// taps in LDS, then the A-operand fragments (rounded to float32, split into
// kTerms bfloat16 vectors at frag[((c * F + f) * kTerms + term) * 64 + lane])
// and lambda^C (lamc[c][g][q][i], mode 16 q + 4 g + i).
template <int DM>
__global__ __launch_bounds__(256) void mfma_setup_kernel(const float2* __restrict__ lam,
                                                         const float2* __restrict__ R,
                                                         const float* __restrict__ h0,
                                                         bf16x8* __restrict__ frag,
                                                         float2* __restrict__ lamc)
{
    constexpr int d = 16 * DM;
    constexpr int F = n_frag(DM);
    __shared__ double pwr[d][kC + 1], pwi[d][kC + 1];
    __shared__ double taps[kC];
    const int c = blockIdx.x;
    const int tid = threadIdx.x;
    const float2* lc = lam + int64_t(c) * d;
    const float2* rc = R + int64_t(c) * d;
    if (tid < d) {  // running float64 products
        const double lr = lc[tid].x, li = lc[tid].y;
        double pr = 1.0, pi = 0.0;
        for (int e = 0; e <= kC; ++e) {
            pwr[tid][e] = pr;
            pwi[tid][e] = pi;
            const double t = pr * lr - pi * li;
            pi = pr * li + pi * lr;
            pr = t;
        }
    }
    __syncthreads();
    if (tid < kC) {  // h_0 = h0, h_m = Re sum_n R_n lambda_n^(m-1)
        double h = 0.0;
        if (tid == 0) {
            h = double(h0[c]);
        } else {
            for (int n = 0; n < d; ++n)
                h += double(rc[n].x) * pwr[n][tid - 1] - double(rc[n].y) * pwi[n][tid - 1];
        }
        taps[tid] = h;
    }
    __syncthreads();
    for (int item = tid; item < F * 64 + d; item += 256) {
        if (item >= F * 64) {
            const int n = item - F * 64;
            const int q = n / 16, g = (n % 16) / 4, i = n % 4;
            lamc[(int64_t(c) * 4 + g) * (4 * DM) + q * 4 + i] =
                make_float2(float(pwr[n][kC]), float(pwi[n][kC]));
            continue;
        }
        const int f = item / 64, lane = item % 64;
        const int g = lane / 16, m = lane % 16;
        bf16x8 t0, t1, t2;
        for (int i = 0; i < 8; ++i) {
            const int k = 8 * g + i;  // K index of this element
            double val;
            if (f < 2 * DM) {  // P tile f: row r = 16 f + m, column j = k
                const int r = 16 * f + m;
                val = r < d ? pwr[r][kC - 1 - k] : pwi[r - d][kC - 1 - k];
            } else if (f < 2 * DM + 2) {  // T tile: row t, column j = k
                const int t = 16 * (f - 2 * DM) + m;
                val = k <= t ? taps[t - k] : 0.0;
            } else {  // W tile mt * DM + q: row t, K index k -> X row of mode n
                const int widx = f - 2 * DM - 2;
                const int mt = widx / DM, q = widx % DM;
                const int t = 16 * mt + m;
                const int n = 16 * q + 4 * g + (i % 4);
                const double rr = rc[n].x, ri = rc[n].y;
                val = i < 4 ? rr * pwr[n][t] - ri * pwi[n][t]      // Re(R lambda^t)
                            : -(rr * pwi[n][t] + ri * pwr[n][t]);  // -Im(R lambda^t)
            }
            __bf16 a, b, cc;
            split3(float(val), a, b, cc);
            t0[i] = a;
            t1[i] = b;
            t2[i] = cc;
        }
        bf16x8* dst = frag + (int64_t(c) * F + f) * kTerms * 64 + lane;
        dst[0] = t0;
        dst[64] = t1;
        dst[128] = t2;
    }
}

// ------------------------------------------------------------- main kernel
// LDS element type of the staged u tile: bfloat16 inputs as they are, float32
// inputs as float32 (split into terms when read as the B operand).
template <typename IO>
struct Stage;
template <>
struct Stage<bf16> {
    typedef __bf16 T;
    static constexpr int kNTU = 1;
};
template <>
struct Stage<float> {
    typedef float T;
    static constexpr int kNTU = kTerms;
};

template <typename IO, int DM, int NBG>
__global__ __launch_bounds__(kThreads) void mfma_prefill_kernel(
    const float2* __restrict__ lam, const IO* __restrict__ u, IO* __restrict__ y,
    float2* __restrict__ state, const bf16x8* __restrict__ frag,
    const float2* __restrict__ lamc, int B, int D, int64_t T, int ncg, int nbg, int nlg,
    int per_xcd)
{
    constexpr int d = 16 * DM;
    constexpr int F = n_frag(DM);
    constexpr int BN = kN * NBG;                      // batch rows per workgroup
    constexpr int NTU = Stage<IO>::kNTU;
    typedef typename Stage<IO>::T ST;
    constexpr int kRowBytes = kW * int(sizeof(IO));   // one (row, step) of 8 channels
    constexpr int kRaw = kRowBytes / 16;              // 16-byte loads per (row, step)
    constexpr int kPairs = BN * kC / 2;               // (row, step pair) items per chunk
    constexpr int kPPT = (kPairs + kThreads - 1) / kThreads;  // items per thread
    constexpr int kYRow = kC * kW + kYPad;            // IO elements per output-stage row
    __shared__ __attribute__((aligned(16))) ST ubuf[1][kW * BN * kC];
    __shared__ __attribute__((aligned(16))) IO ystage[BN * kYRow];

    // ---- workgroup -> (channel group, batch group), XCD-aware
    const int hw = blockIdx.x;
    const int lin = (hw % 8) * per_xcd + hw / 8;
    const int rest = lin / 8;
    const int cg = (rest % nlg) * 8 + lin % 8;
    const int bgw = rest / nlg;
    if (bgw >= nbg || cg >= ncg) return;  // whole workgroup exits together
    const int c0 = cg * kW;
    const int b0 = bgw * BN;

    const int tid = threadIdx.x;
    const int w = tid / 64, lane = tid % 64;
    const int g = lane / 16, n = lane % 16;
    const int c = c0 + w;  // this wave's channel (D % 8 == 0, so c < D)

    // ---- A operands and lambda^C into registers
    bf16x8 A[F][kTerms];
#pragma unroll
    for (int f = 0; f < F; ++f)
#pragma unroll
        for (int s = 0; s < kTerms; ++s)
            A[f][s] = frag[((int64_t(c) * F + f) * kTerms + s) * 64 + lane];
    float lcr[DM][4], lci[DM][4];
#pragma unroll
    for (int q = 0; q < DM; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float2 v = lamc[(int64_t(c) * 4 + g) * (4 * DM) + q * 4 + i];
            lcr[q][i] = v.x;
            lci[q][i] = v.y;
        }
    // carried states: X[bg][mt][i] = row 16 mt + 4 g + i of column n of batch
    // group bg; tiles q < DM hold Re of modes 16 q + 4 g + i, tiles DM + q Im
    f32x4 X[NBG][2 * DM];
#pragma unroll
    for (int bg = 0; bg < NBG; ++bg)
#pragma unroll
        for (int mt = 0; mt < 2 * DM; ++mt) X[bg][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int64_t nch = (T + kC - 1) / kC;

    // ---- u staging: item p (< kPairs) = row p / 16, steps 2 (p % 16) + {0, 1}
    uint4 R0[kPPT][2][kRaw];
    // Loads are unconditional, from addresses clamped into the tensor, so that
    // no control flow surrounds the destination registers and the loads stay
    // in flight until their data is staged two chunks later; rows and steps
    // outside the tensor are zeroed then.
    auto item_ok = [&](int64_t kk, int j, int h) {
        const int p = tid + j * kThreads;
        return p < kPairs && b0 + p / 16 < B && kk * kC + 2 * (p % 16) + h < T;
    };
    // per-item source of chunk 0 (rows clamped into the tensor)
    const IO* src0[kPPT];
#pragma unroll
    for (int j = 0; j < kPPT; ++j) {
        const int p = tid + j * kThreads < kPairs ? tid + j * kThreads : kPairs - 1;
        const int bb = b0 + p / 16 < B ? b0 + p / 16 : B - 1;
        src0[j] = u + (int64_t(bb) * T + 2 * (p % 16)) * D + c0;
    }
    auto load_tile = [&](int64_t kk, uint4 (&Rg)[kPPT][2][kRaw]) {
        if ((kk + 1) * kC <= T) {  // full chunk: every step in range (uniform branch)
            const int64_t off = kk * kC * D;
#pragma unroll
            for (int j = 0; j < kPPT; ++j)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const uint4* src = reinterpret_cast<const uint4*>(src0[j] + off + h * D);
#pragma unroll
                    for (int v = 0; v < kRaw; ++v) Rg[j][h][v] = src[v];
                }
        } else {  // last chunk: steps clamped to T - 1
#pragma unroll
            for (int j = 0; j < kPPT; ++j) {
                const int p = tid + j * kThreads < kPairs ? tid + j * kThreads : kPairs - 1;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int64_t t = kk * kC + 2 * (p % 16) + h;
                    const int64_t tc = (t < T ? t : T - 1) - 2 * (p % 16);
                    const uint4* src = reinterpret_cast<const uint4*>(src0[j] + tc * D);
#pragma unroll
                    for (int v = 0; v < kRaw; ++v) Rg[j][h][v] = src[v];
                }
            }
        }
    };
    auto store_tile = [&](int64_t kk, int buf, const uint4 (&Rg)[kPPT][2][kRaw]) {
#pragma unroll
        for (int j = 0; j < kPPT; ++j) {
            const int p = tid + j * kThreads;
            if (p >= kPairs) continue;
            const int rb = p / 16, sp = p % 16;
            const bool ok0 = item_ok(kk, j, 0), ok1 = item_ok(kk, j, 1);
#pragma unroll
            for (int ch = 0; ch < kW; ++ch) {
                const int e = (ch * BN + rb) * kC + 2 * sp;  // element of step 2 sp
                if constexpr (sizeof(IO) == 2) {
                    const uint32_t w0 = ok0 ? reinterpret_cast<const uint32_t*>(&Rg[j][0][0])[ch / 2] : 0u;
                    const uint32_t w1 = ok1 ? reinterpret_cast<const uint32_t*>(&Rg[j][1][0])[ch / 2] : 0u;
                    const uint32_t lo = ch % 2 == 0 ? (w0 & 0xffffu) : (w0 >> 16);
                    const uint32_t hi = ch % 2 == 0 ? (w1 & 0xffffu) : (w1 >> 16);
                    reinterpret_cast<uint32_t*>(&ubuf[buf][0])[e / 2] = lo | (hi << 16);
                } else {
                    const float v0 = ok0 ? reinterpret_cast<const float*>(&Rg[j][0][0])[ch] : 0.f;
                    const float v1 = ok1 ? reinterpret_cast<const float*>(&Rg[j][1][0])[ch] : 0.f;
                    *reinterpret_cast<float2*>(&ubuf[buf][e]) = make_float2(v0, v1);
                }
            }
        }
    };

    // U operand of batch group bg: steps 8g..8g+7 of row 16 bg + n, channel w
    auto load_u = [&](int buf, int bg, bf16x8 (&U)[NTU]) {
        const int ue = (w * BN + kN * bg + n) * kC + 8 * g;
        if constexpr (NTU == 1) {
            U[0] = *reinterpret_cast<const bf16x8*>(&ubuf[buf][ue]);
        } else {
            const float4 lo = *reinterpret_cast<const float4*>(&ubuf[buf][ue]);
            const float4 hi = *reinterpret_cast<const float4*>(&ubuf[buf][ue + 4]);
            const float uv[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                __bf16 a, b2, c2;
                split3(uv[i], a, b2, c2);
                U[0][i] = a;
                U[1][i] = b2;
                U[2][i] = c2;
            }
        }
    };
    // X_in of batch group bg as the B operand of W X_in (K index 8g + i <->
    // tile q (i < 4), tile DM + q (i >= 4)) in two bfloat16 terms: the
    // correction W X_in then carries a relative error near 2^-16 while the
    // carried state itself stays float32
    auto split_x = [&](int bg, bf16x8 (&XB)[DM][2]) {
#pragma unroll
        for (int q = 0; q < DM; ++q)
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float v = i < 4 ? X[bg][q][i] : X[bg][DM + q][i - 4];
                const __bf16 a = static_cast<__bf16>(v);
                XB[q][0][i] = a;
                XB[q][1][i] = static_cast<__bf16>(v - static_cast<float>(a));
            }
    };
    // Y = T U + W X_in of batch group bg into the output stage
    auto stage_y = [&](int bg, const f32x4 (&Y)[2]) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                io_store(&ystage[(kN * bg + n) * kYRow + (16 * mt + 4 * g + i) * kW + w], Y[mt][i]);
    };
    constexpr int kWX = 4;  // (A term, X term) pairs of W X_in: (0,0) (0,1) (1,0) (2,0)
    constexpr int kWXa[kWX] = {0, 0, 1, 2};
    constexpr int kWXx[kWX] = {0, 1, 0, 0};
    constexpr int G = NBG < 2 ? NBG : 2;  // batch groups whose MFMA chains interleave

    // full chunk: for G batch groups at a time, every product term is issued
    // for all independent accumulators (2 Y tiles and 2 DM S tiles per group)
    auto compute_full = [&](int buf) {
#pragma unroll
        for (int bp = 0; bp < NBG; bp += G) {
            bf16x8 U[G][NTU];
            bf16x8 XB[G][DM][2];
            f32x4 Y[G][2], Sr[G][DM], Si[G][DM];
#pragma unroll
            for (int gg = 0; gg < G; ++gg) {
                load_u(buf, bp + gg, U[gg]);
                split_x(bp + gg, XB[gg]);
                Y[gg][0] = Y[gg][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < DM; ++q) Sr[gg][q] = Si[gg][q] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int ia = 0; ia < kTerms; ++ia)
#pragma unroll
                for (int ju = 0; ju < NTU; ++ju) {
                    if (ia + ju >= kTerms) continue;
#pragma unroll
                    for (int gg = 0; gg < G; ++gg) {
#pragma unroll
                        for (int mt = 0; mt < 2; ++mt)
                            Y[gg][mt] = mfma(A[2 * DM + mt][ia], U[gg][ju], Y[gg][mt]);
#pragma unroll
                        for (int q = 0; q < DM; ++q) {
                            Sr[gg][q] = mfma(A[q][ia], U[gg][ju], Sr[gg][q]);
                            Si[gg][q] = mfma(A[DM + q][ia], U[gg][ju], Si[gg][q]);
                        }
                    }
                }
#pragma unroll
            for (int p = 0; p < kWX; ++p)
#pragma unroll
                for (int q = 0; q < DM; ++q)
#pragma unroll
                    for (int gg = 0; gg < G; ++gg)
#pragma unroll
                        for (int mt = 0; mt < 2; ++mt)
                            Y[gg][mt] = mfma(A[2 * DM + 2 + mt * DM + q][kWXa[p]],
                                             XB[gg][q][kWXx[p]], Y[gg][mt]);
#pragma unroll
            for (int gg = 0; gg < G; ++gg) {
                stage_y(bp + gg, Y[gg]);
#pragma unroll
                for (int q = 0; q < DM; ++q)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {  // carry: X <- lambda^C X + S
                        const float xr = X[bp + gg][q][i], xi = X[bp + gg][DM + q][i];
                        X[bp + gg][q][i] = fmaf(lcr[q][i], xr, fmaf(-lci[q][i], xi, Sr[gg][q][i]));
                        X[bp + gg][DM + q][i] = fmaf(lcr[q][i], xi, fmaf(lci[q][i], xr, Si[gg][q][i]));
                    }
            }
        }
    };

    // last, partial chunk of tr < C steps: outputs as above (the staged
    // inputs past T are zero), end state by the recurrence over its inputs
    auto compute_partial = [&](int buf, int tr) {
#pragma unroll
        for (int bg = 0; bg < NBG; ++bg) {
            bf16x8 U[NTU];
            bf16x8 XB[DM][2];
            load_u(buf, bg, U);
            split_x(bg, XB);
            f32x4 Y[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
            for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
                for (int ia = 0; ia < kTerms; ++ia)
#pragma unroll
                    for (int ju = 0; ju < NTU; ++ju)
                        if (ia + ju < kTerms) Y[mt] = mfma(A[2 * DM + mt][ia], U[ju], Y[mt]);
#pragma unroll
                for (int p = 0; p < kWX; ++p)
#pragma unroll
                    for (int q = 0; q < DM; ++q)
                        Y[mt] = mfma(A[2 * DM + 2 + mt * DM + q][kWXa[p]], XB[q][kWXx[p]], Y[mt]);
            }
            stage_y(bg, Y);
            const int ue0 = (w * BN + kN * bg + n) * kC;
#pragma unroll
            for (int q = 0; q < DM; ++q)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float2 l1 = lam[int64_t(c) * d + 16 * q + 4 * g + i];
                    float xr = X[bg][q][i], xi = X[bg][DM + q][i];
                    for (int j = 0; j < tr; ++j) {
                        const float uv = static_cast<float>(ubuf[buf][ue0 + j]);
                        const float nr = fmaf(l1.x, xr, fmaf(-l1.y, xi, uv));
                        xi = fmaf(l1.x, xi, l1.y * xr);
                        xr = nr;
                    }
                    X[bg][q][i] = xr;
                    X[bg][DM + q][i] = xi;
                }
        }
    };

    // stage -> y: item r = row r / kC, step r % kC (8 channels, 16-byte stores)
    auto write_y = [&](int64_t kk) {
        const int64_t t0 = kk * kC;
#pragma unroll
        for (int j = 0; j < (BN * kC + kThreads - 1) / kThreads; ++j) {
            const int r = tid + j * kThreads;
            const int rb = r / kC, rt = r % kC;
            const int64_t gt = t0 + rt;
            if (r < BN * kC && b0 + rb < B && gt < T) {
                const uint32_t* src = reinterpret_cast<const uint32_t*>(&ystage[rb * kYRow + rt * kW]);
                uint4* dst = reinterpret_cast<uint4*>(y + (int64_t(b0 + rb) * T + gt) * D + c0);
#pragma unroll
                for (int v = 0; v < kRaw; ++v)
                    dst[v] = make_uint4(src[4 * v], src[4 * v + 1], src[4 * v + 2], src[4 * v + 3]);
            }
        }
    };

    // One full chunk kk: compute it from the staged tile, then (after the
    // barrier) stage chunk kk + 1 from the registers it was loaded into one
    // chunk earlier, write chunk kk's outputs and issue the loads of chunk
    // kk + 2.  Loads and stores share one counter on this GPU, so the only
    // outstanding accesses when the registers are consumed are the stores and
    // loads issued a whole compute phase before.  The last, partial chunk is
    // handled after the loop, so that the loop body holds no other path.
    const int64_t nfull = T / kC;
    auto step_full = [&](int64_t kk) {
        compute_full(0);
        lds_barrier();  // tile consumed, stage complete
        if (kk + 1 < nch) store_tile(kk + 1, 0, R0);
        write_y(kk);
        if (kk + 2 < nch) load_tile(kk + 2, R0);
        lds_barrier();  // next tile staged, stage free
    };

    load_tile(0, R0);
    store_tile(0, 0, R0);
    if (nch > 1) load_tile(1, R0);
    lds_barrier();
    for (int64_t kk = 0; kk < nfull; ++kk) step_full(kk);
    if (nch > nfull) {  // chunk nfull (staged)
        compute_partial(0, int(T - nfull * kC));
        lds_barrier();
        write_y(nfull);
    }

    // ---- x_T
#pragma unroll
    for (int bg = 0; bg < NBG; ++bg) {
        const int b = b0 + kN * bg + n;
        if (b < B) {
            float2* dst = state + (int64_t(b) * D + c) * d;
#pragma unroll
            for (int q = 0; q < DM; ++q)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    dst[16 * q + 4 * g + i] = make_float2(X[bg][q][i], X[bg][DM + q][i]);
        }
    }
}

// batch groups of 16 rows per workgroup
int mfma_nbg(int64_t B, int64_t d, bool bf16_io)
{
    if (d != 16) return 1;
    const int cap = 2;  // four groups exceed the register file (the prefetch would spill)
    int nbg = 1;
    while (nbg < cap && B > 16 * nbg) nbg *= 2;
    return nbg;
}

}  // namespace

// Workspace of the MFMA plan: fragments then lambda^C.
size_t mfma_workspace_bytes(int64_t D, int64_t d)
{
    const int DM = int(d / 16);
    const size_t frag = size_t(D) * n_frag(DM) * kTerms * 64 * sizeof(bf16x8);
    const size_t lamc = size_t(D) * d * sizeof(float2);
    return (frag + 255) / 256 * 256 + lamc;
}

bool mfma_supported(int64_t B, int64_t D, int64_t d, int64_t T)
{
    return (d == 16 || d == 32) && D % kW == 0 && T >= 1 && B <= (INT64_C(1) << 30) &&
           D <= (INT64_C(1) << 30);
}

// The matrix-core plan has no parallelism along time: the automatic plan takes
// it when the (channel group, 32-row batch block) pairs alone fill the GPU.
bool mfma_preferred(int64_t B, int64_t D, int64_t d)
{
    (void)d;
    return (D / kW) * ((B + 31) / 32) >= kMinWorkgroups;
}

hipError_t launch_prefill_mfma(const float2* lam, const float2* R, const float* h0,
                               const void* u, bool bf16_io, int64_t B, int64_t D, int64_t d,
                               int64_t T, float2* state, void* y, void* workspace,
                               hipStream_t stream)
{
    (void)hipGetLastError();
    const int DM = int(d / 16);
    const size_t frag_bytes = size_t(D) * n_frag(DM) * kTerms * 64 * sizeof(bf16x8);
    bf16x8* frag = static_cast<bf16x8*>(workspace);
    float2* lamc = reinterpret_cast<float2*>(static_cast<char*>(workspace) +
                                             (frag_bytes + 255) / 256 * 256);
    const int nbgw = mfma_nbg(B, d, bf16_io);  // batch groups per workgroup
    const int ncg = int(D / kW);
    const int nbg = int((B + 16 * nbgw - 1) / (16 * nbgw));
    const int nlg = (ncg + 7) / 8;
    const int64_t groups = int64_t(nlg) * nbg;     // (line group, batch block) pairs
    const int64_t per_xcd = (groups + 7) / 8 * 8;  // logical slots per XCD
    const int64_t grid = 8 * per_xcd;
    if (D > 0x7fffffff || grid > 0x7fffffff) return hipErrorInvalidConfiguration;
    if (DM == 1)
        hipLaunchKernelGGL(mfma_setup_kernel<1>, dim3(uint32_t(D)), dim3(256), 0, stream, lam,
                           R, h0, frag, lamc);
    else
        hipLaunchKernelGGL(mfma_setup_kernel<2>, dim3(uint32_t(D)), dim3(256), 0, stream, lam,
                           R, h0, frag, lamc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
#define LH_MFMA(IO, DMV, NBGV)                                                                  \
    hipLaunchKernelGGL((mfma_prefill_kernel<IO, DMV, NBGV>), dim3(uint32_t(grid)),             \
                       dim3(kThreads), 0, stream, lam, static_cast<const IO*>(u),               \
                       static_cast<IO*>(y), state, frag, lamc, int(B), int(D), T, ncg, nbg, nlg, \
                       int(per_xcd))
    if (bf16_io) {
        if (DM == 2) LH_MFMA(bf16, 2, 1);
        else if (nbgw == 2) LH_MFMA(bf16, 1, 2);
        else LH_MFMA(bf16, 1, 1);
    } else {
        if (DM == 2) LH_MFMA(float, 2, 1);
        else if (nbgw == 2) LH_MFMA(float, 1, 2);
        else LH_MFMA(float, 1, 1);
    }
#undef LH_MFMA
    return hipGetLastError();
}

}  // namespace lh
