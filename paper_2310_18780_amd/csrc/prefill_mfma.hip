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
// Arithmetic: v_mfma_f32_16x16x32_bf16 (float32 accumulation).  A float32
// operand is split into bfloat16 terms a = a1 + a2 (+ a3), each the nearest
// bfloat16 of what the previous terms leave, and a product a b is accumulated
// as the terms ai bj with i + j below the term count.  With float32 inputs
// every operand takes three terms (24 significant bits; six products, an
// error of a few float32 ulps of |a b|).  Bfloat16 inputs are exact in one
// term and their outputs are rounded to bfloat16, so the matrices take two
// terms (relative error near 2^-17, far below the output rounding and the
// float32 state tolerance) and each product two MFMAs.  The carried state
// enters the output correction W X_in in two terms (relative error near 2^-16
// in that correction only; the carry itself stays float32).  The per-channel
// matrices and lambda^C come from float64 powers, rounded once to float32 and
// split by the setup kernel into the workspace, already in the lane order of
// the A operand.
//
// d = 64 (float32 u/y only) takes the same three-term operands: 18 A
// fragments per channel (216 registers per lane), which with the states and
// accumulators need more than the 256 registers of two waves per SIMD, so its
// workgroups have 4 waves (one per SIMD, up to 512 registers: the compiler
// keeps the accumulators in the accumulation registers), one channel and 16
// rows each.
//
// Work layout: a wavefront owns CPW channels (2 for bfloat16 inputs with
// d = 16, else 1) and NBG groups of 16 batch rows (2 for float32 inputs with
// d = 16 and more than 16 rows, else 1), and walks all chunks of the
// prompt, keeping its matrices (A operands) and the carried states in
// registers.  With the 16x16 accumulator layout (lane n + 16 g holds rows
// 4g..4g+3 of column n) and state rows ordered [Re modes | Im modes], the
// real and imaginary parts of a mode sit in the same lane, so the carry is
// lane-local, and X_in itself is the B operand of W X_in once W's columns are
// permuted to match (K index 8g + i <-> the lane's rows).  A workgroup is 8
// waves = 8 CPW consecutive channels (4 waves and channels at d = 64).  The u tile of a chunk is staged
// through LDS (transposed to [channel][row][step]) from registers loaded one
// or two chunks ahead (pf_of); the outputs go back through LDS so that every
// global access is a 16-byte piece of a whole (row, step) segment of the
// workgroup's channels.  Barriers order LDS only, so the prefetch stays in
// flight across them.
// Workgroups are ordered so that each XCD (workgroup i runs on XCD i mod 8)
// owns a contiguous range of channel groups for all batch groups: its L2
// fetches those channels' A operands once, and the channel groups sharing
// 128-byte lines of u and y run on one XCD.
//
// A last chunk shorter than C is computed with zero-padded inputs (causality
// keeps its outputs exact) and its end state by a VALU recurrence from its
// entry state over the staged inputs.
#include "lh_internal.hpp"

namespace lh {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kC = 32;     // chunk length = K of the MFMA
constexpr int kN = 16;     // batch rows per MFMA column block
constexpr int kTerms = 3;  // bfloat16 terms of a split float32
constexpr int kMinWorkgroups = 256;  // automatic plan: at least one workgroup per CU

// A-operand fragments per channel: P (2d/16 tiles), T (2 tiles), W (2 tiles x d/16 K-steps)
__host__ __device__ constexpr int n_frag(int DM) { return 2 * DM + 2 + 2 * DM; }

size_t frag_bytes_of(int64_t D, int DM)
{
    return size_t(D) * n_frag(DM) * kTerms * 64 * sizeof(bf16x8);
}

__device__ __forceinline__ void split3(float v, __bf16& a, __bf16& b, __bf16& c)
{
    a = static_cast<__bf16>(v);
    const float r1 = v - static_cast<float>(a);
    b = static_cast<__bf16>(r1);
    const float r2 = r1 - static_cast<float>(b);
    c = static_cast<__bf16>(r2);
}

// nearest bfloat16 values of a pair (one packed conversion), and the
// bfloat16 residuals of the pair after them
__device__ __forceinline__ bf16x2 to_bf16x2(float a, float b)
{
    return __builtin_convertvector(f32x2{a, b}, bf16x2);
}

__device__ __forceinline__ bf16x2 residual_bf16x2(float a, float b, bf16x2 h)
{
    const f32x2 back = __builtin_convertvector(h, f32x2);
    return to_bf16x2(a - back.x, b - back.y);
}

__device__ __forceinline__ bf16x8 concat4(bf16x2 a, bf16x2 b, bf16x2 c, bf16x2 d)
{
    return __builtin_shufflevector(__builtin_shufflevector(a, b, 0, 1, 2, 3),
                                   __builtin_shufflevector(c, d, 0, 1, 2, 3), 0, 1, 2, 3, 4, 5, 6, 7);
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
// kTerms bfloat16 vectors at frag[((c * F + f) * kTerms + term) * 64 + lane];
// the T and W fragments get only their first tw_terms terms, the ones the
// main kernel reads) and lambda^C (lamc[c][g][q][i], mode 16 q + 4 g + i).
template <int DM>
__global__ __launch_bounds__(256) void mfma_setup_kernel(const float2* __restrict__ lam,
                                                         const float2* __restrict__ R,
                                                         const float* __restrict__ h0,
                                                         bf16x8* __restrict__ frag,
                                                         float2* __restrict__ lamc, int tw_terms)
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
        if (f < 2 * DM || tw_terms > 2) dst[128] = t2;
    }
}

// ------------------------------------------------------------- main kernel
// Tiling per (IO, DM): a wave owns CPW channels and NBG groups of 16 batch
// rows; a workgroup of 8 waves owns CW = 8 CPW consecutive channels, so that
// one (row, step) of its inputs or outputs is a CW-channel segment of a
// 128-byte line.  Lines of u and y are shared by the workgroups of
// neighbouring channel groups, and the data movement, not the arithmetic,
// bounds the kernel: two channels per wave (32-byte segments for bfloat16)
// cut it by about a sixth against one (16-byte segments); 32 channels per
// workgroup, measured with the arithmetic left out, move the data no faster
// than 16 (and their A operands would not fit the registers).
template <typename IO, int DM>
struct Tiling;
template <>
struct Tiling<bf16, 1> {
    static constexpr int CPW = 2;
};
template <>
struct Tiling<bf16, 2> {
    static constexpr int CPW = 1;
};
template <>
struct Tiling<float, 1> {
    static constexpr int CPW = 1;
};
template <>
struct Tiling<float, 2> {
    static constexpr int CPW = 1;
};
template <>
struct Tiling<float, 4> {
    static constexpr int CPW = 1;
};
// Waves per workgroup: 8 (two per SIMD); 4 at d = 64, whose 216 A-operand
// registers per lane and channel need most of a SIMD's register file (one
// wave each, up to 512 registers).
__host__ __device__ constexpr int waves_of(int DM) { return DM == 4 ? 4 : 8; }

// LDS element type of the staged u tile and operand term counts: bfloat16
// inputs are exact in one term and their outputs are rounded to bfloat16, so
// the output operands T and W take two terms (relative error near 2^-17,
// invisible after the rounding), while the state operand P keeps three
// (24 significant bits: the chunk end states, and through the carry x_T, are
// formed at float32 precision); float32 inputs and every A operand take
// three terms.
template <typename IO>
struct Stage;
template <>
struct Stage<bf16> {
    typedef __bf16 T;
    static constexpr int kNTU = 1;
    static constexpr int kNTA = 2;  // T, W
    static constexpr int kNTP = 3;  // P
};
template <>
struct Stage<float> {
    typedef float T;
    static constexpr int kNTU = kTerms;
    static constexpr int kNTA = kTerms;
    static constexpr int kNTP = kTerms;
};

// MODE selects what a column of the MFMA tiles is:
//   kWhole    : a batch row over the whole prompt, from x = 0; writes y and x_T;
//   kSegState : a (batch row b, segment k < nseg - 1) pair over the seg_len steps
//               of segment k, from x = 0; writes only its end state s_k to
//               xs[b][k] (no outputs);
//   kSegOut   : a (b, k < nseg) pair from the entry state xs[b][k] (the carry
//               of the earlier segments); writes y over the segment, and x_T
//               for the last segment.
// Segmented launches need seg_len % C == 0 and T == nseg seg_len.
enum { kWhole = 0, kSegState = 1, kSegOut = 2 };

// Channels per wave: the state-only pass holds only the P operands (a third
// of the A registers), so its waves take more channels and read wider pieces
// of each line of u.
template <typename IO, int DM, int MODE>
constexpr int cpw_of()
{
    return MODE == kSegState && DM < 4 ? (sizeof(IO) == 2 && DM == 1 ? 4 : 2) : Tiling<IO, DM>::CPW;
}

// Chunk tiles of u in flight while a chunk is computed (in registers, one
// per tile): two where the registers allow it without spilling (all but the
// state-only pass and the float32 d = 32 whole-prompt kernel), except at
// d = 64, where a second tile gained 1%.  There are
// only two waves per SIMD, both of one workgroup and meeting at its barrier
// every chunk, so with one tile in flight each chunk waits out most of a
// memory latency; a second tile hides it.
template <typename IO, int DM, int MODE>
constexpr int pf_of()
{
    return MODE == kSegState || DM == 4 || (sizeof(IO) == 4 && DM == 2 && MODE == kWhole) ? 1 : 2;
}

template <typename IO, int DM, int NBG, int MODE>
__global__ __launch_bounds__(64 * waves_of(DM)) void mfma_prefill_kernel(
    const float2* __restrict__ lam, const IO* __restrict__ u, IO* __restrict__ y,
    float2* __restrict__ state, const bf16x8* __restrict__ frag,
    const float2* __restrict__ lamc, int B, int D, int64_t T, int ncg, int nbg, int per_xcd,
    int nseg, int64_t seg_len, float2* __restrict__ xs)
{
    constexpr int d = 16 * DM;
    static_assert(DM < 4 || sizeof(IO) == 4, "d = 64 takes float32 u and y");
    constexpr int F = n_frag(DM);
    constexpr int CPW = cpw_of<IO, DM, MODE>();
    constexpr int NW = waves_of(DM);
    constexpr int NT = 64 * NW;                       // threads
    constexpr int CW = NW * CPW;
    constexpr int BN = kN * NBG;                      // batch rows per workgroup
    constexpr int NTU = Stage<IO>::kNTU;
    constexpr int KT = Stage<IO>::kNTA;               // terms of T and W
    constexpr int KTP = Stage<IO>::kNTP;              // terms of P
    constexpr int KTX = KTP > KT ? KTP : KT;
    typedef typename Stage<IO>::T ST;
    constexpr int ES = int(sizeof(IO));
    constexpr int CPP = 16 / ES;                      // channels per 16-byte piece
    constexpr int PPR = CW / CPP;                     // pieces per (row, step)
    constexpr int NITEM = BN * (kC / 2) * PPR;        // (row, step pair, piece) items
    constexpr int IPT = (NITEM + NT - 1) / NT;  // items per thread
    constexpr int US = kC + 16 / int(sizeof(ST));     // u stage: steps per (channel, row), padded
    // y stage in 32-bit words: (row, step) cells of SD words, rows padded to
    // 4 words past a multiple of 32 and the words of each 16-byte piece
    // permuted by (step >> 2) & 3 (see ysw), so that a wave's stores (16 rows x
    // 4 lane groups, one word each) fall on every LDS bank exactly twice
    constexpr int SD = CW * ES / 4;                   // words per (row, step)
    constexpr int RS = kC * SD + 4;                   // words per row
    constexpr int NYP = BN * kC * PPR;                // 16-byte output pieces per chunk
    // u and y stages: one of each with one tile in flight; with two, two of
    // each, so that a chunk's compute and the staging of its neighbours use
    // different buffers and one barrier per chunk orders them
    constexpr int PF = pf_of<IO, DM, MODE>();
    __shared__ __attribute__((aligned(16))) ST ubuf[PF][CW * BN * US];
    __shared__ __attribute__((aligned(16))) uint32_t ystage[PF][MODE == kSegState ? 1 : BN * RS];
    __shared__ __attribute__((aligned(16))) float2 lcs[CW][4][4 * DM];  // lambda^C per channel, lane group

    // ---- workgroup -> (channel group, batch group).  The CPL channel groups
    // whose pieces make up one 128-byte line of u and y form a line group;
    // logical index lin = (line group * nbg + batch group) * CPL + j, channel
    // group = line group * CPL + j, runs on XCD lin / per_xcd (workgroup i
    // runs on XCD i mod 8).  Each XCD thus owns a contiguous range of line
    // groups for every batch group (its L2 fetches those channels' A operands
    // once), and the workgroups resident together cover whole lines.
    constexpr int CPL = 128 / (CW * ES) > 1 ? 128 / (CW * ES) : 1;
    const int hw = blockIdx.x;
    const int lin = (hw % 8) * per_xcd + hw / 8;
    const int rest = lin / CPL;
    const int lg = rest / nbg;
    const int bgw = rest - lg * nbg;
    const int cg = lg * CPL + (lin - rest * CPL);
    if (cg >= ncg) return;  // whole workgroup exits together
    const int c0 = cg * CW;
    const int b0 = bgw * BN;
    // columns ("rows" below): batch rows, or (batch row, segment) pairs
    // r = b * SV + k, each covering TL steps from time TB(r)
    const int SV = MODE == kWhole ? 1 : MODE == kSegState ? nseg - 1 : nseg;
    const int BV = B * SV;
    const int64_t TL = MODE == kWhole ? T : seg_len;
    auto row_b = [&](int r) { return r / SV; };
    auto row_k = [&](int r) { return r % SV; };

    const int tid = threadIdx.x;
    const int w = tid / 64, lane = tid % 64;
    const int g = lane / 16, n = lane % 16;

    // ---- A operands and lambda^C of this wave's channels (clamped into range;
    // results of channels >= D are never stored)
    bf16x8 A[CPW][F][KTX];
#pragma unroll
    for (int k = 0; k < CPW; ++k) {
        const int cc = min(c0 + w * CPW + k, D - 1);
#pragma unroll
        for (int f = 0; f < F; ++f)
#pragma unroll
            for (int s = 0; s < (f < 2 * DM ? KTP : KT); ++s)
                A[k][f][s] = frag[((int64_t(cc) * F + f) * kTerms + s) * 64 + lane];
        if (n < 4 * DM)  // lambda^C of the modes of lane group g (read back by the carry)
            lcs[w * CPW + k][g][n] = lamc[(int64_t(cc) * 4 + g) * (4 * DM) + n];
    }
    // carried states: X[k][bg][mt][i] = row 16 mt + 4 g + i of column n of
    // batch group bg; tiles q < DM hold Re of modes 16 q + 4 g + i, tiles
    // DM + q their Im
    f32x4 X[CPW][NBG][2 * DM];
#pragma unroll
    for (int k = 0; k < CPW; ++k)
#pragma unroll
        for (int bg = 0; bg < NBG; ++bg) {
#pragma unroll
            for (int mt = 0; mt < 2 * DM; ++mt) X[k][bg][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
            if constexpr (MODE == kSegOut) {  // entry state of the segment
                const int r = min(b0 + kN * bg + n, BV - 1);
                const int cc = min(c0 + w * CPW + k, D - 1);
                const float2* src =
                    xs + ((int64_t(row_b(r)) * nseg + row_k(r)) * D + cc) * d;
#pragma unroll
                for (int q = 0; q < DM; ++q)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float2 v = src[16 * q + 4 * g + i];
                        X[k][bg][q][i] = v.x;
                        X[k][bg][DM + q][i] = v.y;
                    }
            }
        }

    const int64_t nch = (TL + kC - 1) / kC;

    // ---- u staging: item p = tid + j NT holds (row p / (16 PPR), steps
    // 2 ((p / PPR) % 16) + {0, 1}, channels c0 + CPP (p % PPR) ..).  Loads are
    // unconditional, from addresses clamped into the tensor, so that no
    // control flow surrounds the destination registers; rows, steps and
    // channels outside the tensor are zeroed when the tile is staged.
    auto item_of = [&](int j, int& ip, int& itp, int& irb) {
        const int p = min(tid + j * NT, NITEM - 1);
        ip = p % PPR;
        itp = (p / PPR) % (kC / 2);
        irb = p / (PPR * (kC / 2));
    };
    const IO* src0[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        int ip, itp, irb;
        item_of(j, ip, itp, irb);
        const int r = min(b0 + irb, BV - 1);
        src0[j] = u + (int64_t(row_b(r)) * T + int64_t(row_k(r)) * TL + 2 * itp) * D +
                  min(c0 + ip * CPP, D - CPP);
    }
    uint4 RT[PF][IPT][2];  // u tiles in flight
    auto load_tile = [&](int64_t kk, auto& R0) {
        if ((kk + 1) * kC <= TL) {  // full chunk (uniform branch)
            const int64_t off = kk * kC * D;
#pragma unroll
            for (int j = 0; j < IPT; ++j)
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    R0[j][h] = *reinterpret_cast<const uint4*>(src0[j] + off + h * D);
        } else {  // last chunk: steps clamped to T - 1
#pragma unroll
            for (int j = 0; j < IPT; ++j) {
                int ip, itp, irb;
                item_of(j, ip, itp, irb);
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int64_t t = kk * kC + 2 * itp + h;
                    const int64_t tc = (t < TL ? t : TL - 1) - 2 * itp;
                    R0[j][h] = *reinterpret_cast<const uint4*>(src0[j] + tc * D);
                }
            }
        }
    };
    auto store_tile = [&](int64_t kk, const auto& R0, ST* ub) {
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            if (tid + j * NT >= NITEM) continue;
            int ip, itp, irb;
            item_of(j, ip, itp, irb);
            const bool in = b0 + irb < BV && c0 + ip * CPP < D;
            const bool ok0 = in && kk * kC + 2 * itp < TL;
            const bool ok1 = in && kk * kC + 2 * itp + 1 < TL;
            const uint4 z = make_uint4(0u, 0u, 0u, 0u);
            const uint4 s0 = ok0 ? R0[j][0] : z, s1 = ok1 ? R0[j][1] : z;
#pragma unroll
            for (int ch = 0; ch < CPP; ++ch) {
                const int e = ((ip * CPP + ch) * BN + irb) * US + 2 * itp;  // element of step 2 itp
                if constexpr (ES == 2) {  // (step 2 itp, step 2 itp + 1) of channel ch
                    const uint32_t w0 = reinterpret_cast<const uint32_t*>(&s0)[ch / 2];
                    const uint32_t w1 = reinterpret_cast<const uint32_t*>(&s1)[ch / 2];
                    reinterpret_cast<uint32_t*>(ub)[e / 2] =
                        ch % 2 == 0 ? (w0 & 0xffffu) | (w1 << 16) : (w0 >> 16) | (w1 & 0xffff0000u);
                } else {
                    const float v0 = reinterpret_cast<const float*>(&s0)[ch];
                    const float v1 = reinterpret_cast<const float*>(&s1)[ch];
                    *reinterpret_cast<float2*>(&ub[e]) = make_float2(v0, v1);
                }
            }
        }
    };

    // U operand of channel k, batch group bg: steps 8g..8g+7 of row 16 bg + n
    auto load_u = [&](int k, int bg, bf16x8 (&U)[NTU], const ST* ub) {
        const int ue = ((w * CPW + k) * BN + kN * bg + n) * US + 8 * g;
        if constexpr (NTU == 1) {
            U[0] = *reinterpret_cast<const bf16x8*>(&ub[ue]);
        } else {
            const float4 lo = *reinterpret_cast<const float4*>(&ub[ue]);
            const float4 hi = *reinterpret_cast<const float4*>(&ub[ue + 4]);
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
    // X_in as the B operand of W X_in (K index 8g + i <-> tile q (i < 4),
    // tile DM + q (i >= 4)) in two bfloat16 terms: the correction W X_in then
    // carries a relative error near 2^-16 while the carried state itself
    // stays float32
    auto split_x = [&](const f32x4 (&Xs)[2 * DM], bf16x8 (&XB)[DM][2]) {
#pragma unroll
        for (int q = 0; q < DM; ++q) {
            const f32x4 re = Xs[q], im = Xs[DM + q];
            const bf16x2 h0 = to_bf16x2(re[0], re[1]), h1 = to_bf16x2(re[2], re[3]);
            const bf16x2 h2 = to_bf16x2(im[0], im[1]), h3 = to_bf16x2(im[2], im[3]);
            XB[q][0] = concat4(h0, h1, h2, h3);
            XB[q][1] = concat4(residual_bf16x2(re[0], re[1], h0), residual_bf16x2(re[2], re[3], h1),
                               residual_bf16x2(im[0], im[1], h2), residual_bf16x2(im[2], im[3], h3));
        }
    };
    // word of the y stage holding word dw (< SD) of (row, step)
    auto ysw = [&](int row, int step, int dw) { return row * RS + step * SD + (dw ^ ((step >> 2) & 3)); };
    // Y (row 16 bg + n, steps 16 mt + 4 g + i) of this wave's CPW channels
    // into the output stage, adjacent bfloat16 channels packed into one word
    auto stage_y = [&](int bg, const f32x4 (&Y)[CPW][2], uint32_t* ys) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = kN * bg + n, step = 16 * mt + 4 * g + i;
                if constexpr (ES == 2 && CPW == 2) {  // channel 0 in the low half
                    ys[ysw(row, step, w)] =
                        __builtin_bit_cast(uint32_t, to_bf16x2(Y[0][mt][i], Y[1][mt][i]));
                } else if constexpr (ES == 2) {  // one bfloat16 channel: half word w % 2 of word w / 2
                    io_store(reinterpret_cast<IO*>(ys) + 2 * ysw(row, step, w / 2) + w % 2,
                             Y[0][mt][i]);
                } else {
                    reinterpret_cast<float*>(ys)[ysw(row, step, w)] = Y[0][mt][i];
                }
            }
    };
    // (A term, X term) pairs of W X_in: (0,0) (0,1) (1,0), and (2,0) with
    // three-term A operands
    constexpr int kWX = KT == 2 ? 3 : 4;
    constexpr int kWXa[4] = {0, 0, 1, 2};
    constexpr int kWXx[4] = {0, 1, 0, 0};

    // full chunk, one batch group at a time: every product term is issued
    // for all independent accumulators of the wave's channels (2 Y tiles and
    // 2 DM S tiles per channel), then the carry and the output stage
    auto compute_full = [&](const ST* ub, uint32_t* ys) {
#pragma unroll
        for (int bg = 0; bg < NBG; ++bg) {
            bf16x8 U[CPW][NTU];
            bf16x8 XB[CPW][DM][2];
            f32x4 Y[CPW][2], Sr[CPW][DM], Si[CPW][DM];
#pragma unroll
            for (int k = 0; k < CPW; ++k) {
                load_u(k, bg, U[k], ub);
                if constexpr (MODE != kSegState) split_x(X[k][bg], XB[k]);
                Y[k][0] = Y[k][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < DM; ++q) Sr[k][q] = Si[k][q] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int ia = 0; ia < KTX; ++ia)
#pragma unroll
                for (int ju = 0; ju < NTU; ++ju) {
#pragma unroll
                    for (int k = 0; k < CPW; ++k) {
                        if constexpr (MODE != kSegState) {
                            if (ia + ju < KT) {
#pragma unroll
                                for (int mt = 0; mt < 2; ++mt)
                                    Y[k][mt] = mfma(A[k][2 * DM + mt][ia], U[k][ju], Y[k][mt]);
                            }
                        }
                        if (ia + ju < KTP) {
#pragma unroll
                            for (int q = 0; q < DM; ++q) {
                                Sr[k][q] = mfma(A[k][q][ia], U[k][ju], Sr[k][q]);
                                Si[k][q] = mfma(A[k][DM + q][ia], U[k][ju], Si[k][q]);
                            }
                        }
                    }
                }
            if constexpr (MODE != kSegState) {
#pragma unroll
                for (int p = 0; p < kWX; ++p)
#pragma unroll
                    for (int q = 0; q < DM; ++q)
#pragma unroll
                        for (int k = 0; k < CPW; ++k)
#pragma unroll
                            for (int mt = 0; mt < 2; ++mt)
                                Y[k][mt] = mfma(A[k][2 * DM + 2 + mt * DM + q][kWXa[p]],
                                                XB[k][q][kWXx[p]], Y[k][mt]);
            }
#pragma unroll
            for (int k = 0; k < CPW; ++k)
#pragma unroll
                for (int q = 0; q < DM; ++q)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {  // carry: X <- lambda^C X + S
                        const float2 l = lcs[w * CPW + k][g][4 * q + i];
                        const float xr = X[k][bg][q][i], xi = X[k][bg][DM + q][i];
                        X[k][bg][q][i] = fmaf(l.x, xr, fmaf(-l.y, xi, Sr[k][q][i]));
                        X[k][bg][DM + q][i] = fmaf(l.x, xi, fmaf(l.y, xr, Si[k][q][i]));
                    }
            if constexpr (MODE != kSegState) stage_y(bg, Y, ys);
        }
    };

    // last, partial chunk of tr < C steps: outputs as above (the staged
    // inputs past T are zero), end state by the recurrence over its inputs
    auto compute_partial = [&](int tr, const ST* ub, uint32_t* ys) {
#pragma unroll
        for (int bg = 0; bg < NBG; ++bg) {
            f32x4 Y[CPW][2];
#pragma unroll
            for (int k = 0; k < CPW; ++k) {
                bf16x8 U[NTU];
                bf16x8 XB[DM][2];
                load_u(k, bg, U, ub);
                split_x(X[k][bg], XB);
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) {
                    Y[k][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ia = 0; ia < KT; ++ia)
#pragma unroll
                        for (int ju = 0; ju < NTU; ++ju)
                            if (ia + ju < KT) Y[k][mt] = mfma(A[k][2 * DM + mt][ia], U[ju], Y[k][mt]);
#pragma unroll
                    for (int p = 0; p < kWX; ++p)
#pragma unroll
                        for (int q = 0; q < DM; ++q)
                            Y[k][mt] = mfma(A[k][2 * DM + 2 + mt * DM + q][kWXa[p]],
                                            XB[q][kWXx[p]], Y[k][mt]);
                }
            }
            stage_y(bg, Y, ys);
        }
#pragma unroll
        for (int k = 0; k < CPW; ++k) {
            const int cc = min(c0 + w * CPW + k, D - 1);
#pragma unroll
            for (int bg = 0; bg < NBG; ++bg) {
                const int ue0 = ((w * CPW + k) * BN + kN * bg + n) * US;
#pragma unroll
                for (int q = 0; q < DM; ++q)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float2 l1 = lam[int64_t(cc) * d + 16 * q + 4 * g + i];
                        float xr = X[k][bg][q][i], xi = X[k][bg][DM + q][i];
                        for (int j = 0; j < tr; ++j) {
                            const float uv = static_cast<float>(ub[ue0 + j]);
                            const float nr = fmaf(l1.x, xr, fmaf(-l1.y, xi, uv));
                            xi = fmaf(l1.x, xi, l1.y * xr);
                            xr = nr;
                        }
                        X[k][bg][q][i] = xr;
                        X[k][bg][DM + q][i] = xi;
                    }
            }
        }
    };

    // stage -> y: piece r = row r / (kC PPR), step (r / PPR) % kC, channels
    // c0 + CPP (r % PPR) ..
    auto write_y = [&](int64_t kk, const uint32_t* ys) {
        const int64_t t0 = kk * kC;
#pragma unroll
        for (int j = 0; j < (NYP + NT - 1) / NT; ++j) {
            const int r = tid + j * NT;
            const int rp = r % PPR, rt = (r / PPR) % kC, rb = r / (PPR * kC);
            const int64_t gt = t0 + rt;
            if (r < NYP && b0 + rb < BV && gt < TL && c0 + rp * CPP < D) {
                uint4 v = *reinterpret_cast<const uint4*>(&ys[rb * RS + rt * SD + 4 * rp]);
                const int f = (rt >> 2) & 3;  // undo the word permutation of the piece
                if (f & 1) v = make_uint4(v.y, v.x, v.w, v.z);
                if (f & 2) v = make_uint4(v.z, v.w, v.x, v.y);
                const int rv = b0 + rb;
                *reinterpret_cast<uint4*>(y + (int64_t(row_b(rv)) * T + int64_t(row_k(rv)) * TL + gt) * D +
                                          c0 + rp * CPP) = v;
            }
        }
    };

    // One tile in flight (PF = 1): compute chunk kk from the staged tile,
    // then (after a barrier) stage chunk kk + 1 from the registers it was
    // loaded into one chunk earlier, write chunk kk's outputs and issue the
    // loads of chunk kk + 2; a second barrier frees the stages.  Loads and
    // stores share one counter on this GPU, so the only outstanding accesses
    // when the registers are consumed are the stores and loads issued a whole
    // compute phase before.
    //
    // PF >= 2 tiles in flight: chunk kk is computed from u stage kk % PF into
    // y stage kk % PF while chunk kk + 1 goes from its register tile into the
    // next u stage and chunk kk - 1's outputs leave the previous y stage, so
    // one barrier per chunk orders everything and the waves of a workgroup
    // drift apart within it.  Tile t lives in register slot t % PF (the loop
    // is unrolled by PF so that slots and stages have fixed registers and
    // addresses); the slot that frees up takes the loads of chunk kk + 1 + PF.
    // These loads are issued on every path (past the end at the last chunks
    // again) so that the number of accesses issued after each tile is the same
    // on all paths and the wait for one tile leaves the others in flight.
    //
    // The last, partial chunk is handled after the loop, so that the loop
    // body holds no other path.
    const int64_t nfull = TL / kC;
    if constexpr (PF == 1) {
        load_tile(0, RT[0]);
        store_tile(0, RT[0], ubuf[0]);
        if (nch > 1) load_tile(1, RT[0]);
        lds_barrier();
        for (int64_t kk = 0; kk < nfull; ++kk) {
            compute_full(ubuf[0], ystage[0]);
            lds_barrier();  // tile consumed, stage complete
            if (kk + 1 < nch) store_tile(kk + 1, RT[0], ubuf[0]);
            if constexpr (MODE != kSegState) write_y(kk, ystage[0]);
            if (kk + 2 < nch) load_tile(kk + 2, RT[0]);
            lds_barrier();  // next tile staged, stage free
        }
    } else {
        // tile t lives in register slot t % PF; chunk kk uses stage kk % PF
#pragma unroll
        for (int q = 0; q < PF; ++q) load_tile(min(int64_t(q), nch - 1), RT[q]);
        store_tile(0, RT[0], ubuf[0]);
        load_tile(min(int64_t(PF), nch - 1), RT[0]);
        lds_barrier();
        for (int64_t kk = 0; kk < nfull; kk += PF) {
#pragma unroll
            for (int p = 0; p < PF; ++p) {
                const int64_t c = kk + p;  // this phase's chunk
                if (p > 0 && c >= nfull) break;
                const int q = (p + 1) % PF;
                compute_full(ubuf[p], ystage[p]);
                if (c + 1 < nch) store_tile(c + 1, RT[q], ubuf[q]);
                load_tile(min(c + 1 + PF, nch - 1), RT[q]);  // slot q is free again
                if constexpr (MODE != kSegState)
                    if (c > 0) write_y(c - 1, ystage[(p + PF - 1) % PF]);
                lds_barrier();
            }
        }
        if constexpr (MODE != kSegState)
            if (nfull > 0) write_y(nfull - 1, ystage[(nfull - 1) % PF]);
    }
    if constexpr (MODE == kWhole) {
        if (nch > nfull) {  // chunk nfull (staged); segmented launches have none
            compute_partial(int(T - nfull * kC), ubuf[nfull % PF], ystage[nfull % PF]);
            lds_barrier();
            write_y(nfull, ystage[nfull % PF]);
        }
    }

    // ---- x_T
#pragma unroll
    for (int k = 0; k < CPW; ++k) {
        const int c = c0 + w * CPW + k;
#pragma unroll
        for (int bg = 0; bg < NBG; ++bg) {
            const int r = b0 + kN * bg + n;
            if (r < BV && c < D && (MODE != kSegOut || row_k(r) == SV - 1)) {
                // x_T, or the end state s_k of segment k (from zero) in its slot
                float2* dst = MODE == kSegState
                                  ? xs + ((int64_t(row_b(r)) * nseg + row_k(r)) * D + c) * d
                                  : state + (int64_t(row_b(r)) * D + c) * d;
#pragma unroll
                for (int q = 0; q < DM; ++q)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        dst[16 * q + 4 * g + i] = make_float2(X[k][bg][q][i], X[k][bg][DM + q][i]);
            }
        }
    }
}

// batch groups of 16 rows per wave: two when there are more than 16 rows and
// the registers allow (float32 inputs with d = 16, one channel per wave)
int mfma_nbg(int64_t B, int64_t d, bool bf16_io)
{
    return d == 16 && !bf16_io && B > kN ? 2 : 1;
}

template <typename IO, int DM, int NBG, int MODE>
hipError_t launch_main(const float2* lam, const void* u, void* y, float2* state,
                       const bf16x8* frag, const float2* lamc, int64_t B, int64_t D, int64_t T,
                       int nseg, int64_t seg_len, float2* xs, hipStream_t stream)
{
    constexpr int CW = waves_of(DM) * cpw_of<IO, DM, MODE>();
    constexpr int CPL = 128 / (CW * int(sizeof(IO))) > 1 ? 128 / (CW * int(sizeof(IO))) : 1;
    const int64_t sv = MODE == kWhole ? 1 : MODE == kSegState ? nseg - 1 : nseg;
    const int64_t ncg = (D + CW - 1) / CW;
    const int64_t nbg = (B * sv + kN * NBG - 1) / (kN * NBG);
    const int64_t nlg = (ncg + CPL - 1) / CPL;             // line groups
    const int64_t per_xcd = (nlg * CPL * nbg + 7) / 8;  // logical workgroups per XCD
    const int64_t grid = 8 * per_xcd;
    if (grid > 0x7fffffff || B * sv > 0x7fffffff) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((mfma_prefill_kernel<IO, DM, NBG, MODE>), dim3(uint32_t(grid)),
                       dim3(64 * waves_of(DM)), 0, stream, lam, static_cast<const IO*>(u),
                       static_cast<IO*>(y), state, frag, lamc, int(B), int(D), T, int(ncg),
                       int(nbg), int(per_xcd), nseg, seg_len, xs);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_mode(const float2* lam, const void* u, bool bf16_io, int64_t B, int64_t D,
                       int64_t d, int64_t T, float2* state, void* y, const void* workspace,
                       int nseg, int64_t seg_len, float2* xs, hipStream_t stream)
{
    const int DM = int(d / 16);
    const size_t frag_bytes = frag_bytes_of(D, DM);
    const bf16x8* frag = static_cast<const bf16x8*>(workspace);
    const float2* lamc = reinterpret_cast<const float2*>(static_cast<const char*>(workspace) +
                                                         (frag_bytes + 255) / 256 * 256);
    // rows of the MFMA columns: batch rows or (batch row, segment) pairs
    const int64_t rows = MODE == kWhole ? B : MODE == kSegState ? B * (nseg - 1) : B * nseg;
    const bool two = mfma_nbg(rows, d, bf16_io) == 2;
    if (DM == 4) {  // float32 u/y only (mfma_supported), one batch group per wave
        if (bf16_io) return hipErrorInvalidValue;
        return launch_main<float, 4, 1, MODE>(lam, u, y, state, frag, lamc, B, D, T, nseg,
                                              seg_len, xs, stream);
    }
    if (bf16_io)
        return DM == 2 ? launch_main<bf16, 2, 1, MODE>(lam, u, y, state, frag, lamc, B, D, T,
                                                       nseg, seg_len, xs, stream)
                       : launch_main<bf16, 1, 1, MODE>(lam, u, y, state, frag, lamc, B, D, T,
                                                       nseg, seg_len, xs, stream);
    if (DM == 2)
        return launch_main<float, 2, 1, MODE>(lam, u, y, state, frag, lamc, B, D, T, nseg,
                                              seg_len, xs, stream);
    return two ? launch_main<float, 1, 2, MODE>(lam, u, y, state, frag, lamc, B, D, T, nseg,
                                                seg_len, xs, stream)
               : launch_main<float, 1, 1, MODE>(lam, u, y, state, frag, lamc, B, D, T, nseg,
                                                seg_len, xs, stream);
}

}  // namespace

// Workspace of the MFMA plan: fragments then lambda^C.
size_t mfma_workspace_bytes(int64_t D, int64_t d)
{
    const size_t frag = frag_bytes_of(D, int(d / 16));
    const size_t lamc = size_t(D) * d * sizeof(float2);
    return (frag + 255) / 256 * 256 + lamc;
}

bool mfma_supported(int64_t B, int64_t D, int64_t d, int64_t T, bool bf16_io)
{
    const bool tiles = d == 16 || d == 32 ? D % 8 == 0 : d == 64 && !bf16_io && D % 4 == 0;
    return tiles && T >= 1 && B <= (INT64_C(1) << 30) &&
           D <= (INT64_C(1) << 30);
}

// Segmented plan: the fewest segments (a power of two, each a multiple of 32
// and at least 256 steps long) whose (batch row, segment) columns give at
// least kSegWorkgroups workgroups of 8 channels, else the most segments
// allowed.
int64_t mfma_segments(int64_t B, int64_t D, int64_t d, int64_t T)
{
    constexpr int64_t kSegWorkgroups = 1024, kMinSeg = 256;
    const int64_t cw = waves_of(int(d / 16));
    int64_t best = 0;
    for (int64_t s = 2; T % (s * kC) == 0 && T / s >= kMinSeg; s *= 2) {
        best = s;
        if ((B * s + kN - 1) / kN * ((D + cw - 1) / cw) >= kSegWorkgroups) break;
    }
    return best;
}

// The matrix-core plan has no parallelism along time: the automatic plan takes
// it when its workgroups alone fill the GPU, counted as 16 channels x 32 batch
// rows (two rounds of the bfloat16 tiling with d = 16, 16 x 16).  The choice must not depend on the
// input type, which the workspace query does not know.
// Chunk steps of one pass on the busiest CU: its workgroups (one fits per
// CU) run in rounds of kMinWorkgroups, each walking `chunks` chunks for NBG
// groups of 16 columns.  rows = the pass's columns (batch rows, or (batch
// row, segment) pairs).
template <int MODE>
int64_t pass_slots(int64_t rows, int64_t D, int64_t d, bool bf16_io, int64_t chunks)
{
    const int cpw = d == 64   ? 1
                    : bf16_io ? (d == 32 ? cpw_of<bf16, 2, MODE>() : cpw_of<bf16, 1, MODE>())
                              : (d == 32 ? cpw_of<float, 2, MODE>() : cpw_of<float, 1, MODE>());
    const int nbg = mfma_nbg(rows, d, bf16_io);
    const int64_t cw = int64_t(waves_of(int(d / 16))) * cpw, bn = int64_t(kN) * nbg;
    const int64_t wgs = (D + cw - 1) / cw * ((rows + bn - 1) / bn);
    return (wgs + kMinWorkgroups - 1) / kMinWorkgroups * chunks * nbg;
}

bool mfma_preferred(int64_t B, int64_t D, int64_t d, int64_t T, bool bf16_io)
{
    if (((D + 15) / 16) * ((B + 31) / 32) >= kMinWorkgroups) return true;
    // fewer columns: the whole-prompt plan against the segmented one by the
    // chunk steps of their passes on the busiest CU (a chunk step costs about
    // the same in every pass; the segmented plan also pays for its extra
    // launches and second read of u, hence the 7/5 allowance, fitted to
    // measured times of both plans over B = 1..64, D = 768 / 2048, d = 16 /
    // 32, T = 1K..16K, float32 and bfloat16)
    const int64_t nseg = mfma_segments(B, D, d, T);
    if (nseg < 2) return false;
    const int64_t seg_chunks = T / nseg / kC;
    const int64_t whole = pass_slots<kWhole>(B, D, d, bf16_io, (T + kC - 1) / kC);
    const int64_t seg = pass_slots<kSegState>(B * (nseg - 1), D, d, bf16_io, seg_chunks) +
                        pass_slots<kSegOut>(B * nseg, D, d, bf16_io, seg_chunks);
    return 5 * whole <= 7 * seg;
}

int mfma_auto_plan(int64_t B, int64_t D, int64_t d, int64_t T, bool bf16_io)
{
    // d = 64 with fewer than 4 rows and at most 1024 (row, step) pairs: the
    // VALU plan's chunked scan beats both matrix-core plans (measured at D =
    // 768 and 2048)
    if (d == 64 && B < 4 && B * T <= 1024) return 0;
    if (mfma_preferred(B, D, d, T, bf16_io)) return 1;
    if (mfma_segments(B, D, d, T) >= 2) return 2;
    // no segments: at d = 64 the whole prompt beats the VALU plan from 4 rows
    // on (D = 768, T = 256: 0.058 ms against 0.067 ms at 4 rows, 0.13 ms at
    // 16), or once its workgroups (4 channels x 16 rows) fill the GPU
    if (d == 64 && (B >= 4 || (D + 3) / 4 * ((B + kN - 1) / kN) >= kMinWorkgroups)) return 1;
    return 0;
}

hipError_t launch_mfma_setup(const float2* lam, const float2* R, const float* h0, int64_t D,
                             int64_t d, bool bf16_io, void* workspace, hipStream_t stream)
{
    (void)hipGetLastError();
    const int DM = int(d / 16);
    const size_t frag_bytes = frag_bytes_of(D, DM);
    bf16x8* frag = static_cast<bf16x8*>(workspace);
    float2* lamc = reinterpret_cast<float2*>(static_cast<char*>(workspace) +
                                             (frag_bytes + 255) / 256 * 256);
    const int tw = bf16_io ? Stage<bf16>::kNTA : Stage<float>::kNTA;
    if (D > 0x7fffffff) return hipErrorInvalidConfiguration;
    if (DM == 1)
        hipLaunchKernelGGL(mfma_setup_kernel<1>, dim3(uint32_t(D)), dim3(256), 0, stream, lam,
                           R, h0, frag, lamc, tw);
    else if (DM == 4)
        hipLaunchKernelGGL(mfma_setup_kernel<4>, dim3(uint32_t(D)), dim3(256), 0, stream, lam,
                           R, h0, frag, lamc, tw);
    else
        hipLaunchKernelGGL(mfma_setup_kernel<2>, dim3(uint32_t(D)), dim3(256), 0, stream, lam,
                           R, h0, frag, lamc, tw);
    return hipGetLastError();
}

hipError_t launch_prefill_mfma(const float2* lam, const float2* R, const float* h0,
                               const void* u, bool bf16_io, int64_t B, int64_t D, int64_t d,
                               int64_t T, float2* state, void* y, void* workspace,
                               hipStream_t stream)
{
    hipError_t e = launch_mfma_setup(lam, R, h0, D, d, bf16_io, workspace, stream);
    if (e != hipSuccess) return e;
    return launch_mode<kWhole>(lam, u, bf16_io, B, D, d, T, state, y, workspace, 1, T, nullptr,
                               stream);
}

hipError_t launch_mfma_segment_pass(bool outputs, const float2* lam, const void* u,
                                    bool bf16_io, int64_t B, int64_t D, int64_t d, int64_t T,
                                    int nseg, int64_t seg_len, float2* xs, float2* state,
                                    void* y, const void* workspace, hipStream_t stream)
{
    (void)hipGetLastError();
    if (seg_len % kC != 0 || int64_t(nseg) * seg_len != T || nseg < 2)
        return hipErrorInvalidValue;
    return outputs ? launch_mode<kSegOut>(lam, u, bf16_io, B, D, d, T, state, y, workspace, nseg,
                                          seg_len, xs, stream)
                   : launch_mode<kSegState>(lam, u, bf16_io, B, D, d, T, state, y, workspace,
                                            nseg, seg_len, xs, stream);
}

}  // namespace lh
