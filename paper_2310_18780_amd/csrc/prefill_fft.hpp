// Prefill by FFT convolution with the materialised filter and the state by a
// Vandermonde contraction: plan and launcher (internal to liblh).
#pragma once

#include "lh_internal.hpp"

namespace lh {

// Longest prompt of the FFT prefill: the transform length N = 2^m >= 2T - 1
// is cut as N1 x N2 with N1, N2 <= 1024, so N <= 2^20 and T <= 2^19.
constexpr int64_t kFftMaxT = int64_t(1) << 19;

struct FftPlan {
    int logN1;          // row length N1 = 2^logN1 (the second transform pass)
    int logN2;          // column length N2 = 2^logN2 (first and last passes)
    int64_t npair;      // batch rows are transformed in pairs (real, imaginary part)
    int64_t nparts;     // time ranges of the state contraction (summed afterwards)
    int64_t part_len;   // steps per time range (a multiple of the restart length)
    size_t off_tw;      // N-point twiddle table omega_N^k        [N] complex64
    size_t off_polar;   // (log2 |lambda|, arg lambda)             [D, d] 2 x float64
    size_t off_H;       // filter spectrum, [f2][f1][c]            [N, D] complex64
    size_t off_Z;       // spectra of the input pairs, [p][f2][n1][c] (the filter
                        // [T, D] float32 is materialised here first)
    size_t off_parts;   // partial states [nparts, B, D, d] complex64 (nparts > 1)
    size_t ws_bytes;    // 0 when T == 0
};

// False when the sizes are invalid, T > kFftMaxT, or a size overflows.
bool make_fft_plan(int64_t B, int64_t D, int64_t d, int64_t T, FftPlan* plan);

hipError_t launch_prefill_fft(const float2* lam, const float2* R, const float* h0,
                              const void* u, bool bf16_io, int64_t B, int64_t D, int64_t d,
                              int64_t T, float2* state, void* y, const FftPlan& plan,
                              void* workspace, hipStream_t stream);

}  // namespace lh
