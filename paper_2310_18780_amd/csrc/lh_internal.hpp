// Internal declarations of liblh: element helpers shared by the kernels and
// the launchers the C ABI layer calls.  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lh {

// bfloat16 storage type (upper half of a float32)
struct bf16 {
    uint16_t bits;
};

__device__ __forceinline__ float io_load(const float* p) { return *p; }
__device__ __forceinline__ float io_load(const bf16* p) {
    return __uint_as_float(static_cast<uint32_t>(p->bits) << 16);
}
__device__ __forceinline__ void io_store(float* p, float v) { *p = v; }
// float32 -> bfloat16, round to nearest, ties to even (gfx950 converts with
// one v_cvt_pk_bf16_f32; NaN stays NaN).
__device__ __forceinline__ void io_store(bf16* p, float v) {
    p->bits = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
}

// Non-temporal variants (written once, not re-read soon): keep the cache for
// data that is.
__device__ __forceinline__ void io_store_nt(float* p, float v) { __builtin_nontemporal_store(v, p); }
__device__ __forceinline__ void io_store_nt(bf16* p, float v) {
    __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, static_cast<__bf16>(v)), &p->bits);
}

// How the prefill of one call is cut up.
struct PrefillPlan {
    int lpr;          // lanes per (b, c) row: the modes of a row are split over lpr lanes
    int mpl;          // modes per lane (power of two <= 16); lpr * mpl >= d
    int64_t C;        // chunk length (time steps per chunk)
    int64_t nchunks;  // ceil(T / C); 0 when T == 0
    size_t off_pow;   // workspace offset of lambda^C          [D, d] complex64
    size_t off_xin;   // workspace offset of chunk entry states [B, nchunks, D, d] complex64
    size_t ws_bytes;  // total workspace bytes (0 when nchunks <= 1 and no MFMA plan)
    bool mfma;        // matrix-core prefill (automatic plans use it when u and y are
                      // 16-byte aligned, else the VALU plan above)
    bool mfma_forced; // requested explicitly: u and y must be 16-byte aligned
    bool mfma_seg;    // segmented matrix-core plan: the prompt is cut into nchunks
                      // segments of C steps (C % 32 == 0, T == nchunks C); state pass
                      // and output pass on the matrix cores, carry in between (falls
                      // back to the VALU chunked scan with the same C when u or y is
                      // not 16-byte aligned)
    size_t off_mfma;  // workspace offset of the matrix-core tables (segmented plan)
};

// The plan of a prefill call.  request: 0 automatic, > 0 the VALU chunked
// scan with this chunk length, -1 the matrix-core plan, -2 the segmented
// matrix-core plan.  Returns false when the sizes are invalid, overflow or do
// not support the request.  io: 0 float32, 1 bfloat16 u/y, -1 either (the
// automatic plan may differ between them; the workspace size is then the
// larger of the two).
bool make_prefill_plan(int64_t B, int64_t D, int64_t d, int64_t T, int64_t request, int io,
                       PrefillPlan* plan);

// Launchers (asynchronous, on `stream`); they return the launch status.
hipError_t launch_prefill(const float2* lam, const float2* R, const float* h0,
                          const void* u, bool bf16_io, int64_t B, int64_t D, int64_t d,
                          int64_t T, float2* state, void* y, const PrefillPlan& plan,
                          void* workspace, hipStream_t stream);

// Matrix-core prefill: d = 16 or 32 with D a multiple of 8 (bfloat16
// operands), or d = 64 with float32 u/y and D a multiple of 4 (float32
// operands).
bool mfma_supported(int64_t B, int64_t D, int64_t d, int64_t T, bool bf16_io);
// Whether the automatic plan takes the whole-prompt matrix-core plan over the
// segmented one.
bool mfma_preferred(int64_t B, int64_t D, int64_t d, int64_t T, bool bf16_io);
// The automatic plan where the matrix-core plans are supported: 0 the VALU
// scan, 1 the whole-prompt matrix-core plan, 2 the segmented one.
int mfma_auto_plan(int64_t B, int64_t D, int64_t d, int64_t T, bool bf16_io);
size_t mfma_workspace_bytes(int64_t D, int64_t d);
// Segment count of the segmented matrix-core plan (0 when T does not split
// into segments of a multiple of 32 steps, at least 256 long).
int64_t mfma_segments(int64_t B, int64_t D, int64_t d, int64_t T);
// Matrix-core tables of the filters into the workspace (bf16_io: only the
// operand terms the bfloat16 kernels read are written).
hipError_t launch_mfma_setup(const float2* lam, const float2* R, const float* h0, int64_t D,
                             int64_t d, bool bf16_io, void* workspace, hipStream_t stream);
// One pass of the segmented plan: outputs = false writes each segment's end
// state from zero into slot k < nseg - 1 of xs [B, nseg, D, d]; outputs = true
// runs every segment from its entry state in xs, writes y and x_T.
hipError_t launch_mfma_segment_pass(bool outputs, const float2* lam, const void* u,
                                    bool bf16_io, int64_t B, int64_t D, int64_t d, int64_t T,
                                    int nseg, int64_t seg_len, float2* xs, float2* state,
                                    void* y, const void* workspace, hipStream_t stream);
hipError_t launch_prefill_mfma(const float2* lam, const float2* R, const float* h0,
                               const void* u, bool bf16_io, int64_t B, int64_t D, int64_t d,
                               int64_t T, float2* state, void* y, void* workspace,
                               hipStream_t stream);

hipError_t launch_step(const float2* lam, const float2* R, const float* h0, float2* state,
                       const void* u_t, void* y_t, bool bf16_io, int64_t B, int64_t D,
                       int64_t d, bool aligned16, hipStream_t stream);

// Distillation objective: loss and gradients per channel (targets [D, L]).
hipError_t launch_distill(const float* A, const float* theta, const float2* R,
                          const float* target, int64_t D, int64_t d, int64_t L, float* loss,
                          float* dA, float* dtheta, float2* dR, float* hhat, hipStream_t stream);

// Multi-head decode step (state [B, M, N, N, d]; q, k, v, y [B, M N]).
hipError_t launch_mh_step(const float2* lam, const float2* R, const float* h0, float2* state,
                          const void* q, const void* k, const void* v, void* y, bool bf16_io,
                          int64_t B, int64_t M, int64_t N, int64_t d, bool aligned16,
                          hipStream_t stream);

}  // namespace lh
