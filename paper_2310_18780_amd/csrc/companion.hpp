// Companion (rational) form of the distilled filters: launchers (internal to
// liblh).
#pragma once

#include "lh_internal.hpp"

namespace lh {

constexpr int kCompanionMaxModes = 16;  // companion order 2d <= 32

hipError_t launch_companion_coeffs(const float2* lam, const float2* R, int64_t D, int64_t d,
                                   double* a, double* beta, hipStream_t stream);

hipError_t launch_companion_step(const double* a, const double* beta, const float* h0,
                                 double* state, const void* u_t, void* y_t, bool bf16_io,
                                 int64_t B, int64_t D, int64_t d, hipStream_t stream);

// g, the impulse response of 1 / p, for t < T: [T, D] float64 in the workspace
inline size_t companion_init_workspace_bytes(int64_t D, int64_t T)
{
    return T > 0 ? static_cast<size_t>(T) * static_cast<size_t>(D) * sizeof(double) : 0;
}

hipError_t launch_companion_init(const double* a, const void* u, bool bf16_io, int64_t B,
                                 int64_t D, int64_t d, int64_t T, double* state,
                                 void* workspace, hipStream_t stream);

}  // namespace lh
