// dfssm_mamba.hpp -- launchers of the Mamba-2 decode-step kernels around the
// linears (dfssm_mamba.hip).  All return hipSuccess or the launch error;
// shapes are validated by the caller.
#pragma once

#include "dfssm_internal.hpp"

namespace dfssm {

// Largest row the two norm kernels hold in registers: at most 4 float4 per
// thread, on 512 threads up to d = 8192 and on 1024 threads beyond.
constexpr int64_t kNormMaxD = 16384;

// u_out = u + delta (delta may be null; u_out may be null or u), then
// RMSNorm with weight w and the linear's per-token int8 quantisation.
hipError_t launch_add_rmsnorm_quant(const float* u, const float* delta, const float* w, float eps, int64_t M,
                                    int64_t d, float* u_out, int8_t* q, float* s, hipStream_t st);

// g = y * silu(z) (z rows of stride ldz), RMSNorm with weight w, quantisation.
hipError_t launch_gate_norm_quant(const float* y, const float* z, int64_t ldz, const float* w, float eps,
                                  int64_t M, int64_t d, int8_t* q, float* s, hipStream_t st);

// Convolution step (4-slot ring per sequence) and SSM step of one token per
// sequence; heads of 64 channels, d_state 64 or 128, one B/C group.  With
// gate_y the output is y * silu(z) (z = zx[m][0 .. d_inner)), the gated
// norm's first product in the same fp32 rounding, so that the norm itself
// can run as a plain RMSNorm.
hipError_t launch_ssm_step(const float* zx, int64_t ld, int64_t M, int64_t d_inner, int64_t d_state, int64_t step,
                           float* ring, const float* conv_w, const float* conv_b, const float* dt_bias,
                           const float* A_log, const float* D, float* state, float* y, float* xbc,
                           hipStream_t st, bool gate_y = false);

}  // namespace dfssm
