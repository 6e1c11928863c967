// dfssm_int4.hpp -- the scaffold + LoRA linear with int4 LoRA factors:
// A4 [r][K/2] and B4 [N][r/2] bytes of two's-complement nibbles, value 2i in
// the low nibble of byte i.  The few-token kernel reads them directly; the
// other paths expand them to int8 in the workspace first.
#pragma once

#include "dfssm_internal.hpp"

namespace dfssm {

// The few-token kernel (M <= kSkinnyMaxTokens) reading int4 factors.
hipError_t launch_skinny_linear_i4(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                                   int64_t r, const uint32_t* w_bits, const float* alpha,
                                   const uint8_t* A4, const uint8_t* B4, const float* beta, float* y,
                                   int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                                   const LinearWorkspace& ws, hipStream_t st);

// n values from packed nibbles to int8 (dst[i] = value i).
hipError_t launch_unpack_int4(const uint8_t* src, int64_t n, int8_t* dst, hipStream_t st);

// Workspace of an int4 linear: the int8 linear's, then room for the
// expanded factors (A [r][K], B [N][r]) at 256-byte aligned offsets.
inline size_t linear_i4_extra_offset(int64_t M, int64_t K, int64_t r) {
  return (carve_linear_workspace(nullptr, M, K, r).bytes + 255) & ~(size_t)255;
}
inline size_t linear_i4_workspace_bytes(int64_t M, int64_t K, int64_t N, int64_t r) {
  const size_t a = ((size_t)(r * K) + 255) & ~(size_t)255;
  const size_t b = ((size_t)(N * r) + 255) & ~(size_t)255;
  return linear_i4_extra_offset(M, K, r) + a + b;
}

}  // namespace dfssm
