// dfssm_quantize.hip -- per-token absmax int8 activation quantisation (the
// int8 operand of the scaffold product, Sec. 4.1 of the paper), gfx950.
//
// One workgroup of 256 threads per token row.  Pass 1 reduces max|x| over
// the row (wave64 butterfly, then across the 4 waves through LDS); pass 2
// re-reads the row (L2-resident) and writes the codes.  Rows are read with
// 16-byte loads when the row start and stride allow it.
#include <float.h>

#include "dfssm_internal.hpp"

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float to_f32(_Float16 h) { return (float)h; }  // exact widening
__device__ __forceinline__ float to_f32(float f) { return f; }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

__device__ __forceinline__ int8_t code(float v, float inv) {
  float t = v * inv;
  float r = rintf(t);  // v_rndne_f32: round to nearest, ties to even
  r = fminf(fmaxf(r, -127.0f), 127.0f);
  return (int8_t)(int)r;
}

// VEC elements per vector access (16 bytes), or 1.
template <typename T, int VEC>
__global__ __launch_bounds__(kThreads) void quantize_rows(const T* __restrict__ x, int K,
                                                          int64_t ldx, int8_t* __restrict__ q,
                                                          float* __restrict__ s, int scale_mode) {
  const int64_t m = blockIdx.x;
  const T* row = x + m * ldx;
  int8_t* qrow = q + m * (int64_t)K;
  __shared__ float red[kThreads / 64];

  float a = 0.0f;
  if constexpr (VEC > 1) {
    using V = __attribute__((ext_vector_type(VEC))) T;
    for (int k = threadIdx.x * VEC; k < K; k += kThreads * VEC) {
      V v = *reinterpret_cast<const V*>(row + k);
#pragma unroll
      for (int e = 0; e < VEC; ++e) a = fmaxf(a, fabsf(to_f32(v[e])));
    }
  } else {
    for (int k = threadIdx.x; k < K; k += kThreads) a = fmaxf(a, fabsf(to_f32(row[k])));
  }
  a = wave_max(a);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = a;
  __syncthreads();
  a = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));

  if (a < FLT_MIN) {  // all-zero (or subnormal-only) row
    for (int k = threadIdx.x; k < K; k += kThreads) qrow[k] = 0;
    if (threadIdx.x == 0) s[m] = scale_mode ? 1.0f / 127.0f : 0.0f;
    return;
  }
  const float inv = 127.0f / a;  // correctly rounded fp32 division
  if (threadIdx.x == 0) s[m] = scale_mode ? 1.0f / 127.0f : a / 127.0f;

  if constexpr (VEC > 1) {
    using V = __attribute__((ext_vector_type(VEC))) T;
    for (int k = threadIdx.x * VEC; k < K; k += kThreads * VEC) {
      V v = *reinterpret_cast<const V*>(row + k);
      if constexpr (VEC == 8) {
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) lo |= (uint32_t)(uint8_t)code(to_f32(v[e]), inv) << (8 * e);
#pragma unroll
        for (int e = 0; e < 4; ++e) hi |= (uint32_t)(uint8_t)code(to_f32(v[4 + e]), inv) << (8 * e);
        *reinterpret_cast<uint2*>(qrow + k) = make_uint2(lo, hi);
      } else {
        uint32_t w = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) w |= (uint32_t)(uint8_t)code(to_f32(v[e]), inv) << (8 * e);
        *reinterpret_cast<uint32_t*>(qrow + k) = w;
      }
    }
  } else {
    for (int k = threadIdx.x; k < K; k += kThreads) qrow[k] = code(to_f32(row[k]), inv);
  }
}

}  // namespace

namespace dfssm {

hipError_t launch_quantize(const void* x, int x_dtype, int64_t M, int64_t K, int64_t ldx,
                           int8_t* q, float* s, int scale_mode, hipStream_t st) {
  if (M == 0) return hipSuccess;
  dim3 grid((unsigned)M), block(kThreads);
  const uintptr_t xa = reinterpret_cast<uintptr_t>(x);
  if (x_dtype == DFSSM_F16) {
    const bool vec = (xa % 16 == 0) && ((ldx * 2) % 16 == 0) && (K % 8 == 0);
    if (vec)
      quantize_rows<_Float16, 8><<<grid, block, 0, st>>>(static_cast<const _Float16*>(x), (int)K,
                                                         ldx, q, s, scale_mode);
    else
      quantize_rows<_Float16, 1><<<grid, block, 0, st>>>(static_cast<const _Float16*>(x), (int)K,
                                                         ldx, q, s, scale_mode);
  } else {
    const bool vec = (xa % 16 == 0) && ((ldx * 4) % 16 == 0) && (K % 4 == 0);
    if (vec)
      quantize_rows<float, 4><<<grid, block, 0, st>>>(static_cast<const float*>(x), (int)K, ldx,
                                                      q, s, scale_mode);
    else
      quantize_rows<float, 1><<<grid, block, 0, st>>>(static_cast<const float*>(x), (int)K, ldx,
                                                      q, s, scale_mode);
  }
  return hipGetLastError();
}

}  // namespace dfssm
