// dfssm_int4.hip -- expansion of int4 LoRA factors to int8 for the paths
// that read int8 operands (prefill MFMA, popcount GEMV), gfx950.  A thread
// turns 8 packed bytes into 16 values: one 8-byte load, one 16-byte store.
#include <algorithm>

#include "dfssm_int4.hpp"

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t sext_nibbles(uint32_t t) {
  t ^= 0x08080808u;
  return ((t | 0x80808080u) - 0x08080808u) ^ 0x80808080u;
}

__global__ __launch_bounds__(kThreads) void unpack_int4(const uint8_t* __restrict__ src, int64_t n,
                                                        int8_t* __restrict__ dst) {
  const int64_t groups = (n + 15) / 16;
  for (int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x; g < groups; g += (int64_t)gridDim.x * kThreads) {
    const int64_t i0 = 16 * g;
    if (i0 + 16 <= n) {
      const uint2 p = *reinterpret_cast<const uint2*>(src + 8 * g);
      const uint32_t lo0 = p.x & 0x0F0F0F0Fu, hi0 = (p.x >> 4) & 0x0F0F0F0Fu;
      const uint32_t lo1 = p.y & 0x0F0F0F0Fu, hi1 = (p.y >> 4) & 0x0F0F0F0Fu;
      *reinterpret_cast<uint4*>(dst + i0) =
          make_uint4(sext_nibbles(__builtin_amdgcn_perm(hi0, lo0, 0x05010400u)),
                     sext_nibbles(__builtin_amdgcn_perm(hi0, lo0, 0x07030602u)),
                     sext_nibbles(__builtin_amdgcn_perm(hi1, lo1, 0x05010400u)),
                     sext_nibbles(__builtin_amdgcn_perm(hi1, lo1, 0x07030602u)));
    } else {
      for (int64_t i = i0; i < n; ++i) {
        const int byte = src[i >> 1];
        const int nib = (i & 1) ? (byte >> 4) : (byte & 15);
        dst[i] = (int8_t)(nib >= 8 ? nib - 16 : nib);
      }
    }
  }
}

}  // namespace

namespace dfssm {

hipError_t launch_unpack_int4(const uint8_t* src, int64_t n, int8_t* dst, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t groups = ceil_div(n, 16);
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>(ceil_div(groups, kThreads), 4096));
  unpack_int4<<<dim3((unsigned)blocks), dim3(kThreads), 0, st>>>(src, n, dst);
  return hipGetLastError();
}

}  // namespace dfssm
