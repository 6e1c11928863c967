// dfssm_diag.hip -- a diagnostic outside the computation: the time one launch
// takes to read a buffer from memory, the floor under a single linear of the
// same bytes at decode sizes.
#include "dfssm_internal.hpp"

namespace {

constexpr int kReadThreads = 256;
constexpr int kReadU = 2;  // 16-byte loads per thread, all issued before the first use

// Block b reads the 16-byte words b*512 .. b*512+511 (coalesced: load u of
// thread t is word b*512 + 256u + t); wave w of block b stores the XOR of
// the 32-bit words it read into sink[4b + w], so no load can be dropped (one
// word per wave: atomics on a shared word serialise, ~10 ns each).
__global__ __launch_bounds__(kReadThreads) void read_floor(const uint4* __restrict__ p, int64_t n16,
                                                           uint32_t* sink) {
  if (n16 == 0) return;
  const int64_t base = (int64_t)blockIdx.x * (kReadThreads * kReadU) + threadIdx.x;
  uint4 v[kReadU];
#pragma unroll
  for (int u = 0; u < kReadU; ++u) {
    const int64_t i = base + (int64_t)u * kReadThreads;
    v[u] = i < n16 ? p[i] : make_uint4(0, 0, 0, 0);
  }
  uint32_t x = 0;
#pragma unroll
  for (int u = 0; u < kReadU; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x ^= (uint32_t)__shfl_xor((int)x, off, 64);
  if ((threadIdx.x & 63) == 0) sink[blockIdx.x * (kReadThreads / 64) + (threadIdx.x >> 6)] = x;
}

}  // namespace

namespace dfssm {

int64_t read_floor_sink_words(int64_t bytes) {
  return (kReadThreads / 64) * std::max<int64_t>(1, ceil_div(bytes / 16, (int64_t)kReadThreads * kReadU));
}

hipError_t launch_read_floor(const void* p, int64_t bytes, uint32_t* sink, hipStream_t st) {
  const int64_t n16 = bytes / 16;
  const int64_t blocks = n16 == 0 ? 1 : ceil_div(n16, (int64_t)kReadThreads * kReadU);
  read_floor<<<dim3((unsigned)blocks), dim3(kReadThreads), 0, st>>>(reinterpret_cast<const uint4*>(p), n16, sink);
  return hipGetLastError();
}

}  // namespace dfssm
