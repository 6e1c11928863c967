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

// ------------------------------------------------------------ exchange hop
// Workgroups 2i and 2i+1 (on two XCDs: the dispatcher deals workgroups to
// the XCDs in turn) pass one 64-bit word back and forth `iters` times at
// agent scope, as the persistent kernels' exchange words do; with kFence
// the store is a release and the load an acquire (the fence pair a
// release/acquire protocol would need).  Each side records the
// s_memrealtime ticks (100 MHz) of its whole loop.  Waits are bounded: a
// side that gives up sets *fail and leaves, and its partner gives up in turn.
namespace {
constexpr long kPingSpin = 1L << 22;

template <bool kFence>
__global__ __launch_bounds__(64) void exchange_pingpong(uint64_t* words, int iters, int npairs, int64_t* ticks,
                                                        unsigned* fail) {
  const int wg = blockIdx.x;
  if (wg >= 2 * npairs || threadIdx.x != 0) return;
  const int pair = wg >> 1, side = wg & 1;
  uint64_t* mine = words + (int64_t)(2 * pair + side) * 64;  // 512 bytes apart
  const uint64_t* theirs = words + (int64_t)(2 * pair + (side ^ 1)) * 64;
  const int64_t t0 = (int64_t)__builtin_amdgcn_s_memrealtime();
  for (int i = 1; i <= iters; ++i) {
    if (side == 0) {
      if (kFence)
        __hip_atomic_store(mine, (uint64_t)i, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      else
        __hip_atomic_store(mine, (uint64_t)i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    long sp = 0;
    for (;;) {
      const uint64_t v = kFence ? __hip_atomic_load(theirs, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT)
                                : __hip_atomic_load(theirs, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (v == (uint64_t)i) break;
      // every 1024 polls: the bound, and whether the partner gave up
      if ((++sp & 1023) == 0 &&
          (sp > kPingSpin || __hip_atomic_load(fail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)) {
        atomicOr(fail, 1u);
        return;
      }
    }
    if (side == 1) {
      if (kFence)
        __hip_atomic_store(mine, (uint64_t)i, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      else
        __hip_atomic_store(mine, (uint64_t)i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  ticks[wg] = (int64_t)__builtin_amdgcn_s_memrealtime() - t0;
}
}  // namespace

namespace dfssm {

hipError_t launch_exchange_pingpong(int npairs, int iters, bool fence, void* ws, hipStream_t st) {
  char* b = static_cast<char*>(ws);
  uint64_t* words = reinterpret_cast<uint64_t*>(b);
  int64_t* ticks = reinterpret_cast<int64_t*>(b + kPingWordsBytes);
  unsigned* fail = reinterpret_cast<unsigned*>(b + kPingWordsBytes + kPingTicksBytes);
  // every word, tick and the flag start at zero (a fill kernel: no memset
  // node if the caller captures this)
  hipError_t e = launch_zero_words(words, (int64_t)(kPingBytes / 8), st);
  if (e != hipSuccess) return e;
  if (fence)
    exchange_pingpong<true><<<dim3(256), dim3(64), 0, st>>>(words, iters, npairs, ticks, fail);
  else
    exchange_pingpong<false><<<dim3(256), dim3(64), 0, st>>>(words, iters, npairs, ticks, fail);
  return hipGetLastError();
}

}  // namespace dfssm
