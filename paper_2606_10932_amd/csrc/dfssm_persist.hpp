// dfssm_persist.hpp -- device helpers shared by the persistent kernels
// (the re-quantising chain and the fused decode step): 64-bit tagged
// exchange words at agent and XCD scope, wave reductions, direct-to-LDS
// loads, LDS flags and bounded spins.  Every kernel that uses them runs one
// workgroup per CU on the whole chip (256 workgroups, 8 XCDs of 32).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dfssm_px {

constexpr int kGrid = 256;
constexpr int kXcds = 8;
constexpr int kPerXcd = kGrid / kXcds;  // 32 workgroups per XCD
constexpr int kSlices = 8;              // column slices per XCD
constexpr long kSpinLimit = 1L << 20;

// This workgroup's XCD (HW_REG_XCC_ID[3:0]).
__device__ __forceinline__ int xcc_id() {
  return (int)(__builtin_amdgcn_s_getreg((20) | (0 << 6) | ((4 - 1) << 11)) & 7u);
}

// ------------------------------------------------------------ exchange words
// agent scope: the store writes through to memory and the load reads past the
// CU's L1 and the XCD's L2, so a word crosses workgroups on any XCD.  (A
// workgroup-scope store stays in the writer XCD's write-back L2, where
// device-scope loads need not see it, and group-scope loads may keep
// returning a line the reader's L1 holds: neither pairing is used.)
__device__ __forceinline__ uint64_t ll_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void ll_store(uint64_t* p, uint32_t tag, uint32_t v) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}

// The quantiser's code of v for inv = 127/a, where |v| <= a: |v * inv| is
// at most 127 * (1 + 2^-23)^2 < 127.5, so rint() already lands in [-127, 127]
// and the clamp of the definition never changes the result.
__device__ __forceinline__ int code(float v, float inv) { return (int)rintf(v * inv); }
// Eight two's-complement nibbles (value 2i in the low nibble of byte i) as
// two dwords of int8, values 0..3 in x and 4..7 in y: v_perm interleaves
// the low and high nibbles, then bit 3 of each byte is spread over its high
// half (0x08 * 0x1E = 0xF0, no carry between bytes).
__device__ __forceinline__ void unpack_i4x8(uint32_t w, uint32_t& x, uint32_t& y) {
  const uint32_t lo = w & 0x0F0F0F0Fu, hi = (w >> 4) & 0x0F0F0F0Fu;
  x = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
  y = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
  x |= (x & 0x08080808u) * 0x1Eu;
  y |= (y & 0x08080808u) * 0x1Eu;
}

__device__ __forceinline__ int dpp_sum16(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);  // row_mirror
  return v;
}
// Sum over aligned groups of G lanes (G = 1, 2, 4 or 32), in every lane of
// the group.  For 32: the 16-lane rows by DPP, then v_permlane16_swap of a
// value with itself leaves rows (0,0,2,2) in one result and (1,1,3,3) in the
// other, so their sum is the 32-lane half's total.
__device__ __forceinline__ int group_sum(int v, int G) {
  if (G >= 2) v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  if (G >= 4) v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  if (G >= 32) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
    v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);
    const auto p = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
    v = (int)(p[0] + p[1]);
  }
  return v;
}
// Whole-wave reductions with the result as a uniform value: DPP inside each
// 16-lane row, then row_bcast:15 and row_bcast:31, which leave the total in
// lane 63.
__device__ __forceinline__ int wave_sum_u(int v) {
  v = dpp_sum16(v);
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);
  return __builtin_amdgcn_readlane(v, 63);
}
// max of non-negative floats, compared as their bit patterns
__device__ __forceinline__ uint32_t wave_max_bits_u(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false));
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// ------------------------------------------------------------ direct-to-LDS
// Lane i's 16 (or 4) bytes from sbase + voff land at m0 + 16*i (4*i).
// Inline assembly, so the compiler does not make later LDS reads wait for
// them; the loading wave orders them with an explicit vector-memory wait
// before the barrier that hands the slot over.
__device__ __forceinline__ void lds_dma16(uint32_t voff, const void* sbase, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ void lds_dma4(uint32_t voff, const void* sbase, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ void lds_dma(int unit, uint32_t voff, const void* sbase, uint32_t lds) {
  if (unit == 16)
    lds_dma16(voff, sbase, lds);
  else
    lds_dma4(voff, sbase, lds);
}
// s_waitcnt with only the vector-memory counter constrained
#define CHAIN_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(0x0F70 | ((n) & 0xF) | (((n) >> 4) << 14))
// Workgroup barrier for LDS data only: the wave's LDS operations complete
// first, its vector-memory operations do not have to (the loading wave's
// direct-to-LDS loads of the next linears stay in flight; no global data
// crosses a barrier inside a workgroup, every exchange goes through polled
// tagged words)
#define CHAIN_BARRIER() asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory")

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// floor(u / d) for u < 2^11 and d <= 64 without a division: u * ceil(2^20 / d)
// >> 20 (the error term u * (ceil(2^20/d) * d - 2^20) / 2^20 < u * 64 / 2^20
// stays below 1/d, so the floor is exact); m = ceil(2^20 / d) is uniform.
__device__ __forceinline__ uint32_t recip20(uint32_t d) { return ((1u << 20) + d - 1) / d; }
__device__ __forceinline__ int udiv(int u, uint32_t m) { return (int)(((uint32_t)u * m) >> 20); }

// Workgroup flags in LDS, read and written as LDS operations: a volatile
// access through a generic pointer would be a flat access (clang leaves
// volatile accesses in the generic address space), which also counts as a
// vector-memory operation and makes every check wait for the wave's
// outstanding global stores.
typedef __attribute__((address_space(3))) volatile int lds_flag;
#define FLAG(v) (*(lds_flag*)(&(v)))

// One round of a bounded wait: true once the wait has to give up (after
// kSpinLimit rounds, or once another wave of the workgroup has given up:
// abort_flag is a workgroup LDS flag); the caller then leaves its loop.  The
// first time, the wave records `bit` in the status word and raises the flag.
__device__ __forceinline__ bool spin_gives_up(long& spins, int* abort_flag, unsigned* status, unsigned bit) {
  if (++spins > kSpinLimit || FLAG(*abort_flag)) {
    atomicOr(status, bit);
    FLAG(*abort_flag) = 1;
    return true;
  }
  __builtin_amdgcn_s_sleep(1);
  return false;
}

}  // namespace dfssm_px
