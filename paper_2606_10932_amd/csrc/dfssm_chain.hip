// dfssm_chain.hip -- persistent kernel for the re-quantising chain of
// scaffold + LoRA linears at one token (the decode step's projections run
// back to back, Sec. 4.1 of the paper, where a CUDA graph removes launch
// gaps; here one cooperative launch replaces the whole sequence).
//
// Every linear depends on all of the previous linear's output (its absmax
// and its LoRA down-projection are reductions over all of it), so the chain
// is bound by cross-CU communication latency, not by HBM.  The design keeps
// that to two one-way hops per linear and never uses an agent-scope fence
// (on MI355X a release/acquire pair costs ~3.5 us: it writes back and
// invalidates the whole L2):
//
//  * Data crosses workgroups as 64-bit words {tag:32, value:32}, each written
//    with one relaxed agent-scope atomic store and read with relaxed atomic
//    loads, so a consumer polls the data itself: a word is valid once its
//    tag equals the linear's tag.  The exchange region is zeroed before the
//    launch, so tag 0 never matches.
//  * A workgroup is two groups of 4 waves that alternate roles: while one
//    group computes linear l, the other holds (in its own registers) the
//    weights of linear l+1 it loaded during linear l-1.  So the
//    latency-critical waits (which wait for all of a wave's outstanding
//    loads) never wait behind a weight prefetch.
//  * Per linear, the active group: polls y_{l-1}[0:K_l] -> absmax -> Q (the
//    quantiser's fp32 decisions) -> bit-planes in LDS; workgroup j < r
//    computes acc_a[j] = A[j,:].Q and publishes it; the popcount GEMV on the
//    workgroup's rows; waits for the r acc_a words; LoRA up-projection and
//    epilogue; publishes its y rows; then prefetches linear l+2.
//  * Every wait is bounded: on time-out the workgroup records an error in
//    the status word and leaves, so the grid always drains.
//  * The layer table lives in the workspace, written by a setup launch
//    (dfssm_chain_prepare) together with a fingerprint of the table; the
//    kernel compares that fingerprint with the caller's before it reads the
//    table, and leaves (status bit 8) if they differ.
#include <float.h>

#include "dfssm_internal.hpp"

namespace {

constexpr int kGT = 512;              // threads per role group
constexpr int kCT = 2 * kGT;          // threads per workgroup
constexpr int kGW = kGT / 64;         // waves per group
static_assert(kGW == dfssm::kChainWaves, "waves per role group");
constexpr int kMaxSteps = dfssm::kChainMaxSteps;
constexpr int kPollVals = dfssm::kChainMaxK / kGT;
constexpr long kSpinLimit = 1L << 20;
// done and acc_a words are spread one per 128-byte line (16 words), so the
// workgroups polling them do not all hit one memory channel
constexpr int kPad = dfssm::kChainPad;

__device__ __forceinline__ uint64_t ll_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// workgroup scope: may hit a copy in this XCD's L2 (shared by the
// workgroups of the XCD); a stale copy fails the tag check and is re-read
// at agent scope
__device__ __forceinline__ uint64_t ll_load_cached(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void ll_store(uint64_t* p, uint32_t tag, uint32_t v) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}

__device__ __forceinline__ int8_t code(float v, float inv) {
  float r = rintf(v * inv);
  r = fminf(fmaxf(r, -127.0f), 127.0f);
  return (int8_t)(int)r;
}

__device__ __forceinline__ int plane_sum(const int (&c)[8]) {
  int s = c[0] + (c[1] << 1) + (c[2] << 2) + (c[3] << 3) + (c[4] << 4) + (c[5] << 5) + (c[6] << 6);
  return s - (c[7] << 7);
}

__device__ __forceinline__ int chunk_masked_sum(const uint4 w, const uint4 (&P)[8]) {
  int c[8];
#pragma unroll
  for (int b = 0; b < 8; ++b)
    c[b] = __builtin_popcount(w.x & P[b].x) + __builtin_popcount(w.y & P[b].y) +
           __builtin_popcount(w.z & P[b].z) + __builtin_popcount(w.w & P[b].w);
  return plane_sum(c);
}

__device__ __forceinline__ int chunk_qsum(const uint4 (&P)[8]) {
  int c[8];
#pragma unroll
  for (int b = 0; b < 8; ++b)
    c[b] = __builtin_popcount(P[b].x) + __builtin_popcount(P[b].y) + __builtin_popcount(P[b].z) +
           __builtin_popcount(P[b].w);
  return plane_sum(c);
}

__device__ __forceinline__ int dpp_sum16(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);  // row_mirror
  return v;
}

// Sum over aligned groups of G lanes (G = 8..64), result in every lane of
// the group: DPP butterflies inside a 16-lane row, lane swaps across rows.
__device__ __forceinline__ int group_sum(int v, int G) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
  if (G >= 16) v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);
  if (G >= 32) v += __shfl_xor(v, 16, 64);
  if (G >= 64) v += __shfl_xor(v, 32, 64);
  return v;
}

__device__ __forceinline__ int wave_sum(int v) {
  v = dpp_sum16(v);
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}

// max over the wave of non-negative floats, compared as their bit patterns
__device__ __forceinline__ uint32_t wave_max_bits(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));
  v = max(v, (uint32_t)__shfl_xor((int)v, 16, 64));
  v = max(v, (uint32_t)__shfl_xor((int)v, 32, 64));
  return v;
}

// One linear's operands of this workgroup, per lane of a group.  The A row
// is held in the column layout of the codes: a[i] is column gt + kGT * i.
struct Pref {
  uint4 w[kMaxSteps];
  uint32_t b[kMaxSteps];
  float al[kMaxSteps], be[kMaxSteps];
  int32_t a[kPollVals];
};

// Loads go through the global address space (the table's pointers are
// generic, which would otherwise give flat loads) and always read in-range
// addresses; nothing is masked here, so no instruction waits on a prefetched
// value before its use.  Values read for lanes outside the data are harmless
// by construction: lanes past a row's chunks meet all-zero bit-planes, LoRA
// lanes past r meet zero limbs, A bytes past K meet zero codes, and rows
// outside the workgroup's range are never stored.
typedef unsigned v4u __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 gload16(const void* p) {
  v4u v = *(const __attribute__((address_space(1))) v4u*)(p);
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint32_t gload4(const void* p) {
  return *(const __attribute__((address_space(1))) uint32_t*)(p);
}
__device__ __forceinline__ int32_t gload1s(const void* p) {
  return *(const __attribute__((address_space(1))) int8_t*)(p);
}

__device__ __forceinline__ void prefetch(const dfssm::ChainLayerDev& L, int wg, int nwg, int gt,
                                         Pref& p) {
  const int lane = gt & 63, wave = gt >> 6;
  const int G = L.G, g = lane & (G - 1), grp = lane / G;
  const int RW = 64 / G;
  const int R = (L.N + nwg - 1) / nwg;
  const int n0 = wg * R, n1 = min(L.N, n0 + R);
  const int C = L.K >> 7, W = L.K >> 5, r4 = L.r >> 2;
#pragma unroll
  for (int s = 0; s < kMaxSteps; ++s) {
    const int n = n0 + s * kGW * RW + wave * RW + grp;
    const int nc = n < n1 ? n : 0;
    p.w[s] = gload16(L.w_bits + (int64_t)nc * W + 4 * (g < C ? g : 0));
    p.al[s] = __uint_as_float(gload4(L.alpha + nc));
    // the table never holds NULL: with r == 0, A/B/beta point at alpha
    p.b[s] = gload4(L.B + (int64_t)nc * L.r + 4 * (g < r4 ? g : 0));
    p.be[s] = __uint_as_float(gload4(L.beta + nc));
  }
  const int8_t* arow = L.A + (int64_t)(wg < L.r ? wg : 0) * L.K;
#pragma unroll
  for (int i = 0; i < kPollVals; ++i) {
    const int k = gt + i * kGT;
    p.a[i] = gload1s(arow + (k < L.K ? k : 0));
  }
}

__device__ __forceinline__ bool poll_ll(const uint64_t* p, uint32_t tag, uint64_t& wd,
                                        unsigned* status, unsigned code_bit) {
  long spins = 0;
  while ((uint32_t)((wd = ll_load(p)) >> 32) != tag) {
    if (++spins > kSpinLimit) {
      atomicOr(status, code_bit);
      return false;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  return true;
}

__global__ __launch_bounds__(kCT, 1) void chain_persistent(
    const dfssm::ChainLayerDev* __restrict__ layers, int L, const int8_t* __restrict__ q0,
    const float* __restrict__ s0, uint64_t* __restrict__ y_ll, uint64_t* __restrict__ acc_ll,
    uint64_t* __restrict__ done_ll, float* __restrict__ y_all, unsigned* __restrict__ status,
    uint32_t seq, const uint64_t* __restrict__ table_hash, uint64_t expect_hash) {
  // the table was written by a prepare of the same layers, or nothing here
  // is trusted: leave before reading it
  if (*table_hash != expect_hash) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(status, 8u);
    return;
  }
  __shared__ uint4 pl_lds[(dfssm::kChainMaxK / 128) * 8];
  __shared__ int4 acc_lds[dfssm::kMaxRank / 4];
  __shared__ int32_t dot_part[kGW];
  __shared__ uint32_t ymax_lds;
  __shared__ int cnt_dot, cnt_epi;
  __shared__ float inv_lds;
  __shared__ int zero_lds;
  __shared__ int abort_;
  const int wg = blockIdx.x, nwg = gridDim.x;
  const int tid = threadIdx.x;
  const int group = tid / kGT, gt = tid % kGT, lane = gt & 63, wave = gt >> 6;
  if (tid == 0) {
    abort_ = 0;
    cnt_dot = 0;
    cnt_epi = 0;
    ymax_lds = 0;
  }

  Pref pf;
  if (group < L) prefetch(layers[group], wg, nwg, gt, pf);
  __syncthreads();

  // a word written for linear l carries tag(l); seq differs per launch, so a
  // word left from an earlier launch (or a stale cached copy of one) never
  // validates
  auto tag_of = [seq](int l) -> uint32_t { return (seq << 8) | (uint32_t)((l + 1) & 0xff); };

  for (int l = 0; l < L; ++l) {
    const bool active = group == (l & 1);
    const dfssm::ChainLayerDev Ld = layers[l];
    const int K = Ld.K, N = Ld.N, r = Ld.r, G = Ld.G;
    const float s = l == 0 ? s0[0] : 1.0f / 127.0f;

    // ---- 0. wait for the producers of y_{l-1}[0:K]; their done words carry
    //         the absmax of their rows below K, so the scale comes for free
    if (active && l > 0 && wave == 0) {
      const int Rp = (layers[l - 1].N + nwg - 1) / nwg;
      const int P = min(nwg, (K + Rp - 1) / Rp);
      const uint64_t* dn = done_ll + (int64_t)(l - 1) * nwg * kPad;
      // up to 4 producers per lane (nwg <= 256), all polled together
      uint32_t am = 0, need = 0;
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (lane + 64 * t < P) need |= 1u << t;
      long spins = 0;
      while (need) {
        uint64_t wd[4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
          if (need & (1u << t)) wd[t] = ll_load(dn + (lane + 64 * t) * kPad);
#pragma unroll
        for (int t = 0; t < 4; ++t)
          if ((need & (1u << t)) && (uint32_t)(wd[t] >> 32) == tag_of(l - 1)) {
            am = max(am, (uint32_t)wd[t]);
            need &= ~(1u << t);
          }
        if (need) {
          if (++spins > kSpinLimit) {
            atomicOr(status, 1u);
            abort_ = 1;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      am = wave_max_bits(am);
      if (lane == 0) {
        const float a = __uint_as_float(am);
        zero_lds = a < FLT_MIN;
        inv_lds = a < FLT_MIN ? 0.0f : 127.0f / a;
      }
    }
    __syncthreads();  // B0
    if (abort_) return;

    // ---- 1. codes (column gt + kGT*i), LoRA down row j = wg, bit-planes ---
    int q[kPollVals];
    if (active) {
      if (l == 0) {
#pragma unroll
        for (int i = 0; i < kPollVals; ++i) {
          const int k = gt + i * kGT;
          const int c = gload1s(q0 + (k < K ? k : 0));
          q[i] = k < K ? c : 0;
        }
      } else {
        const float inv = inv_lds;
        const bool zero = zero_lds;
        const uint64_t* src = y_ll + layers[l - 1].y_off;
        const uint32_t tag = tag_of(l - 1);
        uint64_t wd[kPollVals];
#pragma unroll
        for (int i = 0; i < kPollVals; ++i)
          wd[i] = gt + i * kGT < K ? ll_load_cached(src + gt + i * kGT) : ((uint64_t)tag << 32);
#pragma unroll
        for (int i = 0; i < kPollVals; ++i) {
          // normally valid on the first read (its producer's done word was
          // seen); a word whose store is not visible yet is polled again
          if ((uint32_t)(wd[i] >> 32) != tag && !poll_ll(src + gt + i * kGT, tag, wd[i], status, 4u))
            abort_ = 1;
          q[i] = (zero || gt + i * kGT >= K) ? 0 : (int)code(__uint_as_float((uint32_t)wd[i]), inv);
        }
      }
      if (wg < r) {  // acc_a[wg]: per-wave partials summed in LDS, last wave publishes
        int acc = 0;
#pragma unroll
        for (int i = 0; i < kPollVals; ++i) acc += pf.a[i] * q[i];
        acc = wave_sum(acc);
        if (lane == 0) {
          dot_part[wave] = acc;
          const int old = __hip_atomic_fetch_add(&cnt_dot, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
          if (old == kGW - 1) {
            int tot = 0;
#pragma unroll
            for (int w = 0; w < kGW; ++w) tot += __hip_atomic_load(&dot_part[w], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            ll_store(acc_ll + ((int64_t)l * dfssm::kMaxRank + wg) * kPad, tag_of(l), (uint32_t)tot);
            cnt_dot = 0;
          }
        }
      }
      // wave `wave` holds columns kGT*i + 64*wave + lane: one ballot per plane
#pragma unroll
      for (int i = 0; i < kPollVals; ++i) {
        if (i * kGT < K) {  // uniform
          uint64_t mk[8];
#pragma unroll
          for (int b = 0; b < 8; ++b) mk[b] = __ballot((q[i] >> b) & 1);
          if (lane < 16) {
            const int b = lane >> 1, h = lane & 1;
            uint64_t m = mk[0];
#pragma unroll
            for (int t = 1; t < 8; ++t) m = (b == t) ? mk[t] : m;
            const int word = (i * kGT + wave * 64) / 32 + h;
            reinterpret_cast<uint32_t*>(pl_lds)[((word >> 2) * 8 + b) * 4 + (word & 3)] = (uint32_t)(m >> (32 * h));
          }
        }
      }
    }
    __syncthreads();  // B2
    if (abort_) return;

    // ---- 2. scaffold GEMV on the prefetched rows; collect acc_a -----------
    const int RW = 64 / G;
    const int R = (N + nwg - 1) / nwg;
    const int steps = (R + kGW * RW - 1) / (kGW * RW);
    const int g = lane & (G - 1);
    int part[kMaxSteps];
    if (active) {
      // one bit-plane at a time: weight c_b = 2^b (b < 7), -128 (b = 7)
      const int C = K >> 7;
      int qpart = 0;
      int dsum[kMaxSteps];
#pragma unroll
      for (int st = 0; st < kMaxSteps; ++st) dsum[st] = 0;
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const uint4 Pb = g < C ? pl_lds[g * 8 + b] : make_uint4(0, 0, 0, 0);
        const int qc = __builtin_popcount(Pb.x) + __builtin_popcount(Pb.y) + __builtin_popcount(Pb.z) +
                       __builtin_popcount(Pb.w);
        qpart += b < 7 ? (qc << b) : -(qc << 7);
#pragma unroll
        for (int st = 0; st < kMaxSteps; ++st) {
          const uint4 w = pf.w[st];
          const int c = __builtin_popcount(w.x & Pb.x) + __builtin_popcount(w.y & Pb.y) +
                        __builtin_popcount(w.z & Pb.z) + __builtin_popcount(w.w & Pb.w);
          dsum[st] += b < 7 ? (c << b) : -(c << 7);
        }
      }
#pragma unroll
      for (int st = 0; st < kMaxSteps; ++st)
        part[st] = st < steps ? group_sum(2 * dsum[st] - qpart, G) : 0;
      if (gt < r) {
        uint64_t wd;
        if (!poll_ll(acc_ll + ((int64_t)l * dfssm::kMaxRank + gt) * kPad, tag_of(l), wd, status, 2u)) abort_ = 1;
        reinterpret_cast<int32_t*>(acc_lds)[gt] = (int32_t)(uint32_t)wd;
      }
    }
    __syncthreads();  // B3
    if (abort_) return;

    // ---- 3. LoRA up-projection, epilogue, publish; prefetch linear l+2 ----
    if (active) {
      const int r4 = (r + 3) >> 2;
      const int grp = lane / G;
      const int n0 = wg * R, n1 = min(N, n0 + R);
      const int Knext = l + 1 < L ? layers[l + 1].K : 0;
      // limbs of acc_a[4g .. 4g+3], packed per limb (j >= r read as 0)
      uint32_t lb0 = 0, lb1 = 0, lb2 = 0, lb3 = 0;
      if (r > 0 && g < r4) {
        const int4 a4 = acc_lds[g];
        const int av[4] = {a4.x, a4.y, a4.z, a4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          int8_t d[4];
          dfssm_dev::split_limbs(4 * g + e < r ? av[e] : 0, d);
          lb0 |= (uint32_t)(uint8_t)d[0] << (8 * e);
          lb1 |= (uint32_t)(uint8_t)d[1] << (8 * e);
          lb2 |= (uint32_t)(uint8_t)d[2] << (8 * e);
          lb3 |= (uint32_t)(uint8_t)d[3] << (8 * e);
        }
      }
      uint32_t ymax = 0;  // |y| of this lane's rows below Knext, as bits
#pragma unroll
      for (int st = 0; st < kMaxSteps; ++st) {
        if (st >= steps) break;
        int elo = 0, ehi = 0;
        if (r > 0) {
          const uint32_t bw = pf.b[st];
          elo = group_sum(sdot4(bw, lb0, 0) + (sdot4(bw, lb1, 0) << 8), G);
          ehi = group_sum(sdot4(bw, lb2, 0) + (sdot4(bw, lb3, 0) << 8), G);
        }
        const int n = n0 + st * kGW * RW + wave * RW + grp;
        if (g == 0 && n < n1) {
          const float y = dfssm_dev::epilogue(s, pf.al[st], pf.be[st], part[st], ehi, elo, r > 0);
          ll_store(y_ll + Ld.y_off + n, tag_of(l), __float_as_uint(y));
          y_all[Ld.y_off + n] = y;
          if (n < Knext) ymax = max(ymax, __float_as_uint(fabsf(y)));
        }
      }
      if (l + 1 < L) {  // done word: last wave to finish publishes the workgroup's max
        ymax = wave_max_bits(ymax);
        if (lane == 0) {
          __hip_atomic_fetch_max(&ymax_lds, ymax, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          const int old = __hip_atomic_fetch_add(&cnt_epi, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
          if (old == kGW - 1) {
            const uint32_t m = __hip_atomic_load(&ymax_lds, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            ll_store(done_ll + ((int64_t)l * nwg + wg) * kPad, tag_of(l), m);
            ymax_lds = 0;
            cnt_epi = 0;
          }
        }
      }
      if (l + 2 < L) prefetch(layers[l + 2], wg, nwg, gt, pf);
    }
    // the next linear's B0 orders every LDS reuse
  }
}

// Writes a chunk of the layer table and zeroes the exchange region.
struct SetupArgs {
  dfssm::ChainLayerDev e[dfssm::kChainSetupChunk];
  dfssm::ChainLayerDev* table;
  uint64_t* zero_base;
  int64_t zero_words;
  uint64_t* hash_dst;
  uint64_t hash;
  int first, count;
};

__global__ void chain_setup(SetupArgs a) {
  const int64_t i0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i0 < a.count) a.table[a.first + i0] = a.e[i0];
  for (int64_t i = i0; i < a.zero_words; i += (int64_t)gridDim.x * blockDim.x) a.zero_base[i] = 0;
  if (a.hash_dst && i0 == 0) *a.hash_dst = a.hash;
}

}  // namespace

namespace dfssm {

int chain_lanes_per_row(int64_t K) {
  const int64_t C = K / 128;
  int G = 8;
  while (G < C && G < 64) G *= 2;
  return G;
}

int chain_grid() { return 256; }  // one workgroup per CU; the done-word poll assumes <= 256

bool chain_persistent_supported(const dfssm_layer* layers, int n_layers, int64_t M, int nwg) {
  if (M != 1) return false;
  for (int l = 0; l < n_layers; ++l) {
    const dfssm_layer& L = layers[l];
    if (L.K % 128 != 0 || L.K > kChainMaxK || L.r % 4 != 0 || L.r > nwg) return false;
    const int G = chain_lanes_per_row(L.K);
    if (L.r / 4 > G) return false;
    const int64_t R = ceil_div(L.N, nwg);
    if (ceil_div(R, kChainWaves * (64 / G)) > kChainMaxSteps) return false;
  }
  return true;
}

hipError_t launch_chain_setup(const ChainLayerDev* table_host, ChainLayerDev* table_dev, int n_layers,
                              uint64_t* exch, int64_t exch_words, uint64_t* hash_dev, uint64_t hash,
                              hipStream_t st) {
  for (int first = 0; first < n_layers; first += kChainSetupChunk) {
    SetupArgs a{};
    a.count = n_layers - first < kChainSetupChunk ? n_layers - first : kChainSetupChunk;
    for (int i = 0; i < a.count; ++i) a.e[i] = table_host[first + i];
    a.table = table_dev;
    a.first = first;
    a.zero_base = exch;
    a.zero_words = first == 0 ? exch_words : 0;
    // the last chunk publishes the table's fingerprint (stream order puts it
    // after every chunk)
    a.hash_dst = first + kChainSetupChunk >= n_layers ? hash_dev : nullptr;
    a.hash = hash;
    chain_setup<<<dim3(first == 0 ? 256 : 1), dim3(256), 0, st>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_chain_run(const ChainLayerDev* table_dev, int n_layers, const int8_t* q0, const float* s0,
                            uint64_t* y_ll, uint64_t* acc_ll, uint64_t* done_ll, float* y_all,
                            unsigned* status, uint32_t seq, const uint64_t* hash_dev, uint64_t hash,
                            hipStream_t st) {
  int L = n_layers;
  void* args[] = {(void*)&table_dev, (void*)&L,      (void*)&q0,       (void*)&s0,
                  (void*)&y_ll,      (void*)&acc_ll, (void*)&done_ll,  (void*)&y_all,
                  (void*)&status,    (void*)&seq,    (void*)&hash_dev, (void*)&hash};
  return hipLaunchCooperativeKernel((const void*)chain_persistent, dim3(chain_grid()), dim3(kCT), args, 0, st);
}

}  // namespace dfssm
