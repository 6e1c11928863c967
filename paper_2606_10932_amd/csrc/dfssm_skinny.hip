// dfssm_skinny.hip -- scaffold + LoRA linear for a few tokens (M <= 32) on
// the gfx950 int8 matrix cores (v_mfma_i32_16x16x64_i8).
//
// At 5..32 tokens the product is still a contraction the matrix cores finish
// in a fraction of the time the sign bits take to stream, but it has too few
// token columns for the prefill tiling (128-token tiles, one long K-loop per
// block).  Here a workgroup owns 16 output rows and every token, and its
// waves split K:
//  * each lane loads, before any arithmetic, 16*S consecutive columns of its
//    row's sign bits (S = 4: one 8-byte load; S = 8: one 16-byte load) and
//    the same columns of its token's codes, then runs S MFMAs per 16-token
//    tile.  Inside one MFMA the order of the 64 contracted columns is free as
//    long as both operands use the same order, so lane (row, kg) feeds
//    columns kc(kg) + 16v .. +15 at step v and token lane (m, kg) feeds the
//    same columns;
//  * the signs are expanded to {0,1} bytes in registers (nibble n -> bytes
//    (n * 0x00204081) & 0x01010101), so the MFMA gives D = sum_{bit=1} Q and
//    acc_s = 2*D - sum_k Q;
//  * the waves' partial tiles are summed in LDS; one wave per token tile then
//    does the LoRA up-projection (four limb MFMAs: E_hi = 256*(B.L3) + B.L2,
//    E_lo = 256*(B.L1) + B.L0, exact int64 acc_b = E_lo + 65536*E_hi) and the
//    fp32 epilogue; its row operands were loaded at the start.
// One launch: the first nb_lora workgroups compute the LoRA down-projection
// acc_a = Q A^T (one wave per rank and 4 tokens) and sum_k Q, and publish
// them as 64-bit words {tag, value} (value: acc_a's 4 signed base-256 limbs
// as bytes, or sum Q) with agent-scope stores; a word is valid once its tag
// is the call's.  A call enqueued directly takes its tag from a host counter
// (bit 31 set).  A call captured into a graph would replay with a frozen
// argument, so there the tag is the call's epoch + 1 (below 2^31), kept on
// the device so that every replay moves it on.  Every reader and writer of the words (each publishing LoRA
// wave, each output workgroup) is a member of the call with an index i, and
// arrives once, at its start, with a 64-bit fetch-add on epoch word i % 64
// of the workspace ({epoch, arrivals}, one per 128-byte line, so that
// arrivals meet at 64 addresses and not one), which hands it the epoch;
// the last member to arrive on a word stores {epoch + 1, 0} there, and
// member 0 stores it into every word no member of this call uses.  All 64
// words start at {0, 0} and each call moves every one of them on by one,
// so all of one call agree on its epoch, the next call (stream-ordered
// after it) starts from the next one, and a word left by an earlier call
// never validates.
// The other workgroups read the words they need after their scaffold
// product.  The wait is bounded:
// a lane whose words have not arrived after `spin` polls computes the values
// itself from A and Q (the integers are the same either way), so no
// workgroup depends on another being scheduled.
#include <algorithm>
#include <atomic>

#include "dfssm_int4.hpp"
#include "dfssm_persist.hpp"

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4i mfma(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ v4i zero4() { return v4i{0, 0, 0, 0}; }

// bits [sh, sh+16) of w -> 16 bytes of {0,1}, byte b of dword t = bit sh+4t+b
__device__ __forceinline__ v4i expand16_at(uint32_t w, uint32_t sh) {
  v4i o;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const uint32_t nib = __builtin_amdgcn_ubfe(w, sh + 4 * t, 4);
    o[t] = (int)((nib * 0x00204081u) & 0x01010101u);
  }
  return o;
}

__device__ __forceinline__ v4i load16(const int8_t* p) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  return v4i{(int)u.x, (int)u.y, (int)u.z, (int)u.w};
}

// 16 bytes of an int8 row, zero outside [0, len)
__device__ __forceinline__ v4i load16_guarded(const int8_t* row, int start, int len, bool aligned) {
  if (start + 16 <= len && aligned) return load16(row + start);
  v4i o = zero4();
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int i = start + e;
    const uint32_t b = (i >= 0 && i < len) ? (uint32_t)(uint8_t)row[i] : 0u;
    o[e >> 2] |= (int)(b << (8 * (e & 3)));
  }
  return o;
}

// int4 factors: two's-complement nibbles, value 2i in the low nibble of byte
// i.  sext_nibbles turns 4 bytes holding nibble values 0..15 into the
// signed values -8..7 (XOR 8, then a subtraction that cannot borrow across
// bytes); expand_i4 turns 8 packed bytes into the 16 int8 values in order.
__device__ __forceinline__ uint32_t sext_nibbles(uint32_t t) {
  t ^= 0x08080808u;
  return ((t | 0x80808080u) - 0x08080808u) ^ 0x80808080u;
}

__device__ __forceinline__ uint4 expand_i4(uint2 p) {
  const uint32_t lo0 = p.x & 0x0F0F0F0Fu, hi0 = (p.x >> 4) & 0x0F0F0F0Fu;
  const uint32_t lo1 = p.y & 0x0F0F0F0Fu, hi1 = (p.y >> 4) & 0x0F0F0F0Fu;
  // v_perm_b32 interleaves the low-nibble and high-nibble bytes
  return make_uint4(sext_nibbles(__builtin_amdgcn_perm(hi0, lo0, 0x05010400u)),
                    sext_nibbles(__builtin_amdgcn_perm(hi0, lo0, 0x07030602u)),
                    sext_nibbles(__builtin_amdgcn_perm(hi1, lo1, 0x05010400u)),
                    sext_nibbles(__builtin_amdgcn_perm(hi1, lo1, 0x07030602u)));
}

// values start .. start+15 (start % 16 == 0) of a factor row, in bytes
// (L4: 8 packed bytes at start/2)
template <bool L4>
__device__ __forceinline__ uint4 load_row16(const int8_t* row, int start) {
  if constexpr (L4) return expand_i4(*reinterpret_cast<const uint2*>(row + start / 2));
  return *reinterpret_cast<const uint4*>(row + start);
}

// 16 values of a factor row of len values, zero outside [0, len)
template <bool L4>
__device__ __forceinline__ v4i load16_row_guarded(const int8_t* row, int start, int len, bool aligned) {
  if constexpr (!L4) {
    return load16_guarded(row, start, len, aligned);
  } else {
    if (start + 16 <= len && aligned) {
      const uint4 u = load_row16<true>(row, start);
      return v4i{(int)u.x, (int)u.y, (int)u.z, (int)u.w};
    }
    v4i o = zero4();
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int i = start + e;
      uint32_t b = 0u;
      if (i >= 0 && i < len) {
        const int byte = (uint8_t)row[i >> 1];
        const int nib = (i & 1) ? (byte >> 4) : (byte & 15);
        b = (uint32_t)(uint8_t)(int8_t)(nib >= 8 ? nib - 16 : nib);
      }
      o[e >> 2] |= (int)(b << (8 * (e & 3)));
    }
    return o;
  }
}

constexpr int kMaxWaves = 8;

struct SkinnyArgs {
  const int8_t* q;
  const float* s;
  int M, K, N, r, rp;
  const uint32_t* w_bits;
  const float* alpha;
  const int8_t* A;
  const int8_t* B;
  const float* beta;
  float* y;
  int32_t* acc_s_out;
  int64_t* acc_b_out;
  int32_t* acc_a;  // [M][r], written by the LoRA workgroups (and by fallback lanes)
  uint64_t* xw;    // [xcopies][xstride]: [M][rp] limb words, then [M] sum-Q words
  int64_t xstride; // M * rp + M, rounded up to 32 words
  int xcopies;     // 8: one copy per XCD (every output workgroup reads the same
                   // words, so the copies spread its polls) at r > 32 when they
                   // fit; else 1
  uint64_t* epoch; // kEpochGroups words {epoch:32, arrivals:32}, kEpochStride apart;
                   // NULL: the call's tag is host_tag
  uint32_t host_tag;
  int arrivals;    // members per call: publishing LoRA waves, then output workgroups
  int lora_members;  // publishing LoRA waves (members 0 .. lora_members - 1)
  int nb_lora;     // LoRA workgroups at the front of the grid
  int spin;        // polls of a missing word before computing it locally
};


__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}

// whole-wave sum, the total in every lane (DPP inside 16-lane rows, then
// gfx950's permlane swaps across rows and halves)
__device__ __forceinline__ int wave_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);  // row_mirror
  auto p = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
  v = (int)(p[0] + p[1]);
  p = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
  return (int)(p[0] + p[1]);
}

// agent scope: the words cross XCDs (each XCD has its own L2)
__device__ __forceinline__ void word_store(uint64_t* p, uint32_t tag, uint32_t v) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t word_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t pack_limbs(int32_t v) {
  int8_t d[4];
  dfssm_dev::split_limbs(v, d);
  return (uint32_t)(uint8_t)d[0] | ((uint32_t)(uint8_t)d[1] << 8) | ((uint32_t)(uint8_t)d[2] << 16) |
         ((uint32_t)(uint8_t)d[3] << 24);
}

// sum_k A[j,k] Q[m,k] (j < r) or sum_k Q[m,k] (j < 0), one lane alone
template <bool L4>
__device__ int lane_dot(const int8_t* __restrict__ A, const int8_t* __restrict__ q, int K, int j, int m) {
  const int8_t* qrow = q + (int64_t)m * K;
  const int8_t* arow = A + (int64_t)(j < 0 ? 0 : j) * (L4 ? K / 2 : K);
  int acc = 0;
  for (int k = 0; k < K; k += 16) {
    const uint4 x = *reinterpret_cast<const uint4*>(qrow + k);
    const uint4 w = j < 0 ? make_uint4(0x01010101u, 0x01010101u, 0x01010101u, 0x01010101u)
                          : load_row16<L4>(arow, k);
    acc = sdot4(w.x, x.x, acc);
    acc = sdot4(w.y, x.y, acc);
    acc = sdot4(w.z, x.z, acc);
    acc = sdot4(w.w, x.w, acc);
  }
  return acc;
}

// LoRA workgroup: wave w takes item b*nw + w = (token group of 4, rank j);
// the wave of rank 0 also sums Q.  Every 16-byte load of a 4 KB column batch
// is issued before the first v_dot4.
constexpr int kPrepTokens = 4;
constexpr int kPrepBatch = 4;
template <bool L4>
__device__ void lora_block(const SkinnyArgs& a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nw = blockDim.x >> 6;
  const int M = a.M, K = a.K, r = a.r, rp = a.rp;
  const int item = (int)blockIdx.x * nw + wave;
  const int j = item % rp, m0 = (item / rp) * kPrepTokens;
  if (m0 >= M) return;
  // a publishing wave arrives once, at its start (device-epoch calls); the
  // epoch is needed only when it publishes
  uint64_t ep_old = 0;
  if (a.epoch && lane == 0) ep_old = dfssm_dev::arrive(a.epoch, item);
  const int mt = min(kPrepTokens, M - m0);
  const bool jr = j < r, qsum = j == 0;
  int acc[kPrepTokens], qs[kPrepTokens];
#pragma unroll
  for (int m = 0; m < kPrepTokens; ++m) acc[m] = qs[m] = 0;
  if (jr || qsum) {
    const int8_t* arow = a.A + (int64_t)(jr ? j : 0) * (L4 ? K / 2 : K);
    for (int kb = 0; kb < K; kb += 1024 * kPrepBatch) {
      // int4: the packed bytes are kept as loaded and expanded at their use,
      // so no expansion waits on a load before the batch's last load issues
      uint4 av[kPrepBatch], x[kPrepTokens][kPrepBatch];
      uint2 araw[kPrepBatch];
#pragma unroll
      for (int u = 0; u < kPrepBatch; ++u) {
        const int k = kb + 1024 * u + 16 * lane;
        const bool ok = k < K;  // K % 32 == 0: a 16-byte chunk is wholly in or out
        if constexpr (L4)
          araw[u] = (jr && ok) ? *reinterpret_cast<const uint2*>(arow + k / 2) : make_uint2(0, 0);
        else
          av[u] = (jr && ok) ? load_row16<false>(arow, k) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int m = 0; m < kPrepTokens; ++m)
          x[m][u] = (ok && m < mt) ? *reinterpret_cast<const uint4*>(a.q + (int64_t)(m0 + m) * K + k)
                                   : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < kPrepBatch; ++u) {
        if constexpr (L4) av[u] = expand_i4(araw[u]);
#pragma unroll
        for (int m = 0; m < kPrepTokens; ++m) {
          acc[m] = sdot4(av[u].x, x[m][u].x, acc[m]);
          acc[m] = sdot4(av[u].y, x[m][u].y, acc[m]);
          acc[m] = sdot4(av[u].z, x[m][u].z, acc[m]);
          acc[m] = sdot4(av[u].w, x[m][u].w, acc[m]);
          if (qsum) {
            qs[m] = sdot4(0x01010101u, x[m][u].x, qs[m]);
            qs[m] = sdot4(0x01010101u, x[m][u].y, qs[m]);
            qs[m] = sdot4(0x01010101u, x[m][u].z, qs[m]);
            qs[m] = sdot4(0x01010101u, x[m][u].w, qs[m]);
          }
        }
      }
    }
  }
  int mine = 0, mine_q = 0;
#pragma unroll
  for (int m = 0; m < kPrepTokens; ++m) {
    if (m < mt) {  // uniform
      const int t = wave_sum(acc[m]);
      mine = lane == m ? t : mine;
      if (qsum) {
        const int tq = wave_sum(qs[m]);
        mine_q = lane == m ? tq : mine_q;
      }
    }
  }
  const uint64_t old = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(ep_old >> 32)) << 32) |
                       (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)ep_old);
  const uint32_t tag = a.epoch ? dfssm_dev::epoch_tag(old) : a.host_tag;
  if (a.xcopies == 1) {
    if (lane < mt) {
      const int m = m0 + lane;
      if (jr) a.acc_a[(int64_t)m * r + j] = mine;
      word_store(a.xw + (int64_t)m * rp + j, tag, pack_limbs(mine));  // zero limbs for ranks in [r, rp)
      if (qsum) word_store(a.xw + (int64_t)M * rp + m, tag, (uint32_t)mine_q);
    }
  } else {
    // lane c*mt + i stores token m0 + i's words into copy c (lane i holds
    // them).  Every instruction here delays the words: this branch's
    // shuffles cost the single copy ~0.3 us a call at r = 16, and a lane
    // modulo in their place cost more.
    const int src = lane % mt;
    const int vm = __shfl(mine, src, 64), vq = __shfl(mine_q, src, 64);
    if (lane < mt && jr) a.acc_a[(int64_t)(m0 + lane) * r + j] = mine;
    if (lane < mt * a.xcopies) {
      const int cpy = lane / mt, m = m0 + (lane - cpy * mt);
      uint64_t* xc = a.xw + (int64_t)cpy * a.xstride;
      word_store(xc + (int64_t)m * rp + j, tag, pack_limbs(vm));  // zero limbs for ranks in [r, rp)
      if (qsum) word_store(xc + (int64_t)M * rp + m, tag, (uint32_t)vq);
    }
  }
  if (a.epoch && lane == 0) dfssm_dev::advance_if_last(a.epoch, item, old, a.arrivals);
}

// The limbs of acc_a[m][j0 + 16kg .. +15] as 4 limb operands (byte e of limb
// t = limb t of rank j0 + 16kg + e) and, when sq is given, sum Q of token m, for
// the lane (rho, kg) of the wave that finishes the token tile starting at t0
// (m = min(t0 + rho, M - 1)): from the LoRA workgroups' words, or computed
// here once `spin` polls have passed.  CP: the words come in one copy per
// XCD, and this wave polls its XCD's copy.
//   - CP and at most NC distinct tokens in the tile (nt): the polls are
//     token-major.  Lane L reads rank j0 + L of each token (one 512-byte
//     load per token), lanes below nt read the sum-Q words, and the words
//     reach their lanes through the wave's LDS tile wx [NC][kWxPitch] (sq:
//     wq [NC]).  More tokens per round hold more loads in registers: 16
//     took 31 more VGPRs (a wave per SIMD), and 4 gave the int4 kernel a
//     stack frame; NC = 4 (int8 factors) or 2 (int4).
//   - otherwise each lane polls its own 16 words and keeps them once in.
constexpr int kWxPitch = 68;  // words per token row of wx (16 bytes of skew)
constexpr int kCoalTokens = 4;

// Token-major polls of n <= NC consecutive tokens from tok0 (tok0 + n <= M)
// in the copy xc: lane L reads rank j0 + L of each, lanes below n the sum-Q
// words (want_sq).  On success the words are in wx rows 0 .. n-1 and wq[0 ..
// n-1]; false once `spin` polls have passed without all of them.
template <int NC>
__device__ bool poll_tokens(const SkinnyArgs& a, uint32_t tag, const uint64_t* xc, int tok0, int n, int j0,
                            bool want_sq, uint32_t* wx, int* wq) {
  const int lane = threadIdx.x & 63;
  const int rp = a.rp;
  const uint64_t* wp = xc + (int64_t)tok0 * rp + j0 + lane;
  const uint64_t* sp = xc + (int64_t)a.M * rp + tok0 + min(lane, n - 1);
  for (int it = 0;; ++it) {
    uint64_t w[NC], wqv = 0;
#pragma unroll
    for (int i = 0; i < NC; ++i)
      if (i < n) w[i] = word_load(wp + (int64_t)i * rp);  // n is uniform
    if (want_sq) wqv = word_load(sp);
    bool ok = !want_sq || (uint32_t)(wqv >> 32) == tag;
#pragma unroll
    for (int i = 0; i < NC; ++i)
      if (i < n) ok = ok && (uint32_t)(w[i] >> 32) == tag;
    if (__all(ok)) {
#pragma unroll
      for (int i = 0; i < NC; ++i)
        if (i < n) wx[i * kWxPitch + lane] = (uint32_t)w[i];
      if (want_sq && lane < n) wq[lane] = (int)(uint32_t)wqv;
      return true;
    }
    if (it >= a.spin) return false;
    __builtin_amdgcn_s_sleep(2);
  }
}

// pre: 0 poll here; 1 the tile's words are already in wx / wq (the
// workgroup's waves polled them together); 2 those polls gave up.
template <bool L4, bool CP>
__device__ void fetch_lora(const SkinnyArgs& a, uint32_t tag, int t0, int j0, int rho, int kg, uint32_t* wx,
                           int* wq, v4i (&lm)[4], int* sq, bool store_acc, int pre) {
  const int lane = threadIdx.x & 63;
  const int M = a.M, rp = a.rp;
  const int nt = max(1, min(16, M - t0));  // distinct tokens of the tile (tokens past M repeat M - 1)
  const int m = min(t0 + min(rho, nt - 1), M - 1);
  const uint64_t* xc = CP ? a.xw + (int64_t)dfssm_px::xcc_id() * a.xstride : a.xw;
  constexpr int NC = L4 ? 2 : kCoalTokens;
  uint32_t val[16], vq = 0;
  bool have = false;
  if (CP && (pre != 0 || nt <= NC)) {  // uniform
    if (pre == 0)
      have = poll_tokens<NC>(a, tag, xc, min(t0, M - 1), nt, j0, sq != nullptr, wx, wq);
    else
      have = pre == 1;
    if (have) {
      // the LDS writes above and these reads are the same wave's, in order
      __builtin_amdgcn_wave_barrier();
      const int rt = min(rho, nt - 1);
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        const uint4 u = *reinterpret_cast<const uint4*>(wx + rt * kWxPitch + 16 * kg + 4 * d);
        val[4 * d] = u.x; val[4 * d + 1] = u.y; val[4 * d + 2] = u.z; val[4 * d + 3] = u.w;
      }
      if (sq) vq = (uint32_t)wq[rt];
      __builtin_amdgcn_wave_barrier();  // wx is written again by the next chunk's call
    }
  } else {
    const uint64_t* wp = xc + (int64_t)m * rp + j0 + 16 * kg;
    const uint64_t* sp = xc + (int64_t)M * rp + m;
    for (int it = 0;; ++it) {
      if (!have) {
        uint64_t w[16], wqv = 0;
#pragma unroll
        for (int e = 0; e < 16; ++e) w[e] = word_load(wp + e);
        if (sq) wqv = word_load(sp);
        bool ok = !sq || (uint32_t)(wqv >> 32) == tag;
#pragma unroll
        for (int e = 0; e < 16; ++e) ok = ok && (uint32_t)(w[e] >> 32) == tag;
        if (ok) {
#pragma unroll
          for (int e = 0; e < 16; ++e) val[e] = (uint32_t)w[e];
          vq = (uint32_t)wqv;
          have = true;
        }
      }
      if (__all(have) || it >= a.spin) break;
      __builtin_amdgcn_s_sleep(2);
    }
  }
  if (!have) {
    // the LoRA workgroups' words did not arrive: compute them here
#pragma unroll 1
    for (int e = 0; e < 16; ++e) {
      const int j = j0 + 16 * kg + e;
      const int v = j < a.r ? lane_dot<L4>(a.A, a.q, a.K, j, m) : 0;
      val[e] = pack_limbs(v);
      if (store_acc && j < a.r) a.acc_a[(int64_t)m * a.r + j] = v;
    }
    if (sq) vq = (uint32_t)lane_dot<L4>(a.A, a.q, a.K, -1, m);
  }
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      uint32_t o = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) o |= ((val[4 * d + b] >> (8 * t)) & 0xffu) << (8 * b);
      lm[t][d] = (int)o;
    }
  if (sq) *sq = (int)vq;
}

// MT token tiles of 16 (M <= 16*MT); S MFMA steps per lane per iteration;
// PM: how the output waves get the LoRA words: 0 from one copy, lane by
// lane; 1 from their XCD's copy (a.xcopies == 8), the finishing wave alone;
// 2 (MT == 1) from their XCD's copy, several waves together.
// Block: 16 output rows, nw = blockDim.x / 64 waves (nw >= MT), wave w takes
// iterations w, w + nw, ... of 64*S columns each.
template <int MT, int S, bool L4, int PM>
__global__ __launch_bounds__(64 * kMaxWaves) void mfma_skinny(SkinnyArgs a) {
  constexpr bool CP = PM > 0;
  __shared__ v4i red[kMaxWaves][MT][64];
  __shared__ __align__(16) uint32_t wx[MT][PM == 2 ? 16 * kWxPitch : (CP ? kCoalTokens * kWxPitch : 4)];
  __shared__ int wq[MT][PM == 2 ? 16 : (CP ? kCoalTokens : 1)];
  __shared__ int gok[PM == 2 ? kMaxWaves : 1];
  __shared__ uint32_t tag_lds;
  if ((int)blockIdx.x < a.nb_lora) {
    if (blockIdx.y == 0) lora_block<L4>(a);  // one set of LoRA workgroups for all tokens
    return;
  }
  // an output workgroup arrives once, at its start (device-epoch calls); the
  // epoch is needed only after the scaffold product
  const int member = a.lora_members + (int)blockIdx.y * (int)(gridDim.x - a.nb_lora) + ((int)blockIdx.x - a.nb_lora);
  uint64_t ep_old = 0;
  if (a.epoch && threadIdx.x == 0) ep_old = dfssm_dev::arrive(a.epoch, member);
  constexpr int KW = 64 * S;  // columns per wave iteration
  constexpr int SW = S / 2;   // sign words per lane per iteration
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nw = blockDim.x >> 6;
  const int rho = lane & 15, kg = lane >> 4;
  const int M = a.M, K = a.K, N = a.N, r = a.r, W = K >> 5;
  const int n0 = 16 * ((int)blockIdx.x - a.nb_lora);
  const int mb = 16 * MT * (int)blockIdx.y;  // first token of this block's chunk (row y of the grid)
  const int nrow = min(n0 + rho, N - 1);  // sign / B row of this lane (rows past N are never stored)
  const uint32_t* wrow = a.w_bits + (int64_t)nrow * W;
  const int nit = (K + KW - 1) / KW;
  const bool wvec = (W % SW) == 0;

  // ---- the row operands of the wave that finishes token tile `wave` go
  //      out first: B bytes of ranks 0..63, row scales, token scales
  const bool fin = wave < MT;
  const int mtok = mb + 16 * wave + rho;  // token of this lane in the finished tile
  const int mc = min(mtok, M - 1);
  const int nb = n0 + 4 * kg;  // this lane's output rows nb .. nb+3
  const bool ba = (r % 16) == 0;
  const int64_t bpitch = L4 ? r / 2 : r;  // bytes per B row
  // int4: the packed B bytes are held as loaded and expanded after the
  // scaffold loop, so the loop's loads do not wait for them
  v4i bop = zero4();
  uint2 braw = make_uint2(0, 0);
  bool bpacked = false;
  float alv[4] = {0.f, 0.f, 0.f, 0.f}, bev[4] = {0.f, 0.f, 0.f, 0.f};
  float sm = 0.f;
  if (fin) {
    if (r > 0) {
      if (L4 && 16 * kg + 16 <= r && ba) {
        braw = *reinterpret_cast<const uint2*>(a.B + (int64_t)nrow * bpitch + 8 * kg);
        bpacked = true;
      } else {
        bop = load16_row_guarded<L4>(a.B + (int64_t)nrow * bpitch, 16 * kg, r, ba);
      }
    }
    if ((N & 3) == 0 && nb + 3 < N) {
      const float4 al4 = *reinterpret_cast<const float4*>(a.alpha + nb);
      alv[0] = al4.x; alv[1] = al4.y; alv[2] = al4.z; alv[3] = al4.w;
      if (r > 0) {
        const float4 be4 = *reinterpret_cast<const float4*>(a.beta + nb);
        bev[0] = be4.x; bev[1] = be4.y; bev[2] = be4.z; bev[3] = be4.w;
      }
    } else {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int n = min(nb + v, N - 1);
        alv[v] = a.alpha[n];
        bev[v] = r > 0 ? a.beta[n] : 0.f;
      }
    }
    sm = a.s[mc];
  }

  // ---- scaffold: this wave's share of K
  v4i acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = zero4();
  for (int it = wave; it < nit; it += nw) {
    const int kc = it * KW + kg * 16 * S;  // first column of this lane (a multiple of 64)
    const int wd0 = kc >> 5;
    uint32_t sw[SW];
    if (wvec && wd0 + SW <= W) {
      if constexpr (S == 8) {
        const uint4 t = *reinterpret_cast<const uint4*>(wrow + wd0);
        sw[0] = t.x; sw[1] = t.y; sw[2] = t.z; sw[3] = t.w;
      } else {
        const uint2 t = *reinterpret_cast<const uint2*>(wrow + wd0);
        sw[0] = t.x; sw[1] = t.y;
      }
    } else {
      // signs past K meet zero codes; only the load has to stay in the row
#pragma unroll
      for (int i = 0; i < SW; ++i) sw[i] = wd0 + i < W ? wrow[wd0 + i] : 0u;
    }
    v4i x[MT][S];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int m = mb + 16 * i + rho;
      const int8_t* qrow = a.q + (int64_t)min(m, M - 1) * K;
#pragma unroll
      for (int v = 0; v < S; ++v) {
        const int col = kc + 16 * v;  // K % 32 == 0: 16 columns are wholly in or out
        x[i][v] = (m < M && col < K) ? load16(qrow + col) : zero4();
      }
    }
#pragma unroll
    for (int v = 0; v < S; ++v) {
      const v4i sg = expand16_at(sw[v >> 1], 16 * (v & 1));
#pragma unroll
      for (int i = 0; i < MT; ++i) acc[i] = mfma(sg, x[i][v], acc[i]);
    }
  }

  // ---- sum the waves' partial tiles; wave i finishes token tile i
#pragma unroll
  for (int i = 0; i < MT; ++i) red[wave][i][lane] = acc[i];
  if (threadIdx.x == 0) {
    if (a.epoch) {
      tag_lds = dfssm_dev::epoch_tag(ep_old);
      dfssm_dev::advance_if_last(a.epoch, member, ep_old, a.arrivals);
    } else {
      tag_lds = a.host_tag;
    }
  }
  __syncthreads();
  const uint32_t tag = tag_lds;
  // with more tokens than one wave's polls take (G), the first ceil(n / G)
  // waves of a one-tile workgroup each poll G tokens into the tile's LDS
  // rows, and all meet at a barrier (one wave holding 16 tokens' loads
  // would take 31 more VGPRs)
  int pre = 0;
  if constexpr (PM == 2 && MT == 1) {
    {
      constexpr int G = L4 ? 2 : kCoalTokens;
      const int ntk = max(1, min(16, M - mb));
      const int ng = (ntk + G - 1) / G;  // <= nw (host)
      if (wave < ng) {
        const uint64_t* xc = a.xw + (int64_t)dfssm_px::xcc_id() * a.xstride;
        const int t = G * wave, n = min(G, ntk - t);
        const bool ok = poll_tokens<G>(a, tag, xc, mb + t, n, 0, true, wx[0] + t * kWxPitch, wq[0] + t);
        if (lane == 0) gok[wave] = ok ? 1 : 0;
      }
      __syncthreads();
      pre = 1;
      for (int w = 0; w < ng; ++w)
        if (gok[w] == 0) pre = 2;
    }
  }
  if (!fin) return;
  v4i d = red[0][wave][lane];
  for (int w = 1; w < nw; ++w) d += red[w][wave][lane];

  // LoRA limbs of ranks 0..63 and sum Q of this lane's token; the first
  // block of each tile row also keeps acc_a for the caller if its words had
  // to be computed here
  v4i lm[4];
  int sq = 0;
  const bool keep = (int)blockIdx.x == a.nb_lora && mtok < M;
  fetch_lora<L4, CP>(a, tag, mb + 16 * wave, 0, rho, kg, wx[wave], wq[wave], lm, &sq, keep, pre);

  // LoRA up-projection, limbs 3, 2, 1, 0 over the 64-rank chunks
  if (L4 && bpacked) {
    // an opaque zero made after the polls: the expansion cannot be moved in
    // front of them, where it would wait for the B load before the first poll
    uint32_t z;
    asm volatile("v_mov_b32 %0, 0" : "=v"(z));
    braw.x ^= z;
    braw.y ^= z;
    const uint4 u = expand_i4(braw);
    bop = v4i{(int)u.x, (int)u.y, (int)u.z, (int)u.w};
  }
  v4i ehi = zero4(), elo = zero4();
  if (r > 0) {
    v4i e3 = mfma(bop, lm[3], zero4()), e2 = mfma(bop, lm[2], zero4());
    v4i e1 = mfma(bop, lm[1], zero4()), e0 = mfma(bop, lm[0], zero4());
    for (int j0 = 64; j0 < a.rp; j0 += 64) {
      const v4i bl = load16_row_guarded<L4>(a.B + (int64_t)nrow * bpitch, j0 + 16 * kg, r, ba);
      v4i lj[4];
      fetch_lora<L4, CP>(a, tag, mb + 16 * wave, j0, rho, kg, wx[wave], wq[wave], lj, nullptr, keep, 0);
      e3 = mfma(bl, lj[3], e3);
      e2 = mfma(bl, lj[2], e2);
      e1 = mfma(bl, lj[1], e1);
      e0 = mfma(bl, lj[0], e0);
    }
    ehi = (e3 << 8) + e2;
    elo = (e1 << 8) + e0;
  }

  // lane (rho, kg) holds D[row nb + v][token mtok]
  if (mtok >= M) return;
  float yv[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int32_t as = 2 * d[v] - sq;
    yv[v] = dfssm_dev::epilogue(sm, alv[v], bev[v], as, ehi[v], elo[v], r > 0);
    if (nb + v < N) {
      if (a.acc_s_out) a.acc_s_out[(int64_t)mtok * N + nb + v] = as;
      if (a.acc_b_out) a.acc_b_out[(int64_t)mtok * N + nb + v] = r > 0 ? (int64_t)elo[v] + ((int64_t)ehi[v] << 16) : 0;
    }
  }
  if (a.y) {
    float* dst = a.y + (int64_t)mtok * N + nb;
    if ((N & 3) == 0 && nb + 3 < N) {
      *reinterpret_cast<float4*>(dst) = make_float4(yv[0], yv[1], yv[2], yv[3]);
    } else {
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (nb + v < N) dst[v] = yv[v];
    }
  }
}

template <int MT, int S, bool L4, int PM>
hipError_t launch_t(const SkinnyArgs& a, int nw, hipStream_t st) {
  // x: LoRA workgroups then 16-row output blocks; y: 32-token chunks
  const int64_t blocks = a.nb_lora + dfssm::ceil_div(a.N, 16);
  const int64_t chunks = dfssm::ceil_div(a.M, 16 * MT);
  mfma_skinny<MT, S, L4, PM><<<dim3((unsigned)blocks, (unsigned)chunks), dim3(64 * nw), 0, st>>>(a);
  return hipGetLastError();
}

// the copy forms (PM > 0) are taken at M <= 8: one token tile
template <bool L4, int PM>
hipError_t launch_tiles(const SkinnyArgs& a, int mt, int S, int nw, hipStream_t st) {
  if (mt == 1) return S == 8 ? launch_t<1, 8, L4, PM>(a, nw, st) : launch_t<1, 4, L4, PM>(a, nw, st);
  if constexpr (PM == 0) {
    if (mt == 2) return S == 8 ? launch_t<2, 8, L4, PM>(a, nw, st) : launch_t<2, 4, L4, PM>(a, nw, st);
    return launch_t<4, 4, L4, PM>(a, nw, st);
  }
  return hipErrorInvalidValue;
}

// Tag of a call enqueued outside graph capture: a process-wide counter with
// bit 31 set, so it never equals a device-epoch tag (below 2^31) or 0.
uint32_t host_tag() {
  static std::atomic<uint32_t> seq{0};
  return 0x80000000u | (seq.fetch_add(1, std::memory_order_relaxed) & 0x7fffffffu);
}

}  // namespace

namespace {

using dfssm::ceil_div;

template <bool L4>
hipError_t skinny_impl(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N, int64_t r,
                       const uint32_t* w_bits, const float* alpha, const int8_t* A, const int8_t* B,
                       const float* beta, float* y, int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                       const dfssm::LinearWorkspace& ws, hipStream_t st) {
  using namespace dfssm;
  if (M == 0 || N == 0) return hipSuccess;
  if (M > kSkinnyChunkedMaxTokens) return hipErrorInvalidValue;
  const int rp = (int)rank_padded(r);
  // 16-byte sign loads (8 MFMA steps) once K gives 4 waves a full one each:
  // at K = 2048 the 1.3B in_proj's 532 workgroups of 4 waves then fit the
  // chip's slots in one round (8 waves of 8-byte loads would not)
  // above 32 tokens, output blocks of 64 tokens (4 token tiles, 8-byte sign
  // loads): each sign operand expanded once feeds 4 tiles (the 1.3B out_proj
  // at M = 256: 31.8 us against 41.3 with 32-token blocks)
  const int S = M > 32 ? 4 : (K >= 2048 ? 8 : 4);
  const int mt = M > 32 ? 4 : (M > 16 ? 2 : 1);
  const int64_t nit = ceil_div(K, 64 * S);
  const int nw = (int)std::max<int64_t>(mt, std::min<int64_t>(kMaxWaves, nit));
  // Test switch local_lora: no LoRA workgroups, every lane computes its LoRA
  // values itself at once (the path a lane takes when the words never
  // arrive).
  const bool local_only = test_switch(DFSSM_TEST_LOCAL_LORA) == 1;
  const int64_t lora_waves = ceil_div(M, kPrepTokens) * rp;
  const int nb_lora = local_only ? 0 : (int)ceil_div(lora_waves, nw);
  const int64_t out_blocks = ceil_div(N, 16) * ceil_div(M, 16 * mt);
  const int arrivals = (int)((local_only ? 0 : lora_waves) + out_blocks);
  // the call's tag: under graph capture from the device epoch (a replay
  // moves it on), otherwise from a host counter (no arrivals at all)
  // (if the query fails, the device epoch, which is right either way; the
  // failed query's error is cleared so that the launch check does not see it)
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(st, &cap) != hipSuccess) {
    (void)hipGetLastError();
    cap = hipStreamCaptureStatusActive;
  }
  const bool device_epoch = cap != hipStreamCaptureStatusNone;
  // One copy of the LoRA words per XCD, each on a 256-byte boundary (no
  // cache line holds words of two copies), when the LoRA down-projection
  // is the longer path (r > 32) at up to kCoalTokens tokens: every output
  // workgroup then waits on the words, and the copies took 1.2-2.3 us off
  // a call at M = 1 to 4 (1.3B projections, r = 64; int4 at M = 3, 4, where
  // the polls go lane by lane: 0.8 us).  At r <= 32 the words are mostly in
  // before the first poll, and from 5 tokens the lane-by-lane polls of one
  // copy were as fast or faster.
  // From G + 1 to 8 tokens (G = 4, or 2 with int4 factors) and one chunk of
  // 64 ranks, the copies are polled by ceil(M / G) waves together (1.3B,
  // r = 64, M = 5 / 8: in_proj 8.6 -> 7.4 / 8.4 -> 8.0 us, out_proj M = 8
  // 8.4 -> 7.7; int4 in_proj M = 4 / 8 8.6 -> 7.6 / ~10 -> 8.4).  At 16
  // tokens they were no faster than one copy polled lane by lane.
  const int64_t xstride = round_up(M * rp + M, 32);
  const int64_t gsize = L4 ? 2 : kCoalTokens;
  const bool group = rp == 64 && M > gsize && M <= 8 && ceil_div(M, gsize) <= nw;
  const int xcopies = r > 32 && (M <= kCoalTokens || group) && 8 * xstride <= kXwWords ? 8 : 1;
  SkinnyArgs a{q, s, (int)M, (int)K, (int)N, (int)r, rp, w_bits, alpha, A, B, beta, y, acc_s, acc_b,
               ws.acc_a, ws.xw, xstride, xcopies, device_epoch ? ws.epoch : nullptr, device_epoch ? 0u : host_tag(),
               arrivals, (int)(local_only ? 0 : lora_waves), nb_lora, local_only ? 0 : (1 << 14)};
  // the two poll forms are separate instantiations: in one kernel their
  // union of registers cost a wave per SIMD and spilled
  hipError_t e = xcopies == 1 ? launch_tiles<L4, 0>(a, mt, S, nw, st)
                 : group       ? launch_tiles<L4, 2>(a, mt, S, nw, st)
                               : launch_tiles<L4, 1>(a, mt, S, nw, st);
  if (e != hipSuccess) return e;
  if (acc_a_out && r > 0)
    e = hipMemcpyAsync(acc_a_out, ws.acc_a, (size_t)(M * r) * 4, hipMemcpyDeviceToDevice, st);
  return e;
}

}  // namespace

namespace dfssm {

hipError_t launch_skinny_linear(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                                int64_t r, const uint32_t* w_bits, const float* alpha,
                                const int8_t* A, const int8_t* B, const float* beta, float* y,
                                int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                                const LinearWorkspace& ws, hipStream_t st) {
  return skinny_impl<false>(q, s, M, K, N, r, w_bits, alpha, A, B, beta, y, acc_s, acc_a_out, acc_b, ws, st);
}

hipError_t launch_skinny_linear_i4(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                                   int64_t r, const uint32_t* w_bits, const float* alpha,
                                   const uint8_t* A4, const uint8_t* B4, const float* beta, float* y,
                                   int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                                   const LinearWorkspace& ws, hipStream_t st) {
  return skinny_impl<true>(q, s, M, K, N, r, w_bits, alpha, reinterpret_cast<const int8_t*>(A4),
                           reinterpret_cast<const int8_t*>(B4), beta, y, acc_s, acc_a_out, acc_b, ws, st);
}

}  // namespace dfssm
