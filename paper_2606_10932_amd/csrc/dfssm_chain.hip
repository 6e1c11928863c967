// dfssm_chain.hip -- persistent kernel for the re-quantising chain of
// scaffold + LoRA linears at one token (the decode step's projections run
// back to back, Sec. 4.1 of the paper, where a CUDA graph removes launch
// gaps; here one cooperative launch replaces the whole sequence).
//
// Every linear depends on all of the previous linear's output (its absmax
// and its LoRA down-projection are reductions over all of it), so the chain
// is bound by cross-CU communication latency, not by HBM.  The design:
//
//  * Data crosses workgroups as 64-bit words {tag:32, value:32}, so a
//    consumer polls the data itself: a word is valid once its tag equals
//    the linear's tag.  Tags carry the launch's epoch, kept on the device:
//    every workgroup arrives once, at its start, on the workspace's epoch
//    words (dfssm_dev::arrive, 64 words so that arrivals meet at 64
//    addresses), and each word's last arrival moves it on; so words left
//    from an earlier launch (or an earlier replay of a captured launch)
//    never validate.  No fences are used (on
//    MI355X a release/acquire pair costs ~3.5 us: it writes back and
//    invalidates the whole L2).
//  * Two levels of exchange.  MI355X has 8 XCDs, each with its own L2; a
//    cross-XCD word needs an agent-scope store and load (~0.9 us round
//    trip), a word inside one XCD only a store into that XCD's L2 and a
//    load that skips the CU's L1 (~0.6 us).  At start every workgroup reads
//    its XCD id (hardware register XCC_ID) and publishes it, so each knows
//    its rank rho among the n_x workgroups of its XCD.  Per linear:
//      - outputs y_{l-1} are stored once at agent scope (y_ll);
//      - workgroup rho of XCD x copies slice rho of y_{l-1}[0:K] from y_ll
//        into x's own region (y_rel[x]) as soon as each word is valid;
//      - every workgroup polls all of y_{l-1}[0:K] in its XCD's region
//        (L2 hits): 1/n_x of the cross-XCD polling traffic of reading y_ll
//        directly;
//      - the LoRA down-projection is computed inside each XCD: workgroup
//        rho computes acc_a[j] for j = rho + n_x*t (t < kChainAccRows) and
//        stores it into x's region, so acc_a never crosses an XCD.
//  * A workgroup is two groups of 8 waves that alternate roles: while one
//    group computes linear l, the other loads the weights of linear l+1
//    into its own registers, once the bit-planes of linear l are built.  A
//    wave's loads complete in order, so a latency-critical wait (a poll)
//    never sits behind a weight load issued shortly before it.
//  * Per linear: the active group relays its slice; all 16 waves poll their
//    words of y_{l-1}[0:K_l], reducing their absmax on the way -> Q (the
//    quantiser's fp32 decisions), the workgroup's acc_a partials and the
//    codes as bytes in LDS; after a barrier, wave 0 publishes the
//    workgroup's acc_a rows at once (the next phase waits on them) while
//    threads p < K/8 build the bit-planes, each transposing the 8x8 bit
//    matrix of codes 8p..8p+7.  Then the active group runs the popcount
//    GEMV on the workgroup's rows, its first wave collects the r acc_a words
//    of the XCD and splits them into limbs in LDS, and the group does the
//    LoRA up-projection and epilogue and stores its y rows.
//  * Row-split constants come precomputed in the layer table, and the loop
//    index is kept uniform, so per-linear set-up runs on the scalar unit.
//  * Every wait is bounded: on time-out the workgroup records an error in
//    the status word and leaves, so the grid always drains.
//  * The layer table lives in the workspace, written by a setup launch
//    (dfssm_chain_prepare) together with a fingerprint of the table; the
//    kernel compares that fingerprint with the caller's before it reads the
//    table, and leaves (status bit 8) if they differ.
#include <float.h>

#include <algorithm>

#include "dfssm_internal.hpp"

namespace {

constexpr int kGT = 512;              // threads per role group
constexpr int kCT = 2 * kGT;          // threads per workgroup
constexpr int kGW = kGT / 64;         // waves per group
static_assert(kGW == dfssm::kChainWaves, "waves per role group");
constexpr int kMaxSteps = dfssm::kChainMaxSteps;
constexpr int kCols = dfssm::kChainMaxK / kCT;  // previous-output columns per thread
constexpr int kChunks = dfssm::kChainMaxK / 128;  // 128-column chunks of the bit-planes
constexpr int kAccRows = dfssm::kChainAccRows;
constexpr int kXcds = dfssm::kChainXcds;
constexpr int kMaxGrid = 256;
constexpr long kSpinLimit = 1L << 20;

// status bits
constexpr unsigned kStY = 1u, kStAcc = 2u, kStPlace = 16u;

// agent scope: crosses XCDs (bypasses the non-coherent per-XCD L2s)
__device__ __forceinline__ uint64_t ll_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void ll_store(uint64_t* p, uint32_t tag, uint32_t v) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// inside one XCD: the store goes through (write-through L1) to the XCD's L2;
// the load is a buffer load with sc0|nt, which skips the CU's L1 and is
// served by that L2 (each poll loop also holds the status atomic, which keeps
// the compiler from hoisting the loads out of it)
__device__ __forceinline__ void xcd_store(uint64_t* p, uint64_t w) {
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
typedef unsigned v2u __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint64_t xcd_load(__amdgpu_buffer_rsrc_t rs, uint32_t word) {
  const v2u v = __builtin_amdgcn_raw_buffer_load_b64(rs, word * 8u, 0, 3);
  return ((uint64_t)v.y << 32) | v.x;
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t xcd_region(uint64_t* base, int64_t words) {
  // dword 3 of the resource: 32-bit data format, as the gfx9 family needs
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, (int)(words * 8), 0x00020000);
}

__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}

// The quantiser's code of v for inv = 127/a, where |v| <= a: |v * inv| is
// at most 127 * (1 + 2^-23)^2 < 127.5, so rint() already lands in [-127, 127]
// and the clamp of the definition never changes the result.
__device__ __forceinline__ int code(float v, float inv) { return (int)rintf(v * inv); }

__device__ __forceinline__ int dpp_sum16(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);  // row_mirror
  return v;
}

// Sum over aligned groups of G lanes (G = 8..64), result in every lane of
// the group: DPP butterflies inside a 16-lane row; across rows, gfx950's
// permlane swaps.  v_permlane16_swap of a value with itself leaves rows
// (0,0,2,2) in one result and (1,1,3,3) in the other, so their sum is the
// 32-lane half's total in every lane; v_permlane32_swap does the same for
// the two halves.
__device__ __forceinline__ int group_sum(int v, int G) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
  if (G >= 16) v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);
  if (G >= 32) {
    const auto p = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
    v = (int)(p[0] + p[1]);
  }
  if (G >= 64) {
    const auto p = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
    v = (int)(p[0] + p[1]);
  }
  return v;
}

// Whole-wave reductions with the result as a uniform value: DPP inside each
// 16-lane row, then row_bcast:15 (rows 1, 3 take lane 15 of the row below)
// and row_bcast:31 (rows 2, 3 take lane 31), which leaves the total in lane
// 63.  No LDS permute on the way.
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

// One linear's operands of this workgroup's rows, per lane of a group.
struct Pref {
  uint4 w[kMaxSteps];
  uint32_t b[kMaxSteps];
  float al[kMaxSteps], be[kMaxSteps];
};

// Loads go through the global address space (the table's pointers are
// generic, which would otherwise give flat loads) and always read in-range
// addresses; nothing is masked here, so no instruction waits on a prefetched
// value before its use.  Values read for lanes outside the data are harmless
// by construction: lanes past a row's chunks meet all-zero bit-planes, LoRA
// lanes past r meet zero limbs, A bytes past K meet zero codes, A rows past
// r are never published, and rows outside the workgroup's range are never
// stored.
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

__device__ __forceinline__ void prefetch(const dfssm::ChainLayerDev& L, int wg, int gt, Pref& p) {
  const int lane = gt & 63, wave = gt >> 6;
  const int G = 1 << L.lgG, g = lane & (G - 1), grp = lane >> L.lgG;
  const int RW = 64 >> L.lgG;
  const int n0 = wg * L.R, n1 = min(L.N, n0 + L.R);
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
}

// This thread's bytes of the LoRA down rows rho + n_x*t (t < kAccRows) of a
// linear, in the column layout of the codes: byte i of a[t] is column
// tid + kCT*i (columns past K read column 0; their codes are 0).
__device__ __forceinline__ void load_a_cols(const dfssm::ChainLayerDev& L, int tid, int rho, int nx,
                                            uint32_t (&a)[kAccRows]) {
  static_assert(kCols == 4, "four bytes per packed word");
#pragma unroll
  for (int t = 0; t < kAccRows; ++t) {
    const int j = rho + nx * t;
    const int8_t* arow = L.A + (int64_t)(j < L.r ? j : 0) * L.K;
    uint32_t w = 0;
#pragma unroll
    for (int i = 0; i < kCols; ++i) {
      const int k = tid + i * kCT;
      w |= (uint32_t)(gload1s(arow + (k < L.K ? k : 0)) & 0xff) << (8 * i);
    }
    a[t] = w;
  }
}

// Bounded polls of one {tag, value} word; they also give up once another
// wave of the workgroup has aborted (abort_ in LDS).
__device__ __forceinline__ bool poll_ll(const uint64_t* p, uint32_t tag, uint64_t& wd,
                                        unsigned* status, unsigned code_bit, const int* abort_flag) {
  long spins = 0;
  while ((uint32_t)((wd = ll_load(p)) >> 32) != tag) {
    if (++spins > kSpinLimit || *(const volatile int*)abort_flag) {
      atomicOr(status, code_bit);
      return false;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  return true;
}
__device__ __forceinline__ bool poll_xcd(__amdgpu_buffer_rsrc_t rs, uint32_t word, uint32_t tag, uint64_t& wd,
                                         unsigned* status, unsigned code_bit, const int* abort_flag) {
  long spins = 0;
  while ((uint32_t)((wd = xcd_load(rs, word)) >> 32) != tag) {
    if (++spins > kSpinLimit || *(const volatile int*)abort_flag) {
      atomicOr(status, code_bit);
      return false;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  return true;
}

__global__ __launch_bounds__(kCT, 1) void chain_persistent(
    const dfssm::ChainLayerDev* __restrict__ layers, int L, const int8_t* __restrict__ q0,
    const float* __restrict__ s0, dfssm::ChainExch ex, float* __restrict__ y_all,
    const uint64_t* __restrict__ table_hash, uint64_t expect_hash) {
  unsigned* const status = ex.status;
  // the table was written by a prepare of the same layers, or nothing here
  // is trusted: leave before reading it
  if (*table_hash != expect_hash) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(status, 8u);
    return;
  }
  // bit-planes, plane-major: the G lanes of a row read consecutive chunks
  __shared__ uint4 pl_lds[8 * kChunks];
  // LoRA down-projection of the current linear as 4 signed base-256 limbs:
  // entry g holds acc_a[4g .. 4g+3], dword t = limb t (r <= 64)
  static_assert(dfssm::kChainAccRows * dfssm::kChainWgPerXcd <= 64, "limb table size");
  __shared__ uint4 limb_lds[16];
  __shared__ int32_t dot_part[kAccRows][64];  // 16-lane row sums of the 16 waves
  static_assert(4 * 2 * kGW == 64, "row sums per rank");
  __shared__ __attribute__((aligned(16))) int8_t code_lds[dfssm::kChainMaxK];
  // absmax of the previous output as {linear, bits}: the largest tag wins,
  // so it needs no reset between linears
  __shared__ uint64_t ymax_lds;
  // phase counters (monotonic): waves of the active group whose bit-planes
  // are in LDS (+kGW per linear) and that have published (+kGW per linear);
  // the linear whose limbs are in LDS (+1 per linear)
  __shared__ int pl_cnt, limb_flag, pub_cnt;
  __shared__ int sumq_lds;
  __shared__ int abort_;
  __shared__ int rho_lds, nx_lds;
  __shared__ uint32_t seq_lds;
  const int wg = blockIdx.x, nwg = gridDim.x;
  const int tid = threadIdx.x;
  const int group = tid / kGT, gt = tid % kGT, lane = gt & 63, wave = gt >> 6;
  const int wave16 = tid >> 6;  // wave index in the workgroup

  // the launch's epoch: one arrival per workgroup; the 24-bit sequence
  // number derived from it is never 0, so zeroed words never validate
  if (tid == 0) {
    const uint64_t old = dfssm_dev::arrive(ex.epoch, wg);
    seq_lds = (uint32_t)((old >> 32) % 0xffffffu) + 1u;
    dfssm_dev::advance_if_last(ex.epoch, wg, old, nwg);
  }
  __syncthreads();
  const uint32_t seq = seq_lds;
  // a word written for linear l carries tag(l)
  auto tag_of = [seq](int l) -> uint32_t { return (seq << 8) | (uint32_t)((l + 1) & 0xff); };
  const uint32_t tag_place = seq << 8;

  // ---- placement: the XCD of every workgroup, this one's rank among the
  //      workgroups of its XCD, and the smallest XCD's size
  const uint32_t xcc = __builtin_amdgcn_s_getreg((20) | (0 << 6) | ((4 - 1) << 11));  // HW_REG_XCC_ID[3:0]
  if (tid == 0) {
    abort_ = 0;
    ymax_lds = 0;
    pl_cnt = 0;
    pub_cnt = 0;
    limb_flag = 0;
    sumq_lds = 0;
    ll_store(ex.xmap + wg, tag_place, xcc);
  }
  if (tid < 64) {
    uint32_t x[kMaxGrid / 64];
    bool ok = true;
#pragma unroll
    for (int t = 0; t < kMaxGrid / 64; ++t) {
      const int w = tid + 64 * t;
      x[t] = 0xffu;
      if (w < nwg) {
        uint64_t wd;
        if (!poll_ll(ex.xmap + w, tag_place, wd, status, kStPlace, &abort_)) ok = false;
        x[t] = (uint32_t)wd;
      }
    }
    int rho = 0, nx = 0, nmin = nwg;
    for (int c = 0; c < 16; ++c) {
      int cnt = 0, below = 0;
#pragma unroll
      for (int t = 0; t < kMaxGrid / 64; ++t) {
        const uint64_t m = __ballot(x[t] == (uint32_t)c);
        cnt += __popcll(m);
        // lanes holding workgroups 64t .. 64t+63 that come before wg
        const int w0 = 64 * t;
        const uint64_t below_mask = wg <= w0 ? 0ull : (wg >= w0 + 64 ? ~0ull : ((1ull << (wg - w0)) - 1));
        below += __popcll(m & below_mask);
      }
      if (cnt > 0) nmin = min(nmin, cnt);
      if (c == (int)xcc) {
        rho = below;
        nx = cnt;
      }
    }
    const bool bad = __ballot(!ok) != 0 || xcc >= (uint32_t)kXcds || (ex.r_max + nmin - 1) / nmin > kAccRows;
    if (tid == 0) {
      rho_lds = rho;
      nx_lds = nx;
      if (bad) {
        atomicOr(status, kStPlace);
        abort_ = 1;
      }
    }
  }
  __syncthreads();
  if (abort_) return;
  const int rho = __builtin_amdgcn_readfirstlane(rho_lds), nx = __builtin_amdgcn_readfirstlane(nx_lds);
  uint64_t* const y_rel = ex.y_rel + (int64_t)xcc * ex.ysum;
  uint64_t* const acc_rel = ex.acc_rel + (int64_t)xcc * L * dfssm::kMaxRank;
  const __amdgpu_buffer_rsrc_t rs_y = xcd_region(y_rel, ex.ysum);
  const __amdgpu_buffer_rsrc_t rs_acc = xcd_region(acc_rel, (int64_t)L * dfssm::kMaxRank);

  Pref pf;
  if (group < L) prefetch(layers[group], wg, gt, pf);

  for (int l = 0; l < L; ++l) {
    const bool active = group == (l & 1);
    // the loop index is uniform: keeps the table reads and the row-split
    // arithmetic on the scalar unit
    const int lu = __builtin_amdgcn_readfirstlane(l);
    const dfssm::ChainLayerDev Ld = layers[lu];
    const int K = Ld.K, N = Ld.N, r = Ld.r, lgG = Ld.lgG, G = 1 << lgG, R = Ld.R;
    const float s = l == 0 ? s0[0] : 1.0f / 127.0f;

    // ---- 0. the active group relays this workgroup's slice of
    //         y_{l-1}[0:K] into the XCD's copy; then every thread loads its
    //         A bytes and polls its words of the copy (columns tid + kCT*i)
    //         until all carry tag(l-1); their absmax is reduced into LDS
    uint32_t av[kAccRows];  // this thread's A bytes of the two rows, column i in byte i
    uint32_t yv[kCols];
    if (l > 0) {
      const int64_t prev = layers[lu - 1].y_off;
      const uint32_t tag = tag_of(l - 1);
      if (active) {
        const int slice = (K + nx - 1) / nx;
        const int k1 = min(K, (rho + 1) * slice);
        for (int k = rho * slice + gt; k < k1; k += kGT) {
          uint64_t wd;
          if (!poll_ll(ex.y_ll + prev + k, tag, wd, status, kStY, &abort_)) {
            abort_ = 1;
            break;
          }
          xcd_store(y_rel + prev + k, wd);
        }
      }
      if (rho < r) load_a_cols(Ld, tid, rho, nx, av);
      // the group active in this linear arrives early (it was idle after the
      // last B1); it starts polling only once its own workgroup has
      // published its rows of y_{l-1}: earlier, its polls would only load
      // the XCD's L2, which the exchange of the previous linear still uses
      if (active) {
        long sp = 0;
        while (__hip_atomic_load(&pub_cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) < kGW * l) {
          if (++sp > kSpinLimit || abort_) break;
          __builtin_amdgcn_s_sleep(1);
        }
      }
      uint32_t pend = 0;
#pragma unroll
      for (int i = 0; i < kCols; ++i)
        if (tid + i * kCT < K) pend |= 1u << i;
      long spins = 0;
      uint32_t m = 0;
      while (pend) {
        uint64_t wd[kCols];
#pragma unroll
        for (int i = 0; i < kCols; ++i)
          if (pend & (1u << i)) wd[i] = xcd_load(rs_y, (uint32_t)(prev + tid + i * kCT));
#pragma unroll
        for (int i = 0; i < kCols; ++i)
          if ((pend & (1u << i)) && (uint32_t)(wd[i] >> 32) == tag) {
            yv[i] = (uint32_t)wd[i];
            m = max(m, yv[i] & 0x7fffffffu);
            pend &= ~(1u << i);
          }
        if (pend) {
          if (++spins > kSpinLimit || abort_) {
            atomicOr(status, kStY);
            abort_ = 1;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      m = wave_max_bits_u(m);
      if (lane == 0)
        __hip_atomic_fetch_max(&ymax_lds, ((uint64_t)l << 32) | m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    } else if (rho < r) {
      load_a_cols(Ld, tid, rho, nx, av);
    }
    __syncthreads();  // B0
    if (abort_) return;

    // ---- 1. codes, LoRA down rows, bit-planes: all 16 waves, columns
    //         tid + kCT*i ----------------------------------------------------
    // column blocks i with tid + kCT*i < K for some thread (uniform)
    int q[kCols];
    if (l == 0) {
#pragma unroll
      for (int i = 0; i < kCols; ++i) {
        q[i] = 0;
        if (i * kCT < K) {
          const int k = tid + i * kCT;
          const int c = gload1s(q0 + (k < K ? k : 0));
          q[i] = k < K ? c : 0;
        }
      }
    } else {
      const float a = __uint_as_float((uint32_t)ymax_lds);
      const bool zero = a < FLT_MIN;
      const float inv = zero ? 0.0f : 127.0f / a;
#pragma unroll
      for (int i = 0; i < kCols; ++i) {
        q[i] = 0;
        if (i * kCT < K) q[i] = (zero || tid + i * kCT >= K) ? 0 : code(__uint_as_float(yv[i]), inv);
      }
    }
    // LoRA down partials of rows rho + nx*t: the 4 codes against the 4 A
    // bytes with one v_dot4, summed over each 16-lane row; the 64 row sums
    // go to LDS.  The codes go to LDS as bytes (bit-planes, sum of codes).
    {
      const uint32_t qp = (uint32_t)(q[0] & 0xff) | ((uint32_t)(q[1] & 0xff) << 8) |
                          ((uint32_t)(q[2] & 0xff) << 16) | ((uint32_t)q[3] << 24);
      if (rho < r) {
#pragma unroll
        for (int t = 0; t < kAccRows; ++t) {
          const int v = dpp_sum16(sdot4(av[t], qp, 0));
          if ((lane & 15) == 0) dot_part[t][4 * wave16 + (lane >> 4)] = v;
        }
      }
#pragma unroll
      for (int i = 0; i < kCols; ++i)
        if (i * kCT < K && tid + i * kCT < K) code_lds[tid + i * kCT] = (int8_t)q[i];
    }
    __syncthreads();  // B1
    if (abort_) return;

    // After B1 the two groups part until the next linear's B0:
    //  * the idle group's first wave publishes this workgroup's LoRA down
    //    rows, sums the codes, collects the XCD's acc_a words into limbs in
    //    LDS and raises limb_flag; the rest of the idle group (and then that
    //    wave) loads the weights of linear l+1;
    //  * the active group builds the bit-planes, waits for all 8 of its
    //    waves to have written them (pl_cnt), runs the GEMV, waits for
    //    limb_flag, and does the LoRA up-projection and epilogue.
    // A wave's LDS operations complete in issue order, so a counter or flag
    // raised after a wave's LDS writes is seen only after those writes; the
    // signal fences keep the compiler from moving LDS accesses across them.
    // Every LDS written here is next written after the next linear's B1, so
    // the next B0 orders its reuse.
    const int RW = 64 >> lgG;
    const int g = lane & (G - 1);
    if (!active) {
      if (gt < 64) {
        if (rho < r) {
          static_assert(kAccRows == 2, "two rows per workgroup below");
          int tot[kAccRows];
#pragma unroll
          for (int t = 0; t < kAccRows; ++t) tot[t] = wave_sum_u(dot_part[t][lane]);
          if (lane < kAccRows) {
            const int j = rho + nx * lane;
            if (j < r)
              xcd_store(acc_rel + (int64_t)l * dfssm::kMaxRank + j,
                        ((uint64_t)tag_of(l) << 32) | (uint32_t)(lane == 0 ? tot[0] : tot[1]));
          }
        }
        {  // sum of the codes, 16 bytes per lane per pass
          int qs = 0;
          for (int k = 16 * lane; k < K; k += 16 * 64) {
            const uint4 c = *reinterpret_cast<const uint4*>(code_lds + k);
            qs = sdot4(c.x, 0x01010101u, qs);
            qs = sdot4(c.y, 0x01010101u, qs);
            qs = sdot4(c.z, 0x01010101u, qs);
            qs = sdot4(c.w, 0x01010101u, qs);
          }
          qs = wave_sum_u(qs);
          if (lane == 0) sumq_lds = qs;
        }
        // lane j collects acc_a[j] (0 past r) and stores its 4 signed
        // base-256 limbs as bytes of limb_lds[j / 4], dword t = limb t
        int32_t v = 0;
        if (gt < r) {
          const uint32_t tag = tag_of(l);
          const uint32_t word = (uint32_t)(l * dfssm::kMaxRank + gt);
          uint64_t wd;
          if (!poll_xcd(rs_acc, word, tag, wd, status, kStAcc, &abort_)) abort_ = 1;
          v = (int32_t)(uint32_t)wd;
        }
        int8_t d[4];
        dfssm_dev::split_limbs(v, d);
        uint8_t* lb = reinterpret_cast<uint8_t*>(limb_lds) + (gt >> 2) * 16 + (gt & 3);
#pragma unroll
        for (int t = 0; t < 4; ++t) lb[4 * t] = (uint8_t)d[t];
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        if (lane == 0) __hip_atomic_store(&limb_flag, l + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
      }
      // the group idle in this linear loads the weights of the next one
      // (it polls nothing more in this linear; its first wave has finished
      // its collect above)
      if (l >= 1 && l + 1 < L) prefetch(layers[lu + 1], wg, gt, pf);
    } else {
      // bit-planes: thread p < K/8 of the group transposes the 8x8 bit
      // matrix of codes 8p .. 8p+7 (byte i = code i) so that byte b holds
      // bit b of the 8 codes, i.e. byte p of plane b (plane-major, 16-byte
      // chunks of 128 columns)
      if (gt < (K >> 3)) {
        const uint2 c = reinterpret_cast<const uint2*>(code_lds)[gt];
        uint32_t lo = c.x, hi = c.y, t;
        t = (lo ^ (lo >> 7)) & 0x00AA00AAu;
        lo ^= t ^ (t << 7);
        t = (hi ^ (hi >> 7)) & 0x00AA00AAu;
        hi ^= t ^ (t << 7);
        t = (lo ^ (lo >> 14)) & 0x0000CCCCu;
        lo ^= t ^ (t << 14);
        t = (hi ^ (hi >> 14)) & 0x0000CCCCu;
        hi ^= t ^ (t << 14);
        t = (lo ^ __builtin_amdgcn_alignbit(hi, lo, 28)) & 0xF0F0F0F0u;
        lo ^= t;
        hi ^= t >> 4;
        uint8_t* pb = reinterpret_cast<uint8_t*>(pl_lds) + gt;
#pragma unroll
        for (int b = 0; b < 4; ++b) pb[b * kChunks * 16] = (uint8_t)(lo >> (8 * b));
#pragma unroll
        for (int b = 0; b < 4; ++b) pb[(4 + b) * kChunks * 16] = (uint8_t)(hi >> (8 * b));
      }
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      if (lane == 0) __hip_atomic_fetch_add(&pl_cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      {
        long spins = 0;
        while (__hip_atomic_load(&pl_cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) < kGW * (l + 1)) {
          if (++spins > kSpinLimit || abort_) {
            atomicOr(status, kStAcc);
            abort_ = 1;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      __atomic_signal_fence(__ATOMIC_SEQ_CST);

      // ---- 2. scaffold GEMV on the prefetched rows: one bit-plane at a
      //      time, weight c_b = 2^b (b < 7), -128 (b = 7); acc_s =
      //      2 * sum_{bit=1} Q - sum Q (sum Q subtracted below)
      int part[kMaxSteps];
      const int C = K >> 7;
      const int n0 = wg * R, n1 = min(N, n0 + R);
#pragma unroll
      for (int st = 0; st < kMaxSteps; ++st) {
        part[st] = 0;
        // uniform per wave: does this wave own rows in step st?
        if (n0 + st * kGW * RW + wave * RW < n1) {
          const uint4 w = pf.w[st];
          int dsum = 0;
#pragma unroll
          for (int b = 0; b < 8; ++b) {
            const uint4 Pb = g < C ? pl_lds[b * kChunks + g] : make_uint4(0, 0, 0, 0);
            const int c = __builtin_popcount(w.x & Pb.x) + __builtin_popcount(w.y & Pb.y) +
                          __builtin_popcount(w.z & Pb.z) + __builtin_popcount(w.w & Pb.w);
            dsum += b < 7 ? (c << b) : -(c << 7);
          }
          part[st] = 2 * group_sum(dsum, G);
        }
      }
      {
        long spins = 0;
        while (__hip_atomic_load(&limb_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) < l + 1) {
          if (++spins > kSpinLimit || abort_) {
            atomicOr(status, kStAcc);
            abort_ = 1;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      __atomic_signal_fence(__ATOMIC_SEQ_CST);

      // ---- 3. LoRA up-projection, epilogue, publish --------------------------
      if (!abort_) {
        const int sq = sumq_lds;
        const int r4 = (r + 3) >> 2;
        const int grp = lane >> lgG;
        // limbs of acc_a[4g .. 4g+3], packed per limb (j >= r read as 0)
        uint32_t lb0 = 0, lb1 = 0, lb2 = 0, lb3 = 0;
        if (r > 0 && g < r4) {
          const uint4 t = limb_lds[g];
          lb0 = t.x;
          lb1 = t.y;
          lb2 = t.z;
          lb3 = t.w;
        }
#pragma unroll
        for (int st = 0; st < kMaxSteps; ++st) {
          if (n0 + st * kGW * RW + wave * RW >= n1) break;  // uniform per wave
          int elo = 0, ehi = 0;
          if (r > 0) {
            const uint32_t bw = pf.b[st];
            elo = group_sum(sdot4(bw, lb0, 0) + (sdot4(bw, lb1, 0) << 8), G);
            ehi = group_sum(sdot4(bw, lb2, 0) + (sdot4(bw, lb3, 0) << 8), G);
          }
          const int n = n0 + st * kGW * RW + wave * RW + grp;
          if (g == 0 && n < n1) {
            const float y = dfssm_dev::epilogue(s, pf.al[st], pf.be[st], part[st] - sq, ehi, elo, r > 0);
            ll_store(ex.y_ll + Ld.y_off + n, tag_of(l), __float_as_uint(y));
            y_all[Ld.y_off + n] = y;
          }
        }
      }
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      if (lane == 0) __hip_atomic_fetch_add(&pub_cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
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

int chain_grid() { return kMaxGrid; }  // one workgroup per CU

bool chain_persistent_supported(const dfssm_layer* layers, int n_layers, int64_t M, int nwg) {
  if (M != 1 || nwg > kMaxGrid) return false;
  for (int l = 0; l < n_layers; ++l) {
    const dfssm_layer& L = layers[l];
    if (L.K % 128 != 0 || L.K > kChainMaxK || L.r % 4 != 0) return false;
    if (L.r > kChainAccRows * kChainWgPerXcd) return false;
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

// A plain launch: one workgroup per CU fits (launch bounds of 1024 threads,
// one block per CU), and the kernel's placement step waits, with a bound,
// for every workgroup to publish its XCD; a grid that is not resident
// together (other work holding CUs for longer than that bound) ends with
// the placement status bit instead of waiting.
hipError_t launch_zero_words(uint64_t* p, int64_t words, hipStream_t st) {
  if (words <= 0) return hipSuccess;
  SetupArgs a{};
  a.zero_base = p;
  a.zero_words = words;
  const int64_t blocks = std::min<int64_t>(1024, ceil_div(words, 256));
  chain_setup<<<dim3((unsigned)blocks), dim3(256), 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_chain_run(const ChainLayerDev* table_dev, int n_layers, const int8_t* q0, const float* s0,
                            const ChainExch& ex, float* y_all, const uint64_t* hash_dev, uint64_t hash,
                            hipStream_t st) {
  chain_persistent<<<dim3(chain_grid()), dim3(kCT), 0, st>>>(table_dev, n_layers, q0, s0, ex, y_all, hash_dev,
                                                            hash);
  return hipGetLastError();
}

}  // namespace dfssm
