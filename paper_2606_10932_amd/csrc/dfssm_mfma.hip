// dfssm_mfma.hip -- prefill-shaped (large M) scaffold + LoRA linear on the
// gfx950 int8 matrix cores (v_mfma_i32_16x16x64_i8).
//
// The sign bits are expanded on chip, in registers, to {0,1} bytes (a
// nibble n becomes bytes via (n * 0x00204081) & 0x01010101), so the MFMA
// computes D[m,n] = sum_{bit=1} Q[m,k] and acc_s = 2*D - sum_k Q[m,k]; the
// expanded signs never touch memory or LDS (the paper expands to int8 "on
// the fly" ahead of a library int8 GEMM, Sec. 4.1).
//
// Operand layout of v_mfma_i32_16x16x64_i8 (wave64): lane l supplies row
// (l % 16) of A and column (l % 16) of B, each as 16 consecutive K-bytes of
// K-group (l / 16); the 16x16 int32 result D has D[4*(l/16)+v][l%16] in
// lane l, register v.  A = Q rows (tokens), B = sign columns (output rows).
//
// LoRA: lora_down computes acc_a = Q * A^T with the same MFMA (K split over
// the 4 waves of a block, reduced in LDS), sum_k Q, and writes acc_a as 4
// signed base-256 int8 limbs.  After the scaffold K-loop the main kernel
// gets the exact int64 acc_b = sum_j B[n,j] acc_a[m,j] from four int8
// MFMAs, E_hi = 256*(L3.B) + L2.B and E_lo = 256*(L1.B) + L0.B (each < 2^31
// for r <= 256), acc_b = E_lo + 65536*E_hi, 16 output rows at a time, so
// the K-loop holds only the scaffold accumulators (3 blocks per CU).
#include "dfssm_internal.hpp"

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

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

// 16 sign bits -> 16 bytes of {0,1}, byte b of dword t = bit 4t+b
__device__ __forceinline__ v4i expand16(uint32_t bits16) {
  v4i o;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    uint32_t nib = (bits16 >> (4 * t)) & 0xfu;
    o[t] = (int)((nib * 0x00204081u) & 0x01010101u);
  }
  return o;
}

__device__ __forceinline__ v4i load16(const int8_t* p) {
  uint4 u = *reinterpret_cast<const uint4*>(p);
  return v4i{(int)u.x, (int)u.y, (int)u.z, (int)u.w};
}

// 16 bytes of an int8 row with bounds (byte granular), zero outside [0, len)
__device__ __forceinline__ v4i load16_guarded(const int8_t* row, int start, int len, bool aligned) {
  if (start + 16 <= len && aligned) return load16(row + start);
  v4i o = zero4();
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int i = start + e;
    uint32_t b = (i >= 0 && i < len) ? (uint32_t)(uint8_t)row[i] : 0u;
    o[e >> 2] |= (int)(b << (8 * (e & 3)));
  }
  return o;
}

// ------------------------------------------------------------ lora_down
// A block owns 16 tokens x 16 ranks (one MFMA tile; blockIdx.y is the rank
// tile, covering rp); its 4 waves split the K steps into quarters and reduce
// their partial sums in LDS.  Loads are issued kLdBatch K-steps at a time.
constexpr int kLdBatch = 4;

__global__ __launch_bounds__(kThreads) void mfma_lora_down(const int8_t* __restrict__ q, int M, int K,
                                                           int r, int rp, const int8_t* __restrict__ A,
                                                           int32_t* __restrict__ acc_a,
                                                           int8_t* __restrict__ limbs,
                                                           int32_t* __restrict__ sumq) {
  __shared__ int32_t part[4][16 * 16];
  __shared__ int32_t qpart[4][16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = lane & 15, kg = lane >> 4;
  const int m0 = blockIdx.x * 16, j0 = blockIdx.y * 16;
  const bool first = blockIdx.y == 0;  // the rank tile that also sums Q
  const int m = m0 + row, j = j0 + row;
  const bool m_ok = m < M, j_ok = j < r;
  const int8_t* qrow = q + (int64_t)(m_ok ? m : 0) * K;
  const int8_t* arow = A + (int64_t)(j_ok ? j : 0) * K;
  const int nks = (K + 63) / 64;
  const int per = (nks + 3) / 4;
  const int ks0 = wave * per, ks1 = min(nks, ks0 + per);

  v4i acc = zero4();
  int qs = 0;
  for (int kb = ks0; kb < ks1; kb += kLdBatch) {
    // all loads of the batch from clamped addresses first, masks after
    v4i a[kLdBatch], b[kLdBatch];
    int ma[kLdBatch], mb[kLdBatch];
#pragma unroll
    for (int u = 0; u < kLdBatch; ++u) {
      const int kk = (kb + u) * 64 + 16 * kg;
      const bool kok = kb + u < ks1 && kk < K;
      const int kc = kok ? kk : 0;
      a[u] = load16(qrow + kc);
      ma[u] = (m_ok && kok) ? -1 : 0;
      b[u] = r > 0 ? load16(arow + kc) : zero4();
      mb[u] = (j_ok && kok) ? -1 : 0;
    }
#pragma unroll
    for (int u = 0; u < kLdBatch; ++u) {
      a[u] &= ma[u];
      b[u] &= mb[u];
      if (first) {
#pragma unroll
        for (int t = 0; t < 4; ++t) qs = __builtin_amdgcn_sdot4(a[u][t], 0x01010101, qs, false);
      }
      acc = mfma(a[u], b[u], acc);
    }
  }
  // D[token 4*kg + v][rank row]
#pragma unroll
  for (int v = 0; v < 4; ++v) part[wave][(4 * kg + v) * 16 + row] = acc[v];
  if (first) {
    qs += __shfl_xor(qs, 16, 64);
    qs += __shfl_xor(qs, 32, 64);
    if (kg == 0) qpart[wave][row] = qs;
  }
  __syncthreads();
  {
    const int i = threadIdx.x;  // 256 threads = 16 tokens x 16 ranks
    const int mi = i >> 4, ji = i & 15;
    const int mm = m0 + mi, jj = j0 + ji;
    if (mm < M) {
      const int32_t val = part[0][i] + part[1][i] + part[2][i] + part[3][i];
      int8_t d[4];
      dfssm_dev::split_limbs(jj < r ? val : 0, d);
#pragma unroll
      for (int l = 0; l < 4; ++l) limbs[((int64_t)l * M + mm) * rp + jj] = d[l];
      if (jj < r) acc_a[(int64_t)mm * r + jj] = val;
    }
  }
  if (first && threadIdx.x < 16 && m0 + threadIdx.x < M)
    sumq[m0 + threadIdx.x] = qpart[0][threadIdx.x] + qpart[1][threadIdx.x] + qpart[2][threadIdx.x] +
                             qpart[3][threadIdx.x];
}

// ------------------------------------------------------------ main GEMM
// Block tile 128 (tokens) x 128 (output rows), 4 waves as 2 x 2 with wave
// tiles of 64 x 64 (4 x 4 MFMA tiles); 64 K per stage.  The K-loop runs a
// 4-stage LDS ring filled by direct-to-LDS loads (global_load_lds: no
// register staging):
//   Q stage: 128 rows x 64 bytes, the four 16-byte chunks of row r stored
//            at chunk slot c ^ ((r >> 2) & 3), so the 16 lanes reading one
//            MFMA operand column hit 16 distinct 4-bank groups;
//   sign stage: 128 rows x 2 words (64 sign bits per row), expanded to
//            {0,1} bytes in registers right before use.
// Each wave issues exactly three loads per stage (two 1 KB Q pieces and
// one 256-byte sign piece), so "stage ks has landed" is a vector-memory
// count; past the last stage the issue repeats the last stage's loads (the
// same bytes into the same slot), which keeps the count uniform.
constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kStages = 4;
constexpr int kLoadsPerStage = 3;
constexpr int kQStage = kBM * kBK;               // 8 KB
constexpr int kWStage = kBN * 2 * 4;             // 1 KB
constexpr int kStageBytes = kQStage + kWStage;
// epilogue: limbs [4][kBM][64] and B [kBN][64] with the same chunk swizzle,
// then one transpose buffer of 16 x kYPitch floats per wave
constexpr int kYPitch = 20;                      // 16 columns + 4: conflict-free both ways
constexpr int kLdsLoop = kStages * kStageBytes;
constexpr int kLdsLora = 4 * kBM * kBK + kBN * kBK + 4 * 16 * kYPitch * 4;
constexpr int kLdsBytes = kLdsLoop > kLdsLora ? kLdsLoop : kLdsLora;
#ifndef DFSSM_MFMA_OCC
#define DFSSM_MFMA_OCC 3
#endif

typedef __attribute__((address_space(3))) void lds_void;

// Direct-to-LDS loads (gfx950 global_load_lds): each lane's 16 (or 4) bytes
// land at m0 + 16*lane (4*lane).  Issued as inline assembly so the compiler
// does not treat every later LDS read as depending on them (it cannot tell
// the ring slots apart and would wait for all loads); the K-loop orders them
// itself with DFSSM_WAIT_VMCNT and the barrier.
// (the address is wave-uniform; readfirstlane puts it in an SGPR for m0)
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(uintptr_t)(const lds_void*)p);
}
__device__ __forceinline__ void lds_dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}
__device__ __forceinline__ void lds_dma4(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}

// s_waitcnt with only the vector-memory counter constrained
#define DFSSM_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(0x0F70 | ((n) & 0xF) | (((n) >> 4) << 14))
// workgroup barrier that does not drain outstanding direct-to-LDS loads
// (the compiler's barrier fence would wait for all of them); LDS visibility
// of the loads is ordered by the DFSSM_WAIT_VMCNT before it
#define DFSSM_BARRIER() asm volatile("s_barrier" ::: "memory")

template <bool kLoraLds>
__global__ __launch_bounds__(kThreads, DFSSM_MFMA_OCC) void mfma_scaffold(
    const int8_t* __restrict__ q, const float* __restrict__ s, int M, int K, int N, int r, int rp,
    const uint32_t* __restrict__ w_bits, const float* __restrict__ alpha,
    const int8_t* __restrict__ limbs, const int8_t* __restrict__ B,
    const float* __restrict__ beta, const int32_t* __restrict__ sumq, float* __restrict__ y,
    int32_t* __restrict__ acc_s_out, int64_t* __restrict__ acc_b_out, int nbm, int nbn) {
  // one LDS buffer, two uses: the K-loop stages (Q tile + sign words, x2),
  // then the LoRA operands of the epilogue (4 limbs x 128 rows + 128 B rows)
  __shared__ __attribute__((aligned(16))) int8_t lds_raw[kLdsBytes];
  int8_t* limb_lds = lds_raw;                       // [4][kBM][64], swizzled
  int8_t* b_lds = lds_raw + 4 * kBM * kBK;          // [kBN][64], swizzled
  __shared__ __attribute__((aligned(16))) float al_lds[kBN], be_lds[kBN], s_lds[kBM];
  __shared__ __attribute__((aligned(16))) int32_t sq_lds[kBM];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = lane & 15, kg = lane >> 4;

  // XCD-aware tile order: blocks are dealt to the 8 XCDs round-robin, so
  // give each XCD a contiguous run of tiles (same n-tile, successive m-tiles:
  // the tile's sign words and the Q tiles stay in that XCD's L2)
  const int nblk = nbm * nbn;
  const int bid = blockIdx.x;
  const int per_xcd = nblk / 8, rem = nblk % 8;
  const int xcd = bid % 8, idx = bid / 8;
  const int tile = xcd < rem ? xcd * (per_xcd + 1) + idx : rem * (per_xcd + 1) + (xcd - rem) * per_xcd + idx;
  const int bm = tile % nbm, bn = tile / nbm;
  const int m0 = bm * kBM, n0 = bn * kBN;
  const int wm0 = m0 + (wave >> 1) * 64, wn0 = n0 + (wave & 1) * 64;
  const int W = K / 32;
  const int nks = (K + kBK - 1) / kBK;

  // per-row and per-column scalars of the tile, staged once in LDS
  if (tid < kBN) {
    const int n = min(n0 + tid, N - 1);
    al_lds[tid] = alpha[n];
    be_lds[tid] = r > 0 ? beta[n] : 0.0f;
  } else {
    const int m = min(m0 + tid - kBN, M - 1);
    s_lds[tid - kBN] = s[m];
    sq_lds[tid - kBN] = sumq[m];
  }
  __syncthreads();

  // ---- scaffold K-loop ------------------------------------------------------
  // loads of stage ks (clamped to the last stage): this wave's Q rows
  // 32*wave + 16*j + lane/4, slot lane%4 <- chunk (lane%4) ^ ((row >> 2) & 3),
  // and sign rows 32*wave + lane/2, word lane%2.  Rows past M or N read the
  // last row (their outputs are never stored); a chunk past K reads the
  // chunk two before it (its sign bits are masked to zero below).
  const int8_t* qrow[2];
  int qchunk[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int rl = 32 * wave + 16 * j + (lane >> 2);
    qrow[j] = q + (int64_t)min(m0 + rl, M - 1) * K;
    qchunk[j] = ((lane & 3) ^ ((rl >> 2) & 3)) * 16;
  }
  const int wrl = 32 * wave + (lane >> 1);
  const uint32_t* wrow = w_bits + (int64_t)min(n0 + wrl, N - 1) * W + (lane & 1);
  auto issue = [&](int ks) {
    ks = min(ks, nks - 1);
    int8_t* base = lds_raw + (ks % kStages) * kStageBytes;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      int kk = ks * kBK + qchunk[j];
      if (kk >= K) kk -= 32;
      lds_dma16(qrow[j] + kk, lds_addr(base + (32 * wave + 16 * j) * kBK));
    }
    lds_dma4(wrow + 2 * ks - ((2 * ks + (lane & 1)) >= W ? 1 : 0), lds_addr(base + kQStage + 32 * wave * 8));
  };

  v4i acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[i][t] = zero4();

  // operand addresses inside a stage: A tile i is rows 64*(wave>>1) + 16*i +
  // row (row & 3 and (row >> 2) & 3 are the same for every i)
  const int am_off = ((wave >> 1) * 64 + row) * kBK + 16 * (kg ^ ((row >> 2) & 3));
  const int bn_off = ((wave & 1) * 64 + row) * 2 + (kg >> 1);
  const int bshift = (kg & 1) * 16;
  // operands of one stage: 4 A tiles (Q rows) and 4 B tiles (expanded signs)
  auto read_stage = [&](int ks, v4i (&a)[4], v4i (&b)[4]) {
    const int8_t* st = lds_raw + (ks % kStages) * kStageBytes;
    const uint32_t* ws = reinterpret_cast<const uint32_t*>(st + kQStage);
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const v4i*>(st + am_off + 16 * i * kBK);
    const bool whole = 2 * ks + 1 < W;  // uniform: only a K tail has a second word past K
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      uint32_t w = ws[bn_off + 32 * t];
      if (!whole && (kg >> 1)) w = 0;  // sign words past K count as 0
      b[t] = expand16_at(w, bshift);
    }
  };
  // Software pipeline: the MFMAs of stage ks are issued together with the
  // LDS reads and sign expansion of stage ks+1 (independent instructions,
  // so the matrix core and the vector ALU work at the same time).  The LDS
  // ring runs three stages ahead of the multiply.
  v4i a0[4], b0[4], a1[4], b1[4];
  auto step = [&](int ks, const v4i (&ac)[4], const v4i (&bc)[4], v4i (&an)[4], v4i (&bn)[4]) {
    // stages ks+1 and ks+2 are in flight here: leaving only stage ks+2's
    // loads outstanding means this wave's loads of stage ks+1 have landed
    DFSSM_WAIT_VMCNT(kLoadsPerStage);
    DFSSM_BARRIER();  // so have every wave's; stage ks-1 is no longer read
    issue(ks + 3);
    read_stage(ks + 1, an, bn);  // past the end: clamped loads, unused
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[i][t] = mfma(ac[i], bc[t], acc[i][t]);
    // interleave: after the LDS reads, one MFMA then three vector ALU ops
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);  // DS reads
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);  // VALU
    }
  };
  issue(0);
  issue(1);
  issue(2);
  DFSSM_WAIT_VMCNT(2 * kLoadsPerStage);  // stage 0 landed, stages 1 and 2 in flight
  DFSSM_BARRIER();
  read_stage(0, a0, b0);
  int ks = 0;
  for (; ks + 1 < nks; ks += 2) {
    step(ks, a0, b0, a1, b1);
    step(ks + 1, a1, b1, a0, b0);
  }
  if (ks < nks) step(ks, a0, b0, a1, b1);
  // the ring is reused below: drain the loads still in flight and wait for
  // every wave to finish its last stage
  DFSSM_WAIT_VMCNT(0);
  __syncthreads();

  // ---- epilogue, one n-subtile (16 output rows) at a time: the LoRA term
  //      from four limb MFMAs (exact int64 acc_b = E_lo + 65536*E_hi) on
  //      operands staged in LDS, then acc_s = 2*D - sum Q and
  //      y = s*(alpha*fs + beta*fb); y leaves through a per-wave LDS
  //      transpose as 16-byte row pieces
  const bool baligned = (r % 16) == 0;
  auto swz = [](int rr) { return (rr >> 2) & 3; };
  // stage 64 LoRA columns [j0, j0+64): limbs of the tile's rows, B of its
  // columns; 10 x 16 bytes per thread, all loads issued before the stores
  auto stage_lora = [&](int j0) {
    uint4 lv[8], bv[2];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int idx = tid + u * kThreads;  // (limb, row, 16-byte chunk)
      const int limb = idx >> 9, ml = (idx >> 2) & 127, c = idx & 3;
      const int m = min(m0 + ml, M - 1);
      lv[u] = *reinterpret_cast<const uint4*>(limbs + ((int64_t)limb * M + m) * rp + j0 + 16 * c);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int idx = tid + u * kThreads;  // (row, 16-byte chunk)
      const int nl = idx >> 2, c = idx & 3;
      const int n = min(n0 + nl, N - 1);
      const v4i b = load16_guarded(B + (int64_t)n * r, j0 + 16 * c, r, baligned);
      bv[u] = make_uint4((uint32_t)b[0], (uint32_t)b[1], (uint32_t)b[2], (uint32_t)b[3]);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int idx = tid + u * kThreads;
      const int limb = idx >> 9, ml = (idx >> 2) & 127, c = idx & 3;
      const uint32_t mk = m0 + ml < M ? ~0u : 0u;
      *reinterpret_cast<uint4*>(limb_lds + (limb * kBM + ml) * kBK + 16 * (c ^ swz(ml))) =
          make_uint4(lv[u].x & mk, lv[u].y & mk, lv[u].z & mk, lv[u].w & mk);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int idx = tid + u * kThreads;
      const int nl = idx >> 2, c = idx & 3;
      const uint32_t mk = n0 + nl < N ? ~0u : 0u;
      *reinterpret_cast<uint4*>(b_lds + nl * kBK + 16 * (c ^ swz(nl))) =
          make_uint4(bv[u].x & mk, bv[u].y & mk, bv[u].z & mk, bv[u].w & mk);
    }
  };
  if (kLoraLds && r > 0) {
    stage_lora(0);
    __syncthreads();
  }
  float* ybuf = reinterpret_cast<float*>(lds_raw + 4 * kBM * kBK + kBN * kBK) + wave * 16 * kYPitch;
  const int sw = 16 * (kg ^ swz(row));
  const bool nvec = (N & 3) == 0;  // rows of y are 16-byte aligned
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    v4i ehi[4], elo[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ehi[i] = elo[i] = zero4();
    const int nl = (wave & 1) * 64 + 16 * t + row;
    const int n = n0 + nl;
    if (r > 0) {
#pragma unroll
      for (int pass = 0; pass < 4; ++pass) {  // limbs 3, 2, 1, 0
        const int limb = 3 - pass;
        if constexpr (kLoraLds) {  // rank <= 64: one chunk, operands in LDS
          const v4i bl = *reinterpret_cast<const v4i*>(b_lds + nl * kBK + sw);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int ml = (wave >> 1) * 64 + 16 * i + row;
            const v4i al = *reinterpret_cast<const v4i*>(limb_lds + (limb * kBM + ml) * kBK + sw);
            if (limb >= 2)
              ehi[i] = mfma(al, bl, ehi[i]);
            else
              elo[i] = mfma(al, bl, elo[i]);
          }
        } else {  // higher rank: operands straight from memory
          for (int j0 = 0; j0 < rp; j0 += 64) {
            const int jj = j0 + 16 * kg;
            const v4i bl = n < N ? load16_guarded(B + (int64_t)n * r, jj, r, baligned) : zero4();
            v4i al[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int m = wm0 + 16 * i + row;
              al[i] = m < M ? load16(limbs + ((int64_t)limb * M + m) * rp + jj) : zero4();
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              if (limb >= 2)
                ehi[i] = mfma(al[i], bl, ehi[i]);
              else
                elo[i] = mfma(al[i], bl, elo[i]);
            }
          }
        }
        if (limb == 3 || limb == 1) {  // scale the high digit's sum by 256
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (limb == 3)
              ehi[i] = ehi[i] << 8;
            else
              elo[i] = elo[i] << 8;
          }
        }
      }
    }
    const float al = al_lds[nl], be = be_lds[nl];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int mlb = (wave >> 1) * 64 + 16 * i + 4 * kg;  // this lane's rows mlb + v
      const float4 s4 = *reinterpret_cast<const float4*>(&s_lds[mlb]);
      const int4 q4 = *reinterpret_cast<const int4*>(&sq_lds[mlb]);
      const float sv[4] = {s4.x, s4.y, s4.z, s4.w};
      const int32_t qv[4] = {q4.x, q4.y, q4.z, q4.w};
      float yv[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int32_t as = 2 * acc[i][t][v] - qv[v];
        const int32_t hi = ehi[i][v], lo = elo[i][v];
        yv[v] = dfssm_dev::epilogue(sv[v], al, be, as, hi, lo, r > 0);
        const int m = m0 + mlb + v;
        if (m < M && n < N) {
          if (acc_s_out) acc_s_out[(int64_t)m * N + n] = as;
          if (acc_b_out) acc_b_out[(int64_t)m * N + n] = r > 0 ? (int64_t)lo + ((int64_t)hi << 16) : 0;
        }
      }
      if (y) {
        // [row 4*kg + v][column row] in, [row lane/4][columns 4*(lane%4)..+3]
        // out; the buffer is this wave's own and LDS instructions of one
        // wave complete in order, so no barrier is involved
#pragma unroll
        for (int v = 0; v < 4; ++v) ybuf[(4 * kg + v) * kYPitch + row] = yv[v];
        const int mr = lane >> 2, nc = 4 * (lane & 3);
        const float4 o = *reinterpret_cast<const float4*>(&ybuf[mr * kYPitch + nc]);
        const int m = m0 + (wave >> 1) * 64 + 16 * i + mr;
        const int nn = n0 + (wave & 1) * 64 + 16 * t + nc;
        if (m < M) {
          float* dst = y + (int64_t)m * N + nn;
          if (nvec && nn + 3 < N) {
            *reinterpret_cast<float4*>(dst) = o;
          } else {
            const float ov[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (nn + e < N) dst[e] = ov[e];
          }
        }
      }
    }
  }
}

}  // namespace

namespace dfssm {

hipError_t launch_mfma_linear(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                              int64_t r, const uint32_t* w_bits, const float* alpha,
                              const int8_t* A, const int8_t* B, const float* beta, float* y,
                              int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                              const LinearWorkspace& ws, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  const int rp = (int)rank_padded(r);
  mfma_lora_down<<<dim3((unsigned)ceil_div(M, 16), (unsigned)(rp / 16)), dim3(kThreads), 0, st>>>(
      q, (int)M, (int)K, (int)r, rp, A, ws.acc_a, ws.limbs, ws.sumq);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (acc_a_out && r > 0) {
    e = hipMemcpyAsync(acc_a_out, ws.acc_a, (size_t)(M * r) * 4, hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
  }
  const int64_t nbm = ceil_div(M, kBM), nbn = ceil_div(N, kBN);
  if (rp == 64)
    mfma_scaffold<true><<<dim3((unsigned)(nbm * nbn)), dim3(kThreads), 0, st>>>(
        q, s, (int)M, (int)K, (int)N, (int)r, rp, w_bits, alpha, ws.limbs, B, beta, ws.sumq, y,
        acc_s, acc_b, (int)nbm, (int)nbn);
  else
    mfma_scaffold<false><<<dim3((unsigned)(nbm * nbn)), dim3(kThreads), 0, st>>>(
        q, s, (int)M, (int)K, (int)N, (int)r, rp, w_bits, alpha, ws.limbs, B, beta, ws.sumq, y,
        acc_s, acc_b, (int)nbm, (int)nbn);
  return hipGetLastError();
}

}  // namespace dfssm
