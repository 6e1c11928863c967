// dfssm_mfma.hip -- prefill-shaped (large M) scaffold + LoRA linear on the
// gfx950 int8 matrix cores (v_mfma_i32_16x16x64_i8).
//
// The sign bits are expanded on chip, in registers, to {0,1} bytes (a
// nibble n becomes bytes via (n * 0x00204081) & 0x01010101), so the MFMA
// computes D[n,m] = sum_{bit=1} Q[m,k] and acc_s = 2*D - sum_k Q[m,k]; the
// expanded signs never touch memory or LDS (the paper expands to int8 "on
// the fly" ahead of a library int8 GEMM, Sec. 4.1).  An expanded operand
// costs 12 vector instructions and feeds 8 MFMAs (a wave covers 128 tokens),
// which keeps the vector ALU below the matrix core.
//
// Operand layout of v_mfma_i32_16x16x64_i8 (wave64): lane l supplies row
// (l % 16) of the first operand and column (l % 16) of the second, each as
// 16 consecutive K-bytes of K-group (l / 16); the 16x16 int32 result D has
// D[4*(l/16)+v][l%16] in lane l, register v.
//
// LoRA: lora_down computes acc_a = Q * A^T with the same MFMA and writes it
// as 4 signed base-256 int8 limbs.  After the scaffold K-loop the main kernel
// gets the exact int64 acc_b = sum_j B[n,j] acc_a[m,j] from four int8 MFMAs
// per 16x16 tile, E_hi = 256*(B.L3) + B.L2 and E_lo = 256*(B.L1) + B.L0
// (each < 2^31 for r <= 256), acc_b = E_lo + 65536*E_hi, so the K-loop holds
// only the scaffold accumulators.
#include <stdlib.h>

#include <algorithm>
#include <atomic>

#include "dfssm_internal.hpp"

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
// acc_a = Q A^T on the same MFMA.  A block owns 16 tokens x 32 ranks (two
// 16-rank tiles; blockIdx.y walks the padded rank range rp); its 16 waves
// split the K steps, each issuing the loads of up to kLdBatch steps before
// its first multiply, and reduce their partial sums in LDS.  The block writes
// acc_a, its 4 signed base-256 int8 limbs (zero for ranks in [r, rp)) and,
// for blockIdx.y == 0, sum_k Q[m,k].
constexpr int kLdThreads = 1024;
constexpr int kLdWaves = kLdThreads / 64;
constexpr int kLdRanks = 32;
constexpr int kLdBatch = 4;
constexpr int kLdPitch = 17;  // padded rank pitch of the partial sums

__global__ __launch_bounds__(kLdThreads) void mfma_lora_down(const int8_t* __restrict__ q, int M, int K,
                                                             int r, int rp, const int8_t* __restrict__ A,
                                                             int32_t* __restrict__ acc_a,
                                                             int8_t* __restrict__ limbs,
                                                             int32_t* __restrict__ sumq) {
  __shared__ int32_t part[kLdWaves][kLdRanks * kLdPitch];
  __shared__ int32_t qpart[kLdWaves][16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = lane & 15, kg = lane >> 4;
  const int m0 = blockIdx.x * 16, j0 = blockIdx.y * kLdRanks;
  const bool first = blockIdx.y == 0;  // the rank block that also sums Q
  const int m = m0 + row;
  const bool m_ok = m < M;
  const int8_t* qrow = q + (int64_t)(m_ok ? m : 0) * K;
  const int8_t* arow[2];
  bool j_ok[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int j = j0 + 16 * u + row;
    j_ok[u] = j < r;
    arow[u] = A + (int64_t)(j_ok[u] ? j : 0) * K;
  }
  const int nks = (K + 63) / 64;
  const int per = (nks + kLdWaves - 1) / kLdWaves;
  const int ks0 = wave * per, ks1 = min(nks, ks0 + per);

  v4i acc[2] = {zero4(), zero4()};
  int qs = 0;
  for (int kb = ks0; kb < ks1; kb += kLdBatch) {
    // every load of the batch first (steps past ks1 are skipped, uniformly)
    v4i b[kLdBatch], a0[kLdBatch], a1[kLdBatch];
#pragma unroll
    for (int u = 0; u < kLdBatch; ++u) {
      b[u] = a0[u] = a1[u] = zero4();
      if (kb + u < ks1) {
        const int kk = (kb + u) * 64 + 16 * kg;
        const int kc = kk < K ? kk : 0;  // K % 32 == 0: a 16-byte chunk is wholly in or out
        b[u] = load16(qrow + kc);
        if (r > 0) {
          a0[u] = load16(arow[0] + kc);
          a1[u] = load16(arow[1] + kc);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kLdBatch; ++u) {
      if (kb + u < ks1) {
        const int kk = (kb + u) * 64 + 16 * kg;
        if (!(m_ok && kk < K)) b[u] = zero4();
        if (!j_ok[0]) a0[u] = zero4();
        if (!j_ok[1]) a1[u] = zero4();
        if (first) {
#pragma unroll
          for (int t = 0; t < 4; ++t) qs = __builtin_amdgcn_sdot4(b[u][t], 0x01010101, qs, false);
        }
        // D[rank][token]: the A rows are the first operand
        acc[0] = mfma(a0[u], b[u], acc[0]);
        acc[1] = mfma(a1[u], b[u], acc[1]);
      }
    }
  }
  // lane (row, kg) holds D[rank 16u + 4kg + v][token row]
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) part[wave][(16 * u + 4 * kg + v) * kLdPitch + row] = acc[u][v];
  if (first) {
    qs += __shfl_xor(qs, 16, 64);
    qs += __shfl_xor(qs, 32, 64);
    if (kg == 0) qpart[wave][row] = qs;
  }
  __syncthreads();
  {
    // thread i: token i / 32, rank i % 32 (consecutive threads, consecutive ranks)
    const int i = threadIdx.x;
    const int ml = i >> 5, jl = i & 31;
    const int mm = m0 + ml, jj = j0 + jl;
    if (ml < 16 && mm < M) {  // threads past 16 tokens x 32 ranks have nothing to reduce
      int32_t val = 0;
#pragma unroll
      for (int w = 0; w < kLdWaves; ++w) val += part[w][jl * kLdPitch + ml];
      int8_t d[4];
      dfssm_dev::split_limbs(jj < r ? val : 0, d);
#pragma unroll
      for (int l = 0; l < 4; ++l) limbs[((int64_t)l * M + mm) * rp + jj] = d[l];
      if (jj < r) acc_a[(int64_t)mm * r + jj] = val;
    }
  }
  if (first && threadIdx.x < 16 && m0 + (int)threadIdx.x < M) {
    int32_t t = 0;
#pragma unroll
    for (int w = 0; w < kLdWaves; ++w) t += qpart[w][threadIdx.x];
    sumq[m0 + threadIdx.x] = t;
  }
}

// ------------------------------------------------------------ scaffold GEMM
// Operand roles: the expanded signs are the MFMA's first operand (rows =
// output rows n) and the codes Q its second (columns = tokens m), so lane
// (rho, kg) of a 16x16 result holds D[n = 4kg + v][m = rho] for v = 0..3:
// four consecutive outputs of one token row, stored as one 16-byte write.
//
// Block: 128 tokens x a run of 16-row "row tiles".  The row tiles of each
// 128-token slice are dealt to blocks in runs whose lengths differ by at most
// one and are at most 17, with enough blocks per slice to fill the chip's
// block slots (two per CU) in whole rounds -- so every block finishes at about
// the same time and no round of leftover tiles follows.  Wave w owns row
// tiles 4w .. 4w+3 of the run (wave tile 128 x 64: each expanded sign operand
// feeds 8 MFMAs, and the Q tile in LDS is shared by the 4 waves); a 17th row
// tile is shared by all 4 waves, wave w taking its token tiles 2w and 2w+1.
// Short forms (every run of the grid at most 4, or at most kShortRun = 8,
// row tiles, e.g. a few hundred tokens): wave w takes token tiles 2w and
// 2w+1 of every row tile of the run and skips token tiles past M, so the 4
// waves share a short run's MFMAs instead of each multiplying its 4 row
// tiles whatever the run (three blocks per CU).  The 8-tile form holds
// twice the accumulators; runs of at most 4 keep the smaller one.
//
// K-loop: 64 K per stage; operands reach LDS by direct-to-LDS loads
// (global_load_lds with a scalar base and a per-lane offset that stays
// fixed, so the loop does no per-lane address arithmetic):
//   Q stage: a kStages-deep ring of 128 rows x 64 bytes, the four 16-byte
//            chunks of row m stored at chunk slot c ^ ((m >> 1) & 3), so each
//            8 lanes of a 16-byte LDS read hit 8 distinct 4-bank groups of
//            the 32 banks;
//   signs:   loaded per "sign group" of kSgStages stages, i.e. 32 bytes of
//            each row, into two alternating buffers: per wave its 64 rows
//            (row tiles 4w .. 4w+3), then the 17th row tile's 16 rows, each
//            row as 8 words.  A load instruction covers 8 whole rows (lane i:
//            word i % 8 of row i / 8), so it touches 8 cache lines where a
//            load of one stage's words of 32 rows touched 32.  Word j of a
//            row (16-row tile position rho) sits at slot j ^ (2*((rho >> 2) & 3)),
//            which makes the per-stage 4-byte reads of 16 rows x 2 words hit
//            32 distinct banks.
// Each wave issues 2 Q loads per stage and 9 sign loads per sign group (the
// 17th tile's words whether or not the run has one), so "stage ks has
// landed" is a count of vector-memory operations.
constexpr int kThreads = 256;
constexpr int kBM = 128;
constexpr int kBK = 64;
constexpr int kStages = 4;
constexpr int kRunMax = 17;                             // row tiles per block
constexpr int kQStage = kBM * kBK;                      // 8 KB
constexpr int kQRing = kStages * kQStage;               // 32 KB
constexpr int kSgStages = 4;                            // stages per sign group (8 words per row)
constexpr int kSgWave = 64 * 32;                        // 2 KB: a wave's 64 rows x 32 bytes
constexpr int kSgBuf = 4 * kSgWave + 16 * 32;           // + the 17th tile's rows: 8.5 KB
constexpr int kLq = 2;                                  // Q loads per wave per stage
constexpr int kLsg = 9;                                 // sign loads per wave per sign group
constexpr int kLdsRing = kQRing + 2 * kSgBuf;           // 49 KB
constexpr int kLimbBytes = 4 * kBM * 64;                // LoRA limbs of the tile, 64 ranks
constexpr int kLdsLora = kLimbBytes + kRunMax * 16 * 64;  // + B rows of the run
constexpr int kLdsBytes = kLdsRing > kLdsLora ? kLdsRing : kLdsLora;
constexpr int kMaxRows = kRunMax * 16;
constexpr int kShortRun = 8;  // row tiles per run, at most, of the short form
static_assert(kSgStages == kStages, "a sign group is one pass over the Q ring");
static_assert(2 * kLq + kLsg + kLq <= 63, "vector-memory counter range");

typedef __attribute__((address_space(3))) void lds_void;

// Direct-to-LDS loads (gfx950 global_load_lds): lane i's 16 (or 4) bytes from
// sbase + voff land at m0 + 16*i (4*i).  Inline assembly, so the compiler does
// not make every later LDS read wait for them; the K-loop orders them with
// DFSSM_WAIT_VMCNT and the barrier.
__device__ __forceinline__ void lds_dma16(uint32_t voff, const void* sbase, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ void lds_dma4(uint32_t voff, const void* sbase, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}

// s_waitcnt with only the vector-memory counter constrained
#define DFSSM_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(0x0F70 | ((n) & 0xF) | (((n) >> 4) << 14))
// s_waitcnt with only the LDS/scalar counter constrained, to zero
#define DFSSM_WAIT_LGKM0() __builtin_amdgcn_s_waitcnt(0xC07F)
// workgroup barrier that does not drain outstanding direct-to-LDS loads
// (the compiler's barrier fence would wait for all of them); LDS visibility
// of the loads is ordered by the DFSSM_WAIT_VMCNT before it
#define DFSSM_BARRIER() asm volatile("s_barrier" ::: "memory")

// A zero the compiler cannot see through: per-lane arithmetic of rarely
// taken edge paths that uses it stays inside the K-loop instead of being
// hoisted into registers that would live across the loop.
__device__ __forceinline__ int opaque_zero() {
  int z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z));
  return z;
}

// 16-byte chunk swizzle of 64-byte rows: conflict-free 16-byte reads of one
// chunk column on gfx950's 32-bank LDS
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 3; }

struct GemmArgs {
  const int8_t* q;
  const float* s;
  int M, K, N, r, rp;
  const uint32_t* w_bits;
  const float* alpha;
  const int8_t* limbs;
  const int8_t* B;
  const float* beta;
  const int32_t* sumq;
  float* y;
  int32_t* acc_s_out;
  int64_t* acc_b_out;
  int nt16;  // row tiles of N: ceil(N / 16)
  int bpm;   // blocks per 128-token slice
};

// Tile index of block b among cnt blocks whose XCD is b % 8: each XCD gets a
// contiguous run of the slice-major block list, so it works on few token rows
// (its Q rows stay in its L2) across all their output rows.
__device__ __forceinline__ int xcd_tile(int b, int cnt) {
  const int per = cnt / 8, rem = cnt % 8;
  const int x = b % 8, idx = b / 8;
  return (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + idx;
}

// LoRA limb products of one 16x16 tile for rank above 64, operands straight
// from memory, 64 ranks at a time
__device__ __forceinline__ void lora_from_memory(const GemmArgs& a, int nrow, int mrow, int kg, v4i& ehi,
                                                 v4i& elo) {
  const bool baligned = (a.r % 16) == 0;
  ehi = zero4();
  elo = zero4();
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {  // limbs 3, 2, 1, 0
    const int limb = 3 - pass;
    v4i e = limb >= 2 ? ehi : elo;
    for (int j0 = 0; j0 < a.rp; j0 += 64) {
      const v4i bl = load16_guarded(a.B + (int64_t)nrow * a.r, j0 + 16 * kg, a.r, baligned);
      const v4i al = load16(a.limbs + ((int64_t)limb * a.M + mrow) * a.rp + j0 + 16 * kg);
      e = mfma(bl, al, e);
    }
    if (limb == 3 || limb == 1) e = e << 8;
    if (limb >= 2)
      ehi = e;
    else
      elo = e;
  }
}

// LDS-side state of a block, shared by the K-loop and the epilogue
struct TileLds {
  int8_t* lds;     // ring, then LoRA staging
  float* al;       // alpha of the run's rows
  float* be;       // beta of the run's rows
  float* sv;       // s of the tile's tokens
  int32_t* sq;     // sum Q of the tile's tokens
};

// Outputs of one 16x16 tile (row tile at row offset nl of the run, token
// tile i): the LoRA term from four limb MFMAs (exact int64 acc_b = E_lo +
// 65536*E_hi, E_hi = 256*(B.L3) + B.L2, E_lo = 256*(B.L1) + B.L0), then
// acc_s = 2*D - sum Q and y = s*(alpha*fs + beta*fb).  kLdsLora: the limbs
// and B rows are in LDS (rank <= 64); otherwise the LoRA operands come from
// memory (rank above 64) or there is no LoRA (rank 0).  kChecked: rows past
// M or N, unaligned rows of y and the accumulator outputs are handled.
template <bool kLdsLora, bool kChecked>
__device__ __forceinline__ void tile_out(const GemmArgs& a, const TileLds& L, const v4i& acc, const v4i& bop,
                                         const v4i (&lm)[4], int m0, int n0, int nl, int i, int rho, int kg) {
  const int M = a.M, N = a.N;
  const bool lora = a.r > 0;
  const int ml = 16 * i + rho;
  const int m = m0 + ml;
  const int n = n0 + nl + 4 * kg;  // this lane's rows n .. n+3
  v4i ehi = zero4(), elo = zero4();
  if (kLdsLora) {
    ehi = mfma(bop, lm[3], ehi);
    ehi = ehi << 8;
    ehi = mfma(bop, lm[2], ehi);
    elo = mfma(bop, lm[1], elo);
    elo = elo << 8;
    elo = mfma(bop, lm[0], elo);
  } else if (lora) {
    lora_from_memory(a, min(n0 + nl + rho, N - 1), min(m, M - 1), kg, ehi, elo);
  }
  const float4 al4 = *reinterpret_cast<const float4*>(&L.al[nl + 4 * kg]);
  const float4 be4 = *reinterpret_cast<const float4*>(&L.be[nl + 4 * kg]);
  const float alv[4] = {al4.x, al4.y, al4.z, al4.w};
  const float bev[4] = {be4.x, be4.y, be4.z, be4.w};
  const float sm = L.sv[ml];
  const int qm = L.sq[ml];
  float yv[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int32_t as = 2 * acc[v] - qm;
    yv[v] = dfssm_dev::epilogue(sm, alv[v], bev[v], as, ehi[v], elo[v], kLdsLora || lora);
    if (kChecked && m < M && n + v < N) {
      if (a.acc_s_out) a.acc_s_out[(int64_t)m * N + n + v] = as;
      if (a.acc_b_out) a.acc_b_out[(int64_t)m * N + n + v] = lora ? (int64_t)elo[v] + ((int64_t)ehi[v] << 16) : 0;
    }
  }
  float* dst = a.y + (int64_t)m * N + n;
  if (!kChecked) {
    *reinterpret_cast<float4*>(dst) = make_float4(yv[0], yv[1], yv[2], yv[3]);
  } else if (m < M) {
    if ((N & 3) == 0 && n + 3 < N) {
      *reinterpret_cast<float4*>(dst) = make_float4(yv[0], yv[1], yv[2], yv[3]);
    } else {
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (n + v < N) dst[v] = yv[v];
    }
  }
}

// Epilogue of the block, per wave: its (up to) 4 row tiles x 8 token tiles,
// then its 2 token tiles (xtok, xtok+1) of the shared row tile at row offset
// xrow of the run.
template <bool kLdsLora, bool kChecked>
__device__ __forceinline__ void block_epilogue(const GemmArgs& a, const TileLds& L, const v4i (&acc)[4][8],
                                               const v4i (&accx)[2], int m0, int n0, int wave, int ntw,
                                               bool extra, int xrow, int xtok, int rho, int kg, int l_off) {
  const int8_t* limb_lds = L.lds;
  const int8_t* b_lds = L.lds + kLimbBytes;
  v4i bop[4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
    bop[t] = kLdsLora ? *reinterpret_cast<const v4i*>(b_lds + (64 * wave + 16 * t) * 64 + l_off) : zero4();
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    v4i lm[4];
#pragma unroll
    for (int l = 0; l < 4; ++l)
      lm[l] = kLdsLora ? *reinterpret_cast<const v4i*>(limb_lds + (l * kBM + 16 * i) * 64 + l_off) : zero4();
    if (ntw == 4) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
        tile_out<kLdsLora, kChecked>(a, L, acc[t][i], bop[t], lm, m0, n0, 64 * wave + 16 * t, i, rho, kg);
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (t < ntw) tile_out<kLdsLora, kChecked>(a, L, acc[t][i], bop[t], lm, m0, n0, 64 * wave + 16 * t, i, rho, kg);
    }
  }
  if (extra) {
    const v4i bx = kLdsLora ? *reinterpret_cast<const v4i*>(b_lds + xrow * 64 + l_off) : zero4();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int i = xtok + h;
      v4i lm[4];
#pragma unroll
      for (int l = 0; l < 4; ++l)
        lm[l] = kLdsLora ? *reinterpret_cast<const v4i*>(limb_lds + (l * kBM + 16 * i) * 64 + l_off) : zero4();
      tile_out<kLdsLora, kChecked>(a, L, accx[h], bx, lm, m0, n0, xrow, i, rho, kg);
    }
  }
}

// Epilogue of a short run (at most kShortRun row tiles), per wave: token
// tiles 2w and 2w+1 of each row tile, held in acc[t][0] and acc[t][1].
template <bool kLdsLora, bool kChecked, int kSR>
__device__ __forceinline__ void short_epilogue(const GemmArgs& a, const TileLds& L, const v4i (&acc)[kSR][2], int m0,
                                               int n0, int wave, int cnt, int ntt, int rho, int kg, int l_off) {
  const int8_t* limb_lds = L.lds;
  const int8_t* b_lds = L.lds + kLimbBytes;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int i = 2 * wave + h;
    if (i >= ntt) continue;  // uniform: no token of the block in this tile
    v4i lm[4];
#pragma unroll
    for (int l = 0; l < 4; ++l)
      lm[l] = kLdsLora ? *reinterpret_cast<const v4i*>(limb_lds + (l * kBM + 16 * i) * 64 + l_off) : zero4();
#pragma unroll
    for (int t = 0; t < kSR; ++t) {
      if (t < cnt) {
        const v4i bop = kLdsLora ? *reinterpret_cast<const v4i*>(b_lds + (16 * t) * 64 + l_off) : zero4();
        tile_out<kLdsLora, kChecked>(a, L, acc[t][h], bop, lm, m0, n0, 16 * t, i, rho, kg);
      }
    }
  }
}

template <bool kLoraLds, int kSR>
__device__ __forceinline__ void scaffold_block(const GemmArgs& a, const TileLds& L, int m0, int rt0, int cnt) {
  const int M = a.M, K = a.K, N = a.N, r = a.r, rp = a.rp;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS addresses of the loads
  const int rho = lane & 15, kg = lane >> 4;
  const int W = K >> 5;
  const int nks = (K + kBK - 1) / kBK;
  const bool ktail = (K & (kBK - 1)) != 0;  // the last stage holds 32 columns
  const int n0 = 16 * rt0;
  const int cmain = min(cnt, 16);
  const int ntw = min(max(cmain - 4 * wave, 0), 4);  // this wave's row tiles
  const bool extra = cnt > 16;                        // the 17th row tile
  // kSR > 0 (every run of the grid holds at most kSR row tiles): wave
  // w multiplies token tiles 2w and 2w+1 of every row tile of the run (the
  // sign words of the areas of waves 0 and 1, which hold the run's rows
  // 0-63 and 64-127), so the 4 waves share the work; token tiles past M are
  // skipped
  constexpr bool kShort = kSR > 0;
  constexpr bool shortrun = kShort;
  // the short forms read only the sign areas of waves 0 (and 1): the other
  // waves load no sign words (and count none in their waits)
  const bool sign_wave = !kShort || wave < (kSR > 4 ? 2 : 1);  // uniform
  const int ntt = min(8, (M - m0 + 15) >> 4);  // token tiles holding tokens
  const int nrows = 16 * cnt;
  int8_t* const lds = L.lds;


  // ---- direct-to-LDS load constants: per-lane offsets fixed for the loop
  //      (rows past M or N read the last row; their outputs are never stored)
  uint32_t voff_q[2], lds_q[2];
  bool hi_chunk[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int slot = 64 * (2 * wave + j) + lane;  // 16-byte slot in the Q stage
    const int m = slot >> 2;
    const int c = (lane & 3) ^ swz(m);
    hi_chunk[j] = c >= 2;
    voff_q[j] = (uint32_t)((min(m0 + m, M - 1) - m0) * K + 16 * c);
    lds_q[j] = 1024u * (2 * wave + j);
  }
  // sign words, per sign group: 8 loads of the wave's rows (lane i: row
  // 8j + i / 8 of the wave's 64, word slot i % 8), then the 17th tile's rows
  // 4w .. 4w+3 (lanes < 32).  Rows 8j + i/8 have (row >> 2) & 3 =
  // (2j + i / 32) & 3, so the swizzled word a lane fetches depends on j only
  // through its parity.  Rows past N read row N - 1 (never stored).
  const bool sg_fast = n0 + 64 * wave + 64 <= N;  // uniform: no row of the wave is clamped
  uint32_t voff_s[2];
#pragma unroll
  for (int jp = 0; jp < 2; ++jp) {
    const int wd = (lane & 7) ^ (2 * ((2 * jp + (lane >> 5)) & 3));
    voff_s[jp] = (uint32_t)((((lane >> 3) + 64 * wave) * W + wd) * 4);
  }
  uint32_t voff_x;
  {
    const int rr = 4 * wave + (lane >> 3);  // row of the 17th tile (< 16 for lanes < 32)
    const int wd = (lane & 7) ^ (2 * ((rr >> 2) & 3));
    const int n = min(n0 + 256 + rr, N - 1);
    voff_x = (uint32_t)(((n - n0) * W + wd) * 4);
  }
  const int8_t* qbase = a.q + (int64_t)m0 * K;
  const uint32_t* wbase = a.w_bits + (int64_t)n0 * W;
  const uint32_t lds0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(uintptr_t)(lds_void*)lds);

  // the sign group of stages 4g .. 4g+3 into buffer g % 2; the last group
  // may reach past the row (K % 256 != 0): its words are clamped to the
  // row's last word, and a stage that would use them does not exist (or has
  // its second word zeroed: K % 64 == 32)
  auto issue_signs = [&](int g) {
    const uint32_t sb = lds0 + kQRing + (g & 1) * kSgBuf;
    const uint32_t* ws = wbase + 8 * g;
    const bool whole = 8 * g + 8 <= W;  // uniform
    if (sg_fast && whole) {
#pragma unroll
      for (int j = 0; j < 8; ++j) lds_dma4(voff_s[j & 1], ws + (int64_t)8 * j * W, sb + kSgWave * wave + 256u * j);
    } else {
      const int ln = lane + opaque_zero();
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int rl = 8 * j + (ln >> 3);  // row of the wave's 64
        const int wd = (ln & 7) ^ (2 * ((rl >> 2) & 3));
        const int n = min(n0 + 64 * wave + rl, N - 1);
        const int wc = min(8 * g + wd, W - 1) - 8 * g;
        lds_dma4((uint32_t)(((n - n0) * W + wc) * 4), ws, sb + kSgWave * wave + 256u * j);
      }
    }
    {
      uint32_t vx = voff_x;
      if (!whole) {
        const int ln = lane + opaque_zero();
        const int rr = 4 * wave + (ln >> 3);
        const int wd = (ln & 7) ^ (2 * ((rr >> 2) & 3));
        const int n = min(n0 + 256 + rr, N - 1);
        vx = (uint32_t)(((n - n0) * W + min(8 * g + wd, W - 1) - 8 * g) * 4);
      }
      if (lane < 32) lds_dma4(vx, ws, sb + 4 * kSgWave + 128u * wave);
    }
  };
  // stage ks's Q into ring slot `slot`, preceded (ks % 4 == 0) by its sign group
  auto issue = [&](int ks, int slot) {
    if (slot == 0 && sign_wave) issue_signs(ks >> 2);
    const int8_t* qs = qbase + ks * kBK;
    const uint32_t sb = lds0 + slot * kQStage;
    if (ktail && ks == nks - 1) {
      // past K: Q chunks 2, 3 re-read chunks 0, 1 (their sign bits are
      // zeroed when the stage is used)
#pragma unroll
      for (int j = 0; j < 2; ++j) lds_dma16(voff_q[j] - (hi_chunk[j] ? 32u : 0u), qs, sb + lds_q[j]);
    } else {
#pragma unroll
      for (int j = 0; j < 2; ++j) lds_dma16(voff_q[j], qs, sb + lds_q[j]);
    }
  };

  // LDS read offsets: the Q operand of token tile i is row 16i + rho, chunk
  // kg; a lane's sign word of stage s (of its group) is word 2s + kg / 2 of
  // rows 16t + rho of its wave's area and of the 17th tile's area, at the
  // swizzled slot
  const int q_off = rho * kBK + 16 * (kg ^ swz(rho));
  // row rho of the wave's area plus the byte of the word slot before the
  // stage's ^ 8s (bits 3-4 of the row offset are zero, so ^ acts on the slot)
  const int w_off = kQRing + kSgWave * (shortrun ? 0 : wave) + 32 * rho + 4 * ((kg >> 1) ^ (2 * ((rho >> 2) & 3)));
  const int x_delta = (4 - wave) * kSgWave;  // uniform: the 17th tile's area
  const uint32_t sh = 16u * (kg & 1);

  typedef uint32_t raw_t __attribute__((ext_vector_type(4)));
  struct Raw {
    raw_t w;
    uint32_t x;
    raw_t w2;  // short form: row tiles 4-7 of the run
  };
  // sign words of stage ks (group ks / 4, stage ks % 4 of it): read one
  // stage ahead of their use
  auto read_signs = [&](int ks) -> Raw {
    const int8_t* st = lds + ((ks >> 2) & 1) * kSgBuf;
    const int wb = w_off ^ (8 * (ks & 3));
    Raw rw;
#pragma unroll
    for (int t = 0; t < 4; ++t) rw.w[t] = *reinterpret_cast<const uint32_t*>(st + wb + 512 * t);
    rw.x = *reinterpret_cast<const uint32_t*>(st + x_delta + wb);
    if constexpr (kSR > 4) {
      if (cnt > 4) {  // uniform
#pragma unroll
        for (int t = 0; t < 4; ++t) rw.w2[t] = *reinterpret_cast<const uint32_t*>(st + wb + kSgWave + 512 * t);
      }
    }
    return rw;
  };

  constexpr int kTT = kShort ? 2 : 8;          // token tiles a wave accumulates
  constexpr int kRT = kShort ? kSR : 4;        // row tiles
  v4i acc[kRT][kTT], accx[2];
#pragma unroll
  for (int t = 0; t < kRT; ++t)
#pragma unroll
    for (int i = 0; i < kTT; ++i) acc[t][i] = zero4();
  accx[0] = accx[1] = zero4();

  // multiply stage ks: the 8 Q operands are read from LDS first; then row
  // tile t's 8 MFMAs run while the vector ALU expands tile t+1's signs
  const bool kg_hi = kg >= 2;
  auto compute = [&](int ks, int slot, const Raw& rw) {
    const int8_t* st = lds + slot * kQStage + q_off;
    raw_t w = rw.w;
    uint32_t wx = rw.x;
    if (ktail && ks == nks - 1) {  // uniform: sign words past K count as 0
#pragma unroll
      for (int t = 0; t < 4; ++t) w[t] = kg_hi ? 0u : w[t];
      wx = kg_hi ? 0u : wx;
    }
    if constexpr (kShort) {
      raw_t w2 = rw.w2;
      if (kSR > 4 && ktail && ks == nks - 1) {
#pragma unroll
        for (int t = 0; t < 4; ++t) w2[t] = kg_hi ? 0u : w2[t];
      }
      if (2 * wave < ntt) {  // uniform
        const v4i qa = *reinterpret_cast<const v4i*>(st + (2 * wave) * 16 * kBK);
        const v4i qb = *reinterpret_cast<const v4i*>(st + (2 * wave + 1) * 16 * kBK);
#pragma unroll
        for (int t = 0; t < kSR; ++t) {
          if (t < cnt) {
            const v4i sg = expand16_at(t < 4 ? w[t] : w2[t - 4], sh);
            acc[t][0] = mfma(sg, qa, acc[t][0]);
            acc[t][1] = mfma(sg, qb, acc[t][1]);
          }
        }
      }
    } else {
    v4i qv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) qv[i] = *reinterpret_cast<const v4i*>(st + i * 16 * kBK);
    {
      // waves owning fewer than 4 row tiles (a short run) multiply all 4
      // anyway: the rows past their run are valid clamped reads and their
      // results are never stored
      v4i sg = expand16_at(w[0], sh);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const v4i sgn = t + 1 < 4 ? expand16_at(w[t + 1], sh) : sg;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[t][i] = mfma(sg, qv[i], acc[t][i]);
        sg = sgn;
      }
      // the LDS reads, the first expansion, then per row tile 8 MFMAs with
      // the next tile's 12 expansion instructions between them
      __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);   // DS reads
      __builtin_amdgcn_sched_group_barrier(0x002, 12, 0);  // VALU
#pragma unroll
      for (int t = 0; t < 3; ++t) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // VALU
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
        }
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    }
    if (extra) {  // uniform: the 17th row tile, token tiles 2w and 2w+1
      const v4i sx = expand16_at(wx, sh);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if ((i >> 1) == wave) accx[i & 1] = mfma(sx, qv[i], accx[i & 1]);
    }
    }
  };

  // one stage: make stage ks+1 visible, refill the ring slot of stage ks-1
  // (every wave has finished reading it: it passed this barrier after its
  // multiplies of stage ks-1) and, at a group start, the sign buffer of the
  // group before last; read stage ks+1's sign words, multiply ks.  Only the
  // loads of stage ks+2 (issued one step earlier, with its sign group when
  // ks+2 starts one) may stay in flight.
  auto step = [&](int ks, int slot, const Raw& wc, Raw& wn_) {
    static_assert(kStages == 4, "wait counts below");
    if (ks + 1 < nks) {
      if (ks + 2 < nks) {
        if ((slot + 2) % kStages == 0 && sign_wave)
          DFSSM_WAIT_VMCNT(kLq + kLsg);
        else
          DFSSM_WAIT_VMCNT(kLq);
      } else {
        DFSSM_WAIT_VMCNT(0);
      }
      DFSSM_BARRIER();
      if (ks + kStages - 1 < nks) issue(ks + kStages - 1, (slot + kStages - 1) % kStages);
      wn_ = read_signs(ks + 1);
    }
    compute(ks, slot, wc);
  };

#pragma unroll
  for (int p = 0; p < kStages - 1; ++p)
    if (p < nks) issue(p, p);
  // per-row and per-token scalars of the block (read after the K-loop's
  // final barrier), loaded while the prologue stages are in flight (the
  // compiler's wait for these loads also covers the stages)
  for (int x = tid; x < nrows; x += kThreads) {
    const int n = min(n0 + x, N - 1);
    L.al[x] = a.alpha[n];
    L.be[x] = r > 0 ? a.beta[n] : 0.0f;
  }
  if (tid < kBM) {
    const int m = min(m0 + tid, M - 1);
    L.sv[tid] = a.s[m];
    L.sq[tid] = a.sumq[m];
  }
  // stage 0 (with sign group 0) has landed once at most the later prologue
  // stages' Q loads are in flight
  if (nks >= 3)
    DFSSM_WAIT_VMCNT(2 * kLq);
  else if (nks == 2)
    DFSSM_WAIT_VMCNT(kLq);
  else
    DFSSM_WAIT_VMCNT(0);
  DFSSM_BARRIER();
  Raw wa = read_signs(0), wb;
  int ks = 0;
  for (; ks + kStages <= nks; ks += kStages) {
    step(ks + 0, 0, wa, wb);
    step(ks + 1, 1, wb, wa);
    step(ks + 2, 2, wa, wb);
    step(ks + 3, 3, wb, wa);
  }
  if (ks < nks) step(ks, 0, wa, wb);
  if (ks + 1 < nks) step(ks + 1, 1, wb, wa);
  if (ks + 2 < nks) step(ks + 2, 2, wa, wb);
  // the ring is reused below: drain and wait for every wave's last stage
  DFSSM_WAIT_VMCNT(0);
  __syncthreads();

  // ---- epilogue: stage the LoRA operands of the block (rank <= 64)
  const bool lora_lds = kLoraLds && r > 0;
  if (lora_lds) {
    int8_t* limb_lds = lds;               // [4][kBM][64], swizzled chunks
    int8_t* b_lds = lds + kLimbBytes;     // [rows of the run][64], swizzled chunks
    const bool baligned = (r % 16) == 0;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int idx = tid + u * kThreads;  // (limb, row, 16-byte chunk)
      const int limb = idx >> 9, ml = (idx >> 2) & 127, c = idx & 3;
      const int m = min(m0 + ml, M - 1);
      *reinterpret_cast<uint4*>(limb_lds + (limb * kBM + ml) * 64 + 16 * (c ^ swz(ml))) =
          *reinterpret_cast<const uint4*>(a.limbs + ((int64_t)limb * M + m) * rp + 16 * c);
    }
    for (int idx = tid; idx < 4 * nrows; idx += kThreads) {  // (row, 16-byte chunk)
      const int nl = idx >> 2, c = idx & 3;
      const int n = min(n0 + nl, N - 1);
      const v4i b = load16_guarded(a.B + (int64_t)n * r, 16 * c, r, baligned);
      *reinterpret_cast<v4i*>(b_lds + nl * 64 + 16 * (c ^ swz(nl))) = b;
    }
    __syncthreads();
  }
  const int l_off = rho * 64 + 16 * (kg ^ swz(rho));
  const bool fast = lora_lds && !a.acc_s_out && !a.acc_b_out && (N & 3) == 0 && m0 + kBM <= M && n0 + nrows <= N;
  if constexpr (kShort) {
    if (fast)
      short_epilogue<true, false, kSR>(a, L, acc, m0, n0, wave, cnt, ntt, rho, kg, l_off);
    else if (lora_lds)
      short_epilogue<true, true, kSR>(a, L, acc, m0, n0, wave, cnt, ntt, rho, kg, l_off);
    else
      short_epilogue<false, true, kSR>(a, L, acc, m0, n0, wave, cnt, ntt, rho, kg, l_off);
  } else {
    if (fast)
      block_epilogue<true, false>(a, L, acc, accx, m0, n0, wave, ntw, extra, 256, 2 * wave, rho, kg, l_off);
    else if (lora_lds)
      block_epilogue<true, true>(a, L, acc, accx, m0, n0, wave, ntw, extra, 256, 2 * wave, rho, kg, l_off);
    else
      block_epilogue<false, true>(a, L, acc, accx, m0, n0, wave, ntw, extra, 256, 2 * wave, rho, kg, l_off);
  }
}

template <bool kLoraLds, int kSR>
__global__ __launch_bounds__(kThreads, 2) void mfma_scaffold(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) int8_t lds[kLdsBytes];
  __shared__ __attribute__((aligned(16))) float al_lds[kMaxRows], be_lds[kMaxRows], s_lds[kBM];
  __shared__ __attribute__((aligned(16))) int32_t sq_lds[kBM];
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int bm = tile / a.bpm, j = tile % a.bpm;
  // row tiles [rt0, rt1) of the slice: runs of equal length up to one
  const int rt0 = (int)((int64_t)j * a.nt16 / a.bpm), rt1 = (int)((int64_t)(j + 1) * a.nt16 / a.bpm);
  const TileLds L{lds, al_lds, be_lds, s_lds, sq_lds};
  scaffold_block<kLoraLds, kSR>(a, L, bm * kBM, rt0, rt1 - rt0);
}


// ------------------------------------------------------------ ping-pong prefill
// One block of 8 waves per CU, two per SIMD, in two groups of 4 (waves 0-3
// and 4-7) that take turns: while one group runs its MFMAs of a stage, the
// other reads its operands of the next stage from LDS, issues the loads of a
// later stage and waits for its own loads of the stage after; a block
// barrier separates the turns, and the second group starts one turn late.
// So at any time one wave of each SIMD is in its MFMA phase.  (Two 4-wave
// blocks per CU cannot arrange that: each block's per-stage barrier and
// loads fell in the same phase on both waves of a SIMD.)
//
// Block: 128 tokens x a run of up to 34 row tiles.  Wave w owns row tiles
// 4w .. 4w+3; the 33rd and 34th are shared, wave w taking token tiles 2i,
// 2i+1 (i = w % 4) of row tile 32 + w / 4.  Per stage each wave issues one
// 16-byte direct-to-LDS load of Q (16 token rows) and, at a sign-group start,
// the 9 loads of its sign rows (its 64 rows, 4 of the 32 shared rows), with
// the layouts of the 4-wave kernel.
constexpr int kPPThreads = 512;
constexpr int kPPRunMax = 34;
constexpr int kPPSgBuf = 8 * kSgWave + 32 * 32;  // 17 KB
constexpr int kPPLdsRing = kQRing + 2 * kPPSgBuf;
constexpr int kPPLdsLora = kLimbBytes + kPPRunMax * 16 * 64;
constexpr int kPPLdsBytes = kPPLdsRing > kPPLdsLora ? kPPLdsRing : kPPLdsLora;
constexpr int kPPMaxRows = kPPRunMax * 16;

template <bool kLoraLds>
__device__ __forceinline__ void scaffold_block_pp(const GemmArgs& a, const TileLds& L, int m0, int rt0, int cnt) {
  const int M = a.M, K = a.K, N = a.N, r = a.r, rp = a.rp;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS addresses of the loads
  const int grp = wave >> 2, wi = wave & 3;
  const int rho = lane & 15, kg = lane >> 4;
  const int W = K >> 5;
  const int nks = (K + kBK - 1) / kBK;
  const bool ktail = (K & (kBK - 1)) != 0;  // the last stage holds 32 columns
  const int n0 = 16 * rt0;
  const int ntw = min(max(min(cnt, 32) - 4 * wave, 0), 4);  // this wave's own row tiles
  const bool extra = cnt > 32 + grp;                         // this wave's shared row tile exists
  const int nrows = 16 * cnt;
  int8_t* const lds = L.lds;

  // ---- direct-to-LDS load constants (rows past M or N read the last row;
  //      their outputs are never stored)
  uint32_t voff_q;
  bool hi_chunk;
  {
    const int m = 16 * wave + (lane >> 2);  // Q row of this lane's 16-byte slot
    const int c = (lane & 3) ^ swz(m);
    hi_chunk = c >= 2;
    voff_q = (uint32_t)((min(m0 + m, M - 1) - m0) * K + 16 * c);
  }
  const bool sg_fast = n0 + 64 * wave + 64 <= N;  // uniform: no own sign row is clamped
  uint32_t voff_s[2];
#pragma unroll
  for (int jp = 0; jp < 2; ++jp) {
    const int wd = (lane & 7) ^ (2 * ((2 * jp + (lane >> 5)) & 3));
    voff_s[jp] = (uint32_t)((((lane >> 3) + 64 * wave) * W + wd) * 4);
  }
  uint32_t voff_x;
  {
    const int rr = 4 * wave + (lane >> 3);  // shared row (< 32 for lanes < 32)
    const int wd = (lane & 7) ^ (2 * ((rr >> 2) & 3));
    const int n = min(n0 + 512 + rr, N - 1);
    voff_x = (uint32_t)(((n - n0) * W + wd) * 4);
  }
  const int8_t* qbase = a.q + (int64_t)m0 * K;
  const uint32_t* wbase = a.w_bits + (int64_t)n0 * W;
  const uint32_t lds0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(uintptr_t)(lds_void*)lds);

  auto issue_signs = [&](int g) {
    const uint32_t sb = lds0 + kQRing + (g & 1) * kPPSgBuf;
    const uint32_t* ws = wbase + 8 * g;
    const bool whole = 8 * g + 8 <= W;  // uniform
    if (sg_fast && whole) {
#pragma unroll
      for (int j = 0; j < 8; ++j) lds_dma4(voff_s[j & 1], ws + (int64_t)8 * j * W, sb + kSgWave * wave + 256u * j);
    } else {
      const int ln = lane + opaque_zero();
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int rl = 8 * j + (ln >> 3);
        const int wd = (ln & 7) ^ (2 * ((rl >> 2) & 3));
        const int n = min(n0 + 64 * wave + rl, N - 1);
        const int wc = min(8 * g + wd, W - 1) - 8 * g;
        lds_dma4((uint32_t)(((n - n0) * W + wc) * 4), ws, sb + kSgWave * wave + 256u * j);
      }
    }
    {
      uint32_t vx = voff_x;
      if (!whole) {
        const int ln = lane + opaque_zero();
        const int rr = 4 * wave + (ln >> 3);
        const int wd = (ln & 7) ^ (2 * ((rr >> 2) & 3));
        const int n = min(n0 + 512 + rr, N - 1);
        vx = (uint32_t)(((n - n0) * W + min(8 * g + wd, W - 1) - 8 * g) * 4);
      }
      if (lane < 32) lds_dma4(vx, ws, sb + 8 * kSgWave + 128u * wave);
    }
  };
  auto issue = [&](int ks, int slot) {
    if (slot == 0) issue_signs(ks >> 2);
    const int8_t* qs = qbase + ks * kBK;
    const uint32_t sb = lds0 + slot * kQStage + 1024u * wave;
    if (ktail && ks == nks - 1)
      lds_dma16(voff_q - (hi_chunk ? 32u : 0u), qs, sb);  // chunks past K re-read 0, 1 (zeroed signs)
    else
      lds_dma16(voff_q, qs, sb);
  };

  // LDS read offsets (as in the 4-wave kernel; the shared tile's rows follow
  // the 8 waves' areas)
  const int q_off = rho * kBK + 16 * (kg ^ swz(rho));
  const int w_off = kQRing + kSgWave * wave + 32 * rho + 4 * ((kg >> 1) ^ (2 * ((rho >> 2) & 3)));
  const int x_delta = 8 * kSgWave + 512 * grp - kSgWave * wave;  // uniform
  const uint32_t sh = 16u * (kg & 1);
  const bool kg_hi = kg >= 2;

  typedef uint32_t raw_t __attribute__((ext_vector_type(4)));
  struct Ops {
    v4i q[8];
    v4i qx[2];  // the shared tile's token tiles 2i, 2i+1 (read again: no register indexing)
    raw_t w;
    uint32_t x;
  };
  auto read_ops = [&](int ks, int slot, Ops& o) {
    const int8_t* qst = lds + slot * kQStage + q_off;
#pragma unroll
    for (int i = 0; i < 8; ++i) o.q[i] = *reinterpret_cast<const v4i*>(qst + i * 16 * kBK);
    if (extra) {
#pragma unroll
      for (int h = 0; h < 2; ++h) o.qx[h] = *reinterpret_cast<const v4i*>(qst + (2 * wi + h) * 16 * kBK);
    }
    const int8_t* st = lds + ((ks >> 2) & 1) * kPPSgBuf;
    const int wb = w_off ^ (8 * (ks & 3));
#pragma unroll
    for (int t = 0; t < 4; ++t) o.w[t] = *reinterpret_cast<const uint32_t*>(st + wb + 512 * t);
    o.x = *reinterpret_cast<const uint32_t*>(st + x_delta + wb);
    if (ktail && ks == nks - 1) {  // uniform: sign words past K count as 0
#pragma unroll
      for (int t = 0; t < 4; ++t) o.w[t] = kg_hi ? 0u : o.w[t];
      o.x = kg_hi ? 0u : o.x;
    }
  };

  v4i acc[4][8], accx[2];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[t][i] = zero4();
  accx[0] = accx[1] = zero4();

  auto compute = [&](const Ops& o) {
    {
      v4i sg = expand16_at(o.w[0], sh);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const v4i sgn = t + 1 < 4 ? expand16_at(o.w[t + 1], sh) : sg;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[t][i] = mfma(sg, o.q[i], acc[t][i]);
        sg = sgn;
      }
      __builtin_amdgcn_sched_group_barrier(0x002, 12, 0);  // VALU: the first expansion
#pragma unroll
      for (int t = 0; t < 3; ++t) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // VALU
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
        }
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    }
    if (extra) {  // uniform: the shared row tile, token tiles 2i and 2i+1
      const v4i sx = expand16_at(o.x, sh);
      accx[0] = mfma(sx, o.qx[0], accx[0]);
      accx[1] = mfma(sx, o.qx[1], accx[1]);
    }
  };

  // loads a wave issues with stage ks: one Q load, plus the sign group's 9
  // when ks starts a group (ks % 4 == 0)
  auto lcount = [](int slot) { return slot == 0 ? 1 + kLsg : 1; };

  // one stage: [memory turn] operands of ks from LDS, the loads of ks+3
  // (into the slot of ks-1, which both groups have read), own loads of ks+1
  // complete; barrier; [MFMA turn] multiply ks; barrier
  auto stage = [&](int ks, int slot) {
    Ops o;
    read_ops(ks, slot, o);
    if (ks + 3 < nks) issue(ks + 3, (slot + 3) % kStages);
    if (ks + 1 < nks) {
      const int c2 = lcount((slot + 2) % kStages), c3 = lcount((slot + 3) % kStages);
      if (ks + 3 < nks) {
        if (c2 + c3 == 2)
          DFSSM_WAIT_VMCNT(2);
        else
          DFSSM_WAIT_VMCNT(2 + kLsg);
      } else if (ks + 2 < nks) {
        if (c2 == 1)
          DFSSM_WAIT_VMCNT(1);
        else
          DFSSM_WAIT_VMCNT(1 + kLsg);
      } else {
        DFSSM_WAIT_VMCNT(0);
      }
    }
    // this wave's LDS reads of ks are complete before the barrier: the other
    // group refills the slot of ks in the turn after next
    DFSSM_WAIT_LGKM0();
    DFSSM_BARRIER();
    __builtin_amdgcn_s_setprio(1);
    compute(o);
    __builtin_amdgcn_s_setprio(0);
    DFSSM_BARRIER();
  };

#pragma unroll
  for (int p = 0; p < kStages - 1; ++p)
    if (p < nks) issue(p, p);
  for (int x = tid; x < nrows; x += kPPThreads) {
    const int n = min(n0 + x, N - 1);
    L.al[x] = a.alpha[n];
    L.be[x] = r > 0 ? a.beta[n] : 0.0f;
  }
  if (tid < kBM) {
    const int m = min(m0 + tid, M - 1);
    L.sv[tid] = a.s[m];
    L.sq[tid] = a.sumq[m];
  }
  // stage 0 (with sign group 0) has landed once at most the Q loads of
  // stages 1 and 2 are in flight
  if (nks >= 3)
    DFSSM_WAIT_VMCNT(2);
  else if (nks == 2)
    DFSSM_WAIT_VMCNT(1);
  else
    DFSSM_WAIT_VMCNT(0);
  DFSSM_BARRIER();
  if (grp == 1) DFSSM_BARRIER();  // the second group starts one turn late
  int ks = 0;
  for (; ks + kStages <= nks; ks += kStages) {
    stage(ks + 0, 0);
    stage(ks + 1, 1);
    stage(ks + 2, 2);
    stage(ks + 3, 3);
  }
  if (ks < nks) stage(ks, 0);
  if (ks + 1 < nks) stage(ks + 1, 1);
  if (ks + 2 < nks) stage(ks + 2, 2);
  if (grp == 0) DFSSM_BARRIER();  // matches the second group's late start
  DFSSM_WAIT_VMCNT(0);
  __syncthreads();

  // ---- epilogue: stage the LoRA operands of the block (rank <= 64)
  const bool lora_lds = kLoraLds && r > 0;
  if (lora_lds) {
    int8_t* limb_lds = lds;            // [4][kBM][64], swizzled chunks
    int8_t* b_lds = lds + kLimbBytes;  // [rows of the run][64], swizzled chunks
    const bool baligned = (r % 16) == 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + u * kPPThreads;  // (limb, row, 16-byte chunk)
      const int limb = idx >> 9, ml = (idx >> 2) & 127, c = idx & 3;
      const int m = min(m0 + ml, M - 1);
      *reinterpret_cast<uint4*>(limb_lds + (limb * kBM + ml) * 64 + 16 * (c ^ swz(ml))) =
          *reinterpret_cast<const uint4*>(a.limbs + ((int64_t)limb * M + m) * rp + 16 * c);
    }
    for (int idx = tid; idx < 4 * nrows; idx += kPPThreads) {  // (row, 16-byte chunk)
      const int nl = idx >> 2, c = idx & 3;
      const int n = min(n0 + nl, N - 1);
      const v4i b = load16_guarded(a.B + (int64_t)n * r, 16 * c, r, baligned);
      *reinterpret_cast<v4i*>(b_lds + nl * 64 + 16 * (c ^ swz(nl))) = b;
    }
    __syncthreads();
  }
  const int l_off = rho * 64 + 16 * (kg ^ swz(rho));
  const int xrow = 512 + 16 * grp, xtok = 2 * wi;
  const bool fast = lora_lds && !a.acc_s_out && !a.acc_b_out && (N & 3) == 0 && m0 + kBM <= M && n0 + nrows <= N;
  if (fast)
    block_epilogue<true, false>(a, L, acc, accx, m0, n0, wave, ntw, extra, xrow, xtok, rho, kg, l_off);
  else if (lora_lds)
    block_epilogue<true, true>(a, L, acc, accx, m0, n0, wave, ntw, extra, xrow, xtok, rho, kg, l_off);
  else
    block_epilogue<false, true>(a, L, acc, accx, m0, n0, wave, ntw, extra, xrow, xtok, rho, kg, l_off);
}

template <bool kLoraLds>
__global__ __launch_bounds__(kPPThreads, 1) void mfma_scaffold_pp(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) int8_t lds[kPPLdsBytes];
  __shared__ __attribute__((aligned(16))) float al_lds[kPPMaxRows], be_lds[kPPMaxRows], s_lds[kBM];
  __shared__ __attribute__((aligned(16))) int32_t sq_lds[kBM];
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int bm = tile / a.bpm, j = tile % a.bpm;
  const int rt0 = (int)((int64_t)j * a.nt16 / a.bpm), rt1 = (int)((int64_t)(j + 1) * a.nt16 / a.bpm);
  const TileLds L{lds, al_lds, be_lds, s_lds, sq_lds};
  scaffold_block_pp<kLoraLds>(a, L, bm * kBM, rt0, rt1 - rt0);
}

// Tiling of the prefill path.  Each 128-token slice's ceil(N/16) row
// tiles are dealt to bpm blocks in runs whose lengths differ by at most
// one; bpm is chosen so the blocks fill the chip's block slots in whole
// rounds where the shape allows.  The 8-wave ping-pong kernel (one block
// per CU, runs of up to 34) is taken where the runs are long enough to keep
// its 8 waves busy (at least 24 row tiles); otherwise the 4-wave kernel (two
// blocks per CU, runs of up to 17), in its short form when every run holds
// at most kShortRun row tiles.  forced: the test switch prefill_kernel (4
// or 8).
enum PrefillForm { kForm8 = 8, kForm4 = 4, kForm4Short = 2 };  // short: runs of at most kShortRun
struct PrefillPlan {
  int64_t nbm, nt16, bpm;
  PrefillForm form;
};
PrefillPlan plan_prefill(int64_t M, int64_t N, int64_t cus, int forced) {
  const int64_t nbm = dfssm::ceil_div(M, kBM);
  const int64_t nt16 = dfssm::ceil_div(N, 16);
  const int64_t bpm8 = std::min(std::max(dfssm::ceil_div(cus, nbm), dfssm::ceil_div(nt16, kPPRunMax)), nt16);
  bool use8 = nt16 >= 24 * bpm8;
  if (forced == 4) use8 = false;
  if (forced == 8) use8 = true;
  if (use8) return {nbm, nt16, bpm8, kForm8};
  const int64_t bpm = std::min(std::max(dfssm::ceil_div(2 * cus, nbm), dfssm::ceil_div(nt16, kRunMax)), nt16);
  return {nbm, nt16, bpm, nt16 <= kShortRun * bpm ? kForm4Short : kForm4};
}

}  // namespace

namespace dfssm {

// Cost of the prefill path (us; both launches), fitted on MI355X to the
// 130M, 1.3B and 2.7B projections at 33 to 512 tokens: a serial K-loop of
// K/64 stages (0.35 us each, plus a share that grows with N), the MFMA work
// of every 128-token slice past the first, and for runs of more than 4 row
// tiles the longer stages of the 4- and 8-wave forms.
double prefill_cost_us(int64_t M, int64_t K, int64_t N) {
  const PrefillPlan p = plan_prefill(M, N, device_cu_count(), 0);
  const double stages = (double)K / 64.0;
  double c = 8.5 + stages * (0.35 + 0.12 * (double)N / 1e4) + 2.2 * (double)N * (double)K * (double)(p.nbm - 1) / 1e7;
  if (p.form != kForm4Short) c += 0.17 * stages * (double)ceil_div(p.nt16, p.bpm) / 4.0;
  return c;
}

int device_cu_count() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v <= 0) {
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

hipError_t launch_mfma_linear(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                              int64_t r, const uint32_t* w_bits, const float* alpha,
                              const int8_t* A, const int8_t* B, const float* beta, float* y,
                              int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                              const LinearWorkspace& ws, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  const int rp = (int)rank_padded(r);
  mfma_lora_down<<<dim3((unsigned)ceil_div(M, 16), (unsigned)(rp / kLdRanks)), dim3(kLdThreads), 0, st>>>(
      q, (int)M, (int)K, (int)r, rp, A, ws.acc_a, ws.limbs, ws.sumq);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (acc_a_out && r > 0) {
    e = hipMemcpyAsync(acc_a_out, ws.acc_a, (size_t)(M * r) * 4, hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
  }
  const PrefillPlan p = plan_prefill(M, N, device_cu_count(), test_switch(DFSSM_TEST_PREFILL_KERNEL));
  const int64_t grid = p.nbm * p.bpm;
  GemmArgs ga{q, s, (int)M, (int)K, (int)N, (int)r, rp, w_bits, alpha, ws.limbs, B, beta, ws.sumq, y,
              acc_s, acc_b, (int)p.nt16, (int)p.bpm};
  if (p.form == kForm8) {
    if (rp == 64)
      mfma_scaffold_pp<true><<<dim3((unsigned)grid), dim3(kPPThreads), 0, st>>>(ga);
    else
      mfma_scaffold_pp<false><<<dim3((unsigned)grid), dim3(kPPThreads), 0, st>>>(ga);
  } else if (p.form == kForm4Short && p.nt16 <= 4 * p.bpm) {  // runs of at most 4 row tiles
    if (rp == 64)
      mfma_scaffold<true, 4><<<dim3((unsigned)grid), dim3(kThreads), 0, st>>>(ga);
    else
      mfma_scaffold<false, 4><<<dim3((unsigned)grid), dim3(kThreads), 0, st>>>(ga);
  } else if (p.form == kForm4Short) {
    if (rp == 64)
      mfma_scaffold<true, kShortRun><<<dim3((unsigned)grid), dim3(kThreads), 0, st>>>(ga);
    else
      mfma_scaffold<false, kShortRun><<<dim3((unsigned)grid), dim3(kThreads), 0, st>>>(ga);
  } else if (rp == 64) {
    mfma_scaffold<true, 0><<<dim3((unsigned)grid), dim3(kThreads), 0, st>>>(ga);
  } else {
    mfma_scaffold<false, 0><<<dim3((unsigned)grid), dim3(kThreads), 0, st>>>(ga);
  }
  return hipGetLastError();
}

}  // namespace dfssm
