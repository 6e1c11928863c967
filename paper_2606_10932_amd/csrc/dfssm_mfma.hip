// dfssm_mfma.hip -- prefill-shaped (large M) scaffold + LoRA linear on the
// gfx950 int8 matrix cores (v_mfma_i32_16x16x64_i8).
//
// The sign bits are expanded on chip, in registers, to {0,1} bytes (a
// nibble n becomes bytes via (n * 0x00204081) & 0x01010101), so the MFMA
// computes D[m,n] = sum_{bit=1} Q[m,k] and acc_s = 2*D - sum_k Q[m,k]; the
// expanded signs never touch memory (the paper expands to int8 "on the fly"
// ahead of a library int8 GEMM, Sec. 4.1).
//
// Operand layout of v_mfma_i32_16x16x64_i8 (wave64): lane l supplies row
// (l % 16) of A and column (l % 16) of B, each as 16 consecutive K-bytes of
// K-group (l / 16); the 16x16 int32 result D has D[4*(l/16)+v][l%16] in
// lane l, register v.  A = Q rows (tokens), B = sign columns (output rows),
// so a lane's 4 results are 4 tokens of one output row, and 16 lanes store
// 16 consecutive output rows of a token.
//
// LoRA: lora_down computes acc_a = Q * A^T with the same MFMA, sum_k Q, and
// writes acc_a as 4 signed base-256 int8 limbs.  The main kernel then gets
// the exact int64 acc_b = sum_j B[n,j] acc_a[m,j] from four int8 MFMAs:
// E_hi = 256*(L3.B) + L2.B and E_lo = 256*(L1.B) + L0.B (each < 2^31 for
// r <= 256), acc_b = E_lo + 65536*E_hi.
#include "dfssm_internal.hpp"

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

__device__ __forceinline__ v4i mfma(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ v4i zero4() { return v4i{0, 0, 0, 0}; }

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
// One wave per (16 tokens, 64 LoRA rows).  Also writes sum_k Q (j-tile 0).
__global__ __launch_bounds__(kThreads) void mfma_lora_down(const int8_t* __restrict__ q, int M,
                                                           int K, int r, int rp,
                                                           const int8_t* __restrict__ A,
                                                           int32_t* __restrict__ acc_a,
                                                           int8_t* __restrict__ limbs,
                                                           int32_t* __restrict__ sumq) {
  const int lane = threadIdx.x & 63;
  const int gw = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int jtiles = rp / 64;
  const int mtile = gw / jtiles, jt = gw % jtiles;
  const int m0 = mtile * 16;
  if (m0 >= M) return;
  const int row = lane & 15, kg = lane >> 4;
  const int m = m0 + row;
  const bool m_ok = m < M;
  const int8_t* qrow = q + (int64_t)(m_ok ? m : 0) * K;

  v4i acc[4] = {zero4(), zero4(), zero4(), zero4()};
  int qs = 0;
  for (int k0 = 0; k0 < K; k0 += 64) {
    const int kk = k0 + 16 * kg;
    v4i a = (m_ok && kk < K) ? load16(qrow + kk) : zero4();
    if (jt == 0) {
#pragma unroll
      for (int t = 0; t < 4; ++t) qs = __builtin_amdgcn_sdot4(a[t], 0x01010101, qs, false);
    }
    if (r > 0) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int j = jt * 64 + 16 * t + row;
        v4i b = (j < r && kk < K) ? load16(A + (int64_t)j * K + kk) : zero4();
        acc[t] = mfma(a, b, acc[t]);
      }
    }
  }
  if (jt == 0) {
    qs += __shfl_xor(qs, 16, 64);
    qs += __shfl_xor(qs, 32, 64);
    if (kg == 0 && m_ok) sumq[m] = qs;
  }
  if (r == 0) return;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int j = jt * 64 + 16 * t + row;  // result column of this lane
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int mm = m0 + 4 * kg + v;
      if (mm >= M) continue;
      const int32_t val = acc[t][v];
      int8_t d[4];
      dfssm_dev::split_limbs(j < r ? val : 0, d);
#pragma unroll
      for (int l = 0; l < 4; ++l) limbs[((int64_t)l * M + mm) * rp + j] = d[l];
      if (j < r) acc_a[(int64_t)mm * r + j] = val;
    }
  }
}

// ------------------------------------------------------------ main GEMM
// Block tile 128 (tokens) x 128 (output rows); 4 waves as 2 x 2, wave tile
// 64 x 64 = 4 x 4 MFMA tiles; K step 64.
constexpr int kBM = 128, kBN = 128, kWM = 64, kWN = 64;

__global__ __launch_bounds__(kThreads) void mfma_scaffold(
    const int8_t* __restrict__ q, const float* __restrict__ s, int M, int K, int N, int r, int rp,
    const uint32_t* __restrict__ w_bits, const float* __restrict__ alpha,
    const int8_t* __restrict__ limbs, const int8_t* __restrict__ B,
    const float* __restrict__ beta, const int32_t* __restrict__ sumq, float* __restrict__ y,
    int32_t* __restrict__ acc_s_out, int64_t* __restrict__ acc_b_out, int n_blocks_n) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = lane & 15, kg = lane >> 4;
  const int bm = blockIdx.x / n_blocks_n, bn = blockIdx.x % n_blocks_n;
  const int wm0 = bm * kBM + (wave >> 1) * kWM;
  const int wn0 = bn * kBN + (wave & 1) * kWN;
  const int W = K / 32;

  const int8_t* qrow[4];
  bool qok[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = wm0 + 16 * i + row;
    qok[i] = m < M;
    qrow[i] = q + (int64_t)(qok[i] ? m : 0) * K;
  }
  const uint32_t* wrow[4];
  bool nok[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int n = wn0 + 16 * t + row;
    nok[t] = n < N;
    wrow[t] = w_bits + (int64_t)(nok[t] ? n : 0) * W;
  }

  v4i acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[i][t] = zero4();

  for (int k0 = 0; k0 < K; k0 += 64) {
    const int kk = k0 + 16 * kg;
    const bool kok = kk < K;  // K % 32 == 0: a K-group is all in or all out
    v4i a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = (qok[i] && kok) ? load16(qrow[i] + kk) : zero4();
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      uint32_t wd = (nok[t] && kok) ? wrow[t][kk >> 5] : 0u;
      b[t] = expand16((wd >> (kk & 16)) & 0xffffu);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[i][t] = mfma(a[i], b[t], acc[i][t]);
  }

  // acc_s = 2*D - sum Q  (in place)
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = wm0 + 16 * i + 4 * kg + v;
      const int sq = m < M ? sumq[m] : 0;
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[i][t][v] = 2 * acc[i][t][v] - sq;
    }

  // LoRA up-projection with limb MFMAs
  v4i ehi[4][4], elo[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t) ehi[i][t] = elo[i][t] = zero4();
  if (r > 0) {
    const bool baligned = (r % 16) == 0;
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {  // limbs 3, 2, 1, 0
      const int limb = 3 - pass;
      for (int j0 = 0; j0 < rp; j0 += 64) {
        const int jj = j0 + 16 * kg;
        v4i bl[4], al[4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
          bl[t] = nok[t] ? load16_guarded(B + (int64_t)(wn0 + 16 * t + row) * r, jj, r, baligned)
                         : zero4();
#pragma unroll
        for (int i = 0; i < 4; ++i)
          al[i] = qok[i] ? load16(limbs + ((int64_t)limb * M + (wm0 + 16 * i + row)) * rp + jj)
                         : zero4();
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            if (limb >= 2)
              ehi[i][t] = mfma(al[i], bl[t], ehi[i][t]);
            else
              elo[i][t] = mfma(al[i], bl[t], elo[i][t]);
          }
      }
      if (limb == 3 || limb == 1) {  // scale the high digit's sum by 256
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            if (limb == 3)
              ehi[i][t] = ehi[i][t] << 8;
            else
              elo[i][t] = elo[i][t] << 8;
          }
      }
    }
  }

  // epilogue
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int n = wn0 + 16 * t + row;
    if (n >= N) continue;
    const float al = alpha[n];
    const float be = r > 0 ? beta[n] : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = wm0 + 16 * i + 4 * kg + v;
        if (m >= M) continue;
        const int32_t as = acc[i][t][v];
        const int32_t hi = ehi[i][t][v], lo = elo[i][t][v];
        if (y) y[(int64_t)m * N + n] = dfssm_dev::epilogue(s[m], al, be, as, hi, lo, r > 0);
        if (acc_s_out) acc_s_out[(int64_t)m * N + n] = as;
        if (acc_b_out) acc_b_out[(int64_t)m * N + n] = r > 0 ? (int64_t)lo + ((int64_t)hi << 16) : 0;
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
  const int64_t waves = ceil_div(M, 16) * (rp / 64);
  mfma_lora_down<<<dim3((unsigned)ceil_div(waves, 4)), dim3(kThreads), 0, st>>>(
      q, (int)M, (int)K, (int)r, rp, A, ws.acc_a, ws.limbs, ws.sumq);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (acc_a_out && r > 0) {
    e = hipMemcpyAsync(acc_a_out, ws.acc_a, (size_t)(M * r) * 4, hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
  }
  const int64_t nbm = ceil_div(M, kBM), nbn = ceil_div(N, kBN);
  mfma_scaffold<<<dim3((unsigned)(nbm * nbn)), dim3(kThreads), 0, st>>>(
      q, s, (int)M, (int)K, (int)N, (int)r, rp, w_bits, alpha, ws.limbs, B, beta, ws.sumq, y,
      acc_s, acc_b, (int)nbn);
  return hipGetLastError();
}

}  // namespace dfssm
