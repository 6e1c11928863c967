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
// A block owns 16 tokens; its 4 waves split the K steps into quarters and
// reduce their partial sums in LDS.  Loads are issued 4 K-steps at a time.
constexpr int kLdBatch = 4;

__global__ __launch_bounds__(kThreads) void mfma_lora_down(const int8_t* __restrict__ q, int M, int K,
                                                           int r, int rp, const int8_t* __restrict__ A,
                                                           int32_t* __restrict__ acc_a,
                                                           int8_t* __restrict__ limbs,
                                                           int32_t* __restrict__ sumq) {
  __shared__ int32_t part[4][16 * 64];
  __shared__ int32_t qpart[4][16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = lane & 15, kg = lane >> 4;
  const int m0 = blockIdx.x * 16;
  const int m = m0 + row;
  const bool m_ok = m < M;
  const int8_t* qrow = q + (int64_t)(m_ok ? m : 0) * K;
  const int nks = (K + 63) / 64;
  const int per = (nks + 3) / 4;
  const int ks0 = wave * per, ks1 = min(nks, ks0 + per);

  for (int jt = 0; jt < rp / 64; ++jt) {
    v4i acc[4] = {zero4(), zero4(), zero4(), zero4()};
    int qs = 0;
    for (int kb = ks0; kb < ks1; kb += kLdBatch) {
      // all loads of the batch from clamped addresses first, masks after
      v4i a[kLdBatch], b[kLdBatch][4];
      int ma[kLdBatch], mb[kLdBatch][4];
#pragma unroll
      for (int u = 0; u < kLdBatch; ++u) {
        const int kk = (kb + u) * 64 + 16 * kg;
        const bool kok = kb + u < ks1 && kk < K;
        const int kc = kok ? kk : 0;
        a[u] = load16(qrow + kc);
        ma[u] = (m_ok && kok) ? -1 : 0;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int j = jt * 64 + 16 * t + row;
          b[u][t] = r > 0 ? load16(A + (int64_t)(j < r ? j : 0) * K + kc) : zero4();
          mb[u][t] = (j < r && kok) ? -1 : 0;
        }
      }
#pragma unroll
      for (int u = 0; u < kLdBatch; ++u) {
        a[u] &= ma[u];
#pragma unroll
        for (int t = 0; t < 4; ++t) b[u][t] &= mb[u][t];
      }
#pragma unroll
      for (int u = 0; u < kLdBatch; ++u) {
        if (jt == 0) {
#pragma unroll
          for (int t = 0; t < 4; ++t) qs = __builtin_amdgcn_sdot4(a[u][t], 0x01010101, qs, false);
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = mfma(a[u], b[u][t], acc[t]);
      }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) part[wave][(4 * kg + v) * 64 + 16 * t + row] = acc[t][v];
    if (jt == 0) {
      qs += __shfl_xor(qs, 16, 64);
      qs += __shfl_xor(qs, 32, 64);
      if (kg == 0) qpart[wave][row] = qs;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 16 * 64; i += kThreads) {
      const int mi = i >> 6, ji = i & 63;
      const int mm = m0 + mi, j = jt * 64 + ji;
      if (mm >= M) continue;
      const int32_t val = part[0][i] + part[1][i] + part[2][i] + part[3][i];
      int8_t d[4];
      dfssm_dev::split_limbs(j < r ? val : 0, d);
#pragma unroll
      for (int l = 0; l < 4; ++l) limbs[((int64_t)l * M + mm) * rp + j] = d[l];
      if (j < r) acc_a[(int64_t)mm * r + j] = val;
    }
    if (jt == 0 && threadIdx.x < 16 && m0 + threadIdx.x < M)
      sumq[m0 + threadIdx.x] = qpart[0][threadIdx.x] + qpart[1][threadIdx.x] + qpart[2][threadIdx.x] +
                               qpart[3][threadIdx.x];
    __syncthreads();
  }
}

// ------------------------------------------------------------ main GEMM
// Block tile 128 (tokens) x 128 (output rows), 4 waves as 2 x 2 with wave
// tiles of 64 x 64 (4 x 4 MFMA tiles); 64 K per stage, two LDS stages.  The
// Q tile is staged with a padded row pitch (80 B) to spread LDS banks; the
// sign words of the tile (1 KB per stage) are staged raw and expanded by
// each wave into its B operands.
constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kQPitch = kBK + 16;
// sign-word stage: 2 x 256 rows, so all 256 threads store (rows >= 128 hold
// masked zeros and are never read): no divergent branch in the K-loop
constexpr int kWRows = 2 * kBN;
constexpr int kLdsLoop = 2 * kBM * kQPitch + 2 * kWRows * 2 * 4;
constexpr int kLdsLora = 4 * kBM * kQPitch + kBN * kQPitch;
constexpr int kLdsBytes = kLdsLoop > kLdsLora ? kLdsLoop : kLdsLora;
#ifndef DFSSM_MFMA_OCC
#define DFSSM_MFMA_OCC 3
#endif

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
  int8_t(*q_lds)[kBM * kQPitch] = reinterpret_cast<int8_t(*)[kBM * kQPitch]>(lds_raw);
  uint32_t(*w_lds)[kWRows * 2] = reinterpret_cast<uint32_t(*)[kWRows * 2]>(lds_raw + 2 * kBM * kQPitch);
  int8_t* limb_lds = lds_raw;                       // [4][kBM][kQPitch]
  int8_t* b_lds = lds_raw + 4 * kBM * kQPitch;      // [kBN][kQPitch]
  __shared__ float al_lds[kBN], be_lds[kBN], s_lds[kBM];
  __shared__ int32_t sq_lds[kBM];
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
  // staging: thread t loads Q row m0 + t/2, bytes (t&1)*32 .. +31 of the
  // stage; threads t < 128 load the two sign words of row n0 + t
  const int qr_row = tid >> 1, qr_off = (tid & 1) * 32;
  const int8_t* qsrc = q + (int64_t)min(m0 + qr_row, M - 1) * K;
  const bool q_row_ok = m0 + qr_row < M;
  const uint32_t* wsrc = w_bits + (int64_t)min(n0 + (tid & 127), N - 1) * W;
  const bool w_row_ok = tid < 128 && n0 + tid < N;
  // Loads read clamped in-range addresses unconditionally; the masks are
  // applied when the data is stored to LDS.  Two register stages: the loads
  // of K-stage ks+2 are issued while stage ks is multiplied and are stored to
  // LDS only at the end of stage ks+1, so each load has two stages of MFMA
  // work to arrive.
  struct Stage {
    uint4 q0, q1;
    uint32_t w0, w1, mq, mw0, mw1;
  };
  // stage indexes past the last K-stage load the last stage's addresses and
  // store zeros (all masks off), so the loop below has no branches and the
  // compiler can count outstanding loads exactly
  auto gload = [&](Stage& st, int ks) {
    const int kk = ks * kBK + qr_off;
    const bool ok = q_row_ok && kk < K;
    const int kc = ok ? kk : 0;
    st.q0 = *reinterpret_cast<const uint4*>(qsrc + kc);
    st.q1 = *reinterpret_cast<const uint4*>(qsrc + kc + 16);
    st.mq = ok ? ~0u : 0u;
    const int w0 = 2 * ks;
    st.w0 = wsrc[w0 < W ? w0 : 0];
    st.w1 = wsrc[w0 + 1 < W ? w0 + 1 : 0];
    st.mw0 = (w_row_ok && w0 < W) ? ~0u : 0u;
    st.mw1 = (w_row_ok && w0 + 1 < W) ? ~0u : 0u;
  };
  auto sstore = [&](int buf, const Stage& st) {
    *reinterpret_cast<uint4*>(&q_lds[buf][qr_row * kQPitch + qr_off]) =
        make_uint4(st.q0.x & st.mq, st.q0.y & st.mq, st.q0.z & st.mq, st.q0.w & st.mq);
    *reinterpret_cast<uint4*>(&q_lds[buf][qr_row * kQPitch + qr_off + 16]) =
        make_uint4(st.q1.x & st.mq, st.q1.y & st.mq, st.q1.z & st.mq, st.q1.w & st.mq);
    w_lds[buf][tid * 2] = st.w0 & st.mw0;
    w_lds[buf][tid * 2 + 1] = st.w1 & st.mw1;
  };

  v4i acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[i][t] = zero4();

  const int am_off = ((wave >> 1) * 64 + row) * kQPitch + 16 * kg;
  const int bn_off = ((wave & 1) * 64 + row) * 2 + (kg >> 1);
  const int bshift = (kg & 1) * 16;
  // one K-stage: refill `ld` with stage ks+2, multiply stage ks (LDS buffer
  // ks & 1), then move stage ks+1 (held in `st`) into the other buffer
  auto kstep = [&](int ks, Stage& ld, const Stage& st) {
    const int cur = ks & 1;
    gload(ld, ks + 2);
    v4i a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const v4i*>(&q_lds[cur][am_off + 16 * i * kQPitch]);
#pragma unroll
    for (int t = 0; t < 4; ++t) b[t] = expand16((w_lds[cur][bn_off + 32 * t] >> bshift) & 0xffffu);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[i][t] = mfma(a[i], b[t], acc[i][t]);
    sstore(cur ^ 1, st);
    __syncthreads();
  };
  Stage s0, s1;
  gload(s0, 0);
  gload(s1, 1);
  sstore(0, s0);
  __syncthreads();
  for (int ks = 0; ks < nks; ks += 2) {  // an odd count runs one zero stage
    kstep(ks, s0, s1);      // stage ks+1 lives in s1, ks+2 -> s0
    kstep(ks + 1, s1, s0);  // stage ks+2 lives in s0, ks+3 -> s1
  }

  // ---- epilogue, one n-subtile (16 output rows) at a time: the LoRA term
  //      from four limb MFMAs (exact int64 acc_b = E_lo + 65536*E_hi) on
  //      operands staged in LDS, then acc_s = 2*D - sum Q and
  //      y = s*(alpha*fs + beta*fb)
  const bool baligned = (r % 16) == 0;
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
      *reinterpret_cast<uint4*>(limb_lds + (limb * kBM + ml) * kQPitch + 16 * c) =
          make_uint4(lv[u].x & mk, lv[u].y & mk, lv[u].z & mk, lv[u].w & mk);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int idx = tid + u * kThreads;
      const int nl = idx >> 2, c = idx & 3;
      const uint32_t mk = n0 + nl < N ? ~0u : 0u;
      *reinterpret_cast<uint4*>(b_lds + nl * kQPitch + 16 * c) =
          make_uint4(bv[u].x & mk, bv[u].y & mk, bv[u].z & mk, bv[u].w & mk);
    }
  };
  if (kLoraLds && r > 0) {
    stage_lora(0);  // the K-loop's last barrier has released the buffer
    __syncthreads();
  }
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
          const v4i bl = *reinterpret_cast<const v4i*>(b_lds + nl * kQPitch + 16 * kg);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int ml = (wave >> 1) * 64 + 16 * i + row;
            const v4i al = *reinterpret_cast<const v4i*>(limb_lds + (limb * kBM + ml) * kQPitch + 16 * kg);
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
    if (n >= N) continue;
    const float al = al_lds[nl], be = be_lds[nl];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int ml = (wave >> 1) * 64 + 16 * i + 4 * kg + v;
        const int m = m0 + ml;
        if (m >= M) continue;
        const int32_t as = 2 * acc[i][t][v] - sq_lds[ml];
        const int32_t hi = ehi[i][v], lo = elo[i][v];
        if (y) y[(int64_t)m * N + n] = dfssm_dev::epilogue(s_lds[ml], al, be, as, hi, lo, r > 0);
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
  mfma_lora_down<<<dim3((unsigned)ceil_div(M, 16)), dim3(kThreads), 0, st>>>(
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
