// dfssm_decode.hip -- decode-shaped (small M) scaffold + LoRA linear, gfx950.
//
// At a few tokens the scaffold product is a matrix-vector product over 1-bit
// weights: HBM-bound (about 12 int-ops per byte), so it runs on the vector
// ALUs, not MFMA.  With Q split into its eight two's-complement bit-planes
// P_b (bit k of P_b is bit b of Q[k]):
//
//   sum_k S[n,k] Q[k] = 2 * sum_{bit=1} Q[k] - sum_k Q[k]
//   sum_{bit=1} Q[k]  = sum_b c_b * popcount(w & P_b),  c_b = 2^b (b < 7),
//                                                      c_7 = -128
//
// so each 32-bit sign word costs 8 v_and_b32 + 8 v_bcnt_u32_b32 per token.
//
// Two kernels:
//  small_prep -- the LoRA down-projection acc_a = Q A^T for few tokens, one
//            wave per rank and 8 tokens, every 16-byte load of its columns
//            issued before the first v_dot4; it writes acc_a, its 4 signed
//            base-256 int8 limbs and sum_k Q.  Further blocks build the
//            bit-planes of Q: a thread transposes the 8x8 bit matrix of 8
//            consecutive codes, so byte b of the result is byte p of plane b.
//  gemv   -- a group of G lanes owns one output row; lane g takes chunks g,
//            g+G, ... of the row.  A block stages the planes and the limbs in
//            LDS once; every lane loads its chunks of the row's signs, its B
//            bytes and the row scales before any arithmetic, so a wave waits
//            for memory once.  Per row: popcounts, the LoRA
//            up-projection (B bytes with v_dot4 against the limbs of acc_a,
//            held in LDS), DPP reductions over the G lanes, and the fp32
//            epilogue.
#include <algorithm>

#include "dfssm_internal.hpp"

namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / 64;

__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}

// Sum over aligned groups of G lanes (G = 8..64), the total in every lane of
// the group: DPP butterflies inside a 16-lane row; across rows gfx950's
// permlane swaps (v_permlane16_swap of a value with itself leaves rows
// (0,0,2,2) in one result and (1,1,3,3) in the other, so their sum is the
// 32-lane half's total; v_permlane32_swap does the same for the halves).
template <int G>
__device__ __forceinline__ int group_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  if (G >= 16) v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);  // row_mirror
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

// ------------------------------------------------------------------ prep
constexpr int kPrepTokens = 8;  // tokens per wave of the LoRA blocks
constexpr int kPrepBatch = 4;   // 1 KB column blocks loaded before the first v_dot4

// 1-D grid: blocks [0, nb_lora) are LoRA blocks, (rank group, token group)
// = (b % nrg, b / nrg) with nrg = rp / 4 (wave w: rank 4*(b % nrg) + w);
// blocks from nb_lora on build the bit-planes.
__global__ __launch_bounds__(kThreads) void small_prep(const int8_t* __restrict__ q, int M, int K, int r,
                                                       int rp, const int8_t* __restrict__ A,
                                                       int32_t* __restrict__ acc_a, int8_t* __restrict__ limbs,
                                                       int32_t* __restrict__ sumq, uint8_t* __restrict__ planes,
                                                       int C, int nb_lora) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if ((int)blockIdx.x < nb_lora) {
    const int nrg = rp >> 2;
    const int j = 4 * ((int)blockIdx.x % nrg) + wave;  // rank of this wave (< rp)
    const int m0 = ((int)blockIdx.x / nrg) * kPrepTokens;
    const int mt = min(kPrepTokens, M - m0);
    const bool jr = j < r;
    const bool qsum = j == 0;  // the wave of rank 0 also sums Q
    int acc[kPrepTokens], qs[kPrepTokens];
#pragma unroll
    for (int m = 0; m < kPrepTokens; ++m) acc[m] = qs[m] = 0;
    if (jr || qsum) {
      const int8_t* arow = A + (int64_t)(jr ? j : 0) * K;
      for (int kb = 0; kb < K; kb += 1024 * kPrepBatch) {
        uint4 a[kPrepBatch], x[kPrepTokens][kPrepBatch];
#pragma unroll
        for (int u = 0; u < kPrepBatch; ++u) {
          const int k = kb + 1024 * u + 16 * lane;
          const bool ok = k < K;  // K % 32 == 0: a 16-byte chunk is wholly in or out
          a[u] = (jr && ok) ? *reinterpret_cast<const uint4*>(arow + k) : make_uint4(0, 0, 0, 0);
#pragma unroll
          for (int m = 0; m < kPrepTokens; ++m)
            x[m][u] = (ok && m < mt) ? *reinterpret_cast<const uint4*>(q + (int64_t)(m0 + m) * K + k)
                                     : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < kPrepBatch; ++u)
#pragma unroll
          for (int m = 0; m < kPrepTokens; ++m) {
            acc[m] = sdot4(a[u].x, x[m][u].x, acc[m]);
            acc[m] = sdot4(a[u].y, x[m][u].y, acc[m]);
            acc[m] = sdot4(a[u].z, x[m][u].z, acc[m]);
            acc[m] = sdot4(a[u].w, x[m][u].w, acc[m]);
            if (qsum) {
              qs[m] = sdot4(0x01010101u, x[m][u].x, qs[m]);
              qs[m] = sdot4(0x01010101u, x[m][u].y, qs[m]);
              qs[m] = sdot4(0x01010101u, x[m][u].z, qs[m]);
              qs[m] = sdot4(0x01010101u, x[m][u].w, qs[m]);
            }
          }
      }
    }
    // wave totals; lane m writes token m0 + m
    int mine = 0, mine_q = 0;
#pragma unroll
    for (int m = 0; m < kPrepTokens; ++m) {
      if (m < mt) {  // uniform
        const int t = group_sum<64>(acc[m]);
        mine = lane == m ? t : mine;
        if (qsum) {
          const int tq = group_sum<64>(qs[m]);
          mine_q = lane == m ? tq : mine_q;
        }
      }
    }
    if (lane < mt) {
      const int m = m0 + lane;
      int8_t d[4];
      dfssm_dev::split_limbs(mine, d);  // zero for ranks in [r, rp)
#pragma unroll
      for (int t = 0; t < 4; ++t) limbs[((int64_t)t * M + m) * rp + j] = d[t];
      if (jr) acc_a[(int64_t)m * r + j] = mine;
      if (qsum) sumq[m] = mine_q;
    }
    return;
  }
  // bit-planes, [M][8 planes][C chunks][16 bytes]: thread (m, p) transposes
  // codes 8p .. 8p+7 (zero at and beyond K) so that byte b holds bit b of the
  // 8 codes, which is byte p % 16 of chunk p / 16 of plane b
  const int64_t per_tok = 16 * (int64_t)C;
  const int64_t total = (int64_t)M * per_tok;
  const int64_t stride = (int64_t)(gridDim.x - nb_lora) * kThreads;
  for (int64_t i = (int64_t)(blockIdx.x - nb_lora) * kThreads + threadIdx.x; i < total; i += stride) {
    const int m = (int)(i / per_tok), p = (int)(i % per_tok);
    uint32_t lo = 0, hi = 0, t;
    if (8 * p < K) {  // K % 32 == 0: all 8 codes are in range
      const uint2 c = *reinterpret_cast<const uint2*>(q + (int64_t)m * K + 8 * p);
      lo = c.x;
      hi = c.y;
    }
    // 8x8 bit transpose: code e in byte e -> bit e of byte b = bit b of code e
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
    uint8_t* dst = planes + (int64_t)m * C * 128 + p;  // plane 0, chunk p / 16, byte p % 16
    const int64_t pstride = 16 * (int64_t)C;
#pragma unroll
    for (int b = 0; b < 4; ++b) dst[b * pstride] = (uint8_t)(lo >> (8 * b));
#pragma unroll
    for (int b = 0; b < 4; ++b) dst[(4 + b) * pstride] = (uint8_t)(hi >> (8 * b));
  }
}

// ------------------------------------------------------------------ gemv
// popcount combine for one 4-word chunk of one token: sum_{bit=1} Q
__device__ __forceinline__ int chunk_masked_sum(const uint4 w, const uint4 (&P)[8]) {
  int c[8];
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    int t = __builtin_popcount(w.x & P[b].x);
    t += __builtin_popcount(w.y & P[b].y);
    t += __builtin_popcount(w.z & P[b].z);
    t += __builtin_popcount(w.w & P[b].w);
    c[b] = t;
  }
  int sum = c[0] + (c[1] << 1) + (c[2] << 2) + (c[3] << 3) + (c[4] << 4) + (c[5] << 5) + (c[6] << 6);
  return sum - (c[7] << 7);
}

// B dwords (4 ranks each) a lane holds: j4 = g + G*i, i < kBWords(G), for
// r <= 256
template <int G>
constexpr int kBWords = (64 + G - 1) / G;

// G lanes per row; CPL chunks per lane held in registers (CPL == 0: planes
// re-read from memory per chunk, any K); MT tokens per pass.
template <int G, int CPL, int MT>
__global__ __launch_bounds__(kThreads) void decode_gemv(
    const uint32_t* __restrict__ w_bits, int W, int N, int r, int rp, const uint32_t* __restrict__ planes,
    int C, const int8_t* __restrict__ limbs, const int32_t* __restrict__ sumq, int M,
    const int8_t* __restrict__ B, const float* __restrict__ alpha, const float* __restrict__ beta,
    const float* __restrict__ s, float* __restrict__ y, int32_t* __restrict__ acc_s_out,
    int64_t* __restrict__ acc_b_out, int m0, int mt) {
  constexpr int RW = 64 / G;  // rows per wave step
  constexpr int BW = kBWords<G>;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, grp = lane / G;
  const bool vec = (W % 4) == 0;
  const bool b4 = (r & 3) == 0;
  const int r4 = (r + 3) / 4;  // dwords of one B row / limb vector
  const int nsteps = (N + RW - 1) / RW;
  const int gwave = blockIdx.x * kWavesPerBlock + wave;
  const int nwaves = gridDim.x * kWavesPerBlock;

  // the first row's signs, B bytes and scales go out before anything else
  auto load_row = [&](int step, uint4 (&wv)[CPL > 0 ? CPL : 1], uint32_t (&bw)[BW], float& al, float& be) {
    const int n = step * RW + grp;
    const bool row_ok = step < nsteps && n < N;
    const int nc = row_ok ? n : 0;
    const uint32_t* wrow = w_bits + (int64_t)nc * W;
#pragma unroll
    for (int c = 0; c < (CPL > 0 ? CPL : 1); ++c) {
      const int ch = g + c * G;
      wv[c] = make_uint4(0, 0, 0, 0);
      if (CPL > 0 && row_ok && ch < C) {
        if (vec) {
          wv[c] = *reinterpret_cast<const uint4*>(wrow + 4 * ch);
        } else {
          uint32_t t[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) t[i] = (4 * ch + i < W) ? wrow[4 * ch + i] : 0u;
          wv[c] = make_uint4(t[0], t[1], t[2], t[3]);
        }
      }
    }
    const int8_t* brow = B + (int64_t)nc * r;
#pragma unroll
    for (int i = 0; i < BW; ++i) {
      const int j4 = g + G * i;
      uint32_t v = 0;
      if (row_ok && j4 < r4) {
        if (b4) {
          v = *reinterpret_cast<const uint32_t*>(brow + 4 * j4);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (4 * j4 + e < r) v |= (uint32_t)(uint8_t)brow[4 * j4 + e] << (8 * e);
        }
      }
      bw[i] = v;
    }
    al = alpha[nc];
    be = r > 0 ? beta[nc] : 0.0f;
  };
  constexpr int CW = CPL > 0 ? CPL : 1;
  uint4 wv[CW];
  uint32_t bw[BW];
  float al, be;
  load_row(gwave, wv, bw, al, be);

  // the tokens' scales and sums of Q
  int sq[MT];
  float sv[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    sq[m] = m < mt ? sumq[m0 + m] : 0;
    sv[m] = m < mt ? s[m0 + m] : 0.0f;
  }

  // LDS: the planes of tokens m0.. (CPL > 0; plane-major, as in memory, so
  // the G lanes of a row read consecutive 16-byte chunks), then the limbs
  // of acc_a: lds_limb[(m*4 + t)*r4 + j4] = bytes 4j4 .. 4j4+3 of limb t (the
  // prep zero-pads ranks up to rp).  One read of each per block instead of
  // one per wave.
  extern __shared__ uint4 lds_dyn[];
  const int npl = CPL > 0 ? MT * 8 * C : 0;  // 16-byte plane chunks staged
  uint4* const lds_pl = lds_dyn;
  uint32_t* const lds_limb = reinterpret_cast<uint32_t*>(lds_dyn + npl);
  if (CPL > 0) {
    const uint4* src = reinterpret_cast<const uint4*>(planes) + (int64_t)m0 * 8 * C;
    for (int i = threadIdx.x; i < npl; i += kThreads)
      lds_pl[i] = i < mt * 8 * C ? src[i] : make_uint4(0, 0, 0, 0);
  }
  if (r > 0) {
    for (int i = threadIdx.x; i < MT * 4 * r4; i += kThreads) {
      const int m = i / (4 * r4), t = (i / r4) % 4, j4 = i % r4;
      lds_limb[i] = m < mt ? *reinterpret_cast<const uint32_t*>(limbs + ((int64_t)t * M + m0 + m) * rp + 4 * j4) : 0u;
    }
  }
  __syncthreads();

  for (int step = gwave; step < nsteps; step += nwaves) {
    const int n = step * RW + grp;
    const bool row_ok = n < N;
    if (step != gwave) load_row(step, wv, bw, al, be);

    int part[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) part[m] = 0;
    if constexpr (CPL > 0) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          const int ch = g + c * G;
          uint4 P[8];
#pragma unroll
          for (int b = 0; b < 8; ++b) P[b] = ch < C ? lds_pl[(m * 8 + b) * C + ch] : make_uint4(0, 0, 0, 0);
          part[m] += chunk_masked_sum(wv[c], P);
        }
    } else {
      const uint32_t* wrow = w_bits + (int64_t)(row_ok ? n : 0) * W;
      for (int ch = g; ch < C; ch += G) {
        uint4 w = make_uint4(0, 0, 0, 0);
        if (row_ok) {
          if (vec) {
            w = *reinterpret_cast<const uint4*>(wrow + 4 * ch);
          } else {
            uint32_t t[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) t[i] = (4 * ch + i < W) ? wrow[4 * ch + i] : 0u;
            w = make_uint4(t[0], t[1], t[2], t[3]);
          }
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          if (m < mt) {
            uint4 Pt[8];
#pragma unroll
            for (int b = 0; b < 8; ++b)
              Pt[b] = *reinterpret_cast<const uint4*>(planes + (((int64_t)(m0 + m) * 8 + b) * C + ch) * 4);
            part[m] += chunk_masked_sum(w, Pt);
          }
        }
      }
    }

    // LoRA up-projection partials: E_lo = D0 + 256*D1, E_hi = D2 + 256*D3
    int elo[MT], ehi[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) elo[m] = ehi[m] = 0;
    if (r > 0) {
#pragma unroll
      for (int i = 0; i < BW; ++i) {
        const int j4 = g + G * i;
        if (j4 < r4) {
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const uint32_t* lm = lds_limb + m * 4 * r4 + j4;
            const int d0 = sdot4(bw[i], lm[0], 0);
            const int d1 = sdot4(bw[i], lm[r4], 0);
            const int d2 = sdot4(bw[i], lm[2 * r4], 0);
            const int d3 = sdot4(bw[i], lm[3 * r4], 0);
            elo[m] += d0 + (d1 << 8);
            ehi[m] += d2 + (d3 << 8);
          }
        }
      }
    }

    // reduce over the G lanes of the row (every lane ends with the totals)
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      part[m] = group_sum<G>(part[m]);
      if (r > 0) {
        elo[m] = group_sum<G>(elo[m]);
        ehi[m] = group_sum<G>(ehi[m]);
      }
    }

    // epilogue: lane g handles token g
    if (row_ok && g < mt) {
      int32_t as = 2 * part[0] - sq[0], hi = ehi[0], lo = elo[0];
      float sm = sv[0];
#pragma unroll
      for (int m = 1; m < MT; ++m)
        if (g == m) {
          as = 2 * part[m] - sq[m];
          hi = ehi[m];
          lo = elo[m];
          sm = sv[m];
        }
      const int mm = m0 + g;
      if (y) y[(int64_t)mm * N + n] = dfssm_dev::epilogue(sm, al, be, as, hi, lo, r > 0);
      if (acc_s_out) acc_s_out[(int64_t)mm * N + n] = as;
      if (acc_b_out) acc_b_out[(int64_t)mm * N + n] = r > 0 ? (int64_t)lo + ((int64_t)hi << 16) : 0;
    }
  }
}

template <int G, int CPL, int MT>
hipError_t launch_gemv_t(const uint32_t* w_bits, int W, int N, int r, int rp, const uint32_t* planes, int C,
                         const int8_t* limbs, const int32_t* sumq, int M, const int8_t* B, const float* alpha,
                         const float* beta, const float* s, float* y, int32_t* acc_s, int64_t* acc_b, int m0,
                         int mt, hipStream_t st) {
  constexpr int RW = 64 / G;
  const int64_t nsteps = (N + RW - 1) / RW;
  // one row step per wave where the grid allows it
  int64_t blocks = (nsteps + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  const size_t lds = (CPL > 0 ? (size_t)MT * 8 * C * 16 : 0) + (size_t)MT * 4 * ((r + 3) / 4) * sizeof(uint32_t);
  decode_gemv<G, CPL, MT><<<dim3((unsigned)blocks), dim3(kThreads), lds, st>>>(
      w_bits, W, N, r, rp, planes, C, limbs, sumq, M, B, alpha, beta, s, y, acc_s, acc_b, m0, mt);
  return hipGetLastError();
}

struct GemvCall {
  const uint32_t* w_bits;
  int W, N, r, rp;
  const uint32_t* planes;
  int C;
  const int8_t* limbs;
  const int32_t* sumq;
  int M;
  const int8_t* B;
  const float *alpha, *beta, *s;
  float* y;
  int32_t* acc_s;
  int64_t* acc_b;
};

template <int G, int CPL, int MT>
hipError_t run_gemv(const GemvCall& c, int m0, int mt, hipStream_t st) {
  return launch_gemv_t<G, CPL, MT>(c.w_bits, c.W, c.N, c.r, c.rp, c.planes, c.C, c.limbs, c.sumq, c.M, c.B,
                                   c.alpha, c.beta, c.s, c.y, c.acc_s, c.acc_b, m0, mt, st);
}

template <int G, int MT>
hipError_t launch_gemv_cpl(const GemvCall& c, int m0, int mt, hipStream_t st) {
  const int cpl = (c.C + G - 1) / G;
  if (cpl <= 1) return run_gemv<G, 1, MT>(c, m0, mt, st);
  if constexpr (MT == 1) {
    if (cpl <= 2) return run_gemv<G, 2, MT>(c, m0, mt, st);
  }
  return run_gemv<G, 0, MT>(c, m0, mt, st);
}

template <int MT>
hipError_t launch_gemv_mt(const GemvCall& c, int m0, int mt, hipStream_t st) {
  // lanes per row: the smallest power of two >= chunks per row, from 8 to 64
  if (c.C <= 8) return launch_gemv_cpl<8, MT>(c, m0, mt, st);
  if (c.C <= 16) return launch_gemv_cpl<16, MT>(c, m0, mt, st);
  if (c.C <= 32) return launch_gemv_cpl<32, MT>(c, m0, mt, st);
  return launch_gemv_cpl<64, MT>(c, m0, mt, st);
}

// acc_a, its limbs, sum Q and the bit-planes of the M tokens into the
// workspace
hipError_t launch_small_prep(const int8_t* q, int64_t M, int64_t K, int64_t r, const int8_t* A,
                             const dfssm::LinearWorkspace& ws, hipStream_t st) {
  if (M == 0) return hipSuccess;
  const int rp = (int)dfssm::rank_padded(r);
  const int C = (int)dfssm::plane_chunks(K);
  const int64_t nb_lora = (int64_t)(rp / 4) * dfssm::ceil_div(M, kPrepTokens);
  const int64_t nb_planes = std::min<int64_t>(dfssm::ceil_div(M * 16 * C, kThreads), 4096);
  if (nb_lora + nb_planes > 0x7fffffff) return hipErrorInvalidValue;
  small_prep<<<dim3((unsigned)(nb_lora + nb_planes)), dim3(kThreads), 0, st>>>(
      q, (int)M, (int)K, (int)r, rp, A, ws.acc_a, ws.limbs, ws.sumq, reinterpret_cast<uint8_t*>(ws.planes), C,
      (int)nb_lora);
  return hipGetLastError();
}

}  // namespace

namespace dfssm {

hipError_t launch_decode_linear(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                                int64_t r, const uint32_t* w_bits, const float* alpha,
                                const int8_t* A, const int8_t* B, const float* beta, float* y,
                                int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                                const LinearWorkspace& ws, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  hipError_t e = launch_small_prep(q, M, K, r, A, ws, st);
  if (e != hipSuccess) return e;
  if (acc_a_out && r > 0) {
    e = hipMemcpyAsync(acc_a_out, ws.acc_a, (size_t)(M * r) * 4, hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
  }
  GemvCall c{w_bits, (int)(K / 32), (int)N, (int)r, (int)rank_padded(r), ws.planes, (int)plane_chunks(K),
             ws.limbs, ws.sumq, (int)M, B, alpha, beta, s, y, acc_s, acc_b};
  for (int64_t m0 = 0; m0 < M; m0 += kDecodeMaxTokens) {
    const int mt = (int)((M - m0) < kDecodeMaxTokens ? (M - m0) : kDecodeMaxTokens);
    if (mt == 1)
      e = launch_gemv_mt<1>(c, (int)m0, mt, st);
    else if (mt == 2)
      e = launch_gemv_mt<2>(c, (int)m0, mt, st);
    else
      e = launch_gemv_mt<4>(c, (int)m0, mt, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace dfssm
