// dfssm_decode.hip -- decode-shaped (small M) scaffold + LoRA linear, gfx950.
//
// At M = 1..4 the scaffold product is a matrix-vector product over 1-bit
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
//  prep   -- blocks [0, r): acc_a[m, j] = sum_k A[j,k] Q[m,k] with v_dot4
//            (16-byte loads of A and Q); blocks [r, ..): bit-planes of Q built
//            with wave ballots into the workspace, laid out so that a GEMV
//            lane fetches the 8 planes of its 4-word chunk as 8 x 16 bytes.
//  gemv   -- a group of G lanes owns one output row at a time; lane g holds
//            the planes of chunks g, g+G, ... in VGPRs for the whole kernel and
//            streams its chunk of every row it visits with one 16-byte load.
//            Per row: popcounts, the LoRA up-projection (B row with v_dot4
//            against acc_a split into 4 int8 limbs, held in LDS), a butterfly
//            reduction over the G lanes, and the fp32 epilogue.
#include "dfssm_internal.hpp"

namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / 64;

__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}

// ------------------------------------------------------------------ prep
// acc_a rows: one block per j.  Plane blocks: each wave turns 64 columns of
// one token into 8 ballots (2 words per plane).
__global__ __launch_bounds__(kThreads) void decode_prep(const int8_t* __restrict__ q, int M, int K,
                                                        int r, const int8_t* __restrict__ A,
                                                        int32_t* __restrict__ acc_a,
                                                        uint32_t* __restrict__ planes, int C) {
  __shared__ int red[kWavesPerBlock];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if ((int)blockIdx.x < r) {
    const int j = blockIdx.x;
    const int8_t* arow = A + (int64_t)j * K;
    for (int m = 0; m < M; ++m) {
      const int8_t* qrow = q + (int64_t)m * K;
      int acc = 0;
      for (int k = threadIdx.x * 16; k < K; k += kThreads * 16) {  // K % 32 == 0
        uint4 a = *reinterpret_cast<const uint4*>(arow + k);
        uint4 x = *reinterpret_cast<const uint4*>(qrow + k);
        acc = sdot4(a.x, x.x, acc);
        acc = sdot4(a.y, x.y, acc);
        acc = sdot4(a.z, x.z, acc);
        acc = sdot4(a.w, x.w, acc);
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
      if (lane == 0) red[wave] = acc;
      __syncthreads();
      if (threadIdx.x == 0) acc_a[(int64_t)m * r + j] = red[0] + red[1] + red[2] + red[3];
      __syncthreads();
    }
    return;
  }
  // planes: global wave index over (token, 64-column group); columns at and
  // beyond K (up to the chunk padding 128*C) read as zero.
  const int groups = 2 * C;  // 64-column groups per token
  const int total = M * groups;
  const int nwaves = (gridDim.x - r) * kWavesPerBlock;
  for (int gw = (blockIdx.x - r) * kWavesPerBlock + wave; gw < total; gw += nwaves) {
    const int m = gw / groups, grp = gw % groups;
    const int col = grp * 64 + lane;
    const int v = col < K ? (int)q[(int64_t)m * K + col] : 0;
    uint64_t mask[8];
#pragma unroll
    for (int b = 0; b < 8; ++b) mask[b] = __ballot((v >> b) & 1);
    if (lane < 16) {
      const int b = lane >> 1, h = lane & 1;
      const int w = grp * 2 + h;  // word index in the row (< 4*C)
      uint64_t mk = mask[0];
#pragma unroll
      for (int t = 1; t < 8; ++t) mk = (b == t) ? mask[t] : mk;
      planes[(((int64_t)m * C + (w >> 2)) * 8 + b) * 4 + (w & 3)] = (uint32_t)(mk >> (32 * h));
    }
  }
}

// ------------------------------------------------------------------ gemv
// popcount combine for one 4-word chunk of one token
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

__device__ __forceinline__ int chunk_qsum(const uint4 (&P)[8]) {
  int c[8];
#pragma unroll
  for (int b = 0; b < 8; ++b)
    c[b] = __builtin_popcount(P[b].x) + __builtin_popcount(P[b].y) + __builtin_popcount(P[b].z) +
           __builtin_popcount(P[b].w);
  int sum = c[0] + (c[1] << 1) + (c[2] << 2) + (c[3] << 3) + (c[4] << 4) + (c[5] << 5) + (c[6] << 6);
  return sum - (c[7] << 7);
}

template <int G>
__device__ __forceinline__ int group_sum(int v) {
#pragma unroll
  for (int off = G / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// G lanes per row; CPL chunks per lane held in registers (CPL == 0: planes
// re-read from memory per chunk, any K); MT tokens per pass.
template <int G, int CPL, int MT>
__global__ __launch_bounds__(kThreads) void decode_gemv(
    const uint32_t* __restrict__ w_bits, int W, int N, int r, const uint32_t* __restrict__ planes,
    int C, const int32_t* __restrict__ acc_a, const int8_t* __restrict__ B,
    const float* __restrict__ alpha, const float* __restrict__ beta, const float* __restrict__ s,
    float* __restrict__ y, int32_t* __restrict__ acc_s_out, int64_t* __restrict__ acc_b_out,
    int m0, int mt, int N_out) {
  constexpr int RW = 64 / G;  // rows per wave step
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, grp = lane / G;
  const bool vec = (W % 4) == 0;
  const int r4 = (r + 3) / 4;  // dwords of one B row / limb vector

  // LoRA limbs of acc_a for tokens m0.. : lds_limb[m][t][j4] packs 4
  // consecutive j of limb t.
  extern __shared__ uint32_t lds_limb[];
  if (r > 0) {
    for (int i = threadIdx.x; i < MT * r4; i += kThreads) {
      const int m = i / r4, j4 = i % r4;
      uint32_t packed[4] = {0, 0, 0, 0};
      if (m < mt) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = 4 * j4 + e;
          if (j < r) {
            int8_t d[4];
            dfssm_dev::split_limbs(acc_a[(int64_t)(m0 + m) * r + j], d);
#pragma unroll
            for (int t = 0; t < 4; ++t) packed[t] |= (uint32_t)(uint8_t)d[t] << (8 * e);
          }
        }
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) lds_limb[(m * 4 + t) * r4 + j4] = packed[t];
    }
    __syncthreads();
  }

  // this lane's planes and its share of sum Q
  constexpr int CR = CPL > 0 ? CPL : 1;
  uint4 P[MT][CR][8];
  int qpart[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    qpart[m] = 0;
#pragma unroll
    for (int c = 0; c < CR; ++c) {
      const int ch = g + c * G;
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        P[m][c][b] = (m < mt && ch < C && CPL > 0)
                         ? *reinterpret_cast<const uint4*>(planes + (((int64_t)(m0 + m) * C + ch) * 8 + b) * 4)
                         : make_uint4(0, 0, 0, 0);
      }
      if (CPL > 0) qpart[m] += chunk_qsum(P[m][c]);
    }
    if (CPL == 0 && m < mt) {
      for (int ch = g; ch < C; ch += G) {
        uint4 Pt[8];
#pragma unroll
        for (int b = 0; b < 8; ++b)
          Pt[b] = *reinterpret_cast<const uint4*>(planes + (((int64_t)(m0 + m) * C + ch) * 8 + b) * 4);
        qpart[m] += chunk_qsum(Pt);
      }
    }
  }

  const int nsteps = (N + RW - 1) / RW;
  const int gwave = blockIdx.x * kWavesPerBlock + wave;
  const int nwaves = gridDim.x * kWavesPerBlock;
  for (int step = gwave; step < nsteps; step += nwaves) {
    const int n = step * RW + grp;
    const bool row_ok = n < N;
    const uint32_t* wrow = w_bits + (int64_t)(row_ok ? n : 0) * W;

    int part[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) part[m] = 0;

    auto load_chunk = [&](int ch) -> uint4 {
      if (!row_ok || ch >= C) return make_uint4(0, 0, 0, 0);
      if (vec) return *reinterpret_cast<const uint4*>(wrow + 4 * ch);
      uint32_t t[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) t[i] = (4 * ch + i < W) ? wrow[4 * ch + i] : 0u;
      return make_uint4(t[0], t[1], t[2], t[3]);
    };

    if constexpr (CPL > 0) {
      uint4 wv[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) wv[c] = load_chunk(g + c * G);
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int c = 0; c < CPL; ++c) part[m] += chunk_masked_sum(wv[c], P[m][c]);
    } else {
      for (int ch = g; ch < C; ch += G) {
        uint4 wv = load_chunk(ch);
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          if (m < mt) {
            uint4 Pt[8];
#pragma unroll
            for (int b = 0; b < 8; ++b)
              Pt[b] = *reinterpret_cast<const uint4*>(planes + (((int64_t)(m0 + m) * C + ch) * 8 + b) * 4);
            part[m] += chunk_masked_sum(wv, Pt);
          }
        }
      }
    }

    // LoRA up-projection partials: E_lo = D0 + 256*D1, E_hi = D2 + 256*D3
    int elo[MT], ehi[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) elo[m] = ehi[m] = 0;
    if (r > 0 && row_ok) {
      const int8_t* brow = B + (int64_t)n * r;
      for (int j4 = g; j4 < r4; j4 += G) {
        uint32_t bw;
        if ((r & 3) == 0) {
          bw = *reinterpret_cast<const uint32_t*>(brow + 4 * j4);
        } else {
          bw = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (4 * j4 + e < r) bw |= (uint32_t)(uint8_t)brow[4 * j4 + e] << (8 * e);
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const int d0 = sdot4(bw, lds_limb[(m * 4 + 0) * r4 + j4], 0);
          const int d1 = sdot4(bw, lds_limb[(m * 4 + 1) * r4 + j4], 0);
          const int d2 = sdot4(bw, lds_limb[(m * 4 + 2) * r4 + j4], 0);
          const int d3 = sdot4(bw, lds_limb[(m * 4 + 3) * r4 + j4], 0);
          elo[m] += d0 + (d1 << 8);
          ehi[m] += d2 + (d3 << 8);
        }
      }
    }

    // reduce over the G lanes of the row (every lane ends with the totals)
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      part[m] = group_sum<G>(2 * part[m] - qpart[m]);
      if (r > 0) {
        elo[m] = group_sum<G>(elo[m]);
        ehi[m] = group_sum<G>(ehi[m]);
      }
    }

    // epilogue: lane g handles token g
    if (row_ok && g < mt) {
      int32_t as = part[0], hi = ehi[0], lo = elo[0];
#pragma unroll
      for (int m = 1; m < MT; ++m)
        if (g == m) {
          as = part[m];
          hi = ehi[m];
          lo = elo[m];
        }
      const int mm = m0 + g;
      if (y)
        y[(int64_t)mm * N_out + n] =
            dfssm_dev::epilogue(s[mm], alpha[n], r > 0 ? beta[n] : 0.0f, as, hi, lo, r > 0);
      if (acc_s_out) acc_s_out[(int64_t)mm * N_out + n] = as;
      if (acc_b_out) acc_b_out[(int64_t)mm * N_out + n] = r > 0 ? (int64_t)lo + ((int64_t)hi << 16) : 0;
    }
  }
}

template <int G, int CPL, int MT>
hipError_t launch_gemv_t(const uint32_t* w_bits, int W, int N, int r, const uint32_t* planes, int C,
                         const int32_t* acc_a, const int8_t* B, const float* alpha,
                         const float* beta, const float* s, float* y, int32_t* acc_s,
                         int64_t* acc_b, int m0, int mt, hipStream_t st) {
  constexpr int RW = 64 / G;
  const int64_t nsteps = (N + RW - 1) / RW;
  // enough waves to give every CU several; each wave walks rows with a
  // grid stride
  int64_t blocks = (nsteps + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  const size_t lds = (size_t)MT * 4 * ((r + 3) / 4) * sizeof(uint32_t);
  decode_gemv<G, CPL, MT><<<dim3((unsigned)blocks), dim3(kThreads), lds, st>>>(
      w_bits, W, N, r, planes, C, acc_a, B, alpha, beta, s, y, acc_s, acc_b, m0, mt, N);
  return hipGetLastError();
}

template <int G, int MT>
hipError_t launch_gemv_cpl(int C, const uint32_t* w_bits, int W, int N, int r,
                           const uint32_t* planes, const int32_t* acc_a, const int8_t* B,
                           const float* alpha, const float* beta, const float* s, float* y,
                           int32_t* acc_s, int64_t* acc_b, int m0, int mt, hipStream_t st) {
  const int cpl = (C + G - 1) / G;
  if (cpl <= 1)
    return launch_gemv_t<G, 1, MT>(w_bits, W, N, r, planes, C, acc_a, B, alpha, beta, s, y, acc_s,
                                   acc_b, m0, mt, st);
  if (cpl <= 2 && MT == 1)
    return launch_gemv_t<G, 2, MT>(w_bits, W, N, r, planes, C, acc_a, B, alpha, beta, s, y, acc_s,
                                   acc_b, m0, mt, st);
  return launch_gemv_t<G, 0, MT>(w_bits, W, N, r, planes, C, acc_a, B, alpha, beta, s, y, acc_s,
                                 acc_b, m0, mt, st);
}

template <int MT>
hipError_t launch_gemv_mt(int C, const uint32_t* w_bits, int W, int N, int r,
                          const uint32_t* planes, const int32_t* acc_a, const int8_t* B,
                          const float* alpha, const float* beta, const float* s, float* y,
                          int32_t* acc_s, int64_t* acc_b, int m0, int mt, hipStream_t st) {
  // lanes per row: the smallest power of two >= chunks per row, from 8 to 64
  if (C <= 8)
    return launch_gemv_cpl<8, MT>(C, w_bits, W, N, r, planes, acc_a, B, alpha, beta, s, y, acc_s,
                                  acc_b, m0, mt, st);
  if (C <= 16)
    return launch_gemv_cpl<16, MT>(C, w_bits, W, N, r, planes, acc_a, B, alpha, beta, s, y, acc_s,
                                   acc_b, m0, mt, st);
  if (C <= 32)
    return launch_gemv_cpl<32, MT>(C, w_bits, W, N, r, planes, acc_a, B, alpha, beta, s, y, acc_s,
                                   acc_b, m0, mt, st);
  return launch_gemv_cpl<64, MT>(C, w_bits, W, N, r, planes, acc_a, B, alpha, beta, s, y, acc_s,
                                 acc_b, m0, mt, st);
}

}  // namespace

namespace dfssm {

hipError_t launch_decode_linear(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                                int64_t r, const uint32_t* w_bits, const float* alpha,
                                const int8_t* A, const int8_t* B, const float* beta, float* y,
                                int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                                const LinearWorkspace& ws, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  const int C = (int)plane_chunks(K);
  // prep: r acc_a blocks + plane blocks (one wave per 64 columns of a token)
  const int64_t plane_waves = M * 2 * C;
  int64_t plane_blocks = (plane_waves + kWavesPerBlock - 1) / kWavesPerBlock;
  if (plane_blocks > 1024) plane_blocks = 1024;
  int32_t* acc_a = ws.acc_a;
  decode_prep<<<dim3((unsigned)(r + plane_blocks)), dim3(kThreads), 0, st>>>(
      q, (int)M, (int)K, (int)r, A, acc_a, ws.planes, C);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (acc_a_out && r > 0) {
    e = hipMemcpyAsync(acc_a_out, acc_a, (size_t)(M * r) * 4, hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
  }
  const int W = (int)(K / 32);
  for (int64_t m0 = 0; m0 < M; m0 += kDecodeMaxTokens) {
    const int mt = (int)((M - m0) < kDecodeMaxTokens ? (M - m0) : kDecodeMaxTokens);
    if (mt == 1)
      e = launch_gemv_mt<1>(C, w_bits, W, (int)N, (int)r, ws.planes, acc_a, B, alpha, beta, s, y,
                            acc_s, acc_b, (int)m0, mt, st);
    else if (mt == 2)
      e = launch_gemv_mt<2>(C, w_bits, W, (int)N, (int)r, ws.planes, acc_a, B, alpha, beta, s, y,
                            acc_s, acc_b, (int)m0, mt, st);
    else
      e = launch_gemv_mt<4>(C, w_bits, W, (int)N, (int)r, ws.planes, acc_a, B, alpha, beta, s, y,
                            acc_s, acc_b, (int)m0, mt, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace dfssm
