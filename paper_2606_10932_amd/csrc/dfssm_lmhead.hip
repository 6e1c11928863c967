// dfssm_lmhead.hip -- the tied int8 embedding table of the model: token
// gather and LM head, gfx950.
//
// The table is int8 per row with a fp32 row scale (Sec. 3.3: the embedding
// is quantised to int8 per row; Table 1: embedding and LM head tied, 103 MB
// for the 1.3B model's 50,280 x 2048).  The LM head takes the final hidden
// state through the same per-token int8 quantiser as the linears:
//
//   acc[m,v]    = sum_k E[v,k] Q[m,k]                 exact int32
//   logits[m,v] = s[m] * (scale[v] * (float)acc)      fp32, this order
//
// At a few tokens the LM head streams the whole table once (2 int-ops per
// byte per token): HBM-bound.  A wave visits R rows at a time (4 KB of the
// table: R = 2 rows of 2 KB at d = 2048); each lane holds its 16-byte slices
// of every token's codes for the whole kernel, and every load of the R rows
// is issued before the first v_dot4.  Waves stride over the row groups, so
// the waves of the grid read neighbouring 4 KB pieces at any moment; the
// table is read once, so its loads are non-temporal (no reuse to keep in the
// caches).  Three workgroups (12 waves) per CU: more waves, bigger visits
// and each wave owning one contiguous range of rows all measured slower.  Row sums go by DPP inside 16-lane
// rows and gfx950's permlane swaps across them.
#include <algorithm>
#include <stdlib.h>

#include "dfssm_internal.hpp"
#include "dfssm_persist.hpp"

namespace {

constexpr int kThreads = 256;

// Tokens from which the LM head runs on the matrix cores (8; the test switch
// lm_head_mfma_tokens moves it).
int lm_head_mfma_tokens() {
  const int v = dfssm::test_switch(DFSSM_TEST_LM_HEAD_MFMA_TOKENS);
  return v > 0 ? v : 8;
}

// Tokens from which the matrix-core path runs the tiled kernel (64; the
// test switch lm_head_tiled_tokens moves it).
int lm_head_tiled_tokens() {
  const int v = dfssm::test_switch(DFSSM_TEST_LM_HEAD_TILED_TOKENS);
  return v > 0 ? v : 64;
}

// rows per wave visit: 4 KB of the table, or one row when rows are longer
template <int NC>
constexpr int rows_per_visit() { return NC >= 4 ? 1 : 4 / NC; }

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 load_stream(const int8_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}

// whole-wave sum, the total in every lane
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

// MT tokens per pass, NC 1 KB chunks of a row (d <= 1024 * NC).  Lane l
// owns bytes 16l + 1024c of every row (zero past d).
template <int MT, int NC>
__global__ __launch_bounds__(kThreads) void lm_head(const int8_t* __restrict__ q, const float* __restrict__ s,
                                                    int d, const int8_t* __restrict__ E,
                                                    const float* __restrict__ scale, int V,
                                                    float* __restrict__ logits, int32_t* __restrict__ acc_out,
                                                    int m0, int mt) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwaves = gridDim.x * (kThreads / 64);
  constexpr int R = rows_per_visit<NC>();
  const int ngroups = (V + R - 1) / R;

  // this lane's slices of the tokens' codes, and their scales
  u32x4 qv[MT][NC];
  float sv[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int k = 16 * lane + 1024 * c;
      qv[m][c] = (m < mt && k < d) ? *reinterpret_cast<const u32x4*>(q + (int64_t)(m0 + m) * d + k)
                                   : u32x4{0, 0, 0, 0};
    }
    sv[m] = m < mt ? s[m0 + m] : 0.0f;
  }

  for (int g = blockIdx.x * (kThreads / 64) + wave; g < ngroups; g += nwaves) {
    const int v0 = g * R;
    // every load of the R rows first (rows past V are not read)
    u32x4 ev[R][NC];
    float sc[R];
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int v = v0 + i;
      const bool ok = v < V;
      const int8_t* row = E + (int64_t)(ok ? v : 0) * d;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int k = 16 * lane + 1024 * c;
        ev[i][c] = (ok && k < d) ? load_stream(row + k) : u32x4{0, 0, 0, 0};
      }
      sc[i] = ok ? scale[v] : 0.0f;
    }
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int v = v0 + i;
      int tot_m = 0;
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        int a = 0;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          a = sdot4(ev[i][c].x, qv[m][c].x, a);
          a = sdot4(ev[i][c].y, qv[m][c].y, a);
          a = sdot4(ev[i][c].z, qv[m][c].z, a);
          a = sdot4(ev[i][c].w, qv[m][c].w, a);
        }
        const int t = wave_sum(a);
        tot_m = lane == m ? t : tot_m;  // lane m keeps token m's sum
      }
      if (lane < mt && v < V) {
        const int m = lane;
        float s_m = sv[0];
#pragma unroll
        for (int mm = 1; mm < MT; ++mm) s_m = m == mm ? sv[mm] : s_m;
        const float fa = (float)tot_m;
        const float t = sc[i] * fa;
        if (logits) logits[(int64_t)(m0 + m) * V + v] = s_m * t;
        if (acc_out) acc_out[(int64_t)(m0 + m) * V + v] = tot_m;
      }
    }
  }
}

template <int MT, int NC>
hipError_t launch_t(const int8_t* q, const float* s, int d, const int8_t* E, const float* scale, int V,
                    float* logits, int32_t* acc, int m0, int mt, hipStream_t st) {
  const int64_t groups = dfssm::ceil_div(V, rows_per_visit<NC>());
  int64_t blocks = dfssm::ceil_div(groups, kThreads / 64);
  blocks = std::max<int64_t>(1, std::min<int64_t>(blocks, 3 * dfssm::device_cu_count()));
  lm_head<MT, NC><<<dim3((unsigned)blocks), dim3(kThreads), 0, st>>>(q, s, d, E, scale, V, logits, acc, m0, mt);
  return hipGetLastError();
}

// ---- many tokens: the matrix cores ------------------------------------
// A workgroup owns 64 vocabulary rows (4 row tiles of 16) and every token:
// its nw waves split d, each holding the E operands of its columns for all
// 4 row tiles in registers, so the table is read once whatever M is.  Token
// tiles of 16 stream Q from L2; the waves' partial tiles are summed in LDS
// and four waves write the logits of one row tile each, in the same fp32
// order as the GEMV kernel.  v_mfma_i32_16x16x64_i8 contracts 64 columns in
// an order of its own; E and Q place column c0 + 16 kg + b in byte b of lane
// (row, kg) alike, so the order is the same on both sides.
typedef int v4i __attribute__((ext_vector_type(4)));
constexpr int kMfmaRows = 64;
constexpr int kMfmaMaxWaves = 8;

__device__ __forceinline__ v4i load16i(const int8_t* p) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  return v4i{(int)u.x, (int)u.y, (int)u.z, (int)u.w};
}

template <int KS>
__global__ __launch_bounds__(64 * kMfmaMaxWaves) void lm_head_mfma(const int8_t* __restrict__ q,
                                                                  const float* __restrict__ s, int M, int d,
                                                                  const int8_t* __restrict__ E,
                                                                  const float* __restrict__ scale, int V,
                                                                  float* __restrict__ logits,
                                                                  int32_t* __restrict__ acc_out) {
  // two buffers of the waves' partial tiles: tile tt + 2 writes the buffer
  // of tile tt only after the barrier of tile tt + 1, which every reader of
  // tile tt passes with its LDS reads done, so one barrier per tile suffices
  __shared__ v4i red[2][kMfmaMaxWaves][4][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nw = blockDim.x >> 6;
  const int rho = lane & 15, kg = lane >> 4;
  const int v0 = blockIdx.x * kMfmaRows;
  const int c0 = wave * KS * 64 + 16 * kg;  // this lane's first column

  v4i e[4][KS];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int row = v0 + 16 * t + rho;
    const bool ok = row < V;
    const int8_t* rp = E + (int64_t)(ok ? row : 0) * d + c0;
#pragma unroll
    for (int k = 0; k < KS; ++k) e[t][k] = ok ? load16i(rp + 64 * k) : v4i{0, 0, 0, 0};
  }
  // the row scales of the tile this wave finishes (waves 0..3: row tile
  // `wave`), loaded once
  const bool vec_store = (V & 3) == 0;  // 4 consecutive rows of a token are 16 aligned bytes
  const int row0 = v0 + 16 * (wave & 3) + 4 * kg;
  float scv[4] = {0.f, 0.f, 0.f, 0.f};
  if (wave < 4) {
    if (vec_store && row0 + 3 < V) {
      const float4 sc = *reinterpret_cast<const float4*>(scale + row0);
      scv[0] = sc.x; scv[1] = sc.y; scv[2] = sc.z; scv[3] = sc.w;
    } else {
#pragma unroll
      for (int vv = 0; vv < 4; ++vv) scv[vv] = row0 + vv < V ? scale[row0 + vv] : 0.f;
    }
  }
  const int ntt = (M + 15) / 16;
  // a tile's token scale goes out just before its Q codes: the wait for the
  // codes before the tile's MFMAs covers it, so the reduction after them
  // never waits for the next tile's loads (a wave's loads complete in order)
  auto load_q = [&](int tt, v4i (&x)[KS], float& sm) {
    const int m = 16 * tt + rho;
    const bool mok = m < M;
    sm = s[mok ? m : 0];
    const int8_t* qp = q + (int64_t)(mok ? m : 0) * d + c0;
#pragma unroll
    for (int k = 0; k < KS; ++k) x[k] = mok ? load16i(qp + 64 * k) : v4i{0, 0, 0, 0};
  };
  v4i x[KS];
  float sm_next;
  load_q(0, x, sm_next);
  for (int tt = 0; tt < ntt; ++tt) {
    const int m = 16 * tt + rho;
    const bool mok = m < M;
    const float sm = sm_next;
    v4i acc[4] = {v4i{0, 0, 0, 0}, v4i{0, 0, 0, 0}, v4i{0, 0, 0, 0}, v4i{0, 0, 0, 0}};
#pragma unroll
    for (int k = 0; k < KS; ++k)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(e[t][k], x[k], acc[t], 0, 0, 0);
    // the next tile's loads go out before this tile's reduction and stores
    if (tt + 1 < ntt) load_q(tt + 1, x, sm_next);
    v4i (&rb)[kMfmaMaxWaves][4][64] = red[tt & 1];
#pragma unroll
    for (int t = 0; t < 4; ++t) rb[wave][t][lane] = acc[t];
    __syncthreads();
    if (wave < 4) {
      // lane (rho, kg) holds D[row 16 wave + 4 kg + vv][token 16 tt + rho]
      v4i sum = rb[0][wave][lane];
      for (int w = 1; w < nw; ++w) sum += rb[w][wave][lane];
      if (mok) {
        if (vec_store && row0 + 3 < V) {
          const float f0 = (float)sum[0], f1 = (float)sum[1], f2 = (float)sum[2], f3 = (float)sum[3];
          const float t0 = scv[0] * f0, t1 = scv[1] * f1, t2 = scv[2] * f2, t3 = scv[3] * f3;
          if (logits)
            *reinterpret_cast<float4*>(logits + (int64_t)m * V + row0) = make_float4(sm * t0, sm * t1, sm * t2, sm * t3);
          if (acc_out) *reinterpret_cast<int4*>(acc_out + (int64_t)m * V + row0) = make_int4(sum[0], sum[1], sum[2], sum[3]);
        } else {
#pragma unroll
          for (int vv = 0; vv < 4; ++vv) {
            const int row = row0 + vv;
            if (row < V) {
              const float fa = (float)sum[vv];
              const float tv = scv[vv] * fa;
              if (logits) logits[(int64_t)m * V + row] = sm * tv;
              if (acc_out) acc_out[(int64_t)m * V + row] = sum[vv];
            }
          }
        }
      }
    }
  }
}

// ---- many tokens, tiled: a GEMM with both operands staged in LDS --------
// A workgroup (4 waves) owns kTlRows vocabulary rows x TB tokens; wave
// (wr, wt) = (w & 1, w >> 1) owns rows 64 wr .. +63 (4 row tiles) and
// tokens TB/2 wt .. +TB/2-1 (TB/32 token tiles).  Each 64-column stage of
// the E rows and the Q rows is brought into a ring of kTlRing LDS slots by
// direct-to-LDS loads, 16-byte chunk c of row r at position c ^ ((r >> 1)
// & 3) (as the prefill kernel's Q tiles: conflict-free reads); one wait and
// one barrier per stage.  E and Q place column 64 st + 16 kg + b in byte b of
// lane (row, kg) alike, so the int32 sums equal the other kernels' and the
// logits keep their fp32 order.  Workgroup id: the ntb token blocks of a row
// block are consecutive ids with the same id mod 8, so they run on one XCD
// back to back and read the row block's 256 KB of the table from HBM once.
constexpr int kTlRows = 128;
constexpr int kTlRing = 3;
constexpr int kTlThreads = 256;

template <int TB>
__global__ __launch_bounds__(kTlThreads, 2) void lm_head_tiled(const int8_t* __restrict__ q,
                                                              const float* __restrict__ s, int M, int d,
                                                              const int8_t* __restrict__ E,
                                                              const float* __restrict__ scale, int V,
                                                              float* __restrict__ logits,
                                                              int32_t* __restrict__ acc_out, int nrb, int ntb) {
  constexpr int kStageE = kTlRows * 64, kStageQ = TB * 64, kStage = kStageE + kStageQ;
  constexpr int NJ = TB / 32;                // token tiles per wave
  constexpr int LE = kTlRows / 64, LQ = TB / 64;  // direct-to-LDS loads per wave per stage (1 KB each)
  __shared__ __align__(16) int8_t ring[kTlRing * kStage];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rho = lane & 15, kg = lane >> 4;
  const int id = (int)blockIdx.x, x = id & 7, k = id >> 3;
  const int tb = k % ntb, rb = (k / ntb) * 8 + x;
  if (rb >= nrb) return;
  const int v0 = rb * kTlRows, m0 = tb * TB;
  // lane offsets of this wave's loads: 16 rows of 64 bytes per load, lane i
  // takes row i / 4 and the chunk that belongs at position i % 4 (rows and
  // tokens past the ends repeat the last one; their results are not stored)
  uint32_t voe[LE], voq[LQ];
#pragma unroll
  for (int u = 0; u < LE; ++u) {
    const int rl = 16 * (LE * wave + u) + (lane >> 2);
    const int c = (lane & 3) ^ ((rl >> 1) & 3);
    voe[u] = (uint32_t)min(v0 + rl, V - 1) * (uint32_t)d + 16u * (uint32_t)c;
  }
#pragma unroll
  for (int u = 0; u < LQ; ++u) {
    const int tl = 16 * (wave + 4 * u) + (lane >> 2);
    const int c = (lane & 3) ^ ((tl >> 1) & 3);
    voq[u] = (uint32_t)min(m0 + tl, M - 1) * (uint32_t)d + 16u * (uint32_t)c;
  }
  const uint32_t ring0 = dfssm_px::lds_addr(ring);
  const int ns = d / 64;
  auto issue = [&](int st) {
    const uint32_t slot = ring0 + (uint32_t)((st % kTlRing) * kStage);
#pragma unroll
    for (int u = 0; u < LE; ++u) dfssm_px::lds_dma16(voe[u], E + 64 * st, slot + (uint32_t)((LE * wave + u) * 1024));
#pragma unroll
    for (int u = 0; u < LQ; ++u)
      dfssm_px::lds_dma16(voq[u], q + 64 * st, slot + (uint32_t)(kStageE + (wave + 4 * u) * 1024));
  };
  const int wr = wave & 1, wt = wave >> 1;
  v4i acc[4][NJ];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = v4i{0, 0, 0, 0};
  for (int st = 0; st < kTlRing - 1 && st < ns; ++st) issue(st);
  for (int st = 0; st < ns; ++st) {
    // this wave's loads of stage st are in once at most the loads of the
    // later stages it has issued remain; the barrier then makes
    // every wave's loads visible and frees the slot of stage st - 1
    static_assert(kTlRing >= 2 && kTlRing <= 6, "wait counts below cover rings of 2 to 6 slots");
    switch (min(ns - 1 - st, kTlRing - 2)) {  // the later stages issued
      case 4: CHAIN_WAIT_VMCNT(4 * (LE + LQ)); break;
      case 3: CHAIN_WAIT_VMCNT(3 * (LE + LQ)); break;
      case 2: CHAIN_WAIT_VMCNT(2 * (LE + LQ)); break;
      case 1: CHAIN_WAIT_VMCNT(LE + LQ); break;
      default: CHAIN_WAIT_VMCNT(0); break;
    }
    CHAIN_BARRIER();
    if (st + kTlRing - 1 < ns) issue(st + kTlRing - 1);
    const int8_t* sl = ring + (st % kTlRing) * kStage;
    v4i a[4], b[NJ];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 64 * wr + 16 * i + rho;
      a[i] = *reinterpret_cast<const v4i*>(sl + r * 64 + 16 * (kg ^ ((r >> 1) & 3)));
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int t = (TB / 2) * wt + 16 * j + rho;
      b[j] = *reinterpret_cast<const v4i*>(sl + kStageE + t * 64 + 16 * (kg ^ ((t >> 1) & 3)));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[i], b[j], acc[i][j], 0, 0, 0);
  }
  // lane (rho, kg) of tile (i, j) holds D[row 64 wr + 16 i + 4 kg + v][token TB/2 wt + 16 j + rho]
  const bool vec_store = (V & 3) == 0;
  float sm[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) sm[j] = s[min(m0 + (TB / 2) * wt + 16 * j + rho, M - 1)];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row0 = v0 + 64 * wr + 16 * i + 4 * kg;
    const bool whole = vec_store && row0 + 3 < V;
    float sc[4];
    if (whole) {
      const float4 t = *reinterpret_cast<const float4*>(scale + row0);
      sc[0] = t.x; sc[1] = t.y; sc[2] = t.z; sc[3] = t.w;
    } else {
#pragma unroll
      for (int v = 0; v < 4; ++v) sc[v] = row0 + v < V ? scale[row0 + v] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int m = m0 + (TB / 2) * wt + 16 * j + rho;
      if (m >= M) continue;
      const v4i sum = acc[i][j];
      if (whole) {
        const float t0 = sc[0] * (float)sum[0], t1 = sc[1] * (float)sum[1];
        const float t2 = sc[2] * (float)sum[2], t3 = sc[3] * (float)sum[3];
        if (logits)
          *reinterpret_cast<float4*>(logits + (int64_t)m * V + row0) =
              make_float4(sm[j] * t0, sm[j] * t1, sm[j] * t2, sm[j] * t3);
        if (acc_out) *reinterpret_cast<int4*>(acc_out + (int64_t)m * V + row0) = make_int4(sum[0], sum[1], sum[2], sum[3]);
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          if (row0 + v < V) {
            const float tv = sc[v] * (float)sum[v];
            if (logits) logits[(int64_t)m * V + row0 + v] = sm[j] * tv;
            if (acc_out) acc_out[(int64_t)m * V + row0 + v] = sum[v];
          }
        }
      }
    }
  }
}

template <int TB>
hipError_t launch_tiled(const int8_t* q, const float* s, int64_t M, int64_t d, const int8_t* E, const float* scale,
                        int64_t V, float* logits, int32_t* acc, hipStream_t st) {
  const int64_t nrb = dfssm::ceil_div(V, kTlRows), ntb = dfssm::ceil_div(M, TB);
  const int64_t blocks = dfssm::ceil_div(nrb, 8) * 8 * ntb;
  lm_head_tiled<TB><<<dim3((unsigned)blocks), dim3(kTlThreads), 0, st>>>(q, s, (int)M, (int)d, E, scale, (int)V, logits,
                                                                         acc, (int)nrb, (int)ntb);
  return hipGetLastError();
}

// MFMA steps per wave for row length d, or 0 when the MFMA kernel does not
// take it (d % 64 != 0, or no split of d / 64 steps over 4..8 waves of at
// most 8 steps)
int mfma_steps(int64_t d) {
  if (d % 64 != 0) return 0;
  const int64_t steps = d / 64;
  for (int ks = 1; ks <= 8; ++ks)
    if (steps % ks == 0 && steps / ks <= kMfmaMaxWaves && steps / ks >= 4) return ks;
  return 0;
}

template <int KS>
hipError_t launch_mfma(const int8_t* q, const float* s, int64_t M, int64_t d, const int8_t* E, const float* scale,
                       int64_t V, float* logits, int32_t* acc, hipStream_t st) {
  const int nw = (int)(d / 64 / KS);
  lm_head_mfma<KS><<<dim3((unsigned)dfssm::ceil_div(V, kMfmaRows)), dim3(64 * nw), 0, st>>>(
      q, s, (int)M, (int)d, E, scale, (int)V, logits, acc);
  return hipGetLastError();
}

template <int NC>
hipError_t launch_nc(const int8_t* q, const float* s, int64_t M, int d, const int8_t* E, const float* scale,
                     int V, float* logits, int32_t* acc, hipStream_t st) {
  // tokens per pass: the codes of a pass stay in registers (MT x NC x 16 B)
  constexpr int MTmax = NC <= 4 ? 4 : (NC <= 8 ? 2 : 1);
  for (int64_t m0 = 0; m0 < M; m0 += MTmax) {
    const int mt = (int)std::min<int64_t>(MTmax, M - m0);
    hipError_t e;
    if (mt == 1)
      e = launch_t<1, NC>(q, s, d, E, scale, V, logits, acc, (int)m0, mt, st);
    else if (mt == 2 && MTmax >= 2)
      e = launch_t<(MTmax >= 2 ? 2 : 1), NC>(q, s, d, E, scale, V, logits, acc, (int)m0, mt, st);
    else
      e = launch_t<MTmax, NC>(q, s, d, E, scale, V, logits, acc, (int)m0, mt, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// x[m, k .. k+15] = scale[t] * E[t, k .. k+15] for one 16-byte piece per thread;
// an id outside [0, V) gives a zero row
__global__ __launch_bounds__(kThreads) void embed_gather(const int8_t* __restrict__ E, const float* __restrict__ scale,
                                                         int V, int d, const int32_t* __restrict__ tok, int64_t M,
                                                         float* __restrict__ x) {
  const int64_t per_row = d / 16;
  const int64_t total = M * per_row;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += (int64_t)gridDim.x * kThreads) {
    const int64_t m = i / per_row;
    const int k = (int)(i % per_row) * 16;
    const int t = tok[m];
    float4* dst = reinterpret_cast<float4*>(x + m * d + k);
    if (t < 0 || t >= V) {
#pragma unroll
      for (int u = 0; u < 4; ++u) dst[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      continue;
    }
    const float sc = scale[t];
    const uint4 e = *reinterpret_cast<const uint4*>(E + (int64_t)t * d + k);
    const uint32_t w[4] = {e.x, e.y, e.z, e.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float a = sc * (float)(int8_t)(w[u] & 0xff);
      const float b = sc * (float)(int8_t)((w[u] >> 8) & 0xff);
      const float c = sc * (float)(int8_t)((w[u] >> 16) & 0xff);
      const float dd = sc * (float)(int8_t)(w[u] >> 24);
      dst[u] = make_float4(a, b, c, dd);
    }
  }
}

}  // namespace

namespace dfssm {

hipError_t launch_lm_head(const int8_t* q, const float* s, int64_t M, int64_t d, const int8_t* E,
                          const float* scale, int64_t V, float* logits, int32_t* acc, hipStream_t st) {
  if (M == 0 || V == 0) return hipSuccess;
  // from 8 tokens on the matrix cores (the table read once),
  // below as GEMV passes of up to 4 tokens
  const int ks = mfma_steps(d);
  if (M >= lm_head_mfma_tokens() && ks > 0) {
    // from 64 tokens the tiled kernel (its load offsets are 32-bit)
    if (M >= lm_head_tiled_tokens() && V * d < (int64_t)1 << 31 && M * d < (int64_t)1 << 31)
      return M >= 128 ? launch_tiled<128>(q, s, M, d, E, scale, V, logits, acc, st)
                      : launch_tiled<64>(q, s, M, d, E, scale, V, logits, acc, st);
    switch (ks) {
      case 1: return launch_mfma<1>(q, s, M, d, E, scale, V, logits, acc, st);
      case 2: return launch_mfma<2>(q, s, M, d, E, scale, V, logits, acc, st);
      case 3: return launch_mfma<3>(q, s, M, d, E, scale, V, logits, acc, st);
      case 4: return launch_mfma<4>(q, s, M, d, E, scale, V, logits, acc, st);
      case 5: return launch_mfma<5>(q, s, M, d, E, scale, V, logits, acc, st);
      case 6: return launch_mfma<6>(q, s, M, d, E, scale, V, logits, acc, st);
      case 7: return launch_mfma<7>(q, s, M, d, E, scale, V, logits, acc, st);
      default: return launch_mfma<8>(q, s, M, d, E, scale, V, logits, acc, st);
    }
  }
  const int64_t nc = ceil_div(d, 1024);
  if (nc <= 1) return launch_nc<1>(q, s, M, (int)d, E, scale, (int)V, logits, acc, st);
  if (nc <= 2) return launch_nc<2>(q, s, M, (int)d, E, scale, (int)V, logits, acc, st);
  if (nc <= 4) return launch_nc<4>(q, s, M, (int)d, E, scale, (int)V, logits, acc, st);
  if (nc <= 8) return launch_nc<8>(q, s, M, (int)d, E, scale, (int)V, logits, acc, st);
  return launch_nc<16>(q, s, M, (int)d, E, scale, (int)V, logits, acc, st);
}

hipError_t launch_embed_gather(const int8_t* E, const float* scale, int64_t V, int64_t d, const int32_t* tok,
                               int64_t M, float* x, hipStream_t st) {
  if (M == 0) return hipSuccess;
  const int64_t total = M * (d / 16);
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, kThreads), 4096));
  embed_gather<<<dim3((unsigned)blocks), dim3(kThreads), 0, st>>>(E, scale, (int)V, (int)d, tok, M, x);
  return hipGetLastError();
}

}  // namespace dfssm
