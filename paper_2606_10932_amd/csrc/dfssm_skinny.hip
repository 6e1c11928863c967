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
//    fp32 epilogue; its operands were loaded at the start.
// The LoRA down-projection, its limbs and sum_k Q come from small_prep.
#include <algorithm>

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

constexpr int kMaxWaves = 8;

struct SkinnyArgs {
  const int8_t* q;
  const float* s;
  int M, K, N, r, rp;
  const uint32_t* w_bits;
  const float* alpha;
  const int8_t* limbs;  // [4][M][rp]
  const int8_t* B;
  const float* beta;
  const int32_t* sumq;
  float* y;
  int32_t* acc_s_out;
  int64_t* acc_b_out;
};

// MT token tiles of 16 (M <= 16*MT); S MFMA steps per lane per iteration.
// Block: 16 output rows, nw = blockDim.x / 64 waves (nw >= MT), wave w takes
// iterations w, w + nw, ... of 64*S columns each.
template <int MT, int S>
__global__ __launch_bounds__(64 * kMaxWaves) void mfma_skinny(SkinnyArgs a) {
  __shared__ v4i red[kMaxWaves][MT][64];
  constexpr int KW = 64 * S;  // columns per wave iteration
  constexpr int SW = S / 2;   // sign words per lane per iteration
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nw = blockDim.x >> 6;
  const int rho = lane & 15, kg = lane >> 4;
  const int M = a.M, K = a.K, N = a.N, r = a.r, W = K >> 5;
  const int n0 = 16 * blockIdx.x;
  const int nrow = min(n0 + rho, N - 1);  // sign / B row of this lane (rows past N are never stored)
  const uint32_t* wrow = a.w_bits + (int64_t)nrow * W;
  const int nit = (K + KW - 1) / KW;
  const bool wvec = (W % SW) == 0;

  // ---- the epilogue operands of the wave that finishes token tile `wave`
  //      go out first: B bytes and limbs of ranks 0..63, row scales, token
  //      scales and sums of Q
  const bool fin = wave < MT;
  const int mtok = 16 * wave + rho;  // token of this lane in the finished tile
  const int mc = min(mtok, M - 1);
  const int nb = n0 + 4 * kg;  // this lane's output rows nb .. nb+3
  const bool ba = (r % 16) == 0;
  v4i bop = zero4(), lm[4] = {zero4(), zero4(), zero4(), zero4()};
  float alv[4] = {0.f, 0.f, 0.f, 0.f}, bev[4] = {0.f, 0.f, 0.f, 0.f};
  float sm = 0.f;
  int sq = 0;
  if (fin) {
    if (r > 0) {
      bop = load16_guarded(a.B + (int64_t)nrow * r, 16 * kg, r, ba);
#pragma unroll
      for (int t = 0; t < 4; ++t) lm[t] = load16(a.limbs + ((int64_t)t * M + mc) * a.rp + 16 * kg);
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
    sq = a.sumq[mc];
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
      const int m = 16 * i + rho;
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
  __syncthreads();
  if (!fin) return;
  v4i d = red[0][wave][lane];
  for (int w = 1; w < nw; ++w) d += red[w][wave][lane];

  // LoRA up-projection, limbs 3, 2, 1, 0 over the 64-rank chunks
  v4i ehi = zero4(), elo = zero4();
  if (r > 0) {
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {
      const int limb = 3 - pass;
      v4i e = limb >= 2 ? ehi : elo;
      e = mfma(bop, lm[limb], e);
      for (int j0 = 64; j0 < a.rp; j0 += 64) {
        const v4i bl = load16_guarded(a.B + (int64_t)nrow * r, j0 + 16 * kg, r, ba);
        const v4i al = load16(a.limbs + ((int64_t)limb * M + mc) * a.rp + j0 + 16 * kg);
        e = mfma(bl, al, e);
      }
      if (limb == 3 || limb == 1) e = e << 8;
      if (limb >= 2)
        ehi = e;
      else
        elo = e;
    }
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

template <int MT, int S>
hipError_t launch_t(const SkinnyArgs& a, int nw, hipStream_t st) {
  const int64_t blocks = dfssm::ceil_div(a.N, 16);
  mfma_skinny<MT, S><<<dim3((unsigned)blocks), dim3(64 * nw), 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace

namespace dfssm {

hipError_t launch_skinny_linear(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                                int64_t r, const uint32_t* w_bits, const float* alpha,
                                const int8_t* A, const int8_t* B, const float* beta, float* y,
                                int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                                const LinearWorkspace& ws, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  if (M > kSkinnyMaxTokens) return hipErrorInvalidValue;
  hipError_t e = launch_small_prep(q, M, K, r, A, ws, false, st);
  if (e != hipSuccess) return e;
  if (acc_a_out && r > 0) {
    e = hipMemcpyAsync(acc_a_out, ws.acc_a, (size_t)(M * r) * 4, hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
  }
  SkinnyArgs a{q, s, (int)M, (int)K, (int)N, (int)r, (int)rank_padded(r), w_bits, alpha, ws.limbs, B, beta,
               ws.sumq, y, acc_s, acc_b};
  // 16-byte sign loads (8 MFMA steps) once K gives every wave a full one
  const int S = K >= 4096 ? 8 : 4;
  const int mt = M > 16 ? 2 : 1;
  const int64_t nit = ceil_div(K, 64 * S);
  const int nw = (int)std::max<int64_t>(mt, std::min<int64_t>(kMaxWaves, nit));
  if (mt == 1) return S == 8 ? launch_t<1, 8>(a, nw, st) : launch_t<1, 4>(a, nw, st);
  return S == 8 ? launch_t<2, 8>(a, nw, st) : launch_t<2, 4>(a, nw, st);
}

}  // namespace dfssm
