// dfssm_mamba.hip -- the Mamba-2 decode step around the scaffold + LoRA
// linears, gfx950: residual add + RMSNorm + int8 quantisation (in_proj's
// input), the convolution step and the SSM step (the two stateful
// operations, Sec. 4.1 and Table 13), and gate-then-norm + quantisation
// (out_proj's input, norm(y * silu(z)) as Table 12 fixes it).
//
// Rounding follows one pinned order so that the int8 codes fed to the
// linears come out the same on every run and on the host: fp32 for every
// elementwise step; exp, log1p, sqrt and the divisions inside silu,
// softplus and the norm's scale in fp64, rounded once to fp32; the norm's
// sum of squares and the SSM output's sum over the state in fp64 over exact
// products.  The library is compiled with contraction off.
//
// The convolution state is a ring of 4 slots per sequence, [M][4][conv_dim]:
// step t reads the inputs of steps t-3, t-2, t-1 from slots (t-3)&3 ..
// (t-1)&3 and writes its own input into slot t&3, the one no reader of step
// t touches.  That is the shift register of the model without moving data,
// and it lets every workgroup read the shared B/C channels while one of them
// appends to them, with no ordering between workgroups.
#include <float.h>

#include <algorithm>

#include "dfssm_mamba.hpp"

namespace {

// ---------------------------------------------------------------- helpers
__device__ __forceinline__ float silu_f(float v) {
  const double x = (double)v;
  return (float)(x / (1.0 + exp(-x)));
}

__device__ __forceinline__ float softplus_f(float v) {
  if (v > 20.0f) return v;
  return (float)log1p(exp((double)v));
}

__device__ __forceinline__ int8_t code(float v, float inv) {
  float r = rintf(v * inv);  // v_rndne_f32: round to nearest, ties to even
  r = fminf(fmaxf(r, -127.0f), 127.0f);
  return (int8_t)(int)r;
}

template <int W>
__device__ __forceinline__ double sum_lanes(double v) {
#pragma unroll
  for (int off = W / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, W);
  return v;
}

__device__ __forceinline__ float max_lanes(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// ---------------------------------------------------------------- norms
constexpr int kNormMaxThreads = 1024;

struct NormArgs {
  const float* a;     // u (residual) or y (SSM output), rows of d
  const float* b;     // delta (rows of d, may be null) or z (rows of ldb)
  int64_t ldb;
  const float* w;     // [d]
  float eps;
  int d;
  float* u_out;       // residual sum, or null (plain norm only)
  int8_t* q;          // [M][d]
  float* s;           // [M]
};

// One workgroup per token row, sized to the row (a multiple of 64 threads,
// at most 512 up to d = 8192, else 1024); VPT float4 per thread held in registers.  The inputs and
// the weight are loaded together, before the reductions, so the row costs
// one memory round trip.  GATE: g = y * silu(z); else g = u + delta.
template <bool GATE, int VPT>
__global__ __launch_bounds__(kNormMaxThreads) void norm_quant(NormArgs a) {
  const int64_t m = blockIdx.x;
  const int tid = threadIdx.x, nt = blockDim.x, nw = nt >> 6;
  const int d = a.d;
  const float* ar = a.a + m * d;
  const float* br = a.b ? a.b + m * a.ldb : nullptr;
  __shared__ double red_ss[kNormMaxThreads / 64];
  __shared__ float red_max[kNormMaxThreads / 64];

  float4 g[VPT], w[VPT], z[VPT];
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int k = 4 * (tid + nt * i);
    const bool in = k < d;
    g[i] = in ? *reinterpret_cast<const float4*>(ar + k) : make_float4(0.f, 0.f, 0.f, 0.f);
    z[i] = (in && br) ? *reinterpret_cast<const float4*>(br + k) : make_float4(0.f, 0.f, 0.f, 0.f);
    w[i] = in ? *reinterpret_cast<const float4*>(a.w + k) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    if (GATE) {
      g[i].x = g[i].x * silu_f(z[i].x);
      g[i].y = g[i].y * silu_f(z[i].y);
      g[i].z = g[i].z * silu_f(z[i].z);
      g[i].w = g[i].w * silu_f(z[i].w);
    } else if (br) {
      g[i].x = g[i].x + z[i].x;
      g[i].y = g[i].y + z[i].y;
      g[i].z = g[i].z + z[i].z;
      g[i].w = g[i].w + z[i].w;
    }
    const int k = 4 * (tid + nt * i);
    if (!GATE && a.u_out && k < d) *reinterpret_cast<float4*>(a.u_out + m * d + k) = g[i];
  }
  // sum of squares in fp64 (each fp32 square is exact there)
  double ss = 0.0;
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    ss += (double)g[i].x * (double)g[i].x;
    ss += (double)g[i].y * (double)g[i].y;
    ss += (double)g[i].z * (double)g[i].z;
    ss += (double)g[i].w * (double)g[i].w;
  }
  ss = sum_lanes<64>(ss);
  if ((tid & 63) == 0) red_ss[tid >> 6] = ss;
  __syncthreads();
  ss = 0.0;
  for (int i = 0; i < nw; ++i) ss += red_ss[i];
  const float r = (float)(1.0 / sqrt(ss / (double)d + (double)a.eps));

  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    g[i].x = (g[i].x * r) * w[i].x;
    g[i].y = (g[i].y * r) * w[i].y;
    g[i].z = (g[i].z * r) * w[i].z;
    g[i].w = (g[i].w * r) * w[i].w;
    amax = fmaxf(amax, fmaxf(fmaxf(fabsf(g[i].x), fabsf(g[i].y)), fmaxf(fabsf(g[i].z), fabsf(g[i].w))));
  }
  amax = max_lanes(amax);
  if ((tid & 63) == 0) red_max[tid >> 6] = amax;
  __syncthreads();
  amax = 0.0f;
  for (int i = 0; i < nw; ++i) amax = fmaxf(amax, red_max[i]);

  int8_t* qr = a.q + m * d;
  if (amax < FLT_MIN) {  // all-zero (or subnormal-only) row
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int k = 4 * (tid + nt * i);
      if (k < d) *reinterpret_cast<uint32_t*>(qr + k) = 0u;
    }
    if (tid == 0) a.s[m] = 0.0f;
    return;
  }
  const float inv = 127.0f / amax;
  if (tid == 0) a.s[m] = amax / 127.0f;
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int k = 4 * (tid + nt * i);
    if (k < d) {
      const uint32_t c = (uint32_t)(uint8_t)code(g[i].x, inv) | (uint32_t)(uint8_t)code(g[i].y, inv) << 8 |
                         (uint32_t)(uint8_t)code(g[i].z, inv) << 16 | (uint32_t)(uint8_t)code(g[i].w, inv) << 24;
      *reinterpret_cast<uint32_t*>(qr + k) = c;
    }
  }
}

template <bool GATE>
hipError_t launch_norm(const NormArgs& a, int64_t M, hipStream_t st) {
  const int64_t vec = dfssm::ceil_div(a.d, 4);   // float4 per row
  // at most 512 threads while 4 float4 per thread cover the row (d <= 8192):
  // the cross-wave reductions then have 8 partials, not 16 (the 1.3B decode
  // step at batch 1: 1.138 against 1.158 ms; 256 or 128 threads: 1.167)
  const int maxt = dfssm::ceil_div(vec, 512) <= 4 ? 512 : kNormMaxThreads;
  const int vpt = (int)dfssm::ceil_div(vec, maxt);
  const int nt = (int)std::min<int64_t>(maxt, dfssm::round_up(dfssm::ceil_div(vec, vpt), 64));
  dim3 grid((unsigned)M), block(nt);
  if (vpt <= 1)
    norm_quant<GATE, 1><<<grid, block, 0, st>>>(a);
  else if (vpt <= 2)
    norm_quant<GATE, 2><<<grid, block, 0, st>>>(a);
  else
    norm_quant<GATE, 4><<<grid, block, 0, st>>>(a);
  return hipGetLastError();
}

// ---------------------------------------------------------------- SSM step
constexpr int kHeadDim = 64;      // P
constexpr int kSsmThreads = 256;

struct SsmArgs {
  const float* zx;    // [M][ld]: z | xBC | dt
  int64_t ld;
  int d_inner, H;
  int64_t step;
  float* ring;        // [M][4][conv_dim]
  const float* conv_w;  // [conv_dim][4]
  const float* conv_b;
  const float* dt_bias;
  const float* A_log;
  const float* D;
  float* state;       // [M][H][P][N]
  float* y;           // [M][d_inner]
  float* xbc;         // [M][conv_dim] or null
  int gate_y;         // y * silu(z) instead of y
};

typedef float f32x4 __attribute__((ext_vector_type(4)));

// The state is read once and written once per step, 4 MB per sequence:
// non-temporal accesses keep it from displacing the step's shared inputs
// in the caches (batch 512: 406 us against 434 with plain accesses).
__device__ __forceinline__ f32x4 load_state(const f32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void store_state(f32x4 v, f32x4* p) { __builtin_nontemporal_store(v, p); }

// Workgroup (m, h, pb): PB channels p = PB pb .. PB pb + PB - 1 of head h,
// whose states are one contiguous PB x N block.  Pass j of thread t holds
// float4 j NT + t of that block: channel (j NT + t) / L and state columns
// 4 (t % L) .. + 3, with L = N / 4 lanes per channel, so every load and
// store of a wave covers 1 KB in one piece; the L lanes of a channel sum
// y[p] over the state.
template <int N, int PB, int NT = kSsmThreads>
__global__ __launch_bounds__(NT) void ssm_step(SsmArgs a) {
  constexpr int L = N / 4;               // lanes per channel
  constexpr int J = PB * L / NT;         // passes
  constexpr int CPJ = NT / L;            // channels per pass
  static_assert(J * NT == PB * L && CPJ * L == NT, "state block tiling");
  constexpr int NBH = kHeadDim / PB;     // workgroups per head
  const int nblk = a.H * NBH;
  const int64_t m = blockIdx.x / nblk;
  const int hb = blockIdx.x % nblk;
  const int h = hb / NBH;
  const int p0 = (hb % NBH) * PB;
  const int tid = threadIdx.x;
  const int pj = tid / L, nc = tid % L;
  const int conv_dim = a.d_inner + 2 * N;
  const float* zr = a.zx + m * a.ld;

  // the state first: it is the bytes that come from HBM
  f32x4* hs = reinterpret_cast<f32x4*>(a.state + ((m * a.H + h) * kHeadDim + p0) * (int64_t)N) + tid;
  f32x4 hv[J];
#pragma unroll
  for (int j = 0; j < J; ++j) hv[j] = load_state(hs + j * NT);

  // convolution step for this workgroup's PB x channels and all B, C channels
  __shared__ float xbc_s[PB + 2 * N];
  __shared__ float gz_s[PB];  // silu(z) of the channels, when gating
  __shared__ float dt_s[2];
  const bool owns_bc = (hb == 0);
  float* ring = a.ring + m * 4 * (int64_t)conv_dim;
  const int s0 = (int)((a.step + 1) & 3), s1 = (int)((a.step + 2) & 3), s2 = (int)((a.step + 3) & 3);
  const int sw = (int)(a.step & 3);
  for (int i = tid; i < PB + 2 * N; i += NT) {
    const int c = i < PB ? h * kHeadDim + p0 + i : a.d_inner + (i - PB);
    const float in = zr[a.d_inner + c];
    const float4 w = *reinterpret_cast<const float4*>(a.conv_w + 4 * (int64_t)c);
    float v = w.x * ring[s0 * (int64_t)conv_dim + c];
    v = v + w.y * ring[s1 * (int64_t)conv_dim + c];
    v = v + w.z * ring[s2 * (int64_t)conv_dim + c];
    v = v + w.w * in;
    v = v + a.conv_b[c];
    const float o = silu_f(v);
    xbc_s[i] = o;
    if (i < PB && a.gate_y) gz_s[i] = silu_f(zr[c]);
    if (i < PB || owns_bc) {
      ring[sw * (int64_t)conv_dim + c] = in;
      if (a.xbc) a.xbc[m * conv_dim + c] = o;
    }
  }
  // dt and dA once per workgroup, by the last wave (the one with the least
  // convolution work), through LDS
  if (tid >= NT - 64) {
    const float dt = softplus_f(zr[a.d_inner + conv_dim + h] + a.dt_bias[h]);
    const float A = (float)(-exp((double)a.A_log[h]));
    if (tid == NT - 64) {
      dt_s[0] = dt;
      dt_s[1] = (float)exp((double)(dt * A));
    }
  }
  __syncthreads();
  const float dt = dt_s[0], dA = dt_s[1];

  const float* Bs = xbc_s + PB + 4 * nc;
  const float* Cs = xbc_s + PB + N + 4 * nc;
  const float b[4] = {Bs[0], Bs[1], Bs[2], Bs[3]};
  const float cc[4] = {Cs[0], Cs[1], Cs[2], Cs[3]};
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int p = j * CPJ + pj;
    const float x = xbc_s[p];
    const float dtx = dt * x;
    float e[4] = {hv[j].x, hv[j].y, hv[j].z, hv[j].w};
    double acc = 0.0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float t1 = e[u] * dA;
      const float t2 = dtx * b[u];
      e[u] = t1 + t2;
      acc += (double)e[u] * (double)cc[u];
    }
    f32x4 o;
    o.x = e[0];
    o.y = e[1];
    o.z = e[2];
    o.w = e[3];
    store_state(o, hs + j * NT);
    acc = sum_lanes<L>(acc);
    if (nc == 0) {
      const int c = h * kHeadDim + p0 + p;
      float yv = (float)(acc + (double)a.D[h] * (double)x);
      if (a.gate_y) yv = yv * gz_s[p];
      a.y[m * a.d_inner + c] = yv;
    }
  }
}

template <int N>
void launch_ssm_n(const SsmArgs& a, int64_t M, hipStream_t st) {
  // More channels per workgroup amortise the B/C convolution every
  // workgroup repeats over more state, and leave fewer workgroups: 64
  // channels (32 KB of state) from 16 sequences, 32 from 5.  Per step of
  // 48 layers' states in a graph (us per call), 32 / 64 channels: batch
  // 8: 8.6 / 9.3; 12: 10.8 / 11.2; 16: 16.6 / 13.1; 32: 28.0 / 28.4; 256:
  // 187 / 182; 512: 375 / 363.  Up to 4 sequences the step is latency and
  // the 16-channel blocks' shorter per-thread chain wins (batch 1: 4.05 us
  // against 4.75).
  if (M <= 4)
    ssm_step<N, 16><<<dim3((unsigned)(M * a.H * (kHeadDim / 16))), dim3(kSsmThreads), 0, st>>>(a);
  else if (M < 16)
    ssm_step<N, 32><<<dim3((unsigned)(M * a.H * (kHeadDim / 32))), dim3(kSsmThreads), 0, st>>>(a);
  else
    ssm_step<N, 64><<<dim3((unsigned)(M * a.H * (kHeadDim / 64))), dim3(kSsmThreads), 0, st>>>(a);
}

}  // namespace

namespace dfssm {

hipError_t launch_add_rmsnorm_quant(const float* u, const float* delta, const float* w, float eps, int64_t M,
                                    int64_t d, float* u_out, int8_t* q, float* s, hipStream_t st) {
  if (M == 0) return hipSuccess;
  NormArgs a{u, delta, d, w, eps, (int)d, u_out, q, s};
  return launch_norm<false>(a, M, st);
}

hipError_t launch_gate_norm_quant(const float* y, const float* z, int64_t ldz, const float* w, float eps,
                                  int64_t M, int64_t d, int8_t* q, float* s, hipStream_t st) {
  if (M == 0) return hipSuccess;
  NormArgs a{y, z, ldz, w, eps, (int)d, nullptr, q, s};
  return launch_norm<true>(a, M, st);
}

hipError_t launch_ssm_step(const float* zx, int64_t ld, int64_t M, int64_t d_inner, int64_t d_state, int64_t step,
                           float* ring, const float* conv_w, const float* conv_b, const float* dt_bias,
                           const float* A_log, const float* D, float* state, float* y, float* xbc,
                           hipStream_t st, bool gate_y) {
  if (M == 0) return hipSuccess;
  const int H = (int)(d_inner / kHeadDim);
  SsmArgs a{zx, ld, (int)d_inner, H, step, ring, conv_w, conv_b, dt_bias, A_log, D, state, y, xbc, gate_y ? 1 : 0};
  if (d_state == 128)
    launch_ssm_n<128>(a, M, st);
  else
    launch_ssm_n<64>(a, M, st);
  return hipGetLastError();
}

}  // namespace dfssm
