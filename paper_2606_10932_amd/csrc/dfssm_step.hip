// dfssm_step.hip -- the decode step of a Mamba-2 model at one token as one
// persistent kernel: every layer's residual add and RMSNorm, in_proj, the
// convolution and SSM step with the gate, the gated RMSNorm and out_proj
// (the paper removes the launch gaps of the batch-1 decode step by capturing
// the forward pass as one CUDA graph, Sec. 4.1; here the layers run inside
// one launch and hand their data over as tagged words).  The token's
// embedding gather, the final norm and the LM head are launched around it.
//
// It carries the re-quantising chain's design (dfssm_chain.hip) from a
// chain of linears to whole layers, for the 1.3B layer shape (d_model 2048,
// d_inner 4096, d_state 128, 64 heads of 64 channels, int8 LoRA, r <= 64):
//  * the same placement (XCD x from XCC_ID, lam = w / 8, column slice
//    kap = lam % 8, row group h = lam / 8), the same slice-split popcount
//    GEMV with XCD-local row and rank partials, the same loading wave and
//    3-slot LDS ring;
//  * a linear's input is normalised before it is quantised.  Its producers
//    publish their values and a partial sum of squares (fp64 as two words);
//    every workgroup sums the 256 partials in one fixed order, so all find
//    the same scale r, forms its slice of (v * r) * w, and the 8 slice maxima
//    of each row group meet in XCD-local words (each row group holds all 8
//    slices, so every workgroup finds the same absmax and token scale);
//  * in_proj's rows are owned so that workgroup g (= 32 x + lam) holds z and
//    x of the 16 channels 16g .. 16g+15 (a quarter of head g / 4), B/C row
//    g and, for g < 64, the dt row of head g.  The convolution, the SSM step
//    of its 16 channels and the gate then run in the workgroup that produced
//    them, after gathering only the 256 B/C values and its head's dt; their
//    state, convolution window and parameters arrive with in_proj's operands
//    through the LDS ring;
//  * out_proj's reducers own 8 rows of the residual stream each and keep
//    them in registers across the layers; they publish the updated rows and
//    their sum of squares for the next layer's norm.
// Every wait is bounded; a workgroup whose wait gives up records a status
// bit and leaves after the next barrier, so the grid always drains.
#include <float.h>
#include <math.h>

#include <algorithm>
#include <cstring>
#include <vector>

#include "dfssm_internal.hpp"
#include "dfssm_persist.hpp"

namespace {

using namespace dfssm_px;

// the layer shape this kernel takes
constexpr int kD = 2048;                       // d_model
constexpr int kDi = 2 * kD;                    // d_inner
constexpr int kDs = 128;                       // d_state
constexpr int kNh = kDi / 64;                  // heads
constexpr int kConv = kDi + 2 * kDs;           // convolution channels (x, B, C)
constexpr int kNin = kDi + kConv + kNh;        // in_proj rows [z | x | B | C | dt]
constexpr int kCpw = kDi / kGrid;              // channels per workgroup: 16
constexpr int kInSlots = 2 * kCpw + 2;         // in_proj row slots per reducer
constexpr int kOutRows = kD / kGrid;           // out_proj rows per reducer: 8
static_assert(kCpw == 16 && kOutRows == 8 && 2 * kDs == kGrid && kNh <= kGrid, "the 1.3B layer shape");
static_assert(64 % kCpw == 0, "a workgroup's channels lie in one head");

constexpr int kWaves = 8;  // 0 reducer, 1 scale/codes/LoRA down, 6 loads; SSM on 1..4
constexpr int kThreads = 64 * kWaves;
constexpr int kAWaves = kWaves - 1;  // phase A: every wave but 1
constexpr int kRowLanes = 64 * kAWaves;
constexpr int kMaxR = 64;
constexpr int kRankGroups = 4;
constexpr int kMaxRh = kMaxR / kRankGroups;
constexpr int kPollLanes = 6 * 64;  // waves 1..5 and 7
constexpr int kBcLane = 48;         // reducer lanes 48 .. 55: the B/C copies
constexpr int kSlotBytes = 40 * 1024;
constexpr int kRing = 3;
constexpr int kMaxKs = kDi / kSlices;  // 512
constexpr int kSetupChunk = 16;
constexpr int kGroups = kPerXcd / kSlices;  // 4 row groups per XCD

// status bits
constexpr unsigned kStIn = 1u, kStAcc = 2u, kStSsm = 4u, kStHash = 8u;

// One linear of the step as the kernel reads it (host-built table).
struct StepLin {
  const uint32_t* w_bits;
  const float* alpha;
  const int8_t* A;  // never NULL (alpha when r == 0)
  const int8_t* B;
  const float* beta;
  const float* nw;  // weight of the norm in front of this linear
  // in_proj: the layer's convolution and SSM parameters
  const float* conv_w;
  const float* conv_b;
  const float* dt_bias;
  const float* A_log;
  const float* Dp;
  int32_t K, N, r, rh;
  int32_t kind;    // 0 in_proj, 1 out_proj
  int32_t rs;      // row slots per reducer
  int32_t us, ub;  // direct-to-LDS units (bytes) of the sign rows and B rows
  int32_t o_a, o_b, o_al, o_be, o_nw;    // slot offsets
  int32_t o_st, o_rg, o_rb, o_cw, o_cb, o_hp;  // in_proj: SSM state, convolution windows (x channels, own
                                              // B/C channel), conv_w, conv_b, head parameters
  int32_t layer;
  int32_t i4;        // 1: A and B are packed int4 (A [r][K/2], B [N][r/2] bytes)
  int64_t part_off;  // XCD-local words [8 slices][N]: row partials
  int64_t p_off;     // XCD-local words [8 XCDs][8 slices][64]: rank partials
  int64_t mx_off;    // XCD-local words [8 XCDs][4 row groups][8 slices]: slice maxima
  int64_t in_off;    // agent words [K]: this linear's input values
  int64_t st_off;    // agent words [8 XCDs][4 row groups][8 slices][8]: each slice's sum of squares and largest entries
  int64_t bc_off;    // in_proj: agent words [8 XCDs][2 d_state]: the B/C rows after the convolution
  int64_t dt_off;    // in_proj: agent words [heads][2]: dt and dA of each head
};

// ---------------------------------------------------------------- helpers
__device__ __forceinline__ float silu_f(float v) {
  const double x = (double)v;
  return (float)(x / (1.0 + exp(-x)));
}
__device__ __forceinline__ float softplus_f(float v) {
  if (v > 20.0f) return v;
  return (float)log1p(exp((double)v));
}
// DPP move of an fp64 value (both halves with the same control); rows the
// mask leaves out read 0.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, kCtrl, kRowMask, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), kCtrl, kRowMask, 0xF, false);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ double readlane_f64(double v, int lane) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), lane);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// Whole-wave fp64 sum, in the same fixed order in every wave: pairs, quads,
// rows, then the row broadcasts that leave the total in lane 63.
__device__ __forceinline__ double wave_sum_f64_u(double v) {
  v = v + dpp_f64<0xB1, 0xF>(v);
  v = v + dpp_f64<0x4E, 0xF>(v);
  v = v + dpp_f64<0x141, 0xF>(v);
  v = v + dpp_f64<0x140, 0xF>(v);
  v = v + dpp_f64<0x142, 0xA>(v);
  v = v + dpp_f64<0x143, 0xC>(v);
  return readlane_f64(v, 63);
}

// Row k of reducer g (-1: none).  in_proj: z and x of channels 16g..16g+15,
// B/C row g, the dt row of head g for g < heads.  out_proj: rows 8g..8g+7.
__device__ __forceinline__ int reducer_row(int kind, int g, int k) {
  if (kind == 1) return k < kOutRows ? kOutRows * g + k : -1;
  if (k < kCpw) return kCpw * g + k;
  if (k < 2 * kCpw) return kDi + kCpw * g + (k - kCpw);
  if (k == 2 * kCpw) return 2 * kDi + g;
  if (k == 2 * kCpw + 1 && g < kNh) return 2 * kDi + 2 * kDs + g;
  return -1;
}
__device__ __forceinline__ int reducer_rows(int kind, int g) {
  return kind == 1 ? kOutRows : 2 * kCpw + 1 + (g < kNh ? 1 : 0);
}
// Row of slot i of row group (x, h): slot i belongs to reducer 32x + 8h +
// i / rs (mrs = recip20(rs)).
__device__ __forceinline__ int group_row(int kind, int rs, uint32_t mrs, int x, int h, int i) {
  const int rho = udiv(i, mrs);
  return reducer_row(kind, kPerXcd * x + kSlices * h + rho, i - rho * rs);
}

// The loading wave's batch for linear L of layer l: this workgroup's sign
// rows (all slots of its row group), its rh A rows' slice, its reducer rows'
// B rows and scales, the norm weight's slice, and for in_proj the SSM
// operands of its 16 channels: their state, the three previous inputs of the
// convolution window of its channels and of the B/C channels, the
// convolution weights and biases of both, its head's dt bias, A_log and D.
// Every address is in range: lanes past the data read the array's first unit.
__device__ void step_batch(const StepLin& L, int x, int kap, int h, int lam, int t, const float* ring_l,
                           const float* state_l, uint32_t sb, int lane) {
  const int K = L.K, Ks = K >> 3, rowbytes = K >> 6, g = kPerXcd * x + lam;
  const uint32_t mrs = recip20((uint32_t)L.rs);
  {  // sign rows of the row group's slots, this slice
    const int us = L.us, upr = rowbytes / us, nunits = kSlices * L.rs * upr, ni = (nunits + 63) >> 6;
    const uint32_t m = recip20((uint32_t)upr);
    for (int tt = 0; tt < ni; ++tt) {
      const int u = 64 * tt + lane;
      uint32_t voff = 0;
      if (u < nunits) {
        const int i = udiv(u, m), q = u - i * upr;
        const int row = group_row(L.kind, L.rs, mrs, x, h, i);
        if (row >= 0) voff = (uint32_t)((int64_t)row * (K >> 3) + kap * rowbytes + q * us);
      }
      lds_dma(us, voff, L.w_bits, sb + (uint32_t)(64 * us * tt));
    }
  }
  if (L.rh > 0) {  // A rows h*rh .. h*rh + rh - 1, the slice's columns (int4: Ks/2 bytes)
    const int sb_a = L.i4 ? Ks >> 1 : Ks, rowb = L.i4 ? K >> 1 : K;
    const int upr = sb_a >> 4, nunits = L.rh * upr, ni = (nunits + 63) >> 6;
    const uint32_t m = recip20((uint32_t)upr);
    for (int tt = 0; tt < ni; ++tt) {
      const int u = 64 * tt + lane;
      uint32_t voff = 0;
      if (u < nunits) {
        const int jj = udiv(u, m), q = u - jj * upr, j = h * L.rh + jj;
        if (j < L.r) voff = (uint32_t)((int64_t)j * rowb + kap * sb_a + 16 * q);
      }
      lds_dma16(voff, L.A, sb + (uint32_t)(L.o_a + 1024 * tt));
    }
  }
  const int R = reducer_rows(L.kind, g);
  if (L.r > 0) {  // B rows of the reducer's rows (int4: r/2 bytes each)
    const int rb = L.i4 ? L.r >> 1 : L.r;
    const int ub = L.ub, upr = rb / ub, nunits = R * upr, ni = (nunits + 63) >> 6;
    const uint32_t m = recip20((uint32_t)upr);
    for (int tt = 0; tt < ni; ++tt) {
      const int u = 64 * tt + lane;
      uint32_t voff = 0;
      if (u < nunits) {
        const int i = udiv(u, m), q = u - i * upr;
        voff = (uint32_t)((int64_t)reducer_row(L.kind, g, i) * rb + q * ub);
      }
      lds_dma(ub, voff, L.B, sb + (uint32_t)(L.o_b + 64 * ub * tt));
    }
  }
  {  // alpha and beta of the reducer's rows
    const uint32_t voff = lane < R ? (uint32_t)reducer_row(L.kind, g, lane) * 4u : 0u;
    lds_dma4(voff, L.alpha, sb + (uint32_t)L.o_al);
    lds_dma4(voff, L.beta, sb + (uint32_t)L.o_be);
  }
  {  // the norm weight's slice (16-byte units)
    const int nunits = Ks >> 2, ni = (nunits + 63) >> 6;
    for (int tt = 0; tt < ni; ++tt) {
      const int u = 64 * tt + lane;
      const uint32_t voff = u < nunits ? (uint32_t)(kap * Ks * 4 + 16 * u) : 0u;
      lds_dma16(voff, L.nw, sb + (uint32_t)(L.o_nw + 1024 * tt));
    }
  }
  if (L.kind == 0) {
    // SSM state of channels 16g..16g+15: [16][d_state] fp32, 8 KB contiguous
    for (int tt = 0; tt < kCpw * kDs * 4 / 1024; ++tt)
      lds_dma16((uint32_t)(g * kCpw * kDs * 4 + 1024 * tt + 16 * lane), state_l,
                sb + (uint32_t)(L.o_st + 1024 * tt));
    // convolution window: for k = 1..3 the ring slot of step t - k: the 16 x
    // channels ([3][16] floats), and the own B/C channel (lane k - 1)
    {
      uint32_t voff = 0;
      if (lane < 12) voff = (uint32_t)(((((t - 1 - (lane >> 2)) & 3) * kConv) + kCpw * g + 4 * (lane & 3)) * 4);
      lds_dma16(voff, ring_l, sb + (uint32_t)L.o_rg);
      const int kk = lane < 3 ? lane : 0;
      lds_dma4((uint32_t)((((t - 1 - kk) & 3) * kConv + kDi + g) * 4), ring_l, sb + (uint32_t)L.o_rb);
    }
    {  // convolution weights [channel][4]: the x channels, then the own B/C channel
      uint32_t voff = 0;
      if (lane < kCpw) voff = (uint32_t)((kCpw * g + lane) * 16);
      if (lane == kCpw) voff = (uint32_t)((kDi + g) * 16);
      lds_dma16(voff, L.conv_w, sb + (uint32_t)L.o_cw);
    }
    {  // convolution biases: the x channels, then the own B/C channel
      uint32_t voff = 0;
      if (lane < kCpw) voff = (uint32_t)((kCpw * g + lane) * 4);
      if (lane == kCpw) voff = (uint32_t)((kDi + g) * 4);
      lds_dma4(voff, L.conv_b, sb + (uint32_t)L.o_cb);
    }
    {  // D of this workgroup's head (its channels lie in head 16g / 64); dt
       // bias and A_log of head g (the dt row this workgroup produces, g < heads)
      const int hd = g < kNh ? g : kNh - 1;
      lds_dma4((uint32_t)((kCpw * g / 64) * 4), L.Dp, sb + (uint32_t)L.o_hp);
      lds_dma4((uint32_t)(hd * 4), L.dt_bias, sb + (uint32_t)(L.o_hp + 256));
      lds_dma4((uint32_t)(hd * 4), L.A_log, sb + (uint32_t)(L.o_hp + 512));
    }
  }
}

// Records 1 + j in bits 16..31 of the status word if no linear is recorded
// there yet (the first linear whose waits gave up).
__device__ __forceinline__ void note_abort_linear(unsigned* status, int j) {
  unsigned old = __hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  while ((old >> 16) == 0) {
    const unsigned want = old | ((unsigned)(j + 1) << 16);
    if (__hip_atomic_compare_exchange_strong(status, &old, want, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      break;
  }
}

// Bounded wait on an LDS flag.
#define STEP_WAIT_FLAG(cond, sp, bit)                          \
  do {                                                         \
    while (!(cond))                                            \
      if (spin_gives_up(sp, &abort_, status, bit)) break;      \
  } while (0)

__global__ __launch_bounds__(kThreads, 1) void step_persistent(
    const StepLin* __restrict__ lins, int L2, int t, const float* __restrict__ u0, float* __restrict__ u_fin,
    float* __restrict__ conv_ring, float* __restrict__ ssm_state, uint64_t* __restrict__ ex, int64_t ex_words,
    unsigned* status, uint64_t* epoch, const uint64_t* __restrict__ table_hash, uint64_t expect_hash, float eps,
    int two_hop) {
  if (*table_hash != expect_hash) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(status, kStHash);
    return;
  }
  __shared__ __attribute__((aligned(16))) uint8_t ring[kRing][kSlotBytes];
  __shared__ __attribute__((aligned(16))) float ys[kMaxKs];       // this slice of the input
  __shared__ __attribute__((aligned(16))) int8_t codes[kMaxKs];   // its codes
  __shared__ __attribute__((aligned(16))) uint32_t planes[8][kMaxKs / 32];
  __shared__ __attribute__((aligned(16))) uint4 limbs[kMaxR / 4];
  __shared__ int red[64 * 17];
  __shared__ float zx_s[2 * kCpw];  // in_proj outputs z, x of this workgroup's channels
  __shared__ float bcc[2 * kDs];    // convolved B and C
  __shared__ float xc[kCpw], szv[kCpw];  // convolved x, silu(z)
  __shared__ float dts[3];          // dt, dA, D of the head
  __shared__ float qs_s;            // the token scale of the current linear's input
  __shared__ int sumq[2];
  __shared__ uint32_t seq_s;
  __shared__ int abort_, rows_done, limbs_ready, pub_done, ssm_cnt, g_cnt;

  const int wg = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int x = xcc_id();
  const int lam = wg / kXcds, kap = lam % kSlices, h = lam / kSlices, g = kPerXcd * x + lam;

  if (tid == 0) {
    FLAG(abort_) = 0;
    FLAG(rows_done) = 0;
    FLAG(limbs_ready) = 0;
    FLAG(pub_done) = 0;
    FLAG(ssm_cnt) = 0;
    FLAG(g_cnt) = 0;
    const uint64_t old = dfssm_dev::arrive(epoch, wg);
    seq_s = (uint32_t)((old >> 32) % 0xffffffu) + 1u;
    dfssm_dev::advance_if_last(epoch, wg, old, kGrid);
  }
  const int64_t ring_stride = 4 * kConv, state_stride = (int64_t)kNh * 64 * kDs;
  const uint32_t sb0 = lds_addr(&ring[0][0]);
  if (wave == 6) {
    step_batch(lins[0], x, kap, h, lam, t, conv_ring, ssm_state, sb0, lane);
    if (L2 > 1) step_batch(lins[1], x, kap, h, lam, t, conv_ring, ssm_state, sb0 + kSlotBytes, lane);
    CHAIN_WAIT_VMCNT(0);
  }
  // the reducer's residual rows, kept across the layers
  float u_reg = wave == 0 && lane < kOutRows ? u0[kOutRows * g + lane] : 0.0f;
  CHAIN_BARRIER();
  if (FLAG(abort_)) return;
  const uint32_t seq = seq_s;
  auto tag_of = [seq](int j) -> uint32_t { return (seq << 8) | (uint32_t)((j + 1) & 0xff); };
  (void)ex_words;

  for (int j = 0; j < L2; ++j) {
    const int ju = __builtin_amdgcn_readfirstlane(j);
    const int l = ju >> 1;
    const StepLin Ld = lins[ju];
    const bool is_in = Ld.kind == 0;
    const int K = Ld.K, Ks = K >> 3, Wr = K >> 8, r = Ld.r;
    const uint8_t* slot = ring[ju % kRing];
    const uint32_t tg = tag_of(ju);

    if (wave >= 1 && wave != 6) {
      const int ct = (wave == 7 ? 5 : wave - 1) * 64 + lane;  // 0 .. 383
      long sp = 0;
      if (ju > 0) STEP_WAIT_FLAG(FLAG(pub_done) >= ju, sp, kStIn);
      if (!is_in && !FLAG(abort_)) {
        // ---- the layer's convolution, SSM step and gate for channels
        //      16g .. 16g+15, from this workgroup's in_proj outputs (zx_s),
        //      the 256 B/C words, the head's dt word and the operands that
        //      came with in_proj's batch (slot of linear j - 1)
        const StepLin Lp = lins[ju - 1];
        const uint8_t* ps = ring[(ju - 1) % kRing];
        const uint32_t tp = tag_of(ju - 1);
        const float* rgw = reinterpret_cast<const float*>(ps + Lp.o_rg);  // [3][x 16]: steps t-1, t-2, t-3
        const float4* cw = reinterpret_cast<const float4*>(ps + Lp.o_cw);  // [x 16 | own B/C]
        const float* cb = reinterpret_cast<const float*>(ps + Lp.o_cb);    // [x 16 | own B/C]
        if (ct < 2 * kDs) {
          // B and C after the convolution, from the workgroup that owns the row
          uint64_t w = 0;
          while (!FLAG(abort_)) {
            w = ll_load(ex + Lp.bc_off + x * 2 * kDs + ct);
            if ((uint32_t)(w >> 32) == tp) break;
            if (spin_gives_up(sp, &abort_, status, kStSsm)) break;
          }
          bcc[ct] = __uint_as_float((uint32_t)w);
        } else if (ct < 2 * kDs + kCpw) {
          // the convolution of this workgroup's x channel p
          const int p = ct - 2 * kDs;
          const float4 wv = cw[p];
          float v = wv.x * rgw[2 * kCpw + p];
          v = v + wv.y * rgw[kCpw + p];
          v = v + wv.z * rgw[p];
          v = v + wv.w * zx_s[kCpw + p];
          v = v + cb[p];
          xc[p] = silu_f(v);
        } else if (ct < 2 * kDs + 2 * kCpw) {
          const int p = ct - 2 * kDs - kCpw;
          szv[p] = silu_f(zx_s[p]);
        } else if (ct == 2 * kDs + 2 * kCpw) {
          // dt and dA of the head, from the workgroup that owns its dt row
          const int hw = kCpw * g / 64;
          uint64_t w0 = 0, w1 = 0;
          while (!FLAG(abort_)) {
            w0 = ll_load(ex + Lp.dt_off + 2 * hw);
            w1 = ll_load(ex + Lp.dt_off + 2 * hw + 1);
            if ((uint32_t)(w0 >> 32) == tp && (uint32_t)(w1 >> 32) == tp) break;
            if (spin_gives_up(sp, &abort_, status, kStSsm)) break;
          }
          dts[0] = __uint_as_float((uint32_t)w0);
          dts[1] = __uint_as_float((uint32_t)w1);
          dts[2] = reinterpret_cast<const float*>(ps + Lp.o_hp)[0];
        }
        // the six waves meet (an LDS counter: waves 0 and 6 are elsewhere)
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's LDS writes are done
        if (lane == 0) __hip_atomic_fetch_add(&ssm_cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        STEP_WAIT_FLAG(FLAG(ssm_cnt) >= 6 * (l + 1), sp, kStSsm);
        if (ct < 256 && !FLAG(abort_)) {
          // SSM step: channel p = ct / 16, states 8 sub .. 8 sub + 7
          const int p = ct >> 4, sub = ct & 15, n0 = 8 * sub;
          const float4* st = reinterpret_cast<const float4*>(ps + Lp.o_st) + (p * kDs + n0) / 4;
          const float4 h0 = st[0], h1 = st[1];
          float hs[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
          const float dt = dts[0], dA = dts[1], xv = xc[p], dtx = dt * xv;
          double acc = 0.0;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float t1 = hs[e] * dA;
            const float t2 = dtx * bcc[n0 + e];
            hs[e] = t1 + t2;
            acc += (double)hs[e] * (double)bcc[kDs + n0 + e];
          }
          // the 16 lanes of the channel (xor butterfly: every lane ends with
          // the same sum)
#pragma unroll
          for (int off = 8; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 16);
          if (sub == 0) {
            const float y = (float)(acc + (double)dts[2] * (double)xv);
            const float gval = y * szv[p];
            ll_store(ex + Ld.in_off + kCpw * g + p, tg, __float_as_uint(gval));
          }
          __builtin_amdgcn_s_waitcnt(0xC07F);
          if (lane == 0) __hip_atomic_fetch_add(&g_cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          // the new state last: a wave's stores complete in order, and the
          // words above are what every other workgroup is waiting for
          float4* dst = reinterpret_cast<float4*>(ssm_state + l * state_stride + (int64_t)(kCpw * g + p) * kDs + n0);
          dst[0] = make_float4(hs[0], hs[1], hs[2], hs[3]);
          dst[1] = make_float4(hs[4], hs[5], hs[6], hs[7]);
        }
      }
      // ---- phase D: this slice of the input
      const int i0 = ct, i1 = ct + kPollLanes;
      if (ju == 0) {
        if (i0 < Ks) ys[i0] = u0[kap * Ks + i0];
        if (i1 < Ks) ys[i1] = u0[kap * Ks + i1];
      } else {
        // out_proj: polls start once this workgroup's own gated outputs are
        // out (the others come at about the same time; earlier polls only
        // load the fabric)
        if (!is_in) STEP_WAIT_FLAG(FLAG(g_cnt) >= 4 * (l + 1), sp, kStSsm);
        uint32_t pend = (i0 < Ks ? 1u : 0u) | (i1 < Ks ? 2u : 0u);
        if (FLAG(abort_)) pend = 0;
        const uint64_t* iw = ex + Ld.in_off + (int64_t)kap * Ks;
        while (pend) {
          uint64_t w0 = 0, w1 = 0;
          if (pend & 1u) w0 = ll_load(iw + i0);
          if (pend & 2u) w1 = ll_load(iw + i1);
          if ((pend & 1u) && (uint32_t)(w0 >> 32) == tg) {
            ys[i0] = __uint_as_float((uint32_t)w0);
            pend &= ~1u;
          }
          if ((pend & 2u) && (uint32_t)(w1 >> 32) == tg) {
            ys[i1] = __uint_as_float((uint32_t)w1);
            pend &= ~2u;
          }
          if (pend && spin_gives_up(sp, &abort_, status, kStIn)) break;
        }
      }
    }
    CHAIN_BARRIER();  // B1
    if (FLAG(abort_)) {
      if (tid == 0) note_abort_linear(status, ju);
      return;
    }

    uint32_t cq0 = 0, cq1 = 0;  // wave 1: codes 8p .. 8p+7 of the slice
    if (wave == 1) {
      // ---- the scale r and the maximum of |(v * r) * w| over the whole
      //      input, from one exchange among the row group's 8 workgroups
      //      (one slice each).  Every workgroup publishes its slice's fp64
      //      sum of squares (wave 2, below) and the entries whose fp32
      //      |v * w| lies within 2^-19 of the slice's largest.  The rounding
      //      of that product and of the two fp32 products of (v * r) * w
      //      moves a value by less than 2^-21 of it, so no other entry can
      //      exceed the largest of these: while values stay in the normal
      //      range (checked below) the maximum over the published entries
      //      is the input's maximum.  Otherwise (more than two such entries
      //      in a slice, values near the ends of the range) the slices'
      //      maxima after r take a second exchange.
      const int p = lane;
      const bool inb = 8 * p < Ks;
      const float* nwv = reinterpret_cast<const float*>(slot + Ld.o_nw);
      const uint64_t* stw = ex + Ld.st_off + (int64_t)(x * kGroups + h) * kSlices * 8;
      // lanes past the slice's end take zeros: they change no maximum and
      // (with a positive largest product) no candidate
      float gq[8], wq[8];
      {
        const float4* y4 = reinterpret_cast<const float4*>(ys) + (inb ? 2 * p : 0);
        const float4* w4 = reinterpret_cast<const float4*>(nwv) + (inb ? 2 * p : 0);
        const float4 ya = y4[0], yb = y4[1], wa = w4[0], wb = w4[1];
        const float z = 0.0f;
        gq[0] = inb ? ya.x : z; gq[1] = inb ? ya.y : z; gq[2] = inb ? ya.z : z; gq[3] = inb ? ya.w : z;
        gq[4] = inb ? yb.x : z; gq[5] = inb ? yb.y : z; gq[6] = inb ? yb.z : z; gq[7] = inb ? yb.w : z;
        wq[0] = inb ? wa.x : z; wq[1] = inb ? wa.y : z; wq[2] = inb ? wa.z : z; wq[3] = inb ? wa.w : z;
        wq[4] = inb ? wb.x : z; wq[5] = inb ? wb.y : z; wq[6] = inb ? wb.z : z; wq[7] = inb ? wb.w : z;
      }
      {
        float ef[8];
        uint32_t em = 0, gm = 0, wm = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          ef[e] = fabsf(gq[e] * wq[e]);
          em = max(em, __float_as_uint(ef[e]));
          gm = max(gm, __float_as_uint(gq[e]) & 0x7fffffffu);
          wm = max(wm, __float_as_uint(wq[e]) & 0x7fffffffu);
        }
        em = wave_max_bits_u(em);
        gm = wave_max_bits_u(gm);
        const float thr = __uint_as_float(em) * (1.0f - 0x1p-19f);
        int cnt = 0;
        float a0 = 0.0f, b0 = 0.0f, a1 = 0.0f, b1v = 0.0f;  // (v, w) of this lane's first two
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const bool hit = ef[e] >= thr;
          a1 = hit && cnt == 1 ? gq[e] : a1;
          b1v = hit && cnt == 1 ? wq[e] : b1v;
          a0 = hit && cnt == 0 ? gq[e] : a0;
          b0 = hit && cnt == 0 ? wq[e] : b0;
          cnt += hit ? 1 : 0;
        }
        // finite values and products, norm weights up to 2^40, at most two
        // candidates
        const uint64_t h1 = __ballot(cnt >= 1), h2 = __ballot(cnt >= 2), h3 = __ballot(cnt >= 3);
        const bool slow_w = gm >= 0x7f800000u || em >= 0x7f800000u || __ballot(wm > 0x53800000u) != 0 ||
                            h3 != 0 || __popcll(h1) + __popcll(h2) > 2;
        uint32_t c0g = 0, c0w = 0, c1g = 0, c1w = 0;
        if (!slow_w) {
          const int la = __builtin_ctzll(h1);
          c0g = (uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(a0), la);
          c0w = (uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(b0), la);
          c1g = c0g;
          c1w = c0w;
          if (h2 != 0) {
            c1g = (uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(a1), la);
            c1w = (uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(b1v), la);
          } else if ((h1 & (h1 - 1)) != 0) {
            const int lb = __builtin_ctzll(h1 & (h1 - 1));
            c1g = (uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(a0), lb);
            c1w = (uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(b0), lb);
          }
        }
        uint32_t v = slow_w ? 1u : 0u;
        v = lane == 6 ? gm : v;
        v = lane == 5 ? c1w : v;
        v = lane == 4 ? c1g : v;
        v = lane == 3 ? c0w : v;
        v = lane == 2 ? c0g : v;
        if (lane >= 2 && lane < 8)
          ll_store(ex + Ld.st_off + (int64_t)((x * kGroups + h) * kSlices + kap) * 8 + lane, tg, v);
      }
      // lane 8k + i: word i of slice k
      uint32_t sv = 0;
      {
        long sp = 0;
        while (!FLAG(abort_)) {
          const uint64_t w = ll_load(stw + lane);
          if ((uint32_t)(w >> 32) == tg) {
            sv = (uint32_t)w;
            break;
          }
          if (spin_gives_up(sp, &abort_, status, kStIn)) break;
        }
      }
      double S = 0.0;
#pragma unroll
      for (int k = 0; k < kSlices; ++k) {
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)sv, 8 * k);
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)sv, 8 * k + 1);
        S += __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
      }
      const float rr = (float)(1.0 / sqrt(S / (double)K + (double)eps));
      float xv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float tv = gq[e] * rr;
        xv[e] = tv * wq[e];
      }
      const int wd = lane & 7;
      // lanes 8k + 3 and 8k + 5 take the entry's v from the lane before
      const uint32_t s_prev = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)sv, 0x111, 0xF, 0xF, false);  // row_shr:1
      uint32_t cand = 0;
      bool fail = false;
      if (wd == 3 || wd == 5) {
        // a published entry: its (v * r) * w, and r * |v| * |w| not below 2^-60
        const float gc = __uint_as_float(s_prev), wc = __uint_as_float(sv);
        const float tv = gc * rr;
        cand = __float_as_uint(tv * wc) & 0x7fffffffu;
        fail = fabs((double)gc * (double)wc) * (double)rr < 0x1p-60;
      } else if (wd == 6) {
        fail = (double)__uint_as_float(sv) * (double)rr > 0x1p80;  // r * max |v| up to 2^80
      } else if (wd == 7) {
        fail = sv != 0;
      }
      uint32_t a_bits = 0;
      if (!two_hop && __ballot(fail) == 0) {
        a_bits = wave_max_bits_u(cand);
      } else {
        uint32_t m = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (inb) m = max(m, __float_as_uint(xv[e]) & 0x7fffffffu);
        m = wave_max_bits_u(m);
        if (lane == 0) ll_store(ex + Ld.mx_off + (x * kGroups + h) * kSlices + kap, tg, m);
        if (lane < kSlices) {
          long sp = 0;
          uint64_t w = 0;
          while (!FLAG(abort_)) {
            w = ll_load(ex + Ld.mx_off + (x * kGroups + h) * kSlices + lane);
            if ((uint32_t)(w >> 32) == tg) break;
            if (spin_gives_up(sp, &abort_, status, kStIn)) break;
          }
          a_bits = (uint32_t)w;
        }
        a_bits = wave_max_bits_u(a_bits);
      }
      const float a = __uint_as_float(a_bits);
      const bool zero = a < FLT_MIN;
      const float inv = zero ? 0.0f : 127.0f / a;
      if (lane == 0) qs_s = zero ? 0.0f : a / 127.0f;
      int qsum = 0;
      if (inb) {
        int q[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) q[e] = zero ? 0 : code(xv[e], inv);
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          lo |= (uint32_t)(q[e] & 0xff) << (8 * e);
          hi |= (uint32_t)(q[4 + e] & 0xff) << (8 * e);
          qsum += q[e] + q[4 + e];
        }
        reinterpret_cast<uint2*>(codes)[p] = make_uint2(lo, hi);
        cq0 = lo;
        cq1 = hi;
        uint32_t tt;
        tt = (lo ^ (lo >> 7)) & 0x00AA00AAu;
        lo ^= tt ^ (tt << 7);
        tt = (hi ^ (hi >> 7)) & 0x00AA00AAu;
        hi ^= tt ^ (tt << 7);
        tt = (lo ^ (lo >> 14)) & 0x0000CCCCu;
        lo ^= tt ^ (tt << 14);
        tt = (hi ^ (hi >> 14)) & 0x0000CCCCu;
        hi ^= tt ^ (tt << 14);
        tt = (lo ^ __builtin_amdgcn_alignbit(hi, lo, 28)) & 0xF0F0F0F0u;
        lo ^= tt;
        hi ^= tt >> 4;
        uint8_t* pb = reinterpret_cast<uint8_t*>(planes) + p;
#pragma unroll
        for (int b = 0; b < 4; ++b) pb[b * (kMaxKs / 8)] = (uint8_t)(lo >> (8 * b));
#pragma unroll
        for (int b = 0; b < 4; ++b) pb[(4 + b) * (kMaxKs / 8)] = (uint8_t)(hi >> (8 * b));
      }
      qsum = wave_sum_u(qsum);
      if (lane == 0) sumq[ju & 1] = qsum;
    } else if (wave == 2) {
      // ---- the slice's fp64 sum of squares (words 0 and 1 of this
      //      workgroup's entry; the same order in every workgroup that holds
      //      the slice)
      const bool inb = 8 * lane < Ks;
      const float4* y4 = reinterpret_cast<const float4*>(ys) + (inb ? 2 * lane : 0);
      const float4 ya = y4[0], yb = y4[1];
      const float gv[8] = {ya.x, ya.y, ya.z, ya.w, yb.x, yb.y, yb.z, yb.w};
      double sq = 0.0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const double d = inb ? (double)gv[e] : 0.0;
        sq = sq + d * d;
      }
      const uint64_t sb = (uint64_t)__double_as_longlong(wave_sum_f64_u(sq));
      if (lane < 2)
        ll_store(ex + Ld.st_off + (int64_t)((x * kGroups + h) * kSlices + kap) * 8 + lane, tg,
                 lane == 0 ? (uint32_t)(sb >> 32) : (uint32_t)sb);
    }
    CHAIN_BARRIER();  // B2
    if (FLAG(abort_)) {
      if (tid == 0) note_abort_linear(status, ju);
      return;
    }

    if (wave != 1) {
      // ---- phase A: slice partials of every slot of the row group (as the
      //      chain; slots without a row are skipped)
      const int G = Wr <= 4 ? 1 : (Wr <= 8 ? 2 : 4);
      // lane blocks of 64 in the order waves 5, 3, 2, 0, 7, 6, 4: the first
      // four sit on four different SIMDs (waves w and w + 4 share one)
      const int ta = 64 * ((0x45061273 >> (4 * wave)) & 0xF) + lane;
      const int gg = ta % G, w0 = 4 * gg;
      uint32_t pw[8][4];
#pragma unroll
      for (int b = 0; b < 8; ++b)
#pragma unroll
        for (int k = 0; k < 4; ++k) pw[b][k] = planes[b][(w0 + k) & (kMaxKs / 32 - 1)];
      uint32_t keep[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) keep[k] = w0 + k < Wr ? ~0u : 0u;
      const int sq = sumq[ju & 1];
      const int nA = kSlices * Ld.rs;
      const uint32_t mrs = recip20((uint32_t)Ld.rs);
      const int per_pass = kRowLanes / G;
      const int rowbytes = K >> 6;
      for (int i0 = 0; i0 < nA; i0 += per_pass) {
        const int i = i0 + ta / G;
        const int ic = i < nA ? i : 0;
        const uint32_t* srow = reinterpret_cast<const uint32_t*>(slot + (size_t)ic * rowbytes);
        uint32_t sw[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) sw[k] = srow[(w0 + k) & 15] & keep[k];
        int d = 0;
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          uint32_t c = 0;
#pragma unroll
          for (int k = 0; k < 4; ++k) c += (uint32_t)__builtin_popcount(sw[k] & pw[b][k]);
          d += b < 7 ? (int)(c << b) : -(int)(c << 7);
        }
        d = group_sum(d, G);
        if (i < nA && gg == 0) {
          const int row = group_row(Ld.kind, Ld.rs, mrs, x, h, i);
          if (row >= 0) ll_store(ex + Ld.part_off + (int64_t)kap * Ld.N + row, tg, (uint32_t)(2 * d - sq));
        }
      }
      if (lane == 0) __hip_atomic_fetch_add(&rows_done, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }

    if (wave == 1) {
      // ---- LoRA down-projection inside the XCD (as the chain)
      const int rh = Ld.rh;
      if (rh > 0) {
        const bool inb = 8 * lane < Ks;
        uint2 aw[kMaxRh];
        if (Ld.i4) {
          // 4 bytes (8 nibbles) per rank and lane, expanded to the int8 pair
          const uint8_t* arow = slot + Ld.o_a + (inb ? 4 * lane : 0);
          uint32_t a4[kMaxRh];
#pragma unroll
          for (int jj = 0; jj < kMaxRh; ++jj)
            a4[jj] = *reinterpret_cast<const uint32_t*>(arow + (jj < rh ? jj : 0) * (Ks >> 1));
#pragma unroll
          for (int jj = 0; jj < kMaxRh; ++jj) unpack_i4x8(a4[jj], aw[jj].x, aw[jj].y);
        } else {
          const uint8_t* arow = slot + Ld.o_a + (inb ? 8 * lane : 0);
#pragma unroll
          for (int jj = 0; jj < kMaxRh; ++jj)
            aw[jj] = *reinterpret_cast<const uint2*>(arow + (jj < rh ? jj : 0) * Ks);
        }
#pragma unroll
        for (int jj = 0; jj < kMaxRh; ++jj)
          red[lane * 17 + jj] = inb ? sdot4(aw[jj].y, cq1, sdot4(aw[jj].x, cq0, 0)) : 0;
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        const int jj = lane >> 2, part = lane & 3;
        int rv[16];
#pragma unroll
        for (int tt = 0; tt < 16; ++tt) rv[tt] = red[(part * 16 + tt) * 17 + jj];
        int v = 0;
#pragma unroll
        for (int tt = 0; tt < 16; ++tt) v += rv[tt];
        v = group_sum(v, 4);
        const int jr = h * rh + jj;
        if (part == 0 && jj < rh && jr < r)
          ll_store(ex + Ld.p_off + (int64_t)(x * kSlices + kap) * kMaxR + jr, tg, (uint32_t)v);
      }
      int acc_a = 0;
      if (r > 0) {
        long sp = 0;
        uint32_t pend = lane < r && !FLAG(abort_) ? 0xffu : 0u;
        while (pend) {
          uint64_t wa[kSlices];
#pragma unroll
          for (int k = 0; k < kSlices; ++k)
            wa[k] = (pend & (1u << k)) ? ll_load(ex + Ld.p_off + (int64_t)(x * kSlices + k) * kMaxR + lane) : 0;
#pragma unroll
          for (int k = 0; k < kSlices; ++k)
            if ((pend & (1u << k)) && (uint32_t)(wa[k] >> 32) == tg) {
              acc_a += (int32_t)(uint32_t)wa[k];
              pend &= ~(1u << k);
            }
          if (pend && spin_gives_up(sp, &abort_, status, kStAcc)) break;
        }
      }
      int8_t dl[4];
      dfssm_dev::split_limbs(lane < r ? acc_a : 0, dl);
      uint8_t* lb = reinterpret_cast<uint8_t*>(limbs) + (lane >> 2) * 16 + (lane & 3);
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) lb[4 * tt] = (uint8_t)dl[tt];
      __builtin_amdgcn_s_waitcnt(0xC07F);
      if (lane == 0) FLAG(limbs_ready) = ju + 1;
    } else if (wave == 0) {
      // ---- reducer: lane k takes row k of this workgroup's rows
      long sp = 0;
      STEP_WAIT_FLAG(FLAG(rows_done) >= kAWaves * (ju + 1), sp, kStAcc);
      const int R = reducer_rows(Ld.kind, g);
      const int rw = r >> 2;
      uint32_t bw[kMaxR / 4];
      if (Ld.i4) {
        // r/2 bytes per row: each dword is 8 nibbles, two dwords of int8
        const uint32_t* brow = reinterpret_cast<const uint32_t*>(slot + Ld.o_b + (lane < R ? lane : 0) * (r >> 1));
        uint32_t b4[kMaxR / 8];
#pragma unroll
        for (int w = 0; w < kMaxR / 8; ++w) b4[w] = 2 * w < rw ? brow[w] : 0u;
#pragma unroll
        for (int w = 0; w < kMaxR / 8; ++w) unpack_i4x8(b4[w], bw[2 * w], bw[2 * w + 1]);
      } else {
        const uint32_t* brow = reinterpret_cast<const uint32_t*>(slot + Ld.o_b + (lane < R ? lane : 0) * r);
#pragma unroll
        for (int w = 0; w < kMaxR / 4; ++w) bw[w] = w < rw ? brow[w] : 0u;
      }
      const float al = reinterpret_cast<const float*>(slot + Ld.o_al)[lane];
      const float be = reinterpret_cast<const float*>(slot + Ld.o_be)[lane];
      const int n = lane < R ? reducer_row(Ld.kind, g, lane) : 0;
      int acc_s = 0;
      uint32_t pend = lane < R && !FLAG(abort_) ? 0xffu : 0u;
      while (pend) {
        uint64_t wp[kSlices];
#pragma unroll
        for (int k = 0; k < kSlices; ++k)
          wp[k] = (pend & (1u << k)) ? ll_load(ex + Ld.part_off + (int64_t)k * Ld.N + n) : 0;
#pragma unroll
        for (int k = 0; k < kSlices; ++k)
          if ((pend & (1u << k)) && (uint32_t)(wp[k] >> 32) == tg) {
            acc_s += (int32_t)(uint32_t)wp[k];
            pend &= ~(1u << k);
          }
        if (pend && spin_gives_up(sp, &abort_, status, kStAcc)) break;
      }
      STEP_WAIT_FLAG(FLAG(limbs_ready) >= ju + 1, sp, kStAcc);
      if (!FLAG(abort_)) {
        uint4 lw[kMaxR / 4];
#pragma unroll
        for (int w = 0; w < kMaxR / 4; ++w) lw[w] = limbs[w];
        int e0 = 0, e1 = 0, e2 = 0, e3 = 0;
#pragma unroll
        for (int w = 0; w < kMaxR / 4; ++w) {
          e0 = sdot4(bw[w], lw[w].x, e0);
          e1 = sdot4(bw[w], lw[w].y, e1);
          e2 = sdot4(bw[w], lw[w].z, e2);
          e3 = sdot4(bw[w], lw[w].w, e3);
        }
        const int elo = e0 + (e1 << 8), ehi = e2 + (e3 << 8);
        const float y = dfssm_dev::epilogue(qs_s, al, be, acc_s, ehi, elo, r > 0);
        if (is_in) {
          // z and x stay here; the B/C and dt rows go out as words; x and
          // B/C inputs enter the convolution window (ring slot t & 3)
          float* ring_t = conv_ring + l * ring_stride + (t & 3) * kConv;
          const float ybc = __shfl(y, 2 * kCpw, 64);
          if (lane < 2 * kCpw) zx_s[lane] = y;
          if (lane >= kCpw && lane < 2 * kCpw) ring_t[kCpw * g + (lane - kCpw)] = y;
          if (lane == 2 * kCpw) ring_t[kDi + g] = y;
          if (lane >= kBcLane && lane < kBcLane + kXcds) {
            // B/C row g after its convolution (window of steps t-3 .. t-1
            // and y), one copy per XCD: every workgroup reads all 256
            const float* rb = reinterpret_cast<const float*>(slot + Ld.o_rb);
            const float4 wv = reinterpret_cast<const float4*>(slot + Ld.o_cw)[kCpw];
            float v = wv.x * rb[2];
            v = v + wv.y * rb[1];
            v = v + wv.z * rb[0];
            v = v + wv.w * ybc;
            v = v + reinterpret_cast<const float*>(slot + Ld.o_cb)[kCpw];
            ll_store(ex + Ld.bc_off + (lane - kBcLane) * 2 * kDs + g, tg, __float_as_uint(silu_f(v)));
          }
          if (lane == 2 * kCpw + 1 && g < kNh) {
            // the dt row of head g: dt = softplus(dt_raw + dt_bias), dA = exp(dt * A)
            const float* hp = reinterpret_cast<const float*>(slot + Ld.o_hp);
            const float dt = softplus_f(y + hp[64]);
            const float A = (float)(-exp((double)hp[128]));
            ll_store(ex + Ld.dt_off + 2 * g, tg, __float_as_uint(dt));
            ll_store(ex + Ld.dt_off + 2 * g + 1, tg, __float_as_uint((float)exp((double)(dt * A))));
          }
          __builtin_amdgcn_s_waitcnt(0xC07F);  // zx_s is in LDS before the flag
        } else {
          // the residual stream: u += delta, then the next layer's input
          if (lane < kOutRows) u_reg = u_reg + y;
          if (ju + 1 < L2) {
            const StepLin& Ln = lins[ju + 1];
            const uint32_t tn = tag_of(ju + 1);
            if (lane < kOutRows) ll_store(ex + Ln.in_off + kOutRows * g + lane, tn, __float_as_uint(u_reg));
          } else if (lane < kOutRows) {
            u_fin[kOutRows * g + lane] = u_reg;
          }
        }
      }
      if (lane == 0) FLAG(pub_done) = ju + 1;
    } else if (wave == 6) {
      // ---- loading: linear j+1's operands have landed once nothing of this
      //      wave is in flight; linear j+2's go into the slot linear j-1 used
      CHAIN_WAIT_VMCNT(0);
      if (ju + 2 < L2) {
        const int l2 = (ju + 2) >> 1;
        step_batch(lins[ju + 2], x, kap, h, lam, t, conv_ring + l2 * ring_stride, ssm_state + l2 * state_stride,
                   sb0 + (uint32_t)(((ju + 2) % kRing) * kSlotBytes), lane);
      }
    }
  }
}

// Writes a chunk of the step's table; the first chunk also zeroes the
// exchange words, the status word and the epochs.
struct StepSetupArgs {
  StepLin e[kSetupChunk];
  StepLin* table;
  uint64_t* zero_base;
  int64_t zero_words;
  uint64_t* hash_dst;
  uint64_t hash;
  int first, count;
};

__global__ void step_setup(StepSetupArgs a) {
  const int64_t i0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i0 < a.count) a.table[a.first + i0] = a.e[i0];
  for (int64_t i = i0; i < a.zero_words; i += (int64_t)gridDim.x * blockDim.x) a.zero_base[i] = 0;
  if (a.hash_dst && i0 == 0) *a.hash_dst = a.hash;
}

// ---------------------------------------------------------------- host side
struct StepPlan {
  std::vector<StepLin> table;
  int64_t ex_words = 0;
  bool ok = false;
};

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// The kernel's table for this model, or ok = false if the model is not the
// shape the kernel takes.
StepPlan make_step_plan(const dfssm_mamba2_model* md) {
  StepPlan p;
  if (!md || !md->layers || md->d_model != kD || md->d_state != kDs || md->n_layers <= 0 || md->n_layers > 120)
    return p;
  const int n = (int)md->n_layers;
  p.table.resize(2 * n);
  int64_t w = 0;
  for (int l = 0; l < n; ++l) {
    const dfssm_mamba2_layer& ML = md->layers[l];
    for (int kind = 0; kind < 2; ++kind) {
      const dfssm_layer& P = kind == 0 ? ML.in_proj : ML.out_proj;
      const int64_t K = kind == 0 ? kD : kDi, N = kind == 0 ? kNin : kD, r = P.r;
      const bool i4 = ML.lora_bits == 4 && r > 0;
      if (P.K != K || P.N != N || r < 0 || r > kMaxR || r % (i4 ? 8 : 4) != 0) return p;
      StepLin& e = p.table[2 * l + kind];
      std::memset(&e, 0, sizeof(e));
      const bool lr = r > 0;
      e.w_bits = P.w_bits;
      e.alpha = P.alpha;
      e.A = lr ? P.A : reinterpret_cast<const int8_t*>(P.alpha);
      e.B = lr ? P.B : reinterpret_cast<const int8_t*>(P.alpha);
      e.beta = lr ? P.beta : P.alpha;
      e.nw = kind == 0 ? ML.norm_w : ML.gate_w;
      e.conv_w = ML.conv_w;
      e.conv_b = ML.conv_b;
      e.dt_bias = ML.dt_bias;
      e.A_log = ML.A_log;
      e.Dp = ML.D;
      e.K = (int32_t)K;
      e.N = (int32_t)N;
      e.r = (int32_t)r;
      e.rh = (int32_t)((r + kRankGroups - 1) / kRankGroups);
      e.kind = kind;
      e.rs = kind == 0 ? kInSlots : kOutRows;
      const int64_t rowbytes = K / 64, Ks = K / 8;
      e.us = rowbytes % 16 == 0 ? 16 : 4;
      e.i4 = i4 ? 1 : 0;
      const int64_t rb = i4 ? r / 2 : r;  // B row bytes
      e.ub = rb % 16 == 0 ? 16 : 4;
      const int64_t rmax = kind == 0 ? kInSlots : kOutRows;
      const int64_t sign_ni = cdiv(kSlices * e.rs * (rowbytes / e.us), 64);
      const int64_t a_ni = cdiv(e.rh * Ks / (i4 ? 32 : 16), 64);
      const int64_t b_ni = lr ? cdiv(rmax * (rb / e.ub), 64) : 0;
      const int64_t nw_ni = cdiv(Ks / 4, 64);
      int64_t o = sign_ni * 64 * e.us;
      e.o_a = (int32_t)o;
      o += a_ni * 1024;
      e.o_b = (int32_t)o;
      o += b_ni * 64 * e.ub;
      e.o_al = (int32_t)o;
      o += 256;
      e.o_be = (int32_t)o;
      o += 256;
      e.o_nw = (int32_t)o;
      o += nw_ni * 1024;
      if (kind == 0) {
        e.o_st = (int32_t)o;
        o += kCpw * kDs * 4;
        e.o_rg = (int32_t)o;
        o += 1024;
        e.o_rb = (int32_t)o;
        o += 256;
        e.o_cw = (int32_t)o;
        o += 1024;
        e.o_cb = (int32_t)o;
        o += 256;
        e.o_hp = (int32_t)o;
        o += 3 * 256;
      }
      if (o > kSlotBytes) return p;
      e.layer = l;
      e.part_off = w;
      w += N * kSlices;
      e.p_off = w;
      w += (int64_t)kXcds * kSlices * kMaxR;
      e.mx_off = w;
      w += (int64_t)kXcds * (kPerXcd / kSlices) * kSlices;
      e.in_off = w;
      w += K;
      e.st_off = w;
      w += (int64_t)kXcds * kGroups * kSlices * 8;
      if (kind == 0) {
        e.bc_off = w;
        w += (int64_t)kXcds * 2 * kDs;
        e.dt_off = w;
        w += 2 * kNh;
      }
    }
  }
  p.ex_words = (w + 31) / 32 * 32;
  p.ok = true;
  return p;
}

// Workspace of the fused step: table, fingerprint, exchange words, status
// word, epoch words, the embedding row u0 and the final residual row.
struct StepLayout {
  size_t off_table, off_hash, off_ex, off_status, off_epoch, off_u0, off_ufin, bytes;
};
StepLayout step_layout(const StepPlan& p) {
  StepLayout o{};
  size_t at = 0;
  auto take = [&](size_t nb) {
    const size_t r = at;
    at += (nb + 255) / 256 * 256;
    return r;
  };
  o.off_table = take(p.table.size() * sizeof(StepLin));
  o.off_hash = take(8);
  o.off_ex = take((size_t)p.ex_words * 8);
  o.off_status = take(4);
  o.off_epoch = take((size_t)dfssm::kEpochGroups * dfssm::kEpochStride * 8);
  o.off_u0 = take(kD * 4);
  o.off_ufin = take(kD * 4);
  o.bytes = at;
  return o;
}

uint64_t step_fingerprint(const StepPlan& p, float eps) {
  uint64_t hsh = 1469598103934665603ull;
  auto mix = [&](const void* q, size_t len) {
    const unsigned char* b = static_cast<const unsigned char*>(q);
    for (size_t i = 0; i < len; ++i) hsh = (hsh ^ b[i]) * 1099511628211ull;
  };
  const int n = (int)p.table.size();
  mix(&n, sizeof(n));
  mix(&eps, sizeof(eps));
  mix(p.table.data(), p.table.size() * sizeof(StepLin));
  return hsh;
}

}  // namespace

namespace dfssm {

StepFusedInfo step_fused_info(const dfssm_mamba2_model* md) {
  StepFusedInfo f{};
  const StepPlan p = make_step_plan(md);
  if (!p.ok) return f;
  const StepLayout o = step_layout(p);
  f.ok = true;
  f.bytes = o.bytes;
  f.off_hash = o.off_hash;
  f.off_ex = o.off_ex;
  f.off_epoch = o.off_epoch;
  f.ex_words = p.ex_words;
  f.off_status = o.off_status;
  f.off_u0 = o.off_u0;
  f.off_ufin = o.off_ufin;
  f.n_linears = (int)p.table.size();
  f.fingerprint = step_fingerprint(p, md->eps);
  return f;
}

hipError_t step_fused_prepare(const dfssm_mamba2_model* md, void* ws, hipStream_t st) {
  const StepPlan p = make_step_plan(md);
  if (!p.ok) return hipErrorInvalidValue;
  const StepLayout o = step_layout(p);
  char* base = static_cast<char*>(ws);
  const uint64_t hsh = step_fingerprint(p, md->eps);
  StepLin* table = reinterpret_cast<StepLin*>(base + o.off_table);
  const int n = (int)p.table.size();
  for (int first = 0; first < n; first += kSetupChunk) {
    StepSetupArgs a{};
    a.count = std::min(kSetupChunk, n - first);
    for (int i = 0; i < a.count; ++i) a.e[i] = p.table[first + i];
    a.table = table;
    a.first = first;
    // the first launch clears the exchange words, the status and the epochs
    a.zero_base = first == 0 ? reinterpret_cast<uint64_t*>(base + o.off_ex) : nullptr;
    a.zero_words = first == 0 ? (int64_t)(o.off_u0 - o.off_ex) / 8 : 0;
    // the last chunk publishes the fingerprint (stream order puts it after
    // every chunk)
    a.hash_dst = first + kSetupChunk >= n ? reinterpret_cast<uint64_t*>(base + o.off_hash) : nullptr;
    a.hash = hsh;
    step_setup<<<dim3(first == 0 ? 1024 : 1), dim3(256), 0, st>>>(a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// A plain launch of one workgroup per CU (its LDS use admits one per CU);
// the whole grid has to be resident at once, and every wait is bounded.
hipError_t step_fused_run(const StepFusedInfo& f, float eps, int64_t step, float* conv_ring, float* ssm_state,
                          void* ws, bool two_hop, hipStream_t st) {
  if (!f.ok) return hipErrorInvalidValue;
  char* base = static_cast<char*>(ws);  // the table sits at the region's start
  step_persistent<<<dim3(kGrid), dim3(kThreads), 0, st>>>(
      reinterpret_cast<const StepLin*>(base), f.n_linears, (int)(step & 3),
      reinterpret_cast<const float*>(base + f.off_u0), reinterpret_cast<float*>(base + f.off_ufin), conv_ring,
      ssm_state, reinterpret_cast<uint64_t*>(base + f.off_ex), f.ex_words,
      reinterpret_cast<unsigned*>(base + f.off_status), reinterpret_cast<uint64_t*>(base + f.off_epoch),
      reinterpret_cast<const uint64_t*>(base + f.off_hash), f.fingerprint, eps, two_hop ? 1 : 0);
  return hipGetLastError();
}

}  // namespace dfssm
