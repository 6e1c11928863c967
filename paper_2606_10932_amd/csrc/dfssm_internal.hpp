// dfssm_internal.hpp -- shared declarations of the HIP implementation of
// include/dfssm.h: workspace layout, kernel launchers and small device
// helpers.  gfx950 (CDNA4) only: wave64, v_mfma_i32_16x16x64_i8,
// v_dot4_i32_i8, v_bcnt_u32_b32.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "dfssm.h"

namespace dfssm {

constexpr int kWave = 64;
constexpr int64_t kMaxK = 65536;
constexpr int64_t kMaxRank = 256;
// Largest M the bit-plane decode kernels take in one pass; larger M on the
// decode path is processed in blocks of this many tokens.
constexpr int kDecodeMaxTokens = 4;
// Automatic dispatch: M <= kDecodeM0 uses the popcount decode kernels, M up
// to kSkinnyMaxTokens the few-token MFMA kernel, larger M the prefill MFMA
// kernel.  Measured on MI355X, the single-launch few-token kernel is the
// faster one from one token on (the popcount GEMV needs a second launch for
// the LoRA down-projection and the bit-planes), so the popcount kernels run
// on request and inside the persistent chain.
constexpr int64_t kDecodeM0 = 0;

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Test switches (dfssm_test_switch), all 0 unless a test sets them: the
// kernel-family choices below read them on the host at each launch.
//   local_lora:           1 = the few-token kernel launches no LoRA
//                         workgroups (every output workgroup computes those
//                         values itself)
//   prefill_kernel:       0 = automatic, 4 or 8 = that prefill kernel
//   lm_head_mfma_tokens:  0 = 8; else the token count from which the LM
//                         head runs on the matrix cores
int test_switch(int which);
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// Per-call workspace (device), every region 256-byte aligned:
//   epoch  uint64 [64][16]        64 words {epoch:32, arrivals:32} of the
//                                 few-token kernel, one per 128-byte line
//   xw     uint64 [kXwWords]      {tag, value} words of the few-token kernel:
//                                 acc_a limbs per (token, rank), then sum Q;
//                                 a region of fixed size at a fixed offset,
//                                 so no other kernel or shape writes over it
//   acc_a  int32 [M][r]           LoRA down-projection
//   limbs  int8  [4][M][rp]       acc_a split into 4 signed base-256 digits,
//                                 rp = r rounded up to 64 (zero padded)
//   sumq   int32 [M]              sum_k Q[m,k]
//   planes uint32 [M][8][C][4]    two's-complement bit-planes of Q, C =
//                                 ceil(K/128) chunks of 4 words (zero padded)
// The epoch word and the words carry state from call to call: the
// workspace must hold zeros before its first use, and after that only the
// library writes it.
struct LinearWorkspace {
  uint64_t* epoch;
  uint64_t* xw;
  int32_t* acc_a;
  int8_t* limbs;
  int32_t* sumq;
  uint32_t* planes;
  size_t bytes;
};

inline int64_t rank_padded(int64_t r) { return round_up(r > 0 ? r : 1, 64); }
inline int64_t plane_chunks(int64_t K) { return ceil_div(K, 128); }

// Few tokens on the matrix cores: the largest M of the one-launch kernel on
// request, and of its automatic use.
constexpr int64_t kSkinnyMaxTokens = 32;
constexpr int64_t kSkinnyChunkedMaxTokens = 512;
// Exchange words of the few-token kernel: M*rp limb words, then M sum-Q
// words, for every M <= kSkinnyChunkedMaxTokens and r <= kMaxRank.
constexpr int64_t kXwWords = kSkinnyChunkedMaxTokens * kMaxRank + kSkinnyChunkedMaxTokens;
// Epoch words of the few-token kernel (its arrivals spread over them) and
// their spacing in 64-bit words.
constexpr int kEpochGroups = 64;
constexpr int kEpochStride = 16;
// Bytes before the first per-call region: the epoch words and the words.
constexpr size_t kLinearStateBytes = (size_t)kEpochGroups * kEpochStride * 8 + (size_t)kXwWords * 8;

inline LinearWorkspace carve_linear_workspace(void* base, int64_t M, int64_t K, int64_t r) {
  LinearWorkspace ws{};
  size_t off = 0;
  auto take = [&](size_t n) {
    size_t o = off;
    off += (size_t)round_up((int64_t)n, 256);
    return o;
  };
  size_t o_ep = take((size_t)kEpochGroups * kEpochStride * 8);
  size_t o_xw = take((size_t)kXwWords * 8);
  size_t o_acc = take((size_t)(M * r) * 4);
  size_t o_limb = take((size_t)(4 * M * rank_padded(r)));
  size_t o_sum = take((size_t)M * 4);
  size_t o_pl = take((size_t)(M * plane_chunks(K) * 128));
  char* b = static_cast<char*>(base);
  ws.epoch = reinterpret_cast<uint64_t*>(b + o_ep);
  ws.xw = reinterpret_cast<uint64_t*>(b + o_xw);
  ws.acc_a = reinterpret_cast<int32_t*>(b + o_acc);
  ws.limbs = reinterpret_cast<int8_t*>(b + o_limb);
  ws.sumq = reinterpret_cast<int32_t*>(b + o_sum);
  ws.planes = reinterpret_cast<uint32_t*>(b + o_pl);
  ws.bytes = off;
  return ws;
}

// ---------------------------------------------------------------- launchers
// All return hipSuccess or the launch error; shapes are validated by the
// caller.

// scale_mode 0: s = absmax/127 (0 for an all-zero row); 1: s = 1/127.
hipError_t launch_quantize(const void* x, int x_dtype, int64_t M, int64_t K, int64_t ldx,
                           int8_t* q, float* s, int scale_mode, hipStream_t st);

// Decode path: prep (acc_a, bit-planes) then the popcount GEMV with the
// fused LoRA up-projection and epilogue.
hipError_t launch_decode_linear(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                                int64_t r, const uint32_t* w_bits, const float* alpha,
                                const int8_t* A, const int8_t* B, const float* beta, float* y,
                                int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                                const LinearWorkspace& ws, hipStream_t st);

// Few tokens (M <= kSkinnyMaxTokens) on the matrix cores, one launch: LoRA
// workgroups publish acc_a and sum Q as tagged words while the others run a
// split-K expanded-sign int8 MFMA product over 16 output rows each, then the
// LoRA up-projection and epilogue.  Above kSkinnyMaxTokens, on request, its
// output blocks take one chunk of tokens each (a second grid dimension).
hipError_t launch_skinny_linear(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                                int64_t r, const uint32_t* w_bits, const float* alpha,
                                const int8_t* A, const int8_t* B, const float* beta, float* y,
                                int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                                const LinearWorkspace& ws, hipStream_t st);

// MFMA path: LoRA down-projection + limbs + sum Q, then the expanded-sign
// int8 MFMA GEMM with the LoRA up-projection and epilogue.
hipError_t launch_mfma_linear(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                              int64_t r, const uint32_t* w_bits, const float* alpha,
                              const int8_t* A, const int8_t* B, const float* beta, float* y,
                              int32_t* acc_s, int32_t* acc_a_out, int64_t* acc_b,
                              const LinearWorkspace& ws, hipStream_t st);

// ---------------------------------------------------------------- embedding
// Largest row length of the int8 embedding table the LM head takes (its
// per-lane slices of the token codes stay in registers).
constexpr int64_t kLmHeadMaxD = 16384;

// Tied int8 embedding table E [V, d] with row scales: token gather
// x = scale[t] * E[t, :] (zero rows for ids outside [0, V)), and the LM head
// logits = s[m] * (scale[v] * (float)(E Q^T)) over all V rows, in passes of
// up to 4 tokens.  d % 16 == 0.
hipError_t launch_embed_gather(const int8_t* E, const float* scale, int64_t V, int64_t d, const int32_t* tok,
                               int64_t M, float* x, hipStream_t st);
hipError_t launch_lm_head(const int8_t* q, const float* s, int64_t M, int64_t d, const int8_t* E,
                          const float* scale, int64_t V, float* logits, int32_t* acc, hipStream_t st);

// Compute units of the current device (cached per device; 256 if the query
// fails).
int device_cu_count();
// modelled duration (us) of the prefill path for an M x K x N linear
double prefill_cost_us(int64_t M, int64_t K, int64_t N);

// ---------------------------------------------------------------- chain
// The persistent chain kernel (M = 1): one launch of one workgroup per CU
// over a prepared workspace.  Workgroups the grid holds.
int chain_grid();
// Whether the persistent kernel takes these linears (M = 1; every K a
// multiple of 256 and <= 4096; r <= 64, r % 4 == 0; each linear's rows and
// operands within the kernel's per-workgroup limits).
bool chain_persistent_supported(const dfssm_layer* layers, int n_layers, int64_t M);
// Workspace bytes of the persistent chain (layer table, fingerprint,
// exchange words, status word, epoch words), 0 if not supported; the
// status word's offset.
size_t chain_persistent_bytes(const dfssm_layer* layers, int n_layers);
size_t chain_status_offset(const dfssm_layer* layers, int n_layers);
// Writes the layer table and its fingerprint and zeroes the rest.
hipError_t chain_persistent_prepare(const dfssm_layer* layers, int n_layers, void* ws, hipStream_t st);
// The chain on a prepared workspace: one kernel launch.
hipError_t chain_persistent_run(const dfssm_layer* layers, int n_layers, const int8_t* q0, const float* s0,
                                float* y_all, void* ws, hipStream_t st);
// The loading schedule of chain_persistent alone (a diagnostic: no
// arithmetic, no exchange, nothing written outside LDS).
hipError_t chain_stream_run(const dfssm_layer* layers, int n_layers, void* ws, hipStream_t st);
// Zeroes `words` 64-bit words at p with a fill kernel (capture-safe).
// The fused decode step at one token (dfssm_step.hip).  Its workspace region
// (bytes; 0 when the model is not the shape it takes) holds its table, the
// table's fingerprint, the exchange words, a status word, the epoch words,
// the gathered embedding row u0 and the final residual row u_fin (offsets
// relative to the region).
struct StepFusedInfo {
  bool ok;
  size_t bytes, off_hash, off_ex, off_status, off_epoch, off_u0, off_ufin;
  int64_t ex_words;
  int n_linears;
  uint64_t fingerprint;
};
StepFusedInfo step_fused_info(const dfssm_mamba2_model* md);
hipError_t step_fused_prepare(const dfssm_mamba2_model* md, void* ws, hipStream_t st);
// two_hop: the input maxima always take the second exchange (for tests;
// results are the same bits either way)
hipError_t step_fused_run(const StepFusedInfo& f, float eps, int64_t step, float* conv_ring, float* ssm_state,
                          void* ws, bool two_hop, hipStream_t st);

hipError_t launch_zero_words(uint64_t* p, int64_t words, hipStream_t st);

// One launch reading `bytes` (a multiple of 16) from p; the XOR of the
// read_floor_sink_words(bytes) words it stores to sink is the XOR of every
// 32-bit word read.  bytes == 0: an empty launch.
int64_t read_floor_sink_words(int64_t bytes);
hipError_t launch_read_floor(const void* p, int64_t bytes, uint32_t* sink, hipStream_t st);

// The exchange ping-pong diagnostic's workspace: 256 x 64 words, 256 tick
// counts, the give-up flag.
constexpr size_t kPingWordsBytes = 256 * 64 * 8, kPingTicksBytes = 256 * 8;
constexpr size_t kPingBytes = kPingWordsBytes + kPingTicksBytes + 256;
hipError_t launch_exchange_pingpong(int npairs, int iters, bool fence, void* ws, hipStream_t st);

}  // namespace dfssm

// ------------------------------------------------------------ device helpers
namespace dfssm_dev {

// Signed base-256 digits of v with every digit in [-128, 127]:
// v = d0 + 256*d1 + 65536*d2 + 16777216*d3, valid for |v| < 2^31 - 2^24.
__device__ __forceinline__ void split_limbs(int32_t v, int8_t d[4]) {
#pragma unroll
  for (int t = 0; t < 3; ++t) {
    int8_t lo = (int8_t)(v & 0xff);
    d[t] = lo;
    v = (v - (int32_t)lo) >> 8;  // exact: v - lo is a multiple of 256
  }
  d[3] = (int8_t)v;
}

// The fixed-order fp32 output scaling y = s*(alpha*fs + beta*fb) with
// acc_b = hi*2^16 + lo.  fb is the int64 acc_b rounded once to fp32: the
// fp64 value hi*65536 + lo is exact (|acc_b| < 2^53), so converting it to
// fp32 is the single round-to-nearest-even of the integer.  The library is
// compiled with -ffp-contract=off, so no multiply-add fuses.
__device__ __forceinline__ float epilogue(float s, float alpha, float beta, int32_t acc_s,
                                          int32_t hi, int32_t lo, bool lora) {
  float fs = (float)acc_s;
  float u = alpha * fs;
  float w = u;
  if (lora) {
    // one fused multiply-add: hi*2^16 + lo is exact in fp64 either way
    double db = __builtin_fma((double)hi, 65536.0, (double)lo);
    float fb = (float)db;
    float v = beta * fb;
    w = u + v;
  }
  return s * w;
}


// Device-side epoch of a kernel's exchange words, kept in kEpochGroups words
// {epoch:32, arrivals:32} kEpochStride words apart: each of a launch's
// `arrivals` members (index i) arrives once with a fetch-add on word
// i % kEpochGroups, which hands it the epoch; the last member of each word
// moves it on to {epoch + 1, 0}, and member 0 moves on the words no member
// uses.  All words start at {0, 0}, so they stay equal between launches.
// Member i's arrival on its epoch word: returns the word before it.
__device__ __forceinline__ uint64_t arrive(uint64_t* ep, int i) {
  return __hip_atomic_fetch_add(ep + (i % dfssm::kEpochGroups) * dfssm::kEpochStride, 1ull, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
}
// Tag of the words of the call whose arrival returned `old`: below 2^31
// and never 0, so zeroed memory never validates.
__device__ __forceinline__ uint32_t epoch_tag(uint64_t old) {
  const uint32_t t = ((uint32_t)(old >> 32) + 1u) & 0x7fffffffu;
  return t ? t : 1u;
}
// After member i's arrival returned `old`: the last member of its word
// moves that word on to {epoch + 1, 0} (every other arrival of the call on
// it precedes this one, so none reads the new epoch); member 0 does the
// same for the words no member uses (calls of fewer than 64 members).
__device__ __forceinline__ void advance_if_last(uint64_t* ep, int i, uint64_t old, int arrivals) {
  constexpr int G = dfssm::kEpochGroups;
  const int g = i % G;
  const int members = arrivals / G + (g < arrivals % G ? 1 : 0);
  const uint64_t next = (uint64_t)((uint32_t)(old >> 32) + 1u) << 32;
  if ((uint32_t)old == (uint32_t)(members - 1))
    __hip_atomic_store(ep + g * dfssm::kEpochStride, next, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (i == 0)
    for (int e = arrivals; e < G; ++e)
      __hip_atomic_store(ep + e * dfssm::kEpochStride, next, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace dfssm_dev
