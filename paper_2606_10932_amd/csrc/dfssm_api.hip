// dfssm_api.hip -- host side of include/dfssm.h: argument validation,
// workspace sizing, kernel-family dispatch, the chain driver and error
// reporting.  Validation is pure host code that runs before any HIP call,
// so a rejected call enqueues nothing.
#include <float.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <vector>

#include "dfssm_internal.hpp"
#include "dfssm_int4.hpp"
#include "dfssm_mamba.hpp"

namespace {

thread_local char g_last_error[512] = "";

void clear_error() { g_last_error[0] = 0; }

dfssm_status fail(dfssm_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

dfssm_status device_fail(hipError_t e, const char* what) {
  return fail(DFSSM_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

dfssm_status check_linear(int64_t M, int64_t K, int64_t N, int64_t r) {
  if (K <= 0 || K % 32 != 0 || K > dfssm::kMaxK)
    return fail(DFSSM_ERR_SHAPE, "K=%lld must be a positive multiple of 32 and <= %lld",
                (long long)K, (long long)dfssm::kMaxK);
  if (M < 0 || N < 0) return fail(DFSSM_ERR_SHAPE, "M=%lld and N=%lld must be >= 0", (long long)M, (long long)N);
  if (M > INT32_MAX / 2 || N > INT32_MAX / 2)
    return fail(DFSSM_ERR_SHAPE, "M=%lld or N=%lld too large", (long long)M, (long long)N);
  if (r < 0 || r > dfssm::kMaxRank)
    return fail(DFSSM_ERR_SHAPE, "r=%lld must be in [0, %lld]", (long long)r, (long long)dfssm::kMaxRank);
  return DFSSM_OK;
}

struct Ptr {
  const void* p;
  const char* name;
};

dfssm_status check_ptrs(std::initializer_list<Ptr> required, std::initializer_list<Ptr> optional) {
  for (const Ptr& x : required) {
    if (!x.p) return fail(DFSSM_ERR_NULL, "%s is NULL", x.name);
    if (!aligned16(x.p)) return fail(DFSSM_ERR_ALIGN, "%s is not 16-byte aligned", x.name);
  }
  for (const Ptr& x : optional)
    if (x.p && !aligned16(x.p)) return fail(DFSSM_ERR_ALIGN, "%s is not 16-byte aligned", x.name);
  return DFSSM_OK;
}

std::atomic<int> g_switch[6];  // dfssm_test_switch values, index = switch id

size_t linear_ws_bytes(int64_t M, int64_t K, int64_t r) {
  return dfssm::carve_linear_workspace(nullptr, M, K, r).bytes;
}

// Kernel family of the automatic path: the popcount GEMV up to kDecodeM0
// tokens (none by default); the one-launch few-token MFMA kernel up to
// kSkinnyMaxTokens; above, whichever of the few-token kernel in 64-token
// blocks and the prefill path a cost model puts lower (us), fitted on
// MI355X to the 130M, 1.3B and 2.7B projections at 33 to 512 tokens:
//   few-token  9.5 + 0.013 B (0.76 + K/2048) + 1.5 ceil(M/64) K/2048,
//              B = ceil(M/16) ceil(N/16) / 4
//   prefill    dfssm::prefill_cost_us (its K-loop stages, its slices and
//              the form its tiling takes)
// The few-token kernel's cost grows with its 16-token tiles (a partly
// filled 64-token block costs its tiles) and its 64-token blocks.  On the
// 72 measured cases the chosen kernel is within 0.9 us (and 5%) of the
// faster one.
int auto_path(int64_t M, int64_t K, int64_t N) {
  if (M <= dfssm::kDecodeM0) return DFSSM_PATH_DECODE;
  if (M <= dfssm::kSkinnyMaxTokens) return DFSSM_PATH_MFMA_FEW;
  if (M > dfssm::kSkinnyChunkedMaxTokens) return DFSSM_PATH_MFMA;
  const double k2 = (double)K / 2048.0;
  const double B = (double)dfssm::ceil_div(M, 16) * (double)dfssm::ceil_div(N, 16) / 4.0;
  const double few = 9.5 + 0.013 * B * (0.76 + k2) + 1.5 * (double)dfssm::ceil_div(M, 64) * k2;
  return few <= dfssm::prefill_cost_us(M, K, N) ? DFSSM_PATH_MFMA_FEW : DFSSM_PATH_MFMA;
}

// Kernel family for a linear (path already chosen or AUTO).
hipError_t launch_linear(int path, const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N, int64_t r,
                         const uint32_t* w_bits, const float* alpha, const int8_t* A, const int8_t* B,
                         const float* beta, float* y, int32_t* acc_s, int32_t* acc_a, int64_t* acc_b,
                         const dfssm::LinearWorkspace& ws, hipStream_t hs) {
  if (path == DFSSM_PATH_AUTO) path = auto_path(M, K, N);
  if (path == DFSSM_PATH_DECODE)
    return dfssm::launch_decode_linear(q, s, M, K, N, r, w_bits, alpha, A, B, beta, y, acc_s, acc_a, acc_b, ws,
                                       hs);
  if (path == DFSSM_PATH_MFMA_FEW)
    return dfssm::launch_skinny_linear(q, s, M, K, N, r, w_bits, alpha, A, B, beta, y, acc_s, acc_a, acc_b, ws,
                                       hs);
  return dfssm::launch_mfma_linear(q, s, M, K, N, r, w_bits, alpha, A, B, beta, y, acc_s, acc_a, acc_b, ws, hs);
}

// The int4 linear after validation: the few-token kernel reads the packed
// factors itself; the other paths run the int8 kernels on factors expanded
// into the workspace (linear_i4_workspace_bytes of it).
hipError_t launch_linear_i4(int path, const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N, int64_t r,
                            const uint32_t* w_bits, const float* alpha, const uint8_t* A4, const uint8_t* B4,
                            const float* beta, float* y, int32_t* acc_s, int32_t* acc_a, int64_t* acc_b,
                            void* workspace, hipStream_t hs) {
  dfssm::LinearWorkspace ws = dfssm::carve_linear_workspace(workspace, M, K, r);
  if (path == DFSSM_PATH_AUTO) path = auto_path(M, K, N);
  hipError_t e;
  if (path == DFSSM_PATH_MFMA_FEW || r == 0) {
    if (path == DFSSM_PATH_MFMA_FEW)
      e = dfssm::launch_skinny_linear_i4(q, s, M, K, N, r, w_bits, alpha, A4, B4, beta, y, acc_s, acc_a, acc_b, ws,
                                         hs);
    else
      e = launch_linear(path, q, s, M, K, N, 0, w_bits, alpha, nullptr, nullptr, nullptr, y, acc_s, acc_a, acc_b,
                        ws, hs);
  } else {
    // the int8 kernels on factors expanded into the workspace
    char* extra = static_cast<char*>(workspace) + dfssm::linear_i4_extra_offset(M, K, r);
    int8_t* A8 = reinterpret_cast<int8_t*>(extra);
    int8_t* B8 = reinterpret_cast<int8_t*>(extra + (((size_t)(r * K) + 255) & ~(size_t)255));
    e = dfssm::launch_unpack_int4(A4, r * K, A8, hs);
    if (e == hipSuccess) e = dfssm::launch_unpack_int4(B4, N * r, B8, hs);
    if (e == hipSuccess)
      e = launch_linear(path, q, s, M, K, N, r, w_bits, alpha, A8, B8, beta, y, acc_s, acc_a, acc_b, ws, hs);
  }
  return e;
}

}  // namespace

namespace dfssm {
int test_switch(int which) { return which > 0 && which < 6 ? g_switch[which].load(std::memory_order_relaxed) : 0; }
}  // namespace dfssm

extern "C" {

dfssm_status dfssm_test_switch(int which, int value) {
  clear_error();
  bool ok = false;
  switch (which) {
    case DFSSM_TEST_LOCAL_LORA: ok = value == 0 || value == 1; break;
    case DFSSM_TEST_PREFILL_KERNEL: ok = value == 0 || value == 4 || value == 8; break;
    case DFSSM_TEST_LM_HEAD_MFMA_TOKENS: ok = value >= 0; break;
    case DFSSM_TEST_STEP_PER_KERNEL: ok = value >= 0 && value <= 2; break;
    case DFSSM_TEST_LM_HEAD_TILED_TOKENS: ok = value >= 0; break;
    default: break;
  }
  if (!ok) return fail(DFSSM_ERR_SHAPE, "test switch %d: value %d", which, value);
  g_switch[which].store(value, std::memory_order_relaxed);
  return DFSSM_OK;
}

const char* dfssm_version(void) { return "dfssm-gfx950 0.1"; }

const char* dfssm_status_string(int status) {
  switch (status) {
    case DFSSM_OK: return "ok";
    case DFSSM_ERR_NULL: return "null pointer";
    case DFSSM_ERR_SHAPE: return "invalid shape";
    case DFSSM_ERR_ALIGN: return "misaligned pointer";
    case DFSSM_ERR_WORKSPACE: return "workspace too small";
    case DFSSM_ERR_DEVICE: return "device error";
    case DFSSM_ERR_UNSUPPORTED: return "unsupported";
    default: return "unknown status";
  }
}

const char* dfssm_last_error(void) { return g_last_error; }

dfssm_status dfssm_quantize_act(const void* x, int x_dtype, int64_t M, int64_t K, int64_t ldx,
                                int8_t* q, float* s, void* stream) {
  clear_error();
  if (x_dtype != DFSSM_F16 && x_dtype != DFSSM_F32) return fail(DFSSM_ERR_SHAPE, "x_dtype=%d", x_dtype);
  if (K <= 0 || K % 32 != 0 || K > dfssm::kMaxK)
    return fail(DFSSM_ERR_SHAPE, "K=%lld must be a positive multiple of 32 and <= %lld", (long long)K,
                (long long)dfssm::kMaxK);
  if (M < 0 || M > INT32_MAX / 2) return fail(DFSSM_ERR_SHAPE, "M=%lld", (long long)M);
  if (ldx < K) return fail(DFSSM_ERR_SHAPE, "ldx=%lld < K=%lld", (long long)ldx, (long long)K);
  if (M == 0) return DFSSM_OK;
  if (!x) return fail(DFSSM_ERR_NULL, "x is NULL");
  const size_t esz = x_dtype == DFSSM_F16 ? 2 : 4;
  if (reinterpret_cast<uintptr_t>(x) % esz) return fail(DFSSM_ERR_ALIGN, "x is not element aligned");
  dfssm_status st = check_ptrs({{q, "q"}, {s, "s"}}, {});
  if (st != DFSSM_OK) return st;
  hipError_t e = dfssm::launch_quantize(x, x_dtype, M, K, ldx, q, s, 0, (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "quantize launch");
}

size_t dfssm_linear_workspace_bytes(int64_t M, int64_t K, int64_t N, int64_t r) {
  (void)N;
  if (M < 0 || K <= 0 || r < 0) return 0;
  return linear_ws_bytes(M, K, r);
}

dfssm_status dfssm_scaffold_lora_linear_ex(const int8_t* q, const float* s, int64_t M, int64_t K,
                                           int64_t N, int64_t r, const uint32_t* w_bits,
                                           const float* alpha, const int8_t* A, const int8_t* B,
                                           const float* beta, float* y, int path, int32_t* acc_s,
                                           int32_t* acc_a, int64_t* acc_b, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  clear_error();
  dfssm_status st = check_linear(M, K, N, r);
  if (st != DFSSM_OK) return st;
  if (path != DFSSM_PATH_AUTO && path != DFSSM_PATH_DECODE && path != DFSSM_PATH_MFMA &&
      path != DFSSM_PATH_MFMA_FEW)
    return fail(DFSSM_ERR_SHAPE, "path=%d", path);
  if (path == DFSSM_PATH_MFMA_FEW && M > dfssm::kSkinnyChunkedMaxTokens)
    return fail(DFSSM_ERR_UNSUPPORTED, "path=%d takes M <= %lld, got M=%lld", path,
                (long long)dfssm::kSkinnyChunkedMaxTokens, (long long)M);
  if (M == 0 || N == 0) return DFSSM_OK;
  st = check_ptrs({{q, "q"}, {s, "s"}, {w_bits, "w_bits"}, {alpha, "alpha"}, {workspace, "workspace"}},
                  {{y, "y"}, {acc_s, "acc_s"}, {acc_a, "acc_a"}, {acc_b, "acc_b"}});
  if (st != DFSSM_OK) return st;
  if (r > 0) {
    st = check_ptrs({{A, "A"}, {B, "B"}, {beta, "beta"}}, {});
    if (st != DFSSM_OK) return st;
  }
  const size_t need = linear_ws_bytes(M, K, r);
  if (workspace_bytes < need)
    return fail(DFSSM_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, need);
  dfssm::LinearWorkspace ws = dfssm::carve_linear_workspace(workspace, M, K, r);
  hipError_t e = launch_linear(path, q, s, M, K, N, r, w_bits, alpha, A, B, beta, y, acc_s, acc_a, acc_b, ws,
                               (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "linear launch");
}

size_t dfssm_linear_i4_workspace_bytes(int64_t M, int64_t K, int64_t N, int64_t r) {
  if (M < 0 || K <= 0 || N < 0 || r < 0) return 0;
  return dfssm::linear_i4_workspace_bytes(M, K, N, r);
}

dfssm_status dfssm_scaffold_lora_linear_i4(const int8_t* q, const float* s, int64_t M, int64_t K, int64_t N,
                                           int64_t r, const uint32_t* w_bits, const float* alpha,
                                           const uint8_t* A4, const uint8_t* B4, const float* beta, float* y,
                                           int path, int32_t* acc_s, int32_t* acc_a, int64_t* acc_b,
                                           void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  dfssm_status st = check_linear(M, K, N, r);
  if (st != DFSSM_OK) return st;
  if (r % 2 != 0) return fail(DFSSM_ERR_SHAPE, "r=%lld must be even for packed int4 factors", (long long)r);
  if (path != DFSSM_PATH_AUTO && path != DFSSM_PATH_DECODE && path != DFSSM_PATH_MFMA &&
      path != DFSSM_PATH_MFMA_FEW)
    return fail(DFSSM_ERR_SHAPE, "path=%d", path);
  if (path == DFSSM_PATH_MFMA_FEW && M > dfssm::kSkinnyChunkedMaxTokens)
    return fail(DFSSM_ERR_UNSUPPORTED, "path=%d takes M <= %lld, got M=%lld", path,
                (long long)dfssm::kSkinnyChunkedMaxTokens, (long long)M);
  if (M == 0 || N == 0) return DFSSM_OK;
  st = check_ptrs({{q, "q"}, {s, "s"}, {w_bits, "w_bits"}, {alpha, "alpha"}, {workspace, "workspace"}},
                  {{y, "y"}, {acc_s, "acc_s"}, {acc_a, "acc_a"}, {acc_b, "acc_b"}});
  if (st != DFSSM_OK) return st;
  if (r > 0) {
    st = check_ptrs({{A4, "A4"}, {B4, "B4"}, {beta, "beta"}}, {});
    if (st != DFSSM_OK) return st;
  }
  const size_t need = dfssm::linear_i4_workspace_bytes(M, K, N, r);
  if (workspace_bytes < need)
    return fail(DFSSM_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, need);
  const hipError_t e = launch_linear_i4(path, q, s, M, K, N, r, w_bits, alpha, A4, B4, beta, y, acc_s, acc_a,
                                        acc_b, workspace, (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "int4 linear launch");
}

dfssm_status dfssm_scaffold_lora_linear(const int8_t* q, const float* s, int64_t M, int64_t K,
                                        int64_t N, int64_t r, const uint32_t* w_bits,
                                        const float* alpha, const int8_t* A, const int8_t* B,
                                        const float* beta, float* y, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  if (!y && M > 0 && N > 0) {
    clear_error();
    return fail(DFSSM_ERR_NULL, "y is NULL");
  }
  return dfssm_scaffold_lora_linear_ex(q, s, M, K, N, r, w_bits, alpha, A, B, beta, y,
                                       DFSSM_PATH_AUTO, nullptr, nullptr, nullptr, workspace,
                                       workspace_bytes, stream);
}

// ---------------------------------------------------------------- no allocation
// Scratch of dfssm_scaffold_lora_linear_noalloc: the linear's workspace as a
// device array of this library, zero at load (the state the workspace
// contract asks for), one copy per GPU, shared by every call on that GPU.
constexpr size_t kScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on device `dev`, looked up once per device
// with that device current.  On the host, `scratch` names a host-side
// stand-in; kernels get this address instead.
hipError_t scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    void* p = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" dfssm_status dfssm_scaffold_lora_linear_noalloc(const int8_t* q, const float* s, int64_t M, int64_t K,
                                                           int64_t N, int64_t r, const uint32_t* w_bits,
                                                           const float* alpha, const int8_t* A, const int8_t* B,
                                                           const float* beta, float* y, void* stream) {
  clear_error();
  dfssm_status st = check_linear(M, K, N, r);
  if (st != DFSSM_OK) return st;
  if (M == 0 || N == 0) return DFSSM_OK;
  st = check_ptrs({{q, "q"}, {s, "s"}, {w_bits, "w_bits"}, {alpha, "alpha"}, {y, "y"}}, {});
  if (st != DFSSM_OK) return st;
  if (r > 0) {
    st = check_ptrs({{A, "A"}, {B, "B"}, {beta, "beta"}}, {});
    if (st != DFSSM_OK) return st;
  }
  const size_t need = linear_ws_bytes(M, K, r);
  if (need > kScratchBytes)
    return fail(DFSSM_ERR_WORKSPACE,
                "M=%lld K=%lld r=%lld needs %zu bytes of scratch; the allocation-free linear holds %zu "
                "(use dfssm_scaffold_lora_linear with a workspace)",
                (long long)M, (long long)K, (long long)r, need, kScratchBytes);
  hipStream_t hs = (hipStream_t)stream;
  int dev = 0;
  hipError_t e = hs ? hipStreamGetDevice(hs, &dev) : hipGetDevice(&dev);
  void* base = nullptr;
  if (e == hipSuccess) e = scratch_address(dev, &base);
  if (e != hipSuccess) return device_fail(e, "scratch address");
  dfssm::LinearWorkspace ws = dfssm::carve_linear_workspace(base, M, K, r);
  e = launch_linear(DFSSM_PATH_AUTO, q, s, M, K, N, r, w_bits, alpha, A, B, beta, y, nullptr, nullptr, nullptr, ws,
                    hs);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "linear launch");
}

extern "C" size_t dfssm_noalloc_scratch_bytes(void) { return kScratchBytes; }

// ---------------------------------------------------------------- chain
// Workspace of the host-sequenced chain: Q [M, Kmax] int8, s [M] fp32, one
// linear workspace sized for the largest layer.  Workspace of the persistent
// chain (M = 1): its layer table, fingerprint, exchange words, status word
// and epoch words (dfssm::chain_persistent_bytes).  The larger of the two is
// required.
struct ChainLayout {
  size_t off_s, off_lin, seq_bytes, pers_bytes;
  bool persistent;
};

static ChainLayout chain_layout(const dfssm_layer* layers, int n_layers, int64_t M) {
  ChainLayout c{};
  int64_t kmax = 0;
  for (int l = 0; l < n_layers; ++l) kmax = std::max(kmax, layers[l].K);
  size_t o = (size_t)dfssm::round_up(M * kmax, 256);
  c.off_s = o;
  o += (size_t)dfssm::round_up(M * 4, 256);
  c.off_lin = o;
  size_t lin = 0;
  for (int l = 0; l < n_layers; ++l) lin = std::max(lin, linear_ws_bytes(M, layers[l].K, layers[l].r));
  c.seq_bytes = o + lin;
  c.persistent = dfssm::chain_persistent_supported(layers, n_layers, M);
  c.pers_bytes = c.persistent ? dfssm::chain_persistent_bytes(layers, n_layers) : 0;
  return c;
}

static dfssm_status validate_chain(const dfssm_layer* layers, int n_layers, int64_t M) {
  if (n_layers < 0) return fail(DFSSM_ERR_SHAPE, "n_layers=%d", n_layers);
  if (n_layers == 0 || M == 0) return DFSSM_OK;
  if (!layers) return fail(DFSSM_ERR_NULL, "layers is NULL");
  if (M < 0 || M > 4) return fail(M < 0 ? DFSSM_ERR_SHAPE : DFSSM_ERR_UNSUPPORTED, "chain M=%lld (1..4)", (long long)M);
  for (int l = 0; l < n_layers; ++l) {
    const dfssm_layer& L = layers[l];
    char why[256];
    dfssm_status st = check_linear(M, L.K, L.N, L.r);
    if (st != DFSSM_OK) {
      snprintf(why, sizeof(why), "%s", g_last_error);
      return fail(st, "layer %d: %s", l, why);
    }
    if (L.N <= 0) return fail(DFSSM_ERR_SHAPE, "layer %d: N must be > 0", l);
    if (L.lora_bits != 0 && L.lora_bits != 8 && L.lora_bits != 4)
      return fail(DFSSM_ERR_SHAPE, "layer %d: lora_bits=%lld: 8 (or 0) or 4", l, (long long)L.lora_bits);
    if (L.lora_bits == 4 && L.r % 2 != 0)
      return fail(DFSSM_ERR_SHAPE, "layer %d: r=%lld must be even for packed int4 factors", l, (long long)L.r);
    if (l > 0 && L.K > layers[l - 1].N)
      return fail(DFSSM_ERR_SHAPE, "layer %d: K=%lld > previous N=%lld", l, (long long)L.K,
                  (long long)layers[l - 1].N);
    st = check_ptrs({{L.w_bits, "w_bits"}, {L.alpha, "alpha"}}, {});
    if (st == DFSSM_OK && L.r > 0) st = check_ptrs({{L.A, "A"}, {L.B, "B"}, {L.beta, "beta"}}, {});
    if (st != DFSSM_OK) {
      snprintf(why, sizeof(why), "%s", g_last_error);
      return fail(st, "layer %d: %s", l, why);
    }
  }
  return DFSSM_OK;
}

size_t dfssm_chain_workspace_bytes(const dfssm_layer* layers, int n_layers, int64_t M) {
  if (!layers || n_layers <= 0 || M <= 0) return 0;
  ChainLayout c = chain_layout(layers, n_layers, M);
  return std::max(c.seq_bytes, c.pers_bytes);
}

static dfssm_status chain_common(const dfssm_layer* layers, int n_layers, int64_t M, void* workspace,
                                 size_t workspace_bytes, ChainLayout* c) {
  dfssm_status st = check_ptrs({{workspace, "workspace"}}, {});
  if (st != DFSSM_OK) return st;
  *c = chain_layout(layers, n_layers, M);
  const size_t need = std::max(c->seq_bytes, c->pers_bytes);
  if (workspace_bytes < need)
    return fail(DFSSM_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, need);
  return DFSSM_OK;
}

dfssm_status dfssm_chain_prepare(const dfssm_layer* layers, int n_layers, int64_t M, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  clear_error();
  dfssm_status st = validate_chain(layers, n_layers, M);
  if (st != DFSSM_OK || n_layers == 0 || M == 0) return st;
  ChainLayout c;
  st = chain_common(layers, n_layers, M, workspace, workspace_bytes, &c);
  if (st != DFSSM_OK) return st;
  char* base = static_cast<char*>(workspace);
  hipError_t e;
  if (c.persistent)
    e = dfssm::chain_persistent_prepare(layers, n_layers, workspace, (hipStream_t)stream);
  else  // the host-sequenced chain: its linears' epoch words and exchange words
    e = dfssm::launch_zero_words(reinterpret_cast<uint64_t*>(base + c.off_lin),
                                 (int64_t)(dfssm::kLinearStateBytes / 8), (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "chain prepare launch");
}

dfssm_status dfssm_chain_run(const dfssm_layer* layers, int n_layers, int64_t M, const int8_t* q0,
                             const float* s0, float* y_all, void* workspace, size_t workspace_bytes,
                             void* stream) {
  clear_error();
  dfssm_status st = validate_chain(layers, n_layers, M);
  if (st != DFSSM_OK || n_layers == 0 || M == 0) return st;
  st = check_ptrs({{q0, "q0"}, {s0, "s0"}, {y_all, "y_all"}}, {});
  if (st != DFSSM_OK) return st;
  ChainLayout c;
  st = chain_common(layers, n_layers, M, workspace, workspace_bytes, &c);
  if (st != DFSSM_OK) return st;
  hipStream_t hs = (hipStream_t)stream;
  char* base = static_cast<char*>(workspace);

  if (c.persistent) {
    hipError_t e = dfssm::chain_persistent_run(layers, n_layers, q0, s0, y_all, workspace, hs);
    return e == hipSuccess ? DFSSM_OK : device_fail(e, "chain run launch");
  }

  int8_t* qbuf = reinterpret_cast<int8_t*>(base);
  float* sbuf = reinterpret_cast<float*>(base + c.off_s);
  float* y_prev = nullptr;
  float* y_cur = y_all;
  for (int l = 0; l < n_layers; ++l) {
    const dfssm_layer& L = layers[l];
    const int8_t* ql = q0;
    const float* sl = s0;
    if (l > 0) {
      hipError_t e = dfssm::launch_quantize(y_prev, DFSSM_F32, M, L.K, layers[l - 1].N, qbuf, sbuf, 1, hs);
      if (e != hipSuccess) return device_fail(e, "chain quantize launch");
      ql = qbuf;
      sl = sbuf;
    }
    dfssm::LinearWorkspace ws = dfssm::carve_linear_workspace(base + c.off_lin, M, L.K, L.r);
    // M <= 4: int4 factors go to the few-token kernel, which reads them packed
    hipError_t e = L.lora_bits == 4 && L.r > 0
                       ? dfssm::launch_skinny_linear_i4(ql, sl, M, L.K, L.N, L.r, L.w_bits, L.alpha,
                                                        reinterpret_cast<const uint8_t*>(L.A),
                                                        reinterpret_cast<const uint8_t*>(L.B), L.beta, y_cur,
                                                        nullptr, nullptr, nullptr, ws, hs)
                       : launch_linear(DFSSM_PATH_AUTO, ql, sl, M, L.K, L.N, L.r, L.w_bits, L.alpha, L.A, L.B,
                                       L.beta, y_cur, nullptr, nullptr, nullptr, ws, hs);
    if (e != hipSuccess) return device_fail(e, "chain linear launch");
    y_prev = y_cur;
    y_cur += M * L.N;
  }
  return DFSSM_OK;
}

dfssm_status dfssm_scaffold_lora_chain(const dfssm_layer* layers, int n_layers, int64_t M,
                                       const int8_t* q0, const float* s0, float* y_all,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  // everything the run checks is checked before the prepare enqueues
  clear_error();
  dfssm_status st = validate_chain(layers, n_layers, M);
  if (st != DFSSM_OK || n_layers == 0 || M == 0) return st;
  st = check_ptrs({{q0, "q0"}, {s0, "s0"}, {y_all, "y_all"}}, {});
  if (st != DFSSM_OK) return st;
  ChainLayout c;
  st = chain_common(layers, n_layers, M, workspace, workspace_bytes, &c);
  if (st != DFSSM_OK) return st;
  st = dfssm_chain_prepare(layers, n_layers, M, workspace, workspace_bytes, stream);
  if (st != DFSSM_OK) return st;
  return dfssm_chain_run(layers, n_layers, M, q0, s0, y_all, workspace, workspace_bytes, stream);
}

dfssm_status dfssm_chain_status(const dfssm_layer* layers, int n_layers, int64_t M, const void* workspace,
                                size_t workspace_bytes, unsigned* status, void* stream) {
  clear_error();
  if (!status) return fail(DFSSM_ERR_NULL, "status is NULL");
  *status = 0;
  dfssm_status st = validate_chain(layers, n_layers, M);
  if (st != DFSSM_OK || n_layers == 0 || M == 0) return st;
  ChainLayout c;
  st = chain_common(layers, n_layers, M, const_cast<void*>(workspace), workspace_bytes, &c);
  if (st != DFSSM_OK) return st;
  if (!c.persistent) return DFSSM_OK;
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e == hipSuccess)
    e = hipMemcpy(status, static_cast<const char*>(workspace) + dfssm::chain_status_offset(layers, n_layers),
                  sizeof(unsigned), hipMemcpyDeviceToHost);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "chain status read");
}

dfssm_status dfssm_chain_stream_floor(const dfssm_layer* layers, int n_layers, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  clear_error();
  dfssm_status st = validate_chain(layers, n_layers, 1);
  if (st != DFSSM_OK || n_layers == 0) return st;
  ChainLayout c;
  st = chain_common(layers, n_layers, 1, workspace, workspace_bytes, &c);
  if (st != DFSSM_OK) return st;
  if (!c.persistent) return fail(DFSSM_ERR_UNSUPPORTED, "the persistent chain kernel does not take these layers");
  hipError_t e = dfssm::chain_stream_run(layers, n_layers, workspace, (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "chain stream launch");
}

size_t dfssm_exchange_pingpong_bytes(void) { return dfssm::kPingBytes; }

dfssm_status dfssm_exchange_pingpong(int npairs, int iters, int fence, void* workspace, size_t workspace_bytes,
                                     double* ns_per_round_trip, void* stream) {
  clear_error();
  if (!ns_per_round_trip) return fail(DFSSM_ERR_NULL, "ns_per_round_trip is NULL");
  *ns_per_round_trip = 0.0;
  if (npairs < 1 || npairs > 128 || iters < 1 || iters > 100000)
    return fail(DFSSM_ERR_SHAPE, "npairs=%d (1..128), iters=%d (1..100000)", npairs, iters);
  const dfssm_status st = check_ptrs({{workspace, "workspace"}}, {});
  if (st != DFSSM_OK) return st;
  if (workspace_bytes < dfssm::kPingBytes)
    return fail(DFSSM_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, dfssm::kPingBytes);
  hipStream_t hs = (hipStream_t)stream;
  hipError_t e = dfssm::launch_exchange_pingpong(npairs, iters, fence != 0, workspace, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  std::vector<int64_t> ticks(256);
  unsigned failed = 0;
  const char* b = static_cast<const char*>(workspace);
  if (e == hipSuccess)
    e = hipMemcpy(ticks.data(), b + dfssm::kPingWordsBytes, 256 * 8, hipMemcpyDeviceToHost);
  if (e == hipSuccess)
    e = hipMemcpy(&failed, b + dfssm::kPingWordsBytes + dfssm::kPingTicksBytes, 4, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return device_fail(e, "exchange ping-pong");
  if (failed) return fail(DFSSM_ERR_DEVICE, "exchange ping-pong: a bounded wait gave up");
  // the pinging side's loop, median over the pairs, in ns (100 MHz ticks)
  std::vector<int64_t> ping;
  for (int p = 0; p < npairs; ++p) ping.push_back(ticks[2 * p]);
  std::sort(ping.begin(), ping.end());
  *ns_per_round_trip = (double)ping[ping.size() / 2] * 10.0 / iters;
  return DFSSM_OK;
}

size_t dfssm_read_floor_sink_words(size_t bytes) { return (size_t)dfssm::read_floor_sink_words((int64_t)bytes); }

dfssm_status dfssm_read_floor(const void* p, size_t bytes, uint32_t* sink, size_t sink_words, void* stream) {
  clear_error();
  if (bytes % 16 != 0) return fail(DFSSM_ERR_SHAPE, "bytes=%zu must be a multiple of 16", bytes);
  if (!sink) return fail(DFSSM_ERR_NULL, "sink is NULL");
  if (sink_words < (size_t)dfssm::read_floor_sink_words((int64_t)bytes))
    return fail(DFSSM_ERR_WORKSPACE, "sink holds %zu words < %lld needed", sink_words,
                (long long)dfssm::read_floor_sink_words((int64_t)bytes));
  if (reinterpret_cast<uintptr_t>(sink) % 4 != 0) return fail(DFSSM_ERR_ALIGN, "sink is not 4-byte aligned");
  if (bytes > 0) {
    const dfssm_status st = check_ptrs({{p, "p"}}, {});
    if (st != DFSSM_OK) return st;
  }
  const hipError_t e = dfssm::launch_read_floor(p, (int64_t)bytes, sink, (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "read floor launch");
}

dfssm_status dfssm_embed_gather(const int8_t* E, const float* scale, int64_t V, int64_t d, const int32_t* tok,
                                int64_t M, float* x, void* stream) {
  clear_error();
  if (d <= 0 || d % 16 != 0 || d > dfssm::kMaxK)
    return fail(DFSSM_ERR_SHAPE, "d=%lld must be a positive multiple of 16 and <= %lld", (long long)d,
                (long long)dfssm::kMaxK);
  if (V <= 0 || V > INT32_MAX / 2) return fail(DFSSM_ERR_SHAPE, "V=%lld must be in [1, 2^30)", (long long)V);
  if (M < 0 || M > INT32_MAX / 2) return fail(DFSSM_ERR_SHAPE, "M=%lld", (long long)M);
  if (M == 0) return DFSSM_OK;
  dfssm_status st = check_ptrs({{E, "E"}, {scale, "scale"}, {tok, "tok"}, {x, "x"}}, {});
  if (st != DFSSM_OK) return st;
  hipError_t e = dfssm::launch_embed_gather(E, scale, V, d, tok, M, x, (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "embed gather launch");
}

dfssm_status dfssm_lm_head(const int8_t* q, const float* s, int64_t M, int64_t d, const int8_t* E,
                           const float* scale, int64_t V, float* logits, int32_t* acc, void* stream) {
  clear_error();
  if (d <= 0 || d % 16 != 0 || d > dfssm::kLmHeadMaxD)
    return fail(DFSSM_ERR_SHAPE, "d=%lld must be a positive multiple of 16 and <= %lld", (long long)d,
                (long long)dfssm::kLmHeadMaxD);
  if (V < 0 || V > INT32_MAX / 2) return fail(DFSSM_ERR_SHAPE, "V=%lld must be in [0, 2^30)", (long long)V);
  if (M < 0 || M > INT32_MAX / 2) return fail(DFSSM_ERR_SHAPE, "M=%lld", (long long)M);
  if (M == 0 || V == 0) return DFSSM_OK;
  dfssm_status st = check_ptrs({{q, "q"}, {s, "s"}, {E, "E"}, {scale, "scale"}}, {{logits, "logits"}, {acc, "acc"}});
  if (st != DFSSM_OK) return st;
  if (!logits && !acc) return fail(DFSSM_ERR_NULL, "logits and acc are both NULL");
  hipError_t e = dfssm::launch_lm_head(q, s, M, d, E, scale, V, logits, acc, (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "lm head launch");
}

dfssm_status dfssm_add_rmsnorm_quant(const float* u, const float* delta, const float* w, float eps, int64_t M,
                                     int64_t d, float* u_out, int8_t* q, float* s, void* stream) {
  clear_error();
  if (d <= 0 || d % 4 != 0 || d > dfssm::kNormMaxD)
    return fail(DFSSM_ERR_SHAPE, "d=%lld must be a positive multiple of 4 and <= %lld", (long long)d,
                (long long)dfssm::kNormMaxD);
  if (M < 0 || M > INT32_MAX / 2) return fail(DFSSM_ERR_SHAPE, "M=%lld", (long long)M);
  if (!(eps >= 0.0f) || eps > FLT_MAX) return fail(DFSSM_ERR_SHAPE, "eps must be finite and >= 0");
  if (M == 0) return DFSSM_OK;
  dfssm_status st = check_ptrs({{u, "u"}, {w, "w"}, {q, "q"}, {s, "s"}}, {{delta, "delta"}, {u_out, "u_out"}});
  if (st != DFSSM_OK) return st;
  hipError_t e = dfssm::launch_add_rmsnorm_quant(u, delta, w, eps, M, d, u_out, q, s, (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "rmsnorm launch");
}

dfssm_status dfssm_gate_norm_quant(const float* y, const float* z, int64_t ldz, const float* w, float eps,
                                   int64_t M, int64_t d, int8_t* q, float* s, void* stream) {
  clear_error();
  if (d <= 0 || d % 4 != 0 || d > dfssm::kNormMaxD)
    return fail(DFSSM_ERR_SHAPE, "d=%lld must be a positive multiple of 4 and <= %lld", (long long)d,
                (long long)dfssm::kNormMaxD);
  if (ldz < d || ldz % 4 != 0) return fail(DFSSM_ERR_SHAPE, "ldz=%lld must be >= d and a multiple of 4", (long long)ldz);
  if (M < 0 || M > INT32_MAX / 2) return fail(DFSSM_ERR_SHAPE, "M=%lld", (long long)M);
  if (!(eps >= 0.0f) || eps > FLT_MAX) return fail(DFSSM_ERR_SHAPE, "eps must be finite and >= 0");
  if (M == 0) return DFSSM_OK;
  dfssm_status st = check_ptrs({{y, "y"}, {z, "z"}, {w, "w"}, {q, "q"}, {s, "s"}}, {});
  if (st != DFSSM_OK) return st;
  hipError_t e = dfssm::launch_gate_norm_quant(y, z, ldz, w, eps, M, d, q, s, (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "gate norm launch");
}

dfssm_status dfssm_ssm_step(const float* zxbcdt, int64_t ld, int64_t M, int64_t d_inner, int64_t d_state,
                            int64_t headdim, int64_t step, float* conv_ring, const float* conv_w,
                            const float* conv_b, const float* dt_bias, const float* A_log, const float* D,
                            float* ssm_state, float* y, float* xbc, void* stream) {
  clear_error();
  if (headdim != 64) return fail(DFSSM_ERR_UNSUPPORTED, "headdim=%lld: heads of 64 channels only", (long long)headdim);
  if (d_state != 64 && d_state != 128)
    return fail(DFSSM_ERR_UNSUPPORTED, "d_state=%lld: 64 or 128 only", (long long)d_state);
  if (d_inner <= 0 || d_inner % headdim != 0 || d_inner > 65536)
    return fail(DFSSM_ERR_SHAPE, "d_inner=%lld must be a positive multiple of headdim and <= 65536",
                (long long)d_inner);
  const int64_t H = d_inner / headdim, conv_dim = d_inner + 2 * d_state;
  if (ld < d_inner + conv_dim + H)
    return fail(DFSSM_ERR_SHAPE, "ld=%lld < 2 d_inner + 2 d_state + nheads = %lld", (long long)ld,
                (long long)(d_inner + conv_dim + H));
  if (M < 0 || M * H * 4 > INT32_MAX) return fail(DFSSM_ERR_SHAPE, "M=%lld", (long long)M);
  if (step < 0) return fail(DFSSM_ERR_SHAPE, "step=%lld must be >= 0", (long long)step);
  if (M == 0) return DFSSM_OK;
  dfssm_status st = check_ptrs({{zxbcdt, "zxbcdt"}, {conv_ring, "conv_ring"}, {conv_w, "conv_w"}, {conv_b, "conv_b"},
                                {dt_bias, "dt_bias"}, {A_log, "A_log"}, {D, "D"}, {ssm_state, "ssm_state"}, {y, "y"}},
                               {{xbc, "xbc"}});
  if (st != DFSSM_OK) return st;
  hipError_t e = dfssm::launch_ssm_step(zxbcdt, ld, M, d_inner, d_state, step, conv_ring, conv_w, conv_b, dt_bias,
                                        A_log, D, ssm_state, y, xbc, (hipStream_t)stream);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "ssm step launch");
}

}  // extern "C"

// ---------------------------------------------------------------- model step
namespace {

struct ModelDims {
  int64_t d_model, d_inner, N, H, conv_dim, ld;
};

dfssm_status check_model(const dfssm_mamba2_model* md, int64_t M, ModelDims* dims) {
  if (!md) return fail(DFSSM_ERR_NULL, "model is NULL");
  // d_model % 128 keeps in_proj's row (4 d_model + 2 d_state + d_model / 32
  // values) a whole number of 16-byte words for the gated norm's z loads
  if (md->d_model <= 0 || md->d_model % 128 != 0 || md->d_model > 8192)
    return fail(DFSSM_ERR_SHAPE, "d_model=%lld must be a positive multiple of 128, <= 8192", (long long)md->d_model);
  if (md->d_state != 64 && md->d_state != 128)
    return fail(DFSSM_ERR_UNSUPPORTED, "d_state=%lld: 64 or 128 only", (long long)md->d_state);
  if (md->n_layers <= 0 || md->n_layers > 4096) return fail(DFSSM_ERR_SHAPE, "n_layers=%lld", (long long)md->n_layers);
  if (md->vocab <= 0 || md->vocab > INT32_MAX / 2) return fail(DFSSM_ERR_SHAPE, "vocab=%lld", (long long)md->vocab);
  if (!(md->eps >= 0.0f) || md->eps > FLT_MAX) return fail(DFSSM_ERR_SHAPE, "eps must be finite and >= 0");
  if (M <= 0 || M > 65536) return fail(DFSSM_ERR_SHAPE, "M=%lld must be in [1, 65536]", (long long)M);
  ModelDims d;
  d.d_model = md->d_model;
  d.d_inner = 2 * md->d_model;
  d.N = md->d_state;
  d.H = d.d_inner / 64;
  d.conv_dim = d.d_inner + 2 * d.N;
  d.ld = d.d_inner + d.conv_dim + d.H;
  *dims = d;
  return DFSSM_OK;
}

dfssm_status check_model_pointers(const dfssm_mamba2_model* md, const ModelDims& d) {
  dfssm_status st = check_ptrs({{md->E, "E"}, {md->E_scale, "E_scale"}, {md->norm_f, "norm_f"}}, {});
  if (st != DFSSM_OK) return st;
  if (!md->layers) return fail(DFSSM_ERR_NULL, "layers is NULL");
  for (int64_t l = 0; l < md->n_layers; ++l) {
    const dfssm_mamba2_layer& L = md->layers[l];
    char why[256];
    st = check_ptrs({{L.norm_w, "norm_w"}, {L.conv_w, "conv_w"}, {L.conv_b, "conv_b"}, {L.dt_bias, "dt_bias"},
                     {L.A_log, "A_log"}, {L.D, "D"}, {L.gate_w, "gate_w"}},
                    {});
    if (st == DFSSM_OK && L.lora_bits != 0 && L.lora_bits != 8 && L.lora_bits != 4)
      st = fail(DFSSM_ERR_SHAPE, "lora_bits=%lld: 8 (or 0) or 4", (long long)L.lora_bits);
    const dfssm_layer* pr[2] = {&L.in_proj, &L.out_proj};
    const int64_t want_k[2] = {d.d_model, d.d_inner}, want_n[2] = {d.ld, d.d_model};
    for (int i = 0; i < 2 && st == DFSSM_OK; ++i) {
      const dfssm_layer& P = *pr[i];
      if (P.K != want_k[i] || P.N != want_n[i])
        st = fail(DFSSM_ERR_SHAPE, "%s is %lld x %lld, the model needs %lld x %lld", i ? "out_proj" : "in_proj",
                  (long long)P.K, (long long)P.N, (long long)want_k[i], (long long)want_n[i]);
      else
        st = check_linear(1, P.K, P.N, P.r);
      if (st == DFSSM_OK && L.lora_bits == 4 && P.r % 2 != 0)
        st = fail(DFSSM_ERR_SHAPE, "%s: r=%lld must be even for packed int4 factors", i ? "out_proj" : "in_proj",
                  (long long)P.r);
      if (st == DFSSM_OK && P.lora_bits != 0 && (P.lora_bits == 4) != (L.lora_bits == 4))
        st = fail(DFSSM_ERR_SHAPE, "%s: lora_bits=%lld differs from the layer's %lld", i ? "out_proj" : "in_proj",
                  (long long)P.lora_bits, (long long)L.lora_bits);
      if (st == DFSSM_OK) st = check_ptrs({{P.w_bits, "w_bits"}, {P.alpha, "alpha"}}, {});
      if (st == DFSSM_OK && P.r > 0) st = check_ptrs({{P.A, "A"}, {P.B, "B"}, {P.beta, "beta"}}, {});
    }
    if (st != DFSSM_OK) {
      snprintf(why, sizeof(why), "%s", g_last_error);
      return fail(st, "layer %lld: %s", (long long)l, why);
    }
  }
  return DFSSM_OK;
}

struct ModelWs {
  float *u, *delta, *zx, *y, *s;
  int8_t* q;
  char* lin;
  char* fused;  // the fused step's region (M = 1, models of its shape), or null
  dfssm::StepFusedInfo fi;
  size_t lin_bytes, bytes;
};

ModelWs carve_model_ws(void* base, const dfssm_mamba2_model* md, const ModelDims& d, int64_t M) {
  ModelWs w{};
  size_t off = 0;
  auto take = [&](size_t n) {
    size_t o = off;
    off += (n + 255) & ~(size_t)255;
    return o;
  };
  const size_t o_u = take((size_t)(M * d.d_model) * 4), o_d = take((size_t)(M * d.d_model) * 4);
  const size_t o_zx = take((size_t)(M * d.ld) * 4), o_y = take((size_t)(M * d.d_inner) * 4);
  const size_t o_s = take((size_t)M * 4), o_q = take((size_t)(M * d.d_inner));
  size_t lin = 0;
  for (int64_t l = 0; md->layers && l < md->n_layers; ++l) {
    const dfssm_mamba2_layer& L = md->layers[l];
    if (L.lora_bits == 4) {
      lin = std::max(lin, dfssm::linear_i4_workspace_bytes(M, d.d_model, d.ld, L.in_proj.r));
      lin = std::max(lin, dfssm::linear_i4_workspace_bytes(M, d.d_inner, d.d_model, L.out_proj.r));
    } else {
      lin = std::max(lin, linear_ws_bytes(M, d.d_model, L.in_proj.r));
      lin = std::max(lin, linear_ws_bytes(M, d.d_inner, L.out_proj.r));
    }
  }
  const size_t o_lin = take(lin);
  w.fi = M == 1 ? dfssm::step_fused_info(md) : dfssm::StepFusedInfo{};
  const size_t o_fused = w.fi.ok ? take(w.fi.bytes) : 0;
  char* b = static_cast<char*>(base);
  w.fused = w.fi.ok ? b + o_fused : nullptr;
  w.u = reinterpret_cast<float*>(b + o_u);
  w.delta = reinterpret_cast<float*>(b + o_d);
  w.zx = reinterpret_cast<float*>(b + o_zx);
  w.y = reinterpret_cast<float*>(b + o_y);
  w.s = reinterpret_cast<float*>(b + o_s);
  w.q = reinterpret_cast<int8_t*>(b + o_q);
  w.lin = b + o_lin;
  w.lin_bytes = lin;
  w.bytes = off;
  return w;
}

// Workspaces whose fused-step region dfssm_mamba2_prepare wrote, with the
// fingerprint of the table it wrote there.
std::mutex g_prep_mu;
std::vector<std::pair<const void*, uint64_t>> g_prepared;

void note_prepared(const void* ws, uint64_t fp) {
  std::lock_guard<std::mutex> lk(g_prep_mu);
  for (auto& e : g_prepared)
    if (e.first == ws) {
      e.second = fp;
      return;
    }
  g_prepared.emplace_back(ws, fp);
}
void forget_prepared(const void* ws) {
  std::lock_guard<std::mutex> lk(g_prep_mu);
  for (size_t i = 0; i < g_prepared.size(); ++i)
    if (g_prepared[i].first == ws) {
      g_prepared.erase(g_prepared.begin() + (std::ptrdiff_t)i);
      return;
    }
}
bool is_prepared(const void* ws, uint64_t fp) {
  std::lock_guard<std::mutex> lk(g_prep_mu);
  for (const auto& e : g_prepared)
    if (e.first == ws) return e.second == fp;
  return false;
}

}  // namespace

extern "C" {

dfssm_status dfssm_mamba2_state_bytes(const dfssm_mamba2_model* model, int64_t M, size_t* conv_ring_bytes,
                                      size_t* ssm_state_bytes) {
  clear_error();
  ModelDims d;
  dfssm_status st = check_model(model, M, &d);
  if (st != DFSSM_OK) return st;
  if (conv_ring_bytes) *conv_ring_bytes = (size_t)(model->n_layers * M * 4 * d.conv_dim) * 4;
  if (ssm_state_bytes) *ssm_state_bytes = (size_t)(model->n_layers * M * d.H * 64 * d.N) * 4;
  return DFSSM_OK;
}

size_t dfssm_mamba2_workspace_bytes(const dfssm_mamba2_model* model, int64_t M) {
  ModelDims d;
  if (check_model(model, M, &d) != DFSSM_OK) return 0;
  return carve_model_ws(nullptr, model, d, M).bytes;
}

dfssm_status dfssm_mamba2_decode_step(const dfssm_mamba2_model* model, int64_t M, const int32_t* tok,
                                      int64_t step, float* conv_ring, float* ssm_state, float* logits,
                                      void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  ModelDims d;
  dfssm_status st = check_model(model, M, &d);
  if (st != DFSSM_OK) return st;
  if (step < 0) return fail(DFSSM_ERR_SHAPE, "step=%lld must be >= 0", (long long)step);
  st = check_model_pointers(model, d);
  if (st != DFSSM_OK) return st;
  st = check_ptrs({{tok, "tok"}, {conv_ring, "conv_ring"}, {ssm_state, "ssm_state"}, {logits, "logits"},
                   {workspace, "workspace"}},
                  {});
  if (st != DFSSM_OK) return st;
  const ModelWs w = carve_model_ws(workspace, model, d, M);
  if (workspace_bytes < w.bytes)
    return fail(DFSSM_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, w.bytes);
  hipStream_t hs = (hipStream_t)stream;
  const float eps = model->eps;
  const int step_switch = dfssm::test_switch(DFSSM_TEST_STEP_PER_KERNEL);
  if (w.fused && step_switch != 1 && is_prepared(workspace, w.fi.fingerprint)) {
    // the fused step: gather, one persistent launch for all layers, final
    // norm, LM head
    float* u0 = reinterpret_cast<float*>(w.fused + w.fi.off_u0);
    float* ufin = reinterpret_cast<float*>(w.fused + w.fi.off_ufin);
    hipError_t e = dfssm::launch_embed_gather(model->E, model->E_scale, model->vocab, d.d_model, tok, 1, u0, hs);
    if (e == hipSuccess)
      e = dfssm::step_fused_run(w.fi, eps, step, conv_ring, ssm_state, w.fused, step_switch == 2, hs);
    if (e == hipSuccess)
      e = dfssm::launch_add_rmsnorm_quant(ufin, nullptr, model->norm_f, eps, 1, d.d_model, nullptr, w.q, w.s, hs);
    if (e == hipSuccess)
      e = dfssm::launch_lm_head(w.q, w.s, 1, d.d_model, model->E, model->E_scale, model->vocab, logits, nullptr, hs);
    return e == hipSuccess ? DFSSM_OK : device_fail(e, "decode step launch");
  }
  const int64_t ring_stride = M * 4 * d.conv_dim, state_stride = M * d.H * 64 * d.N;
  hipError_t e = dfssm::launch_embed_gather(model->E, model->E_scale, model->vocab, d.d_model, tok, M, w.u, hs);
  for (int64_t l = 0; l < model->n_layers && e == hipSuccess; ++l) {
    const dfssm_mamba2_layer& L = model->layers[l];
    e = dfssm::launch_add_rmsnorm_quant(w.u, l > 0 ? w.delta : nullptr, L.norm_w, eps, M, d.d_model, w.u, w.q, w.s, hs);
    if (e != hipSuccess) break;
    const bool i4 = L.lora_bits == 4;
    const dfssm_layer& I = L.in_proj;
    if (i4)
      e = launch_linear_i4(DFSSM_PATH_AUTO, w.q, w.s, M, I.K, I.N, I.r, I.w_bits, I.alpha,
                           reinterpret_cast<const uint8_t*>(I.A), reinterpret_cast<const uint8_t*>(I.B), I.beta,
                           w.zx, nullptr, nullptr, nullptr, w.lin, hs);
    else
      e = launch_linear(DFSSM_PATH_AUTO, w.q, w.s, M, I.K, I.N, I.r, I.w_bits, I.alpha, I.A, I.B, I.beta, w.zx,
                        nullptr, nullptr, nullptr, dfssm::carve_linear_workspace(w.lin, M, I.K, I.r), hs);
    if (e != hipSuccess) break;
    // the SSM step applies the gate (y * silu(z), one fp32 product per
    // channel, spread over its workgroups), so the norm after it is a plain
    // RMSNorm: at batch 1 the gated norm's single workgroup otherwise spends
    // ~1.2 us on the row's 2 d_model fp64 silus
    e = dfssm::launch_ssm_step(w.zx, d.ld, M, d.d_inner, d.N, step, conv_ring + l * ring_stride, L.conv_w, L.conv_b,
                               L.dt_bias, L.A_log, L.D, ssm_state + l * state_stride, w.y, nullptr, hs, true);
    if (e != hipSuccess) break;
    e = dfssm::launch_add_rmsnorm_quant(w.y, nullptr, L.gate_w, eps, M, d.d_inner, nullptr, w.q, w.s, hs);
    if (e != hipSuccess) break;
    const dfssm_layer& O = L.out_proj;
    if (i4)
      e = launch_linear_i4(DFSSM_PATH_AUTO, w.q, w.s, M, O.K, O.N, O.r, O.w_bits, O.alpha,
                           reinterpret_cast<const uint8_t*>(O.A), reinterpret_cast<const uint8_t*>(O.B), O.beta,
                           w.delta, nullptr, nullptr, nullptr, w.lin, hs);
    else
      e = launch_linear(DFSSM_PATH_AUTO, w.q, w.s, M, O.K, O.N, O.r, O.w_bits, O.alpha, O.A, O.B, O.beta, w.delta,
                        nullptr, nullptr, nullptr, dfssm::carve_linear_workspace(w.lin, M, O.K, O.r), hs);
  }
  if (e == hipSuccess)
    e = dfssm::launch_add_rmsnorm_quant(w.u, w.delta, model->norm_f, eps, M, d.d_model, w.u, w.q, w.s, hs);
  if (e == hipSuccess)
    e = dfssm::launch_lm_head(w.q, w.s, M, d.d_model, model->E, model->E_scale, model->vocab, logits, nullptr, hs);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "decode step launch");
}

dfssm_status dfssm_mamba2_prepare(const dfssm_mamba2_model* model, int64_t M, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  clear_error();
  ModelDims d;
  dfssm_status st = check_model(model, M, &d);
  if (st != DFSSM_OK) return st;
  st = check_model_pointers(model, d);
  if (st != DFSSM_OK) return st;
  st = check_ptrs({{workspace, "workspace"}}, {});
  if (st != DFSSM_OK) return st;
  const ModelWs w = carve_model_ws(workspace, model, d, M);
  if (workspace_bytes < w.bytes)
    return fail(DFSSM_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, w.bytes);
  if (!w.fused) return DFSSM_OK;
  const hipError_t e = dfssm::step_fused_prepare(model, w.fused, (hipStream_t)stream);
  if (e != hipSuccess) return device_fail(e, "decode step prepare launch");
  note_prepared(workspace, w.fi.fingerprint);
  return DFSSM_OK;
}

dfssm_status dfssm_mamba2_release(const void* workspace) {
  clear_error();
  if (workspace) forget_prepared(workspace);
  return DFSSM_OK;
}

dfssm_status dfssm_mamba2_fused_path(const dfssm_mamba2_model* model, int64_t M, const void* workspace,
                                     size_t workspace_bytes, int* fused) {
  clear_error();
  if (!fused) return fail(DFSSM_ERR_NULL, "fused is NULL");
  *fused = 0;
  ModelDims d;
  dfssm_status st = check_model(model, M, &d);
  if (st != DFSSM_OK) return st;
  st = check_ptrs({{workspace, "workspace"}}, {});
  if (st != DFSSM_OK) return st;
  const ModelWs w = carve_model_ws(const_cast<void*>(workspace), model, d, M);
  if (workspace_bytes < w.bytes)
    return fail(DFSSM_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, w.bytes);
  *fused = w.fused && dfssm::test_switch(DFSSM_TEST_STEP_PER_KERNEL) != 1 && is_prepared(workspace, w.fi.fingerprint)
               ? 1
               : 0;
  return DFSSM_OK;
}

dfssm_status dfssm_mamba2_status(const dfssm_mamba2_model* model, int64_t M, const void* workspace,
                                 size_t workspace_bytes, unsigned* status, void* stream) {
  clear_error();
  if (!status) return fail(DFSSM_ERR_NULL, "status is NULL");
  *status = 0;
  ModelDims d;
  dfssm_status st = check_model(model, M, &d);
  if (st != DFSSM_OK) return st;
  st = check_ptrs({{workspace, "workspace"}}, {});
  if (st != DFSSM_OK) return st;
  const ModelWs w = carve_model_ws(const_cast<void*>(workspace), model, d, M);
  if (workspace_bytes < w.bytes)
    return fail(DFSSM_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, w.bytes);
  if (!w.fused || !is_prepared(workspace, w.fi.fingerprint)) return DFSSM_OK;
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e == hipSuccess) e = hipMemcpy(status, w.fused + w.fi.off_status, sizeof(unsigned), hipMemcpyDeviceToHost);
  return e == hipSuccess ? DFSSM_OK : device_fail(e, "decode step status read");
}

}  // extern "C"
