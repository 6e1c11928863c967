/*
 * dfssm.h -- C ABI of the DF-SSM scaffold + int8 LoRA linear for AMD
 * Instinct MI355X (gfx950).
 *
 * The operation (paper: Sec. 3.2, Eq. 3 -- a frozen scaffold plus a low-rank
 * correction; Sec. 3.3 and Table 1 -- the scaffold stored at 1 bit per
 * weight, the LoRA factors in int8 with per-channel scales; Sec. 4.1 -- int8
 * activations feeding an int8 x int8 scaffold product), with the scaffold
 * binarised to sign(W) and a per-output-row scale:
 *
 *     y = diag(alpha) * S * q(x)  +  diag(beta) * B * (A * q(x))
 *
 * where q(x) = s * Q is per-token absmax int8 quantisation of x.
 *
 * Conventions for every entry point:
 *  - All array pointers are DEVICE pointers (hipMalloc'd or torch tensors)
 *    unless a comment says host.  The caller owns every buffer; the library
 *    never allocates or frees device memory in these calls.
 *  - Arrays are dense row-major with the shapes given; base pointers must be
 *    16-byte aligned (DFSSM_ERR_ALIGN otherwise).
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls are
 *    stream-ordered and asynchronous: they validate on the host, enqueue
 *    kernels and return.  A validation failure returns before anything is
 *    enqueued.  A launch failure returns DFSSM_ERR_DEVICE.  Faults inside a
 *    kernel surface at the caller's next synchronisation.
 *  - Outputs must not alias inputs.  Inputs must be finite; the kernels do
 *    not check this and the output for non-finite input is unspecified.
 *  - Results are bitwise deterministic run to run (integer arithmetic, no
 *    floating-point atomics).
 *  - No C++ exception crosses this interface.  dfssm_last_error() returns a
 *    thread-local message describing the last failure on the calling thread.
 *
 * Layouts:
 *   x      [M, ldx]  fp16 or fp32 activations, row stride ldx >= K elements
 *   q      [M, K]    int8 codes Q, |Q| <= 127
 *   s      [M]       fp32 per-token scale
 *   w_bits [N, K/32] uint32; bit j of word w of row n is S[n, 32*w + j],
 *                    1 -> +1, 0 -> -1 (little-endian, least significant bit
 *                    first)
 *   alpha  [N]       fp32 scaffold row scale
 *   A      [r, K]    int8 LoRA down-projection (the paper's W_B)
 *   B      [N, r]    int8 LoRA up-projection   (the paper's W_A)
 *   beta   [N]       fp32 LoRA row scale (per-channel int8 scales and the
 *                    scalar LoRA gain folded together)
 *   y      [M, N]    fp32 output
 * Limits: 0 < K <= 65536, K % 32 == 0; M, N >= 0 (0 is a no-op);
 *         0 <= r <= 256.  When r == 0, A, B and beta may be NULL.
 *
 * Arithmetic (exact where it is integer):
 *   acc_s = Q * S^T  (int32), acc_a = Q * A^T (int32),
 *   acc_b = acc_a * B^T (int64, exact), then per element in fp32 with one
 *   rounding per operation: fs=(float)acc_s; u=alpha*fs; fb=(float)acc_b;
 *   v=beta*fb; w=u+v; y=s*w   (r == 0: y = s*u).
 */
#ifndef DFSSM_H
#define DFSSM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DFSSM_OK = 0,
  DFSSM_ERR_NULL = 1,        /* a required pointer is NULL */
  DFSSM_ERR_SHAPE = 2,       /* a size or stride is outside the limits */
  DFSSM_ERR_ALIGN = 3,       /* a pointer is not 16-byte aligned */
  DFSSM_ERR_WORKSPACE = 4,   /* workspace missing or smaller than required */
  DFSSM_ERR_DEVICE = 5,      /* a HIP call failed (see dfssm_last_error) */
  DFSSM_ERR_UNSUPPORTED = 6  /* valid request this build does not handle */
} dfssm_status;

typedef enum { DFSSM_F16 = 0, DFSSM_F32 = 1 } dfssm_dtype;

/* Kernel family selection for dfssm_scaffold_lora_linear_ex. */
typedef enum {
  DFSSM_PATH_AUTO = 0,     /* few-token MFMA for M <= 32; for 33..512 the
                              few-token kernel in 64-token blocks or the
                              prefill kernel, by a cost model of the two
                              (see the implementation); prefill MFMA
                              above 512 */
  DFSSM_PATH_DECODE = 1,   /* bit-plane popcount GEMV (any M, best for M <= 4) */
  DFSSM_PATH_MFMA = 2,     /* sign bits expanded on chip + int8 MFMA, tiles of
                              128 tokens (prefill): an 8-wave ping-pong
                              kernel where each block gets at least 24 row
                              tiles of 16, a 4-wave kernel otherwise
                              (dfssm_test_switch can force one of them). */
  DFSSM_PATH_MFMA_FEW = 3  /* the same expansion and MFMA for M <= 512 in
                              one launch: 16 output rows and up to 32
                              tokens per workgroup (64 above 32 tokens), K
                              split over its waves, the LoRA
                              down-projection in workgroups of the same
                              grid; M > 512 gives DFSSM_ERR_UNSUPPORTED. */
} dfssm_path;

/* Per-token absmax int8 quantisation of the activations (the int8 operand
 * of the scaffold product, Sec. 4.1).  For each row m:
 *   a = max_k |x[m,k]|;  a < FLT_MIN -> Q[m,:] = 0, s[m] = 0;
 *   else s[m] = a/127, inv = 127/a, Q[m,k] = clamp(rint(x[m,k]*inv), +-127)
 * with fp32 operations rounded to nearest-even (fp16 input is widened to
 * fp32 exactly first).
 *   x       device [M, ldx], element type x_dtype (DFSSM_F16 or DFSSM_F32)
 *   q       device [M, K] int8 output;  s  device [M] fp32 output
 * Errors: NULL/SHAPE/ALIGN (x needs only element alignment: 2 B for fp16,
 * 4 B for fp32), DEVICE. */
dfssm_status dfssm_quantize_act(const void* x, int x_dtype, int64_t M, int64_t K,
                                int64_t ldx, int8_t* q, float* s, void* stream);

/* Bytes of device workspace dfssm_scaffold_lora_linear needs for (M,K,N,r):
 * about 1 MB of state kept from call to call, plus per-call staging. */
size_t dfssm_linear_workspace_bytes(int64_t M, int64_t K, int64_t N, int64_t r);

/* The scaffold + LoRA linear (Eq. 3 with a binary scaffold), on already
 * quantised activations (q, s).  Writes y [M,N].  `workspace` is device
 * memory of at least dfssm_linear_workspace_bytes(M,K,N,r) bytes, used for
 * acc_a, per-token staging and the exchange words of the few-token path.
 * The workspace must hold zeros before its first use (hipMemset, or a
 * zero-filled tensor); after that it belongs to the library: pass it back
 * unchanged to later calls, of any shape and path, and do not run two
 * calls on one workspace at the same time.  The exchange words are tagged
 * per call: from a host counter for a call enqueued directly, and, for a
 * call captured into a graph, from an epoch that the kernels themselves
 * advance once per replay; so a captured call replayed any number of
 * times, with new inputs, computes each replay from that replay's inputs.
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, DEVICE. */
dfssm_status dfssm_scaffold_lora_linear(const int8_t* q, const float* s, int64_t M,
                                        int64_t K, int64_t N, int64_t r,
                                        const uint32_t* w_bits, const float* alpha,
                                        const int8_t* A, const int8_t* B,
                                        const float* beta, float* y, void* workspace,
                                        size_t workspace_bytes, void* stream);

/* The same linear with no workspace argument, for callers that cannot
 * allocate device memory (code under graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, results and errors as
 * dfssm_scaffold_lora_linear, minus the workspace: the library keeps one
 * scratch array of dfssm_noalloc_scratch_bytes() bytes (16 MiB) per GPU, in
 * device memory of the loaded library that stays until the process ends,
 * and this call allocates nothing.  A call whose workspace would exceed it
 * (dfssm_linear_workspace_bytes(M, K, N, r) > that size; e.g. M*K above
 * about 14 M at r = 64) returns DFSSM_ERR_WORKSPACE.  Every call on one GPU
 * shares its array: calls that overlap on one GPU (two streams, two
 * threads) race and give unspecified results; calls in one stream are
 * ordered and fine.
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, DEVICE. */
dfssm_status dfssm_scaffold_lora_linear_noalloc(const int8_t* q, const float* s, int64_t M,
                                                int64_t K, int64_t N, int64_t r,
                                                const uint32_t* w_bits, const float* alpha,
                                                const int8_t* A, const int8_t* B,
                                                const float* beta, float* y, void* stream);
/* Size of the scratch array dfssm_scaffold_lora_linear_noalloc uses. */
size_t dfssm_noalloc_scratch_bytes(void);

/* Same operation with an explicit kernel family and optional integer
 * accumulator outputs (each may be NULL): acc_s int32 [M,N], acc_a int32
 * [M,r], acc_b int64 [M,N].  y may be NULL too.  The accumulators are the
 * exact integers defined above, identical on every path. */
dfssm_status dfssm_scaffold_lora_linear_ex(const int8_t* q, const float* s, int64_t M,
                                           int64_t K, int64_t N, int64_t r,
                                           const uint32_t* w_bits, const float* alpha,
                                           const int8_t* A, const int8_t* B,
                                           const float* beta, float* y, int path,
                                           int32_t* acc_s, int32_t* acc_a,
                                           int64_t* acc_b, void* workspace,
                                           size_t workspace_bytes, void* stream);

/* The same linear with int4 LoRA factors (Table 4: the scaffold with an
 * int4 LoRA; the paper gives no format).  Each factor value is a
 * two's-complement 4-bit integer in [-8, 7], two per byte, value 2i in the
 * low nibble of byte i:
 *   A4 [r][K/2] bytes (row j holds A[j, 0..K-1])
 *   B4 [N][r/2] bytes (row n holds B[n, 0..r-1])
 * r must be even.  Every other argument, output and result is as in
 * dfssm_scaffold_lora_linear_ex on the unpacked A and B (the same exact
 * integers).  The few-token path (M <= 32) reads the packed bytes directly,
 * half the LoRA bytes of int8; the prefill MFMA and popcount paths first
 * expand the factors to int8 inside the workspace.  The workspace must hold
 * dfssm_linear_i4_workspace_bytes(M, K, N, r) bytes.
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, UNSUPPORTED, DEVICE. */
size_t dfssm_linear_i4_workspace_bytes(int64_t M, int64_t K, int64_t N, int64_t r);
dfssm_status dfssm_scaffold_lora_linear_i4(const int8_t* q, const float* s, int64_t M, int64_t K,
                                           int64_t N, int64_t r, const uint32_t* w_bits,
                                           const float* alpha, const uint8_t* A4, const uint8_t* B4,
                                           const float* beta, float* y, int path, int32_t* acc_s,
                                           int32_t* acc_a, int64_t* acc_b, void* workspace,
                                           size_t workspace_bytes, void* stream);

/* One projection of a chain (host struct; the pointers in it are device
 * pointers with the layouts above). */
typedef struct {
  const uint32_t* w_bits;
  const float* alpha;
  const int8_t* A;
  const int8_t* B;
  const float* beta;
  int64_t K, N, r;
  int64_t lora_bits;  /* 0 or 8: A [r][K] and B [N][r] int8; 4: A and B are
                         packed int4 (Table 4): A [r][K/2], B [N][r/2] bytes
                         of two's-complement nibbles, value 2i in the low
                         nibble of byte i (as dfssm_scaffold_lora_linear_i4);
                         r even */
} dfssm_layer;

/* Bytes of device workspace dfssm_scaffold_lora_chain needs. */
size_t dfssm_chain_workspace_bytes(const dfssm_layer* layers, int n_layers, int64_t M);

/* A chain of linears run back to back on one stream, each output
 * re-quantised as the next input (the decode sweep over a model's
 * projections, Sec. 4.1):
 *   linear 0 consumes (q0 [M,K_0], s0 [M]);
 *   linear l >= 1 consumes Q_l = quantise(y_{l-1}[:, 0:K_l]) (fp32, row
 *   stride N_{l-1}, same rule as dfssm_quantize_act) with s_l = 1/127 for
 *   every token, standing in for the normalisation between projections.
 * Requires K_l <= N_{l-1}.  y_all (device) receives every linear's y back
 * to back: sum_l M*N_l floats, linear l at offset sum_{i<l} M*N_i.
 * `layers` is a HOST array of n_layers entries.  M must be 1..4.  Layers
 * may mix int8 and packed int4 LoRA factors (lora_bits); at M = 1 the
 * persistent kernel takes int4 layers with r % 8 == 0, others run the
 * host-sequenced path.
 * Equivalent to dfssm_chain_prepare followed by dfssm_chain_run.
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, UNSUPPORTED, DEVICE. */
dfssm_status dfssm_scaffold_lora_chain(const dfssm_layer* layers, int n_layers, int64_t M,
                                       const int8_t* q0, const float* s0, float* y_all,
                                       void* workspace, size_t workspace_bytes,
                                       void* stream);

/* Prepares `workspace` for dfssm_chain_run with these layers: writes the
 * persistent kernel's layer table and its 64-bit fingerprint into the
 * workspace and clears the exchange region and the status word
 * (stream-ordered, asynchronous).  Needed once per (layers, workspace): a
 * prepared workspace can be run any number of times, as long as nothing
 * but dfssm_chain_run writes to it in between.  The persistent kernel
 * takes chains at M = 1 with, for every linear, K % 256 == 0, K <= 4096,
 * r <= 64, r % 4 == 0, N >= 4, the next linear's K a multiple of 256, at
 * most 64 output rows per workgroup and operands that fit its LDS ring;
 * other chains run as a sequence of quantise and linear launches, and for
 * them preparation clears the linears' exchange state in the workspace.
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, UNSUPPORTED, DEVICE. */
dfssm_status dfssm_chain_prepare(const dfssm_layer* layers, int n_layers, int64_t M,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* Runs the chain (same contract as dfssm_scaffold_lora_chain) on a
 * workspace prepared for exactly these layers: at M = 1 one kernel launch
 * of one workgroup per compute unit, which needs the whole grid resident at
 * once (nothing else holding the GPU's compute units; otherwise its bounded
 * waits end it with a status bit, see dfssm_chain_status).  If the
 * workspace's fingerprint does not match these layers, the kernel leaves
 * before reading the table, writes nothing and sets status bit 8.  The
 * kernel advances an epoch in the workspace once per run, so a run captured
 * in a graph can be replayed with new inputs.
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, UNSUPPORTED, DEVICE. */
dfssm_status dfssm_chain_run(const dfssm_layer* layers, int n_layers, int64_t M, const int8_t* q0,
                             const float* s0, float* y_all, void* workspace,
                             size_t workspace_bytes, void* stream);

/* Synchronises `stream` and reads the persistent chain's status word into
 * *status (host): 0 = fine; bit 1 = a wait for a previous output timed out;
 * bit 2 = a wait for a row or rank partial timed out (a workgroup of the
 * grid was not resident, or another one left early); bit 8 = the workspace
 * was not prepared for these layers.  After a nonzero status the outputs of
 * that run are incomplete.  Bits accumulate over runs until the next
 * dfssm_chain_prepare.
 * Always 0 for chains that do not use the persistent kernel.
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, UNSUPPORTED, DEVICE. */
dfssm_status dfssm_chain_status(const dfssm_layer* layers, int n_layers, int64_t M,
                                const void* workspace, size_t workspace_bytes, unsigned* status,
                                void* stream);

/* Diagnostic, not part of the computation: runs only the persistent
 * chain's operand loads -- each workgroup's direct-to-LDS loads of its sign
 * words, A slice, B rows and row scales for every linear, with the chain
 * kernel's placement and LDS ring, back to back (one linear in flight while
 * the previous lands) -- with no arithmetic, no exchange and no output.
 * One launch takes the time that streaming the chain's weights alone sets,
 * the floor under dfssm_chain_run on the same layers.  Needs a workspace
 * prepared by dfssm_chain_prepare for these layers at M = 1 (it only reads
 * the layer table; a fingerprint mismatch sets status bit 8 and loads
 * nothing).
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, UNSUPPORTED (layers the persistent
 * kernel does not take), DEVICE. */
dfssm_status dfssm_chain_stream_floor(const dfssm_layer* layers, int n_layers, void* workspace,
                                      size_t workspace_bytes, void* stream);

/* Diagnostic, not part of the computation: one launch that reads `bytes`
 * bytes from the device buffer p (16-byte loads, every thread's loads issued
 * before their first use, enough workgroups to cover the buffer at once).
 * Each wave stores the XOR of the 32-bit words it read into its own word of
 * sink, so the XOR of the first dfssm_read_floor_sink_words(bytes) words
 * of sink is the XOR of the buffer's words.  Its duration is the floor
 * under a single-launch linear whose weights take the same bytes (Table 13
 * prices a decode linear by the bytes it moves).  bytes == 0 makes an empty
 * launch: the launch floor.
 *   p      16-byte aligned device buffer (may be NULL when bytes == 0)
 *   sink   4-byte aligned device uint32 [sink_words]
 * Errors: NULL, SHAPE (bytes not a multiple of 16), ALIGN, WORKSPACE (sink
 * too small), DEVICE. */
size_t dfssm_read_floor_sink_words(size_t bytes);

/* Diagnostic, not part of the computation: the cost of one exchange hop of
 * the persistent kernels (Sec. 4.1: the decode path is bound by latency,
 * not by bytes).  npairs pairs of workgroups, the two of a pair on
 * different XCDs, pass one 64-bit word back and forth iters times with
 * agent-scope stores and polling loads (fence != 0: a release store and
 * acquire loads instead); *ns_per_round_trip (host) receives the median over
 * the pairs of one round trip (two hops).  Synchronises `stream` to read
 * the result.  Every wait is bounded.
 *   workspace  device, dfssm_exchange_pingpong_bytes() bytes, 16-byte
 *              aligned; its contents on entry do not matter
 * Errors: NULL, SHAPE (npairs outside 1..128, iters outside 1..100000),
 * ALIGN, WORKSPACE, DEVICE (also when a wait gave up). */
size_t dfssm_exchange_pingpong_bytes(void);
dfssm_status dfssm_exchange_pingpong(int npairs, int iters, int fence, void* workspace, size_t workspace_bytes,
                                     double* ns_per_round_trip, void* stream);
dfssm_status dfssm_read_floor(const void* p, size_t bytes, uint32_t* sink, size_t sink_words, void* stream);

/* The tied int8 embedding table (Sec. 3.3 and Table 1: the token embedding
 * is stored in int8 with one fp32 scale per row and shared with the LM
 * head):
 *   E      [V, d]  int8 table
 *   scale  [V]     fp32 row scale
 *
 * Token gather (the model's input rows):
 *   tok    [M]     int32 token ids;  x [M, d] fp32 output
 *   x[m,k] = scale[t] * (float)E[t,k] with t = tok[m] (one fp32 rounding).
 * The ids are read on the device: an id outside [0, V) is not an error, it
 * gives a zero row.
 * Limits: 0 < d <= 65536, d % 16 == 0; 0 < V < 2^30; M >= 0 (0 is a no-op).
 * Errors: NULL, SHAPE, ALIGN, DEVICE. */
dfssm_status dfssm_embed_gather(const int8_t* E, const float* scale, int64_t V, int64_t d,
                                const int32_t* tok, int64_t M, float* x, void* stream);

/* LM head on the tied table: the logits of M tokens over the whole
 * vocabulary from the int8-quantised final hidden state (q [M, d], s [M],
 * as dfssm_quantize_act makes them):
 *   acc[m,v]    = sum_k E[v,k] * Q[m,k]                  (int32, exact)
 *   logits[m,v] = s[m] * (scale[v] * (float)acc[m,v])    (fp32, rounded
 *                 after each operation, in this order)
 *   logits [M, V] fp32 output, or NULL;  acc [M, V] int32 output, or NULL
 *   (not both NULL).
 * Below 8 tokens, GEMV passes of up to 4 tokens (fewer for d > 4096), each
 * streaming the table once; from 8 tokens, when d is a multiple of 64 that
 * splits into 4..8 waves of at most 8 steps of 64 (d = 256 .. 4096), one
 * pass on the matrix cores that reads the table once for all tokens; from
 * 64 tokens (and V * d, M * d < 2^31) a tiled matrix-core kernel that
 * stages both operands in LDS (dfssm_test_switch can move both thresholds).
 * All choices give the same bits.
 * Limits: 0 < d <= 16384, d % 16 == 0; 0 <= V < 2^30; M >= 0 (M or V == 0
 * is a no-op).
 * Errors: NULL, SHAPE, ALIGN, DEVICE. */
dfssm_status dfssm_lm_head(const int8_t* q, const float* s, int64_t M, int64_t d, const int8_t* E,
                           const float* scale, int64_t V, float* logits, int32_t* acc, void* stream);

/* The Mamba-2 decode step around the two linears (Sec. 4.1: the convolution
 * step is a stateful shift register and the SSM step a stateful recurrence;
 * Table 13 lists them with RMSNorm and gate + norm; Table 12 fixes the
 * step's semantics: the input enters the state as (x * dt) outer B, d_state
 * is 128 for the 1.3B model, and the gate comes before the norm).  The
 * other sizes follow the public Mamba-2 design: d_inner = 2 d_model, heads
 * of 64 channels, one B/C group, a width-4 convolution, and in_proj's output
 * row laid out as [z | x | B | C | dt] (d_inner, d_inner, N, N, nheads).
 *
 * Rounding, the same on every run: fp32 for every elementwise step; exp,
 * log1p, sqrt and the divisions inside silu(v) = v / (1 + exp(-v)),
 * softplus(v) = v > 20 ? v : log1p(exp(v)) and the norm's scale in fp64,
 * rounded once to fp32; the norm's sum of squares and the SSM output's sum
 * over the state accumulated in fp64.  Results may differ from another
 * summation order only when an fp64 sum falls within its last bits of an
 * fp32 rounding boundary. */

/* Residual add, RMSNorm and the linear's per-token quantisation: the input
 * of in_proj, and the final norm before the LM head.
 *   u'  = u + delta  (fp32; u' = u when delta is NULL)
 *   r   = (float)(1 / sqrt(sum_k u'^2 / d + eps))
 *   o   = (u' * r) * w
 *   (q, s) = dfssm_quantize_act's rule applied to o
 *   u, delta, u_out [M, d] fp32; w [d] fp32; q [M, d] int8; s [M] fp32
 * u_out (may be NULL) receives u'; u_out == u (in place) is allowed.
 * Limits: 0 < d <= 16384, d % 4 == 0; eps finite, >= 0; M >= 0.
 * Errors: NULL, SHAPE, ALIGN, DEVICE. */
dfssm_status dfssm_add_rmsnorm_quant(const float* u, const float* delta, const float* w, float eps,
                                     int64_t M, int64_t d, float* u_out, int8_t* q, float* s,
                                     void* stream);

/* Gate then norm, and quantisation: the input of out_proj.
 *   g = y * silu(z);  r = (float)(1 / sqrt(sum_k g^2 / d + eps));
 *   o = (g * r) * w;  (q, s) = quantise(o)
 *   y [M, d] fp32 (the SSM output); z rows of stride ldz fp32 (in_proj's
 *   output row holds z at its start: pass it with ldz = its row length);
 *   w [d]; q [M, d] int8; s [M].
 * Limits: 0 < d <= 16384, d % 4 == 0; ldz >= d, ldz % 4 == 0; eps finite,
 * >= 0.  Errors: NULL, SHAPE, ALIGN, DEVICE. */
dfssm_status dfssm_gate_norm_quant(const float* y, const float* z, int64_t ldz, const float* w, float eps,
                                   int64_t M, int64_t d, int8_t* q, float* s, void* stream);

/* The convolution step and the SSM step for one token of each of M
 * sequences, updating their state in place.
 *   zxbcdt  [M, ld] fp32 in_proj's output rows; xBC (conv_dim = d_inner +
 *           2 d_state values) at column d_inner, dt (nheads) at column
 *           d_inner + conv_dim
 *   conv_ring [M][4][conv_dim] fp32 convolution state as a ring: before the
 *           call with step t, slot (t - k) & 3 holds the xBC input of step
 *           t - k (k = 1..3; zeros for steps before the first).  The call
 *           reads those three slots and writes this step's input into slot
 *           t & 3.  In the model's shift-register form [conv_dim][4] the
 *           register's position j is ring slot (t - 4 + j) & 3 before step t.
 *           Advance t by one per call; a new sequence starts from zeros.
 *   conv_w [conv_dim][4] fp32 (tap 3 meets the newest input), conv_b
 *           [conv_dim]; dt_bias, A_log, D [nheads] fp32
 *   ssm_state [M][nheads][headdim][d_state] fp32, updated
 *   y       [M, d_inner] fp32 out; xbc [M, conv_dim] fp32 out or NULL (the
 *           convolution outputs)
 * Per channel c:  v = (((w0 s_{t-3} + w1 s_{t-2}) + w2 s_{t-1}) + w3 s_t)
 *                 + b;  xbc = silu(v)
 * Per head h (x = xbc[h*64 + p], B = xbc[d_inner + n], C = xbc[d_inner +
 * d_state + n]):  dt = softplus(dt_raw + dt_bias); A = -exp(A_log);
 *   dA = exp(dt * A);  h[p][n] = h[p][n] * dA + (dt * x) * B[n];
 *   y[h*64 + p] = sum_n h[p][n] C[n] + D x
 * Limits: headdim == 64 and d_state in {64, 128} (else UNSUPPORTED);
 * d_inner a positive multiple of 64, <= 65536; ld >= 2 d_inner + 2 d_state
 * + nheads; step >= 0.  Outputs must not alias the inputs.
 * Errors: NULL, SHAPE, ALIGN, UNSUPPORTED, DEVICE. */
dfssm_status dfssm_ssm_step(const float* zxbcdt, int64_t ld, int64_t M, int64_t d_inner, int64_t d_state,
                            int64_t headdim, int64_t step, float* conv_ring, const float* conv_w,
                            const float* conv_b, const float* dt_bias, const float* A_log,
                            const float* D, float* ssm_state, float* y, float* xbc, void* stream);

/* ---- the whole decode step of the model ------------------------------- */

/* One Mamba-2 layer of the distilled model (host struct of device pointers).
 * conv_dim = d_inner + 2 d_state, nheads = d_inner / 64, d_inner = 2 d_model. */
typedef struct {
  const float* norm_w;   /* [d_model]  RMSNorm before the mixer */
  dfssm_layer in_proj;   /* K = d_model, N = 2 d_inner + 2 d_state + nheads */
  const float* conv_w;   /* [conv_dim][4] */
  const float* conv_b;   /* [conv_dim] */
  const float* dt_bias;  /* [nheads] */
  const float* A_log;    /* [nheads] */
  const float* D;        /* [nheads] */
  const float* gate_w;   /* [d_inner]  weight of the gated norm */
  dfssm_layer out_proj;  /* K = d_inner, N = d_model */
  int64_t lora_bits;     /* 8 (or 0): A and B of both projections are int8,
                            as for dfssm_scaffold_lora_linear; 4: they are
                            packed int4 as for dfssm_scaffold_lora_linear_i4
                            (A [r][K/2], B [N][r/2] bytes; r even) */
} dfssm_mamba2_layer;

/* The model: tied int8 embedding / LM head table, n_layers layers, final
 * norm.  `layers` is a HOST array of n_layers entries. */
typedef struct {
  int64_t d_model, d_state, n_layers, vocab;
  float eps;                         /* RMSNorm epsilon (1e-5 in Mamba-2) */
  const int8_t* E;                   /* [vocab][d_model] int8 */
  const float* E_scale;              /* [vocab] */
  const float* norm_f;               /* [d_model] */
  const dfssm_mamba2_layer* layers;  /* host array */
} dfssm_mamba2_model;

/* Bytes of the per-sequence state for M sequences (caller-allocated, device):
 *   conv_ring [n_layers][M][4][conv_dim] fp32 and
 *   ssm_state [n_layers][M][nheads][64][d_state] fp32,
 * zero for sequences that start with the next step (their step counter then
 * counts from there; only step & 3 matters to the ring).  Either output may
 * be NULL.  Returns DFSSM_OK or SHAPE. */
dfssm_status dfssm_mamba2_state_bytes(const dfssm_mamba2_model* model, int64_t M, size_t* conv_ring_bytes,
                                      size_t* ssm_state_bytes);

/* Bytes of device workspace dfssm_mamba2_decode_step needs for M tokens
 * (at M = 1, for a model of the shape the fused step takes, this includes
 * the fused step's region: about 39 MB for 48 layers). */
size_t dfssm_mamba2_workspace_bytes(const dfssm_mamba2_model* model, int64_t M);

/* One decode step of M sequences, all on `stream` (Sec. 4.1: the paper
 * captures the whole 48-layer forward pass as one CUDA graph, with the SSM
 * and convolution states preallocated and kept across tokens):
 *   x = embed_gather(tok); for each layer l:
 *     u += delta (l > 0);  (q, s) = quantise(rmsnorm(u) * norm_w)
 *     zx = in_proj(q, s);  y = ssm_step(zx, step, state_l)
 *     (q, s) = quantise(rmsnorm(y * silu(z)) * gate_w);  delta = out_proj(q, s)
 *   u += delta;  (q, s) = quantise(rmsnorm(u) * norm_f);  logits = lm_head(q, s)
 * with the entry points above (in_proj and out_proj on the automatic path,
 * through the int4 linear for layers with lora_bits = 4).  The gate's
 * product y * silu(z) is taken inside the SSM step's kernel, in the same
 * fp32 rounding, so the results are those of the entry points bit for bit.
 *   tok     [M] int32 device token ids (outside [0, vocab) -> a zero row)
 *   step    this token's position; only step & 3 is used (the ring slot)
 *   conv_ring, ssm_state   the state, updated in place
 *   logits  [M][vocab] fp32 device output
 * The workspace must hold zeros before its first use and belongs to the
 * library after that, as dfssm_scaffold_lora_linear's does.
 * Graph capture: nothing here allocates, copies or synchronises, so the call
 * can be captured.  A captured step keeps its step & 3 (capture four graphs,
 * one per value, and replay the one for each token); its linears advance
 * their exchange epoch on the device, so every replay computes from its own
 * token ids and state.
 * Limits: d_model a multiple of 128 (<= 8192); d_state 64 or 128; every
 * layer's projections of those shapes; M >= 1; vocab >= 1.
 * The fused step: at M = 1, on a workspace that dfssm_mamba2_prepare has
 * prepared for this model, and for models of the 1.3B layer shape (d_model
 * 2048, d_state 128, LoRA factors with r <= 64 in every projection and
 * r % 4 == 0 for int8, r % 8 == 0 for int4), the layers run as one
 * persistent launch of one workgroup per compute unit (between the gather
 * and the final norm and LM head), with the same arithmetic; every other
 * case runs the per-kernel sequence above.  The fused launch needs the whole grid resident at once;
 * its waits are bounded and record a status bit (dfssm_mamba2_status) if
 * they give up, after which that step's outputs are incomplete.
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, UNSUPPORTED, DEVICE. */
dfssm_status dfssm_mamba2_decode_step(const dfssm_mamba2_model* model, int64_t M, const int32_t* tok,
                                      int64_t step, float* conv_ring, float* ssm_state, float* logits,
                                      void* workspace, size_t workspace_bytes, void* stream);

/* Prepares `workspace` for the fused step at M = 1 (see
 * dfssm_mamba2_decode_step): writes the layer table and its fingerprint
 * into the fused region and clears its exchange words, status and epochs
 * (stream-ordered, asynchronous), and records on the host that this
 * workspace holds this model's table.  Needed once per (model, workspace)
 * before decode steps at M = 1 take the fused path.  Call
 * dfssm_mamba2_release before freeing a prepared workspace: the record is
 * kept by address, and a new workspace at the same address would otherwise
 * be taken for a prepared one.  A no-op (DFSSM_OK) for M > 1 or models of
 * another shape.
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, UNSUPPORTED, DEVICE. */
dfssm_status dfssm_mamba2_prepare(const dfssm_mamba2_model* model, int64_t M, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* Drops the host-side record that dfssm_mamba2_prepare made for
 * `workspace` (host call, no device work; a no-op if there is none): the
 * next step on it runs the per-kernel sequence until it is prepared again.
 * Errors: none. */
dfssm_status dfssm_mamba2_release(const void* workspace);

/* *fused = 1 if dfssm_mamba2_decode_step on this model, M and workspace
 * takes the fused step (one persistent launch for the layers), else 0
 * (host call, no device work).
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE. */
dfssm_status dfssm_mamba2_fused_path(const dfssm_mamba2_model* model, int64_t M, const void* workspace,
                                     size_t workspace_bytes, int* fused);

/* Synchronises `stream` and reads the fused step's status word into
 * *status (host): 0 = fine; bit 1 = a wait for a linear's input timed out;
 * bit 2 = a wait for a row or rank partial timed out; bit 4 = a wait in the
 * SSM stage (B/C, dt or the partners' progress) timed out; bit 8 = the
 * fused region does not hold this model's table; bits 16..31 = 1 + the
 * index of the first linear (2 per layer) at which a workgroup gave up.
 * Bits accumulate until the next dfssm_mamba2_prepare.  0 when the fused
 * step is not in use.
 * Errors: NULL, SHAPE, ALIGN, WORKSPACE, DEVICE. */
dfssm_status dfssm_mamba2_status(const dfssm_mamba2_model* model, int64_t M, const void* workspace,
                                 size_t workspace_bytes, unsigned* status, void* stream);

/* ---- test switches ------------------------------------------------------ */

/* For tests only: forces a kernel-family choice that the automatic path
 * would otherwise make, for the whole process (all switches start at 0,
 * which leaves every choice automatic; a test sets a switch, runs its
 * calls, and sets it back to 0).  Results are the same integers and bits
 * on every choice; only the kernels that compute them change.
 *   DFSSM_TEST_LOCAL_LORA          1: the few-token kernel launches no LoRA
 *                                  workgroups; every output workgroup
 *                                  computes acc_a itself (the path it takes
 *                                  when the exchange words never arrive)
 *   DFSSM_TEST_PREFILL_KERNEL      4 or 8: the 4-wave or the 8-wave prefill
 *                                  kernel on the prefill path
 *   DFSSM_TEST_LM_HEAD_MFMA_TOKENS n > 0: the LM head runs on the matrix
 *                                  cores from n tokens instead of 8
 *   DFSSM_TEST_LM_HEAD_TILED_TOKENS n > 0: on the matrix cores, the tiled
 *                                  kernel (both operands staged in LDS)
 *                                  from n tokens instead of 64
 *   DFSSM_TEST_STEP_PER_KERNEL     1: the decode step at M = 1 runs the
 *                                  per-kernel sequence on a prepared
 *                                  workspace too; 2: the fused step takes
 *                                  every input maximum from the second
 *                                  exchange (its path for inputs with
 *                                  many near-equal largest entries)
 * Errors: SHAPE for an unknown switch or value. */
typedef enum {
  DFSSM_TEST_LOCAL_LORA = 1,
  DFSSM_TEST_PREFILL_KERNEL = 2,
  DFSSM_TEST_LM_HEAD_MFMA_TOKENS = 3,
  DFSSM_TEST_STEP_PER_KERNEL = 4,
  DFSSM_TEST_LM_HEAD_TILED_TOKENS = 5
} dfssm_test_switch_id;
dfssm_status dfssm_test_switch(int which, int value);

/* Static text for a status code. */
const char* dfssm_status_string(int status);
/* Thread-local description of the last failure on this thread ("" if none). */
const char* dfssm_last_error(void);
/* Library version string. */
const char* dfssm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DFSSM_H */
