/*
 * dfssm_ref.h -- CPU oracle for the DF-SSM scaffold + int8 LoRA linear.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, obviously-correct host
 * implementation used to check the GPU library.  Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load it.  The
 * product path (include/dfssm.h and its HIP kernels) never calls, links or
 * includes anything from this directory, and this directory includes nothing
 * from the product.
 *
 * What is computed (paper: Sec. 3.2, Eq. 3, frozen scaffold plus low-rank
 * correction; Sec. 3.3 and Table 1, 1-bit packed scaffold and int8 LoRA with
 * per-channel scales; Sec. 4.1, int8 activations fed to an int8 x int8
 * product), with the scaffold binarised to sign(W) and a per-row scale:
 *
 *     y = diag(alpha) * S * q(x)  +  diag(beta) * B * (A * q(x))
 *
 *   S      [N,K]  +-1 signs, stored 1 bit each, uint32 words [N][K/32],
 *                 bit j of word w is column 32*w + j, bit 1 means +1.
 *   A      [r,K]  int8 LoRA down-projection (the paper's W_B).
 *   B      [N,r]  int8 LoRA up-projection   (the paper's W_A).
 *   alpha  [N]    fp32 per-row scaffold scale.
 *   beta   [N]    fp32 per-row LoRA scale (per-channel int8 scales and the
 *                 scalar LoRA gain folded together).
 *   q(x)   = s * Q, per-token absmax int8 quantisation of x.
 *
 * Integer accumulators (exact):
 *   acc_s[m,n] = sum_k S[n,k] * Q[m,k]          int32
 *   acc_a[m,j] = sum_k A[j,k] * Q[m,k]          int32
 *   acc_b[m,n] = sum_j B[n,j] * acc_a[m,j]      int64
 *
 * Output:
 *   y64[m,n] = s[m] * (alpha[n]*acc_s + beta[n]*acc_b)   evaluated in fp64
 *   y32[m,n] = the same in fp32, one rounding per operation, in the order
 *              fs=(float)acc_s; u=alpha*fs; fb=(float)acc_b; v=beta*fb;
 *              w=u+v; y=s*w   (r==0: y=s*u).  This is the order in which
 *              the GPU library evaluates it; the chain needs it bit-exact
 *              because each output is re-quantised into the next input.
 *
 * Parity status: every function here is pinned by the CPU tests (brute
 * force, closed forms, invariants, hand-derived fixtures).
 *
 * Also here: the tied int8 embedding gather and LM head, and the Mamba-2
 * decode-step operations around the linears (below).
 */
#ifndef DFSSM_REF_H
#define DFSSM_REF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  DFSSM_REF_OK = 0,
  DFSSM_REF_ERR_NULL = 1,
  DFSSM_REF_ERR_SHAPE = 2,
  DFSSM_REF_ERR_NONFINITE = 7
};

enum { DFSSM_REF_F16 = 0, DFSSM_REF_F32 = 1 };

/* IEEE 754 binary16 bit pattern -> the binary32 value it denotes (exact). */
float dfssm_ref_f16_to_f32(uint16_t h);

/* Per-token absmax quantisation of x [M rows, row stride ldx elements] to
 * Q int8 [M,K] and s fp32 [M]:
 *   a = max_k |x[m,k]|
 *   a < FLT_MIN  ->  Q[m,:] = 0, s[m] = 0
 *   otherwise       s[m] = a/127, inv = 127/a, Q = clamp(rint(x*inv), -127, 127)
 * every step one fp32 operation rounded to nearest-even.
 * Returns DFSSM_REF_ERR_NONFINITE if any x is Inf/NaN. */
int dfssm_ref_quantize_act(const void* x, int x_dtype, int64_t M, int64_t K,
                           int64_t ldx, int8_t* q, float* s);

/* The linear.  All outputs are written (acc_* and y32/y64 may be NULL to
 * skip them).  K > 0, K % 32 == 0, M >= 0, N >= 0, 0 <= r <= 256. */
int dfssm_ref_scaffold_lora_linear(const int8_t* q, const float* s,
                                   int64_t M, int64_t K, int64_t N, int64_t r,
                                   const uint32_t* w_bits, const float* alpha,
                                   const int8_t* A, const int8_t* B,
                                   const float* beta,
                                   int32_t* acc_s, int32_t* acc_a,
                                   int64_t* acc_b, float* y32, double* y64);

/* A chain of linears in which each output is re-quantised as the next
 * input: linear 0 consumes (q0, s0); linear l >= 1 consumes
 * Q_l = quantise(y32_{l-1}[:, 0:K_l]) (fp32 input, row stride N_{l-1}) with
 * its scale fixed to s_l = 1/127, standing in for the normalisation that
 * sits between projections in the model.  Requires K_l <= N_{l-1}.
 * y_all receives every linear's y32 back to back (sum_l M*N_l floats);
 * q_all (optional) every linear's Q (sum_l M*K_l bytes). */
int dfssm_ref_chain(int n_layers, int64_t M, const int64_t* K,
                    const int64_t* N, const int64_t* r,
                    const uint32_t* const* w_bits, const float* const* alpha,
                    const int8_t* const* A, const int8_t* const* B,
                    const float* const* beta, const int8_t* q0,
                    const float* s0, float* y_all, int8_t* q_all);

/* The tied int8 embedding / LM head (Sec. 3.3: the embedding matrix is
 * quantised to int8 per row; Table 1: embedding and LM head are one tied
 * int8 table of 103 MB).  E [V,d] int8, scale [V] fp32: row v stands for
 * scale[v] * E[v,:].
 *
 * Embedding gather of token ids tok [M] (0 <= tok < V, else
 * DFSSM_REF_ERR_SHAPE):   x[m,k] = scale[tok[m]] * (float)E[tok[m],k]
 * (one fp32 multiply, exact inputs).  d > 0. */
int dfssm_ref_embed_gather(const int8_t* E, const float* scale, int64_t V, int64_t d,
                           const int32_t* tok, int64_t M, float* x);

/* LM head on per-token int8 hidden states (q, s) = quantise(h), the same
 * quantiser as the linear's input:
 *   acc[m,v]    = sum_k E[v,k] * Q[m,k]                 int32, exact
 *   logits[m,v] = s[m] * (scale[v] * (float)acc[m,v])   fp32, this order,
 *                                                       one rounding each
 * (float)acc rounds to nearest-even (|acc| <= 127^2 d may exceed 2^24).
 * acc or logits may be NULL.  d > 0, M >= 0, V >= 0. */
int dfssm_ref_lm_head(const int8_t* q, const float* s, int64_t M, int64_t d,
                      const int8_t* E, const float* scale, int64_t V,
                      int32_t* acc, float* logits);

/* ---- int4 LoRA factors -------------------------------------------------
 * Table 4 lists the scaffold with an int4 LoRA (perplexity 52.9 against
 * 49.1 for int8) without giving its format.  Reading: each factor value is
 * a two's-complement 4-bit integer in [-8, 7], two per byte, value 2i in
 * the low nibble of byte i and value 2i+1 in the high nibble, rows packed
 * along their contracted length (A [r][K/2] bytes, B [N][r/2] bytes, r
 * even); per-channel scales stay folded into beta.  The linear is then the
 * int8 linear above on the unpacked values, with the same exact integers.
 *
 * Unpacks n values from `packed` (ceil(n/2) bytes) into out[n]. */
int dfssm_ref_unpack_int4(const uint8_t* packed, int64_t n, int8_t* out);

/* ---- the Mamba-2 decode step around the linears ------------------------
 *
 * The paper keeps Mamba-2's layer and lists what runs around the two
 * projections at batch 1 (Sec. 4.1 and Table 13: RMSNorm, the convolution
 * step as a stateful shift register, the SSM step as a stateful recurrence,
 * and gate + norm), with three fixes to the step's semantics (Table 12):
 * the input enters the state as (x * dt) outer B, d_state is 128 for the
 * 1.3B model, and the gate is applied before the norm, norm(y * silu(z)).
 * The remaining sizes follow the public Mamba-2 design: d_inner = 2 d_model,
 * heads of P = 64 channels (H = d_inner / P), one B/C group, d_conv = 4, and
 * in_proj's output laid out as [z | x | B | C | dt] (d_inner, d_inner, N, N,
 * H values).
 *
 * Precision (one rounding per operation, in the order written):
 *   fp32   every elementwise step;
 *   fp64   exp, log1p, sqrt and divisions inside silu, softplus and the
 *          norm's scale, each rounded once to fp32 where it is used;
 *   fp64   the two reductions, sum g^2 of the norms and sum_n h C of the
 *          SSM output, over exact products of fp32 values, rounded once.
 *   silu(v)     = (float)(v / (1 + exp(-v)))                  in fp64
 *   softplus(v) = v > 20 ? v : (float)log1p(exp(v))            in fp64
 */

/* Residual add + RMSNorm + the linear's quantiser (in_proj's input, and the
 * final norm before the LM head):
 *   u'  = u + delta           (fp32; u' = u when delta is NULL)
 *   r   = (float)(1 / sqrt(sum_k (double)u'^2 / d + eps))
 *   o   = (u' * r) * w        (fp32)
 *   (Q, s) = quantise(o)      (dfssm_ref_quantize_act's rule)
 * u_out and o may be NULL; u_out may equal u.  d > 0. */
int dfssm_ref_add_rmsnorm_quant(const float* u, const float* delta, const float* w, float eps,
                                int64_t M, int64_t d, float* u_out, float* o, int8_t* q,
                                float* s);

/* The convolution step and the SSM step of one token per sequence.
 *   zxbcdt   [M, ld]  in_proj's output: z at 0, xBC at d_inner (conv_dim =
 *                     d_inner + 2N values), dt at d_inner + conv_dim (H values)
 *   conv_state [M][conv_dim][4]   shift register, updated: position 3 is the
 *                     newest input.  Each step shifts it one place towards
 *                     position 0 and writes the new xBC at position 3; then
 *                     c_out = silu((((w0 s0 + w1 s1) + w2 s2) + w3 s3) + b)
 *   conv_w [conv_dim][4], conv_b [conv_dim]
 *   dt_bias, A_log, D [H]
 *   ssm_state [M][H][P][N] fp32, updated
 *   y [M, d_inner] out; xbc [M, conv_dim] out (the conv outputs) or NULL
 * Per head h (x = c_out[h P + p], B = c_out[d_inner + n], C = c_out[d_inner +
 * N + n]):
 *   dt = softplus(dt_raw + dt_bias)     A = (float)(-exp(A_log))
 *   dA = (float)exp(dt * A)             (dt * A in fp32)
 *   h[p][n] = h[p][n] * dA + (dt * x) * B[n]
 *   y[h P + p] = (float)(sum_n (double)h[p][n] C[n] + (double)D x)
 * d_inner = H * P; P = headdim. */
int dfssm_ref_ssm_step(const float* zxbcdt, int64_t ld, int64_t M, int64_t d_inner,
                       int64_t d_state, int64_t headdim, float* conv_state,
                       const float* conv_w, const float* conv_b, const float* dt_bias,
                       const float* A_log, const float* D, float* ssm_state, float* y,
                       float* xbc);

/* Gate then norm, and the linear's quantiser (out_proj's input):
 *   g = y * silu(z)   (fp32);  r = (float)(1 / sqrt(sum_k (double)g^2 / d + eps))
 *   o = (g * r) * w   (fp32);  (Q, s) = quantise(o)
 * y [M, d]; z rows of stride ldz; o may be NULL.  d > 0. */
int dfssm_ref_gate_norm_quant(const float* y, const float* z, int64_t ldz, const float* w,
                              float eps, int64_t M, int64_t d, float* o, int8_t* q, float* s);

/* Number of OpenMP threads the row loops use (1 without OpenMP). */
int dfssm_ref_threads(void);
/* Sets the number of OpenMP threads later calls use (n > 0; no effect
 * without OpenMP).  For timing the oracle single-threaded. */
void dfssm_ref_set_threads(int n);

#ifdef __cplusplus
}
#endif

#endif /* DFSSM_REF_H */
