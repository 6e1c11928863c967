/*
 * dfssm_ref.c -- CPU oracle for the DF-SSM scaffold + int8 LoRA linear.
 *
 * TEST INFRASTRUCTURE ONLY (see dfssm_ref.h).  Plain loops, one output
 * element at a time, written from the definitions; nothing here is blocked,
 * fused or reordered.  Build: gcc -O2 -ffp-contract=off (no fast-math), so
 * every fp32 expression below is evaluated with one IEEE rounding per
 * operation and no fused multiply-add.
 */
#include "dfssm_ref.h"

#include <float.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

int dfssm_ref_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void dfssm_ref_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* IEEE 754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction
 * bits.  exponent 0 -> subnormal f * 2^-24; exponent 31 -> Inf/NaN;
 * otherwise (1024 + f) * 2^(e - 25).  Every binary16 value is exactly
 * representable in binary32, so ldexpf is exact here. */
float dfssm_ref_f16_to_f32(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1f;
  int f = h & 0x3ff;
  float mag;
  if (e == 0) {
    mag = ldexpf((float)f, -24);
  } else if (e == 31) {
    mag = (f == 0) ? INFINITY : NAN;
  } else {
    mag = ldexpf((float)(1024 + f), e - 25);
  }
  return sign ? -mag : mag;
}

static float load_x(const void* x, int x_dtype, int64_t idx) {
  if (x_dtype == DFSSM_REF_F16) return dfssm_ref_f16_to_f32(((const uint16_t*)x)[idx]);
  return ((const float*)x)[idx];
}

/* Per-token absmax quantisation (the int8 activation operand the paper's
 * int8 x int8 scaffold product consumes, Sec. 4.1; the scheme itself is
 * symmetric per-token absmax to +-127 with round-half-even). */
int dfssm_ref_quantize_act(const void* x, int x_dtype, int64_t M, int64_t K,
                           int64_t ldx, int8_t* q, float* s) {
  if (M < 0 || K <= 0 || ldx < K) return DFSSM_REF_ERR_SHAPE;
  if (x_dtype != DFSSM_REF_F16 && x_dtype != DFSSM_REF_F32) return DFSSM_REF_ERR_SHAPE;
  if (M > 0 && (!x || !q || !s)) return DFSSM_REF_ERR_NULL;
  for (int64_t m = 0; m < M; ++m) {
    float a = 0.0f;
    for (int64_t k = 0; k < K; ++k) {
      float v = load_x(x, x_dtype, m * ldx + k);
      if (!isfinite(v)) return DFSSM_REF_ERR_NONFINITE;
      float av = fabsf(v);
      if (av > a) a = av;
    }
    if (a < FLT_MIN) {
      s[m] = 0.0f;
      for (int64_t k = 0; k < K; ++k) q[m * K + k] = 0;
      continue;
    }
    s[m] = a / 127.0f;
    float inv = 127.0f / a;
    for (int64_t k = 0; k < K; ++k) {
      float v = load_x(x, x_dtype, m * ldx + k);
      float t = v * inv;
      float rq = rintf(t); /* default rounding mode: nearest, ties to even */
      if (rq > 127.0f) rq = 127.0f;
      if (rq < -127.0f) rq = -127.0f;
      q[m * K + k] = (int8_t)rq;
    }
  }
  return DFSSM_REF_OK;
}

/* One scaffold sign, read straight off the packed words (Table 1: 1 bit per
 * scaffold weight).  Bit (k mod 32) of word k/32 of row n; 1 -> +1, 0 -> -1. */
static int scaffold_sign(const uint32_t* w_bits, int64_t words_per_row,
                         int64_t n, int64_t k) {
  uint32_t word = w_bits[n * words_per_row + k / 32];
  return ((word >> (k % 32)) & 1u) ? +1 : -1;
}

static int check_linear_args(int64_t M, int64_t K, int64_t N, int64_t r) {
  if (M < 0 || N < 0 || K <= 0 || (K % 32) != 0) return DFSSM_REF_ERR_SHAPE;
  if (r < 0 || r > 256) return DFSSM_REF_ERR_SHAPE;
  return DFSSM_REF_OK;
}

/* Eq. 3 (Sec. 3.2) with a binary scaffold and int8 LoRA factors. */
int dfssm_ref_scaffold_lora_linear(const int8_t* q, const float* s,
                                   int64_t M, int64_t K, int64_t N, int64_t r,
                                   const uint32_t* w_bits, const float* alpha,
                                   const int8_t* A, const int8_t* B,
                                   const float* beta,
                                   int32_t* acc_s, int32_t* acc_a,
                                   int64_t* acc_b, float* y32, double* y64) {
  int st = check_linear_args(M, K, N, r);
  if (st != DFSSM_REF_OK) return st;
  if (M == 0 || N == 0) return DFSSM_REF_OK;
  if (!q || !s || !w_bits || !alpha) return DFSSM_REF_ERR_NULL;
  if (r > 0 && (!A || !B || !beta)) return DFSSM_REF_ERR_NULL;
  const int64_t wpr = K / 32;

  /* LoRA down-projection: acc_a = Q * A^T, int32.  |A|,|Q| <= 127, so
   * |acc_a| <= 127*127*K, which fits int32 for K below 133,000. */
  int32_t* a_buf = (int32_t*)malloc((size_t)(M * r > 0 ? M * r : 1) * sizeof(int32_t));
  if (!a_buf) return DFSSM_REF_ERR_NULL;
  for (int64_t m = 0; m < M; ++m) {
    for (int64_t j = 0; j < r; ++j) {
      int64_t sum = 0;
      for (int64_t k = 0; k < K; ++k) sum += (int64_t)A[j * K + k] * (int64_t)q[m * K + k];
      a_buf[m * r + j] = (int32_t)sum;
      if (acc_a) acc_a[m * r + j] = (int32_t)sum;
    }
  }

#ifdef _OPENMP
#pragma omp parallel for schedule(static)
#endif
  for (int64_t n = 0; n < N; ++n) {
    for (int64_t m = 0; m < M; ++m) {
      /* scaffold product, one sign at a time */
      int64_t ss = 0;
      for (int64_t k = 0; k < K; ++k)
        ss += (int64_t)scaffold_sign(w_bits, wpr, n, k) * (int64_t)q[m * K + k];
      /* LoRA up-projection, exact in int64 (127 * 127^2 * K * r can
       * exceed 2^31) */
      int64_t sb = 0;
      for (int64_t j = 0; j < r; ++j) sb += (int64_t)B[n * r + j] * (int64_t)a_buf[m * r + j];

      if (acc_s) acc_s[m * N + n] = (int32_t)ss;
      if (acc_b) acc_b[m * N + n] = sb;

      /* output scaling: y = s * (alpha*acc_s + beta*acc_b) */
      if (y64) {
        double d = (double)alpha[n] * (double)ss;
        if (r > 0) d = d + (double)beta[n] * (double)sb;
        y64[m * N + n] = (double)s[m] * d;
      }
      if (y32) {
        float fs = (float)ss; /* exact: |acc_s| <= 127*K < 2^24 */
        float u = alpha[n] * fs;
        float w;
        if (r > 0) {
          float fb = (float)sb; /* int64 -> fp32, round to nearest even */
          float v = beta[n] * fb;
          w = u + v;
        } else {
          w = u;
        }
        y32[m * N + n] = s[m] * w;
      }
    }
  }
  free(a_buf);
  return DFSSM_REF_OK;
}

int dfssm_ref_chain(int n_layers, int64_t M, const int64_t* K,
                    const int64_t* N, const int64_t* r,
                    const uint32_t* const* w_bits, const float* const* alpha,
                    const int8_t* const* A, const int8_t* const* B,
                    const float* const* beta, const int8_t* q0,
                    const float* s0, float* y_all, int8_t* q_all) {
  if (n_layers < 0 || M < 0) return DFSSM_REF_ERR_SHAPE;
  if (n_layers == 0 || M == 0) return DFSSM_REF_OK;
  for (int l = 0; l < n_layers; ++l) {
    int st = check_linear_args(M, K[l], N[l], r[l]);
    if (st != DFSSM_REF_OK) return st;
    if (l > 0 && K[l] > N[l - 1]) return DFSSM_REF_ERR_SHAPE;
  }
  int64_t kmax = 0;
  for (int l = 0; l < n_layers; ++l) kmax = K[l] > kmax ? K[l] : kmax;
  int8_t* qbuf = (int8_t*)malloc((size_t)(M * kmax));
  float* sbuf = (float*)malloc((size_t)M * sizeof(float));
  if (!qbuf || !sbuf) { free(qbuf); free(sbuf); return DFSSM_REF_ERR_NULL; }

  int64_t y_off = 0, q_off = 0, y_prev_off = 0;
  int st = DFSSM_REF_OK;
  for (int l = 0; l < n_layers && st == DFSSM_REF_OK; ++l) {
    if (l == 0) {
      memcpy(qbuf, q0, (size_t)(M * K[0]));
      memcpy(sbuf, s0, (size_t)M * sizeof(float));
    } else {
      st = dfssm_ref_quantize_act(y_all + y_prev_off, DFSSM_REF_F32, M, K[l],
                                  N[l - 1], qbuf, sbuf);
      if (st != DFSSM_REF_OK) break;
      for (int64_t m = 0; m < M; ++m) sbuf[m] = 1.0f / 127.0f;
    }
    if (q_all) memcpy(q_all + q_off, qbuf, (size_t)(M * K[l]));
    st = dfssm_ref_scaffold_lora_linear(qbuf, sbuf, M, K[l], N[l], r[l], w_bits[l],
                                        alpha[l], A[l], B[l], beta[l], NULL, NULL,
                                        NULL, y_all + y_off, NULL);
    y_prev_off = y_off;
    y_off += M * N[l];
    q_off += M * K[l];
  }
  free(qbuf);
  free(sbuf);
  return st;
}

/* ---- tied int8 embedding / LM head ------------------------------------- */

int dfssm_ref_embed_gather(const int8_t* E, const float* scale, int64_t V, int64_t d,
                           const int32_t* tok, int64_t M, float* x) {
  if (d <= 0 || V < 0 || M < 0) return DFSSM_REF_ERR_SHAPE;
  if (M == 0) return DFSSM_REF_OK;
  if (!E || !scale || !tok || !x) return DFSSM_REF_ERR_NULL;
  for (int64_t m = 0; m < M; ++m)
    if (tok[m] < 0 || (int64_t)tok[m] >= V) return DFSSM_REF_ERR_SHAPE;
  for (int64_t m = 0; m < M; ++m) {
    const int64_t v = tok[m];
    for (int64_t k = 0; k < d; ++k) x[m * d + k] = scale[v] * (float)E[v * d + k];
  }
  return DFSSM_REF_OK;
}

int dfssm_ref_lm_head(const int8_t* q, const float* s, int64_t M, int64_t d,
                      const int8_t* E, const float* scale, int64_t V,
                      int32_t* acc, float* logits) {
  if (d <= 0 || V < 0 || M < 0) return DFSSM_REF_ERR_SHAPE;
  if (M == 0 || V == 0) return DFSSM_REF_OK;
  if (!q || !s || !E || !scale) return DFSSM_REF_ERR_NULL;
#ifdef _OPENMP
#pragma omp parallel for schedule(static)
#endif
  for (int64_t v = 0; v < V; ++v) {
    for (int64_t m = 0; m < M; ++m) {
      int64_t sum = 0;
      for (int64_t k = 0; k < d; ++k) sum += (int64_t)E[v * d + k] * (int64_t)q[m * d + k];
      if (acc) acc[m * V + v] = (int32_t)sum;
      if (logits) {
        float fa = (float)(int32_t)sum;
        float t = scale[v] * fa;
        logits[m * V + v] = s[m] * t;
      }
    }
  }
  return DFSSM_REF_OK;
}

/* ---- int4 LoRA factors ------------------------------------------------- */

int dfssm_ref_unpack_int4(const uint8_t* packed, int64_t n, int8_t* out) {
  if (n < 0) return DFSSM_REF_ERR_SHAPE;
  if (n == 0) return DFSSM_REF_OK;
  if (!packed || !out) return DFSSM_REF_ERR_NULL;
  for (int64_t i = 0; i < n; ++i) {
    const int byte = packed[i / 2];
    const int nib = (i % 2 == 0) ? (byte & 0x0f) : (byte >> 4);
    out[i] = (int8_t)(nib >= 8 ? nib - 16 : nib);
  }
  return DFSSM_REF_OK;
}

/* ---- the Mamba-2 decode step around the linears ------------------------ */

static float silu_f(float v) {
  const double x = (double)v;
  return (float)(x / (1.0 + exp(-x)));
}

static float softplus_f(float v) {
  if (v > 20.0f) return v;
  return (float)log1p(exp((double)v));
}

/* r = 1 / sqrt(mean of squares + eps), the sum in fp64 over exact squares. */
static float rms_scale(const float* v, int64_t d, float eps) {
  double ss = 0.0;
  for (int64_t k = 0; k < d; ++k) ss += (double)v[k] * (double)v[k];
  return (float)(1.0 / sqrt(ss / (double)d + (double)eps));
}

int dfssm_ref_add_rmsnorm_quant(const float* u, const float* delta, const float* w, float eps,
                                int64_t M, int64_t d, float* u_out, float* o, int8_t* q,
                                float* s) {
  if (M < 0 || d <= 0 || !(eps >= 0.0f)) return DFSSM_REF_ERR_SHAPE;
  if (M == 0) return DFSSM_REF_OK;
  if (!u || !w || !q || !s) return DFSSM_REF_ERR_NULL;
  float* res = (float*)malloc((size_t)d * sizeof(float));
  float* on = (float*)malloc((size_t)(M * d) * sizeof(float));
  if (!res || !on) {
    free(res);
    free(on);
    return DFSSM_REF_ERR_NULL;
  }
  for (int64_t m = 0; m < M; ++m) {
    for (int64_t k = 0; k < d; ++k) res[k] = delta ? u[m * d + k] + delta[m * d + k] : u[m * d + k];
    const float r = rms_scale(res, d, eps);
    for (int64_t k = 0; k < d; ++k) {
      const float t = res[k] * r;
      on[m * d + k] = t * w[k];
    }
    if (u_out)
      for (int64_t k = 0; k < d; ++k) u_out[m * d + k] = res[k];
  }
  int st = dfssm_ref_quantize_act(on, DFSSM_REF_F32, M, d, d, q, s);
  if (o && st == DFSSM_REF_OK) memcpy(o, on, (size_t)(M * d) * sizeof(float));
  free(res);
  free(on);
  return st;
}

int dfssm_ref_ssm_step(const float* zxbcdt, int64_t ld, int64_t M, int64_t d_inner,
                       int64_t d_state, int64_t headdim, float* conv_state,
                       const float* conv_w, const float* conv_b, const float* dt_bias,
                       const float* A_log, const float* D, float* ssm_state, float* y,
                       float* xbc) {
  if (M < 0 || d_inner <= 0 || d_state <= 0 || headdim <= 0 || d_inner % headdim) return DFSSM_REF_ERR_SHAPE;
  const int64_t N = d_state, P = headdim, H = d_inner / headdim;
  const int64_t conv_dim = d_inner + 2 * N;
  if (ld < d_inner + conv_dim + H) return DFSSM_REF_ERR_SHAPE;
  if (M == 0) return DFSSM_REF_OK;
  if (!zxbcdt || !conv_state || !conv_w || !conv_b || !dt_bias || !A_log || !D || !ssm_state || !y)
    return DFSSM_REF_ERR_NULL;
  float* c_out = (float*)malloc((size_t)conv_dim * sizeof(float));
  if (!c_out) return DFSSM_REF_ERR_NULL;
  for (int64_t m = 0; m < M; ++m) {
    const float* row = zxbcdt + m * ld;
    /* convolution step: shift the register, append the new input, filter */
    for (int64_t c = 0; c < conv_dim; ++c) {
      float* st = conv_state + (m * conv_dim + c) * 4;
      st[0] = st[1];
      st[1] = st[2];
      st[2] = st[3];
      st[3] = row[d_inner + c];
      const float* wc = conv_w + c * 4;
      float v = wc[0] * st[0];
      v = v + wc[1] * st[1];
      v = v + wc[2] * st[2];
      v = v + wc[3] * st[3];
      v = v + conv_b[c];
      c_out[c] = silu_f(v);
    }
    if (xbc) memcpy(xbc + m * conv_dim, c_out, (size_t)conv_dim * sizeof(float));
    const float* Bv = c_out + d_inner;
    const float* Cv = c_out + d_inner + N;
    /* SSM step, head by head */
    for (int64_t h = 0; h < H; ++h) {
      const float dt = softplus_f(row[d_inner + conv_dim + h] + dt_bias[h]);
      const float A = (float)(-exp((double)A_log[h]));
      const float dA = (float)exp((double)(dt * A));
      for (int64_t p = 0; p < P; ++p) {
        const float x = c_out[h * P + p];
        const float dtx = dt * x;
        float* hs = ssm_state + ((m * H + h) * P + p) * N;
        double acc = 0.0;
        for (int64_t n = 0; n < N; ++n) {
          const float t1 = hs[n] * dA;
          const float t2 = dtx * Bv[n];
          hs[n] = t1 + t2;
          acc += (double)hs[n] * (double)Cv[n];
        }
        y[m * d_inner + h * P + p] = (float)(acc + (double)D[h] * (double)x);
      }
    }
  }
  free(c_out);
  return DFSSM_REF_OK;
}

int dfssm_ref_gate_norm_quant(const float* y, const float* z, int64_t ldz, const float* w,
                              float eps, int64_t M, int64_t d, float* o, int8_t* q, float* s) {
  if (M < 0 || d <= 0 || ldz < d || !(eps >= 0.0f)) return DFSSM_REF_ERR_SHAPE;
  if (M == 0) return DFSSM_REF_OK;
  if (!y || !z || !w || !q || !s) return DFSSM_REF_ERR_NULL;
  float* g = (float*)malloc((size_t)d * sizeof(float));
  float* on = (float*)malloc((size_t)(M * d) * sizeof(float));
  if (!g || !on) {
    free(g);
    free(on);
    return DFSSM_REF_ERR_NULL;
  }
  for (int64_t m = 0; m < M; ++m) {
    for (int64_t k = 0; k < d; ++k) g[k] = y[m * d + k] * silu_f(z[m * ldz + k]);
    const float r = rms_scale(g, d, eps);
    for (int64_t k = 0; k < d; ++k) on[m * d + k] = (g[k] * r) * w[k];
  }
  int st = dfssm_ref_quantize_act(on, DFSSM_REF_F32, M, d, d, q, s);
  if (o && st == DFSSM_REF_OK) memcpy(o, on, (size_t)(M * d) * sizeof(float));
  free(g);
  free(on);
  return st;
}
