/*
 * CPU oracle for the batch-1 decode step.  TEST INFRASTRUCTURE ONLY: see
 * oracle.h for what it computes, its precision, and who may call it.
 *
 * Written for reading, not speed: each function follows the definition of
 * one step in order.  OpenMP only spreads independent output rows, heads and
 * vocabulary entries across threads; every single sum runs in index order.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* bf16 is the upper half of an IEEE binary32; widening is exact. */
float orc_bf16_to_f32(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* Round a float to bf16, nearest-even (the KV cache storage rule). */
uint16_t orc_f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u); /* NaN */
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

/* IEEE binary16 -> float, exact (all binary16 values are floats). */
float orc_fp16_to_f32(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1f;
  int m = h & 0x3ff;
  double v;
  if (e == 0) v = ldexp((double)m, -24);
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = ldexp((double)(m | 0x400), e - 25);
  return (float)(sign ? -v : v);
}

/* RMSNorm: out_i = x_i / sqrt(mean_j x_j^2 + eps) * g_i.  eps sits inside
 * the square root and the gain multiplies after normalising. */
void orc_rmsnorm(const float* x, const uint16_t* g, int d, float eps, float* out) {
  double ss = 0.0;
  for (int i = 0; i < d; ++i) ss += (double)x[i] * (double)x[i];
  double inv = 1.0 / sqrt(ss / (double)d + (double)eps);
  for (int i = 0; i < d; ++i) out[i] = (float)((double)x[i] * inv * (double)orc_bf16_to_f32(g[i]));
}

/* y = W x with W [n_out][n_in] row-major.  bf16: W[n,k] widened to float.
 * int8 (W8A16, symmetric per output channel): W[n,k] = q[n,k] * s_n with s_n
 * an fp16 scale, so y_n = s_n * sum_k q[n,k] x_k. */
void orc_gemv(const void* w, const uint16_t* scale, int wfmt, int n_out, int n_in,
              const float* x, float* y) {
#pragma omp parallel for schedule(static)
  for (int n = 0; n < n_out; ++n) {
    double acc = 0.0;
    if (wfmt == ORC_BF16) {
      const uint16_t* row = (const uint16_t*)w + (size_t)n * (size_t)n_in;
      for (int k = 0; k < n_in; ++k) acc += (double)orc_bf16_to_f32(row[k]) * (double)x[k];
    } else {
      const int8_t* row = (const int8_t*)w + (size_t)n * (size_t)n_in;
      for (int k = 0; k < n_in; ++k) acc += (double)row[k] * (double)x[k];
      acc *= (double)orc_fp16_to_f32(scale[n]);
    }
    y[n] = (float)acc;
  }
}

/* Rotary position embedding, rotate-half convention, in place on one head:
 * for i < hd/2, theta_i = base^(-2i/hd), phi = pos * theta_i,
 *   u'_i        = u_i cos(phi) - u_{i+hd/2} sin(phi)
 *   u'_{i+hd/2} = u_{i+hd/2} cos(phi) + u_i sin(phi).
 * cos and sin are evaluated in double and rounded to float. */
void orc_rope(float* u, int head_dim, int pos, double base) {
  int half = head_dim / 2;
  for (int i = 0; i < half; ++i) {
    double theta = pow(base, -2.0 * (double)i / (double)head_dim);
    double phi = (double)pos * theta;
    double c = (double)(float)cos(phi);
    double s = (double)(float)sin(phi);
    double a = u[i], b = u[i + half];
    u[i] = (float)(a * c - b * s);
    u[i + half] = (float)(b * c + a * s);
  }
}

/* One query head against n_keys cached rows (bf16 [n_keys][hd] each):
 * s_j = (q . K_j) / sqrt(hd); a = softmax(s) = exp(s - max) / sum;
 * out = sum_j a_j V_j. */
void orc_attention_head(const float* q, const uint16_t* k_rows, const uint16_t* v_rows,
                        int n_keys, int head_dim, float* out) {
  double* s = (double*)malloc(sizeof(double) * (size_t)(n_keys > 0 ? n_keys : 1));
  double scale = 1.0 / sqrt((double)head_dim);
  double mx = -INFINITY;
  for (int j = 0; j < n_keys; ++j) {
    const uint16_t* kr = k_rows + (size_t)j * (size_t)head_dim;
    double dot = 0.0;
    for (int i = 0; i < head_dim; ++i) dot += (double)q[i] * (double)orc_bf16_to_f32(kr[i]);
    s[j] = dot * scale;
    if (s[j] > mx) mx = s[j];
  }
  double den = 0.0;
  for (int j = 0; j < n_keys; ++j) {
    s[j] = exp(s[j] - mx);
    den += s[j];
  }
  /* out_i = sum_j s_j V_ji / den, each sum over j in ascending order */
  double* acc = (double*)calloc((size_t)head_dim, sizeof(double));
  for (int j = 0; j < n_keys; ++j) {
    const uint16_t* vr = v_rows + (size_t)j * (size_t)head_dim;
    for (int i = 0; i < head_dim; ++i) acc[i] += s[j] * (double)orc_bf16_to_f32(vr[i]);
  }
  for (int i = 0; i < head_dim; ++i) out[i] = (float)(acc[i] / den);
  free(acc);
  free(s);
}

/* silu(z) = z / (1 + e^-z). */
double orc_silu(double z) { return z / (1.0 + exp(-z)); }

/* Index of the maximum; the lowest index wins ties; NaN ranks above
 * everything (the first NaN wins). */
int orc_argmax(const float* x, int n) {
  int best = 0;
  for (int i = 0; i < n; ++i) {
    if (isnan(x[i])) return i;
    if (x[i] > x[best]) best = i;
  }
  return best;
}

static const void* lin(const orc_layer* L, int which) {
  const void* p[7] = {L->wq, L->wk, L->wv, L->wo, L->w_gate, L->w_up, L->w_down};
  return p[which];
}
static const uint16_t* lin_scale(const orc_layer* L, int which) {
  const uint16_t* p[7] = {L->sq, L->sk, L->sv, L->so, L->s_gate, L->s_up, L->s_down};
  return p[which];
}

int orc_decode_step(const orc_model* m, uint16_t* kv, int token, int pos, float* logits) {
  return orc_decode_step_row(m, kv, token, pos, NULL, NULL, logits);
}

int orc_decode_step_row(const orc_model* m, uint16_t* kv, int token, int pos,
                        const uint16_t* row_in, uint16_t* row_out, float* logits) {
  const int d = m->d_model, H = m->n_heads, Hkv = m->n_kv_heads, hd = m->head_dim;
  const int F = m->ffn_dim, V = m->vocab, G = H / Hkv;
  if (token < 0 || token >= V || pos < 0 || pos >= m->max_ctx) return -1;
  const size_t head_stride = (size_t)m->max_ctx * (size_t)hd;   /* one kv head */
  const size_t kv_stride = (size_t)Hkv * head_stride;            /* K or V of a layer */

  float* x = (float*)malloc(sizeof(float) * (size_t)d);
  float* h = (float*)malloc(sizeof(float) * (size_t)d);
  float* q = (float*)malloc(sizeof(float) * (size_t)(H * hd));
  float* k = (float*)malloc(sizeof(float) * (size_t)(Hkv * hd));
  float* v = (float*)malloc(sizeof(float) * (size_t)(Hkv * hd));
  float* o = (float*)malloc(sizeof(float) * (size_t)(H * hd));
  float* y = (float*)malloc(sizeof(float) * (size_t)(d > F ? d : F));
  float* gt = (float*)malloc(sizeof(float) * (size_t)F);
  float* up = (float*)malloc(sizeof(float) * (size_t)F);
  float* mm = (float*)malloc(sizeof(float) * (size_t)F);

  /* 1. embedding row, widened to fp32 */
  for (int i = 0; i < d; ++i) x[i] = orc_bf16_to_f32(m->embed[(size_t)token * (size_t)d + (size_t)i]);

  for (int l = 0; l < m->n_layers; ++l) {
    const orc_layer* L = &m->layers[l];
    uint16_t* Kc = kv + (size_t)l * 2 * kv_stride;
    uint16_t* Vc = Kc + kv_stride;

    /* 2a. pre-attention RMSNorm */
    orc_rmsnorm(x, L->attn_norm, d, m->rms_eps, h);
    /* 2b. q, k, v projections */
    orc_gemv(lin(L, 0), lin_scale(L, 0), m->wfmt, H * hd, d, h, q);
    orc_gemv(lin(L, 1), lin_scale(L, 1), m->wfmt, Hkv * hd, d, h, k);
    orc_gemv(lin(L, 2), lin_scale(L, 2), m->wfmt, Hkv * hd, d, h, v);
    /* 2c. RoPE on every query and key head at this position */
    for (int hh = 0; hh < H; ++hh) orc_rope(q + hh * hd, hd, pos, m->rope_base);
    for (int g = 0; g < Hkv; ++g) orc_rope(k + g * hd, hd, pos, m->rope_base);
    /* 2d. append k, v to the bf16 cache at pos (or the supplied row's entries,
     * after handing out the step's own) */
    const size_t row_l = (size_t)l * 2 * (size_t)(Hkv * hd);
    for (int g = 0; g < Hkv; ++g) {
      for (int i = 0; i < hd; ++i) {
        uint16_t kb = orc_f32_to_bf16(k[g * hd + i]);
        uint16_t vb = orc_f32_to_bf16(v[g * hd + i]);
        const size_t rk = row_l + (size_t)(g * hd + i), rv = rk + (size_t)(Hkv * hd);
        if (row_out) { row_out[rk] = kb; row_out[rv] = vb; }
        if (row_in) { kb = row_in[rk]; vb = row_in[rv]; }
        Kc[(size_t)g * head_stride + (size_t)pos * hd + i] = kb;
        Vc[(size_t)g * head_stride + (size_t)pos * hd + i] = vb;
      }
    }
    /* 2e. each query head h attends over cached keys [0, pos] of kv head h/G */
#pragma omp parallel for schedule(static)
    for (int hh = 0; hh < H; ++hh) {
      int g = hh / G;
      orc_attention_head(q + hh * hd, Kc + (size_t)g * head_stride, Vc + (size_t)g * head_stride,
                         pos + 1, hd, o + hh * hd);
    }
    /* 2f. output projection and residual */
    orc_gemv(lin(L, 3), lin_scale(L, 3), m->wfmt, d, H * hd, o, y);
    for (int i = 0; i < d; ++i) x[i] = (float)((double)x[i] + (double)y[i]);
    /* 2g. pre-FFN RMSNorm, SwiGLU: m = silu(W_gate h) * (W_up h) */
    orc_rmsnorm(x, L->ffn_norm, d, m->rms_eps, h);
    orc_gemv(lin(L, 4), lin_scale(L, 4), m->wfmt, F, d, h, gt);
    orc_gemv(lin(L, 5), lin_scale(L, 5), m->wfmt, F, d, h, up);
    for (int i = 0; i < F; ++i) mm[i] = (float)(orc_silu((double)gt[i]) * (double)up[i]);
    /* 2h. down projection and residual */
    orc_gemv(lin(L, 6), lin_scale(L, 6), m->wfmt, d, F, mm, y);
    for (int i = 0; i < d; ++i) x[i] = (float)((double)x[i] + (double)y[i]);
  }
  /* 3. final RMSNorm and LM head */
  orc_rmsnorm(x, m->final_norm, d, m->rms_eps, h);
  orc_gemv(m->lm_head, m->s_lm_head, m->wfmt, V, d, h, logits);

  free(x); free(h); free(q); free(k); free(v); free(o); free(y); free(gt); free(up); free(mm);
  return 0;
}

int orc_verify(const orc_model* m, uint16_t* kv, const int32_t* tokens, int n, int pos,
               float* logits) {
  if (n < 1 || pos < 0 || pos + n > m->max_ctx) return -1;
  for (int i = 0; i < n; ++i) {
    int rc = orc_decode_step(m, kv, tokens[i], pos + i, logits + (size_t)i * (size_t)m->vocab);
    if (rc) return rc;
  }
  return 0;
}

int orc_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
