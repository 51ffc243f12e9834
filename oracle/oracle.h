/*
 * CPU oracle for the batch-1 decode step of a dense decoder-only transformer.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  It shares no code
 * with the GPU path and the GPU path never calls it.
 *
 * What it computes.  The paper (A-IO, Section 2.1 "The Memory-Bound Dilemma"
 * and Section 3.1 "System Architecture and Bandwidth Conservation") rests on
 * the autoregressive decode step, in which each generated token reads every
 * weight and the KV cache once.  It does not spell out the architecture, so
 * the decoder is the Llama-style one of the synthetic workloads: pre-norm
 * RMSNorm, rotate-half RoPE, grouped-query attention, SwiGLU FFN, untied LM
 * head, no biases.  W8A16 storage (Section 2.4 and Section 4.2 "Quantization")
 * is symmetric per-output-channel int8 with an fp16 scale.  Prompt-lookup
 * verification (Section 3.3 "Strategy Routing", Section 4.2 "PLD
 * Configuration") scores k drafts in one forward; here it is defined as the
 * k+1 sequential decode steps it must equal.
 *
 * Precision: weights are widened exactly to float; every activation stored
 * between steps is fp32 (as on the device); every sum (dot products, mean of
 * squares, softmax normaliser, attention-weighted values) accumulates in
 * double and is rounded to float once.  The KV cache holds bf16, rounded to
 * nearest even from the fp32 key/value.
 *
 * Parity status: each function below is pinned by the CPU tests against
 * closed forms, numpy fp64 brute force or a full causal recompute.
 */
#ifndef AIO_ORACLE_H
#define AIO_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_BF16 = 0, ORC_INT8 = 1 };

typedef struct orc_layer {
  const uint16_t* attn_norm; /* bf16 [d] */
  const uint16_t* ffn_norm;  /* bf16 [d] */
  /* bf16 [out][in] or int8 [out][in]; scales fp16 [out] for int8 */
  const void *wq, *wk, *wv, *wo, *w_gate, *w_up, *w_down;
  const uint16_t *sq, *sk, *sv, *so, *s_gate, *s_up, *s_down;
} orc_layer;

typedef struct orc_model {
  int n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  int max_ctx;
  int wfmt; /* ORC_BF16 or ORC_INT8 */
  float rms_eps;
  double rope_base;
  const uint16_t* embed;      /* bf16 [vocab][d] */
  const uint16_t* final_norm; /* bf16 [d] */
  const void* lm_head;        /* bf16 or int8 [vocab][d] */
  const uint16_t* s_lm_head;  /* fp16 [vocab] (int8 only) */
  const orc_layer* layers;    /* [n_layers] */
} orc_model;

/* ---- single operations (each used by the decode step) ---- */
float orc_bf16_to_f32(uint16_t b);
uint16_t orc_f32_to_bf16(float f);
float orc_fp16_to_f32(uint16_t h);
void orc_rmsnorm(const float* x, const uint16_t* g, int d, float eps, float* out);
void orc_gemv(const void* w, const uint16_t* scale, int wfmt, int n_out, int n_in,
              const float* x, float* y);
void orc_rope(float* u, int head_dim, int pos, double base);
void orc_attention_head(const float* q, const uint16_t* k_rows, const uint16_t* v_rows,
                        int n_keys, int head_dim, float* out);
double orc_silu(double z);
int orc_argmax(const float* x, int n);

/* ---- the decode step and its verify variant ----
 * kv: bf16 [n_layers][2][n_kv_heads][max_ctx][head_dim], read at positions
 * [0, pos] and written at pos.  logits: fp32 [vocab].  Returns 0, or -1 for an
 * out-of-range token or position. */
int orc_decode_step(const orc_model* m, uint16_t* kv, int token, int pos, float* logits);

/* The same step with the entries cached at pos supplied from outside: the
 * step's own bf16 K and V of every layer are written to row_out (layout
 * [n_layers][2][n_kv_heads][head_dim]) and row_in's entries, not the step's,
 * are stored at pos before that layer attends.  With row_in = the step's own
 * row this is orc_decode_step exactly.  It lets a comparison start every
 * position from identical state: a cache entry is a bf16 rounding, and two
 * correct fp32 evaluations may round one entry to neighbouring values. */
int orc_decode_step_row(const orc_model* m, uint16_t* kv, int token, int pos,
                        const uint16_t* row_in, uint16_t* row_out, float* logits);

/* rows = [tokens[0..n)] at positions pos..pos+n-1; logits fp32 [n][vocab]. */
int orc_verify(const orc_model* m, uint16_t* kv, const int32_t* tokens, int n, int pos,
               float* logits);

/* Threads OpenMP will use (reported beside the CPU timing). */
int orc_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
