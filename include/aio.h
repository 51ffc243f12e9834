/*
 * aio.h -- C ABI of the batch-1 decode step on MI355X (gfx950).
 *
 * The operation.  A-IO (arXiv 2604.09752) routes requests between a 1B probe
 * and a 7B backbone because batch-1 autoregressive decoding is bound by HBM
 * bandwidth: every generated token fetches the full weight set (Section 2.1,
 * "The Memory-Bound Dilemma"; Section 3.1, about 14 GB per token for the 7B
 * and 2 GB for the 1B).  This library is that decode step for a dense
 * decoder-only transformer -- pre-norm RMSNorm, rotate-half RoPE,
 * grouped-query attention, SwiGLU FFN, untied LM head, no biases -- in
 * hand-written HIP kernels.  It also provides the two variants the paper
 * toggles per request (Section 3.3 "Strategy Routing", Section 4.2): W8A16
 * storage-only quantization (int8 weights, fp16 per-output-channel scales,
 * dequantised inside the matrix-vector kernels) and the one-forward
 * verification of prompt-lookup drafts.
 *
 * Conventions.
 *  - Every pointer named *_dev is a device pointer on the current HIP device;
 *    the caller allocates and owns it (weights, KV cache, workspace, logits,
 *    token buffers).  The library only borrows them, never frees them, and
 *    keeps using the weight, KV and workspace pointers until aio_model_free.
 *  - The library owns only the model handle, a RoPE cos/sin table and any
 *    captured graph; aio_model_free releases exactly those.
 *  - Weight matrices are row-major [out][in] (y = W x).  bf16 is stored as
 *    uint16 bit patterns, fp16 scales likewise.
 *  - Device pointers must be 16-byte aligned (the workspace 256-byte
 *    aligned); d_model and ffn_dim must be multiples of 64.
 *  - All calls are asynchronous on the stream given at load time: a return of
 *    AIO_OK means the work is enqueued.  Results are valid after a stream
 *    synchronisation; device faults surface there.
 *  - Every argument is checked on the host before anything is enqueued; a
 *    rejected call enqueues nothing and changes nothing.  No call aborts or
 *    exits the process and no C++ exception crosses this interface.
 *  - A handle is not thread-safe; distinct handles are independent (a 1B and a
 *    7B model can be resident together, as in the paper's Section 3.1).
 *  - Decode state is (KV cache contents, position), owned by the caller.  Rows
 *    of the cache beyond the current position are never read, so rolling back
 *    after a rejected draft is just calling again at the earlier position.
 */
#ifndef AIO_H
#define AIO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- errors */
enum {
  AIO_OK = 0,
  AIO_EINVAL = -1,       /* null or misaligned pointer, inconsistent config */
  AIO_ERANGE = -2,       /* token or position out of range, k out of range  */
  AIO_EUNSUPPORTED = -3, /* shape or device this build does not handle      */
  AIO_EHIP = -4,         /* a HIP runtime or launch error; see aio_last_hip_error */
  AIO_ENOMEM = -5,       /* the library's own small allocations failed      */
  AIO_EDEVICE = -6       /* a bounded wait inside the persistent decode kernel
                            gave up (aio_device_status); the handle's results
                            from then on are invalid: free it and load again */
};

/* Weight storage formats. */
enum {
  AIO_WFMT_BF16 = 0, /* every projection and the LM head in bf16            */
  AIO_WFMT_INT8 = 1  /* W8A16: int8 [out][in] + fp16 scale [out], symmetric,
                        no zero point, W[n,k] = q[n,k] * s[n]; embedding and
                        norm gains stay bf16                                 */
};

/* Largest number of rows (the current token plus drafts) one aio_verify call
 * scores. */
#define AIO_MAX_VERIFY_ROWS 10

typedef struct aio_config {
  int32_t n_layers;   /* L                                                  */
  int32_t d_model;    /* d, multiple of 64                                  */
  int32_t n_heads;    /* H query heads                                      */
  int32_t n_kv_heads; /* Hkv key/value heads, H % Hkv == 0                  */
  int32_t head_dim;   /* hd, 64 or 128                                      */
  int32_t ffn_dim;    /* F, multiple of 64                                  */
  int32_t vocab;      /* V                                                  */
  int32_t max_ctx;    /* positions the KV cache holds                       */
  int32_t max_verify; /* rows per aio_verify call, 1..AIO_MAX_VERIFY_ROWS   */
  int32_t wfmt;       /* AIO_WFMT_BF16 or AIO_WFMT_INT8                     */
  float rms_eps;      /* RMSNorm epsilon (inside the square root)           */
  float rope_base;    /* RoPE base; theta_i = base^(-2i/hd)                 */
} aio_config;

/* Per-layer weights (device pointers).  Norm gains are bf16 [d].  With
 * AIO_WFMT_BF16 the projections are bf16 and the s_* scales must be NULL; with
 * AIO_WFMT_INT8 they are int8 and every s_* is an fp16 [out] array. */
typedef struct aio_layer_weights {
  const void* attn_norm; /* [d]                  */
  const void* ffn_norm;  /* [d]                  */
  const void* wq;        /* [H*hd][d]            */
  const void* wk;        /* [Hkv*hd][d]          */
  const void* wv;        /* [Hkv*hd][d]          */
  const void* wo;        /* [d][H*hd]            */
  const void* w_gate;    /* [F][d]               */
  const void* w_up;      /* [F][d]               */
  const void* w_down;    /* [d][F]               */
  const void *sq, *sk, *sv, *so, *s_gate, *s_up, *s_down;
} aio_layer_weights;

typedef struct aio_weights {
  const void* embed;               /* bf16 [V][d]                             */
  const void* final_norm;          /* bf16 [d]                                */
  const void* lm_head;             /* bf16 or int8 [V][d] (untied)            */
  const void* s_lm_head;           /* fp16 [V] for int8, else NULL            */
  const aio_layer_weights* layers; /* HOST array of n_layers entries; copied   */
} aio_weights;

typedef struct aio_model aio_model;

/* ----------------------------------------------------------- pure host calls */

/* Bytes of the KV cache: bf16 [n_layers][2 (K, V)][n_kv_heads][max_ctx][head_dim].
 * Returns 0 for an invalid config. */
size_t aio_kv_bytes(const aio_config* cfg);

/* Bytes of device workspace the model needs (activations, split-KV partials,
 * a small state block).  Returns 0 for an invalid config. */
size_t aio_workspace_bytes(const aio_config* cfg);

/* AIO_OK, or the error aio_model_load would return for this config. */
int aio_check_config(const aio_config* cfg);

/* Checks of one call's scalar arguments against a config, exactly as the entry
 * points make them (AIO_OK, AIO_EINVAL or AIO_ERANGE). */
int aio_check_decode(const aio_config* cfg, int32_t token, int32_t pos);
int aio_check_verify(const aio_config* cfg, int32_t token, const int32_t* drafts, int32_t k,
                     int32_t pos);

const char* aio_strerror(int code);

/* The last hipError_t this library saw on the calling thread (0 if none). */
int aio_last_hip_error(void);

/* ---------------------------------------------------------- model lifecycle */

/* Binds a model to caller-owned device memory.  One handle is one resident
 * model; the paper keeps its 1B probe and 7B backbone resident together in
 * full precision and switches between them per request (Section 3.1,
 * "System Architecture and Bandwidth Conservation"; Section 5.3), which here
 * is two handles.
 *  cfg, w      host structs; copied.
 *  kv_dev      aio_kv_bytes(cfg) bytes; positions the caller has not written
 *              are never read before a decode or verify call writes them.
 *  ws_dev      aio_workspace_bytes(cfg) bytes, used only by this handle.
 *  hip_stream  hipStream_t every later call enqueues on (NULL = default stream).
 *  out         receives the handle.
 * Allocates and fills the RoPE table (fp32 cos/sin of angles computed in
 * double on the host), so it synchronises once.  Fails with AIO_EUNSUPPORTED
 * on a device that is not gfx950. */
int aio_model_load(const aio_config* cfg, const aio_weights* w, void* kv_dev, void* ws_dev,
                   void* hip_stream, aio_model** out);

void aio_model_free(aio_model* m);

/* ------------------------------------------------------------- the hot path */

/* One decode step (Section 2.1, Section 3.1): consume `token` at position
 * `pos` (0-based; the cache must hold positions 0..pos-1), write its K and V
 * at `pos` in every layer, attend over positions [0, pos], and write fp32
 * logits [vocab] to logits_dev.
 * AIO_ERANGE: token not in [0, vocab) or pos not in [0, max_ctx). */
int aio_decode_step(aio_model* m, int32_t token, int32_t pos, float* logits_dev);

/* Prompt-lookup verification in one forward (Section 3.3, Section 4.2): rows
 * are [token, drafts[0..k-1]] (drafts is a HOST array) at positions
 * pos..pos+k.  Writes K/V of all k+1 rows; row i of logits_dev (fp32
 * [k+1][vocab]) equals the logits of aio_decode_step on row i's token after
 * rows 0..i-1, i.e. row i attends over positions [0, pos+i].
 * AIO_ERANGE: k < 0, k+1 > max_verify, pos < 0, pos+k >= max_ctx, or a token
 * outside [0, vocab). */
int aio_verify(aio_model* m, int32_t token, const int32_t* drafts, int32_t k, int32_t pos,
               float* logits_dev);

/* Greedy argmax of `rows` rows of `n` fp32 values each (row-major), one
 * int32 index per row into out_dev: the next token of greedy decoding, and
 * for a verify forward the per-row ids that prompt-lookup acceptance
 * compares with the drafts (Section 3.3, Strategy Routing; Section 4.2, PLD
 * Configuration).  The lowest index wins ties; NaN ranks above +Inf (the
 * first NaN wins), as torch.argmax orders them.  logits_dev and out_dev
 * 4-byte aligned.  AIO_ERANGE: rows outside [1, 65535] or n outside
 * [1, 2^30]. */
int aio_argmax(aio_model* m, const float* logits_dev, int32_t rows, int32_t n, int32_t* out_dev);

/* Device-resident greedy decoding for timing: consume `token` at `pos`, then
 * feed each step's argmax as the next token, for n_steps steps, with no host
 * round trip inside the loop (the persistent step kernel reads the token and
 * position from device state and advances them; the per-operation path
 * replays a captured HIP graph unless AIO_GRAPH is "0").  tokens_dev (int32 [n_steps]) receives the
 * argmax of every step; logits_dev (fp32 [vocab]) holds the last step's
 * logits.  AIO_ERANGE if pos + n_steps > max_ctx. */
int aio_decode_greedy(aio_model* m, int32_t token, int32_t pos, int32_t n_steps,
                      int32_t* tokens_dev, float* logits_dev);

/* Profiling: one aio_decode_step with a HIP event recorded on the model's
 * stream before the first kernel and after every kernel, then a wait for the
 * last event.  kernel_ms (host, max_kernels floats) receives each kernel's
 * event-to-event time in launch order -- one entry for the persistent step
 * kernel, else per layer: qkv, attention, split merge, o-projection,
 * gate/up, down; then the LM head -- and *n_kernels the count written.
 * Synchronises; not for the timed loop. */
int aio_profile_step(aio_model* m, int32_t token, int32_t pos, float* logits_dev,
                     float* kernel_ms, int32_t max_kernels, int32_t* n_kernels);

/* 1 if this handle runs each decode step as the single persistent kernel
 * (the default where the shape allows it and AIO_MEGA is not "0"), else 0
 * (a sequence of per-operation kernels). */
int aio_uses_step_kernel(const aio_model* m);

/* Phase timing of one decode step of the persistent kernel: the same work as
 * aio_decode_step, with workgroup 0 recording the device clock as it
 * publishes the outputs of each phase.  phase_us (host, max_phases doubles)
 * receives the time between consecutive phases' outputs, i.e. per layer:
 * attention, O projection, gate/up, down, next layer's QKV; *n_phases the
 * count written.  Synchronises.  AIO_EUNSUPPORTED when the handle does not
 * use that kernel. */
int aio_trace_step(aio_model* m, int32_t token, int32_t pos, float* logits_dev, double* phase_us,
                   int32_t max_phases, int32_t* n_phases);

/* Per-workgroup timing of one step of the persistent kernel, device clock
 * (100 MHz).  Phase k = 5 l + 1 .. 5 l + 5 of layer l is QKV, attention, O,
 * gate/up, down.  arrive[k][b] receives the time workgroup b published its
 * outputs of phase k, leave[k][b] the time it had the inputs of phase k + 1
 * (entry 0 unused).  With max_entries >= 4 (5 L + 1) x blocks, arrive also
 * carries, after its first (5 L + 1) x blocks entries, [phase][workgroup][2]
 * the start and end of each workgroup's weight loop (attention: the end of
 * its splits and of its merge).  n_barriers and n_blocks receive the
 * dimensions (5 L + 1 and blocks).  Allocates a device buffer and
 * synchronises; a profiling aid.  AIO_EUNSUPPORTED when the handle does not
 * use that kernel. */
int aio_trace_barriers(aio_model* m, int32_t token, int32_t pos, float* logits_dev,
                       uint64_t* arrive, uint64_t* leave, int32_t max_entries,
                       int32_t* n_barriers, int32_t* n_blocks);

/* Calibrates the persistent kernel's split of the gate/up rows over its
 * workgroups: runs `rounds` decode steps of `token` at `pos` (so it writes
 * that cache row, like aio_decode_step) with every workgroup timing its
 * gate/up loops, and after each moves every workgroup's share of rows
 * halfway towards its measured streaming rate (CUs and XCDs stream at
 * slightly different rates, steadily; an even split waits for the slowest).
 * The split stays with the handle for all later steps; results are
 * unchanged up to fp32 rounding order, which does not depend on the split.
 * Synchronises.  AIO_ERANGE: rounds outside [1, 64] or a bad token or pos;
 * AIO_EUNSUPPORTED when the handle does not use the persistent kernel. */
int aio_tune_step(aio_model* m, int32_t token, int32_t pos, float* logits_dev, int32_t rounds);

/* Synchronises the model's stream and reports the device-side status word:
 * 0, or 1 if a bounded wait of the persistent kernel for another
 * workgroup's data gave up.  The word is sticky: once set, the results of
 * that step and of every later call on the handle are invalid (free the
 * handle and load again).  Synchronises. */
int aio_device_status(aio_model* m, int32_t* status);

/* ------------------------------------------ prompt-lookup decoding (host) */

/* Prompt-lookup drafts: the draft source of PLD, which Section 3.3
 * ("Dynamic Policy Routing and Execution", Strategy Routing) enables per
 * request and Section 4.2 ("Models and Baselines", PLD Configuration)
 * configures by an n-gram window and a look-ahead length.  Pure host
 * function, no device work.  For n from min(ngram_max, n_hist - 1) down to
 * ngram_min, looks for the last n tokens of hist[0..n_hist) earlier in hist;
 * the earliest earlier occurrence that is followed by at least one token
 * wins, and the up to k tokens that follow it are the drafts.  drafts (host,
 * k int32) receives them and *n_drafts their count (0 when no n-gram
 * recurs).
 * AIO_EINVAL: a null pointer.  AIO_ERANGE: n_hist < 0, k < 0, ngram_min < 1
 * or ngram_max < ngram_min. */
int aio_pld_match(const int32_t* hist, int32_t n_hist, int32_t ngram_max, int32_t ngram_min,
                  int32_t k, int32_t* drafts, int32_t* n_drafts);

typedef struct aio_pld_stats {
  int32_t forwards; /* model forwards: verify calls plus single decode steps */
  int32_t verifies; /* forwards that scored drafts                          */
  int32_t drafted;  /* draft tokens scored                                  */
  int32_t accepted; /* draft tokens accepted                                */
} aio_pld_stats;

/* Greedy generation with prompt-lookup decoding (Section 3.3, Strategy
 * Routing; Section 4.2, PLD Configuration).  history (host, pos int32) holds
 * the tokens at positions 0..pos-1, whose K/V the cache already holds;
 * `token` is consumed at pos.  Each round drafts up to k tokens with
 * aio_pld_match over everything consumed so far plus `token` (never more
 * drafts than tokens still wanted, nor past the end of the cache), scores
 * [token, drafts] in one aio_verify (or one aio_decode_step when nothing
 * matches), takes each row's greedy argmax on the device, and accepts the
 * longest prefix of drafts in which every draft equals the argmax of the row
 * before it.  The argmax of the row after the last accepted draft is the
 * next token, consumed by the next round at pos + accepted + 1 (cache rows
 * written past that are overwritten later, never read).  out (host, n_new
 * int32) receives the generated tokens; they are the tokens plain greedy
 * decoding produces from the same state, whatever the acceptance.
 * logits_dev (fp32 [k+1][vocab], 16-byte aligned) and argmax_dev (int32
 * [k+1]) are scratch.  stats may be NULL.  Synchronises the model's stream
 * once per round and returns when all n_new tokens are generated, or with
 * AIO_EDEVICE as soon as a round finds the device status word set.
 * AIO_ERANGE: token outside [0, vocab), pos < 0, n_new < 1,
 * pos + n_new > max_ctx, k < 0, k + 1 > max_verify, ngram_min < 1 or
 * ngram_max < ngram_min.  AIO_EINVAL: a null pointer or a history token
 * outside [0, vocab). */
int aio_pld_generate(aio_model* m, const int32_t* history, int32_t pos, int32_t token,
                     int32_t n_new, int32_t ngram_max, int32_t ngram_min, int32_t k,
                     float* logits_dev, int32_t* argmax_dev, int32_t* out, aio_pld_stats* stats);

/* -------------------------------------------- the probe's front end (host) */

/* The probe's single forward over its templated request (Section 3.2,
 * "Probe-Based Request-Level Intent Sensing"; its cost is the "1B
 * Single-Token Prefill" of Section 5.3): consumes tokens[0..n) (host) at
 * positions pos .. pos+n-1 in prompt-length matrix products (up to 2048
 * rows per pass over the weights) with causal attention, writes every
 * token's K/V in every layer, and writes the logits after the last token,
 * fp32 [vocab], to logits_dev (16-byte aligned).  The result equals n
 * aio_decode_step calls up to rounding.  A single token is one decode step
 * (the kernels of aio_decode_step), and a prompt of 2 to max_verify tokens
 * goes through the verify forward (the kernels of aio_verify); neither takes
 * scratch beyond the workspace.  The scratch
 * (4 (1 + 2 d + H hd + max(d, H hd) + F) + d / 16 bytes per row, for up to
 * 2048 rows) is allocated by the library on the first call that needs more
 * and kept until
 * aio_model_free, so such a call synchronises once.  Asynchronous
 * otherwise, like aio_verify.
 * AIO_ERANGE: n < 1, pos < 0, pos + n > max_ctx or a token outside
 * [0, vocab); AIO_EINVAL: a null pointer; AIO_ENOMEM: the scratch could not
 * be allocated. */
int aio_prefill(aio_model* m, const int32_t* tokens, int32_t n, int32_t pos, float* logits_dev);

/* Bytes of the device array aio_prefill_noalloc takes its scratch from. */
#define AIO_PREFILL_NOALLOC_SCRATCH_BYTES (32u << 20)

/* aio_prefill for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops, harnesses that forbid allocation): the
 * same operation and kernels, with the scratch taken from a fixed array of
 * AIO_PREFILL_NOALLOC_SCRATCH_BYTES in the library's device memory instead
 * of library-allocated memory.  It calls no hipMalloc, hipFree or other
 * allocating routine.  The prompt goes through in passes of at most
 * aio_prefill_noalloc_rows(cfg) rows (the array divided by the scratch of
 * one row: 4 (1 + d + H hd + max(d, H hd) + F) bytes, and at most 2048),
 * so any n works; results equal aio_prefill's up to rounding (bit-identical
 * where both take the prompt in one pass; a prompt of at most max_verify
 * tokens takes aio_prefill's verify route and needs none of the array).
 * Every GPU holds one such array
 * for the whole process, shared by all calls on that GPU: calls that
 * overlap on one GPU (handles on different streams) race and must be
 * serialised by the caller.  Nothing in the array needs to start at zero:
 * each call writes every region before reading it.  Asynchronous like
 * aio_verify; the tokens are copied from host memory on the model's stream.
 * Errors as aio_prefill, and AIO_EUNSUPPORTED when a prompt of more than
 * max_verify tokens meets a config whose one row's scratch exceeds the
 * array (aio_prefill_noalloc_rows(cfg) == 0). */
int aio_prefill_noalloc(aio_model* m, const int32_t* tokens, int32_t n, int32_t pos,
                        float* logits_dev);

/* Rows aio_prefill_noalloc takes per pass for this config (0 for an
 * invalid config or when one row's scratch exceeds the array). */
int aio_prefill_noalloc_rows(const aio_config* cfg);

/* The probe's routing decision (Section 3.2 and Section 3.3, "Dynamic
 * Policy Routing and Execution"), pure host: the categories' scores are the
 * probe's logits of the n_categories label tokens (host array).  The
 * category is their argmax (lowest index on ties) and H(X) the Shannon
 * entropy, in nats, of their softmax.  The request goes to the small model
 * (return 1) when the category is `code_category`, ctx_len <= ctx_limit and
 * H(X) <= tau; otherwise to the large one (return 0).  *entropy and
 * *category receive H(X) and the category when not NULL.  Negative error
 * code (AIO_EINVAL: null logits; AIO_ERANGE: n_categories < 1 or
 * code_category outside [0, n_categories)) on bad arguments. */
int aio_probe_route(const float* category_logits, int32_t n_categories, int32_t code_category,
                    int32_t ctx_len, int32_t ctx_limit, float tau, float* entropy,
                    int32_t* category);

/* The probe's category scores on the device (Section 3.2): reads the
 * logits of the n_labels label tokens label_ids[0 .. n_labels) (host array
 * of vocabulary indices) from logits_dev (one fp32 row, e.g. what
 * aio_prefill wrote) and writes out_dev[0] = H(X), the Shannon entropy in
 * nats of their softmax, and out_dev[1] = the category (argmax, lowest index
 * on ties) as a float; the same values aio_probe_route computes on the host
 * from the same logits.  Enqueued on the model's stream; only the two floats
 * need to cross to the host for the routing decision (Section 3.3).
 * Returns AIO_EINVAL on null or misaligned pointers, AIO_ERANGE when
 * n_labels is outside [1, AIO_MAX_CATEGORIES] or a label id outside
 * [0, vocab). */
#define AIO_MAX_CATEGORIES 64
int aio_category_entropy(aio_model* m, const float* logits_dev, const int32_t* label_ids,
                         int32_t n_labels, float* out_dev);

/* ------------------------------------- draft-model speculative decoding */

typedef struct aio_spec_stats {
  int32_t rounds;      /* target forwards (verify calls plus single decode steps) */
  int32_t drafted;     /* draft tokens scored by the target                       */
  int32_t accepted;    /* draft tokens accepted                                   */
  int32_t draft_steps; /* decode steps of the draft model                         */
} aio_spec_stats;

/* Greedy generation with a draft model (Section 4.2, the DraftModel
 * baseline: the 1B model drafts for the 7B).  `target` and `draft` are two
 * resident models with the same vocabulary whose caches both hold the
 * sequence at positions 0..pos-1; `token` is consumed at pos.  Each round
 * the draft decodes up to k tokens greedily from the current token, the
 * target scores [token, drafts] in one aio_verify (one aio_decode_step when
 * no draft is wanted), and the longest prefix of drafts in which every draft
 * equals the target's argmax of the row before it is accepted; the target's
 * argmax after it is the next token.  When every draft is accepted the
 * draft model also consumes the last draft, so both caches hold the
 * sequence; rows past the accepted prefix are overwritten later, never
 * read.  out (host, n_new int32) receives the generated tokens, which equal
 * those of plain greedy decoding of the target.  target_logits_dev (fp32
 * [k+1][vocab]), draft_logits_dev (fp32 [vocab]), argmax_dev (int32 [k+1])
 * and draft_tokens_dev (int32 [k]) are scratch, each 16-byte aligned (the
 * int32 buffers 4-byte aligned); stats may be NULL.  Synchronises both
 * models' streams twice per round; returns AIO_EDEVICE as soon as either
 * model's device status word is found set.
 * AIO_EINVAL: a null handle or buffer, or vocabularies that differ.
 * AIO_ERANGE: token outside [0, vocab), pos < 0, n_new < 1, pos + n_new
 * beyond either cache, k < 0 or k + 1 > the target's max_verify. */
int aio_spec_generate(aio_model* target, aio_model* draft, int32_t pos, int32_t token,
                      int32_t n_new, int32_t k, float* target_logits_dev,
                      float* draft_logits_dev, int32_t* argmax_dev, int32_t* draft_tokens_dev,
                      int32_t* out, aio_spec_stats* stats);

#ifdef __cplusplus
}
#endif
#endif /* AIO_H */
