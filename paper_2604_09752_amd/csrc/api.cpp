// Host side of the C ABI declared in include/aio.h: argument checks, the
// workspace layout, model load (RoPE table), and launch sequencing.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "aio_internal.h"

// Scratch of aio_prefill_noalloc: one array per GPU the library runs on,
// held until the process ends.  In host code `scratch` is only a stand-in
// for the symbol; its device address on each GPU comes from
// hipGetSymbolAddress (g_scratch_dev), and only that address is ever used.
static __device__ __align__(256) char scratch[AIO_PREFILL_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_dev[kMaxDevices];  // device address of `scratch` on each GPU (null until set up)

// The device address of `scratch` on the current device, resolved once per
// device (with that device current).
hipError_t scratch_address(int dev, char** out) {
  *out = nullptr;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_dev[dev] = (char*)p;
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}

thread_local int g_last_hip = 0;

int hip_fail(hipError_t e) {
  g_last_hip = (int)e;
  return AIO_EHIP;
}

size_t align256(size_t v) { return (v + 255u) & ~(size_t)255u; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int env_int(const char* name, int dflt) {
  const char* s = getenv(name);
  if (!s || !*s) return dflt;
  return atoi(s);
}

// Split-KV partitions per head for the per-operation and verify attention:
// (split, kv head) workgroups to cover the 256 CUs once for caches of up to
// 8K positions (a workgroup's fixed cost then outweighs its keys; measured
// on the 7B verify at 2K: 4, 8, 16 splits 5.48, 5.24, 5.85 ms) and about
// twice beyond (at 32K: 16 splits 11.3 ms, 32 splits 12.4 ms), but no split
// shorter than 64 keys at full context.
int choose_splits(const aio_config& c) {
  int s = env_int("AIO_SPLITS", 0);
  if (s <= 0) {
    const int wgs = c.max_ctx <= 8192 ? 256 : 512;
    s = (wgs + c.n_kv_heads - 1) / c.n_kv_heads;
    int cap = c.max_ctx / 64;
    if (cap < 1) cap = 1;
    if (s > cap) s = cap;
  }
  if (s > 256) s = 256;
  if (s < 1) s = 1;
  return s;
}

}  // namespace

WsLayout aio_ws_layout(const aio_config& c) {
  WsLayout L{};
  const size_t MV = (size_t)c.max_verify, d = (size_t)c.d_model, F = (size_t)c.ffn_dim;
  const size_t Hd = (size_t)c.n_heads * (size_t)c.head_dim;
  L.splits = choose_splits(c);
  // verify attention: at least 4 key blocks of 32 per split, at most 64 splits
  L.vsplits = (int)std::min<size_t>(64, std::max<size_t>(1, ((size_t)c.max_ctx + 127) / 128));
  const size_t SP = (size_t)std::max(L.splits, L.vsplits);
  size_t ka = d > Hd ? d : Hd;
  if (F > ka) ka = F;
  L.ka = (int)ka;
  size_t off = 0;
  L.state = off; off = align256(off + sizeof(aio_state));
  L.x = off; off = align256(off + MV * d * 4);
  L.q = off; off = align256(off + MV * Hd * 4);
  L.o = off; off = align256(off + MV * Hd * 4);
  L.m = off; off = align256(off + F * 4);
  L.part_o = off; off = align256(off + MV * (size_t)c.n_heads * SP * c.head_dim * 4);
  L.part_ml = off; off = align256(off + MV * (size_t)c.n_heads * SP * 2 * 4);
  L.act = off; off = align256(off + 2 * 32 * ka * 2);  // two split-activation buffers
  L.vpart = off; off = align256(off + (size_t)kVerifyMaxKs * MV * d * 4);
  L.vss = off; off = align256(off + MV * (d / 64) * 4);
  L.vcnt = off; off = align256(off + (d / 64) * 4);
  L.sk_tiles = (F + 31) / 32;
  L.skpart = off;
  off = align256(off + L.sk_tiles * kVerifySkMaxC * AIO_MAX_VERIFY_ROWS * 64 * 4);
  L.skcnt = off; off = align256(off + L.sk_tiles * 4);
  // prefill K split (products with fewer tiles than two per CU): room for
  // 512 partial tiles of 128 x 64 fp32 and 1024 tile counters
  L.pfix_bytes = (size_t)512 * 128 * 64 * 4;
  L.pfix = off; off = align256(off + L.pfix_bytes);
  L.pcnt_n = 1024;
  L.pcnt = off; off = align256(off + L.pcnt_n * 4);
  L.vacnt = off; off = align256(off + (size_t)c.n_heads * 4);
  L.amax = off; off = align256(off + MV * 4);
  L.sync = off; off = align256(off + (size_t)kSyncWords * 4);
  // split-KV partitions per kv head in the step kernel: one per workgroup,
  // but at most 16.  With fewer kv heads the splits get short and the merge
  // of their partials long: the 1B (8 kv heads) at 2K positions, 32 splits
  // of 64 keys, 1204 tokens/s; 16 splits 1232; 8 splits 1197; 4 splits 1113.
  // (Fixed per model: a partial slot's previous contents must always come
  // from the previous layer, which its version tag tells apart.)
  L.mega_splits = std::min(AIO_STEP_MAX_BLOCKS / c.n_kv_heads, 16);
  if (L.mega_splits < 1) L.mega_splits = 1;
  L.mega_xa = off; off = align256(off + d * 4);
  L.mega_xb = off; off = align256(off + d * 4);
  L.mega_q = off; off = align256(off + Hd * 4);
  L.mega_kvn = off; off = align256(off + 2 * (size_t)c.n_kv_heads * c.head_dim * 4);
  L.mega_o = off; off = align256(off + Hd * 4);
  L.mega_m = off; off = align256(off + F * 4);
  L.mega_part = off;
  off = align256(off + (size_t)c.n_heads * (size_t)L.mega_splits * ((size_t)c.head_dim + 2) * 4);
  L.mega_end = off;
  L.total = off;
  return L;
}

extern "C" {

int aio_check_config(const aio_config* c) {
  if (!c) return AIO_EINVAL;
  if (c->n_layers < 1 || c->d_model < 64 || c->n_heads < 1 || c->n_kv_heads < 1 ||
      c->ffn_dim < 64 || c->vocab < 1 || c->max_ctx < 1 || c->head_dim < 1)
    return AIO_EINVAL;
  if (c->n_heads % c->n_kv_heads) return AIO_EINVAL;
  if (c->d_model % 64 || c->ffn_dim % 64) return AIO_EINVAL;
  if (c->wfmt != AIO_WFMT_BF16 && c->wfmt != AIO_WFMT_INT8) return AIO_EINVAL;
  if (!(c->rms_eps > 0.f) || !isfinite(c->rms_eps)) return AIO_EINVAL;
  if (!(c->rope_base > 1.f) || !isfinite(c->rope_base)) return AIO_EINVAL;
  if (c->max_verify < 1 || c->max_verify > AIO_MAX_VERIFY_ROWS) return AIO_EINVAL;
  if (c->head_dim != 64 && c->head_dim != 128) return AIO_EUNSUPPORTED;
  const int G = c->n_heads / c->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) return AIO_EUNSUPPORTED;
  if (c->max_ctx > (1 << 24) || c->vocab > (1 << 24) || c->d_model > (1 << 16) ||
      c->ffn_dim > (1 << 16) || c->n_layers > 1024 || c->n_heads > 1024)
    return AIO_EUNSUPPORTED;
  if ((size_t)c->n_heads * c->head_dim > 65536) return AIO_EUNSUPPORTED;
  return AIO_OK;
}

size_t aio_kv_bytes(const aio_config* c) {
  if (aio_check_config(c) != AIO_OK) return 0;
  return (size_t)c->n_layers * 2 * (size_t)c->n_kv_heads * (size_t)c->max_ctx *
         (size_t)c->head_dim * 2;
}

size_t aio_workspace_bytes(const aio_config* c) {
  if (aio_check_config(c) != AIO_OK) return 0;
  return aio_ws_layout(*c).total;
}

int aio_check_decode(const aio_config* c, int32_t token, int32_t pos) {
  int rc = aio_check_config(c);
  if (rc) return rc;
  if (token < 0 || token >= c->vocab) return AIO_ERANGE;
  if (pos < 0 || pos >= c->max_ctx) return AIO_ERANGE;
  return AIO_OK;
}

int aio_check_verify(const aio_config* c, int32_t token, const int32_t* drafts, int32_t k,
                     int32_t pos) {
  int rc = aio_check_config(c);
  if (rc) return rc;
  if (k < 0 || k + 1 > c->max_verify) return AIO_ERANGE;
  if (k > 0 && !drafts) return AIO_EINVAL;
  if (pos < 0 || (int64_t)pos + k >= (int64_t)c->max_ctx) return AIO_ERANGE;
  if (token < 0 || token >= c->vocab) return AIO_ERANGE;
  for (int i = 0; i < k; ++i)
    if (drafts[i] < 0 || drafts[i] >= c->vocab) return AIO_ERANGE;
  return AIO_OK;
}

const char* aio_strerror(int code) {
  switch (code) {
    case AIO_OK: return "ok";
    case AIO_EINVAL: return "invalid argument (null or misaligned pointer, inconsistent config)";
    case AIO_ERANGE: return "argument out of range (token, position or draft count)";
    case AIO_EUNSUPPORTED: return "unsupported shape or device";
    case AIO_EHIP: return "HIP runtime error";
    case AIO_ENOMEM: return "out of host or device memory";
    case AIO_EDEVICE: return "a bounded device-side wait gave up; the handle's results are invalid";
    default: return "unknown error";
  }
}

int aio_last_hip_error(void) { return g_last_hip; }

static int check_weights(const aio_config& c, const aio_weights* w) {
  if (!w || !w->layers) return AIO_EINVAL;
  const bool int8 = c.wfmt == AIO_WFMT_INT8;
  auto need = [](const void* p) { return p && aligned16(p); };
  auto scale_ok = [&](const void* s) { return int8 ? need(s) : s == nullptr; };
  if (!need(w->embed) || !need(w->final_norm) || !need(w->lm_head) || !scale_ok(w->s_lm_head))
    return AIO_EINVAL;
  for (int l = 0; l < c.n_layers; ++l) {
    const aio_layer_weights& L = w->layers[l];
    const void* mats[] = {L.wq, L.wk, L.wv, L.wo, L.w_gate, L.w_up, L.w_down};
    const void* scs[] = {L.sq, L.sk, L.sv, L.so, L.s_gate, L.s_up, L.s_down};
    if (!need(L.attn_norm) || !need(L.ffn_norm)) return AIO_EINVAL;
    for (int i = 0; i < 7; ++i)
      if (!need(mats[i]) || !scale_ok(scs[i])) return AIO_EINVAL;
  }
  return AIO_OK;
}

int aio_model_load(const aio_config* cfg, const aio_weights* w, void* kv_dev, void* ws_dev,
                   void* hip_stream, aio_model** out) {
  if (!out) return AIO_EINVAL;
  *out = nullptr;
  int rc = aio_check_config(cfg);
  if (rc) return rc;
  if ((rc = check_weights(*cfg, w))) return rc;
  if (!kv_dev || !ws_dev || !aligned16(kv_dev) || ((uintptr_t)ws_dev & 255u)) return AIO_EINVAL;

  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e);
  hipDeviceProp_t prop;
  if ((e = hipGetDeviceProperties(&prop, dev)) != hipSuccess) return hip_fail(e);
  if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) return AIO_EUNSUPPORTED;

  char* static_scratch = nullptr;
  if ((e = scratch_address(dev, &static_scratch)) != hipSuccess) return hip_fail(e);

  aio_model* m = new (std::nothrow) aio_model();
  if (!m) return AIO_ENOMEM;
  m->cfg = *cfg;
  m->static_scratch = static_scratch;
  m->layers.assign(w->layers, w->layers + cfg->n_layers);
  m->embed = w->embed;
  m->final_norm = w->final_norm;
  m->lm_head = w->lm_head;
  m->s_lm_head = w->s_lm_head;
  m->kv = (uint16_t*)kv_dev;
  m->ws = (char*)ws_dev;
  m->stream = (hipStream_t)hip_stream;
  m->lay = aio_ws_layout(*cfg);
  m->num_cus = prop.multiProcessorCount;
  m->greedy_exec = nullptr;
  m->greedy_logits = nullptr;
  m->greedy_tokens = nullptr;
  const char* g = getenv("AIO_GRAPH");
  m->use_graph = !(g && strcmp(g, "0") == 0) && hip_stream != nullptr;
  const char* mg = getenv("AIO_MEGA");
  m->use_mega = !(mg && strcmp(mg, "0") == 0) && aio_step_kernel_supports(*cfg) &&
                prop.cooperativeLaunch;
  m->mega_blocks = prop.multiProcessorCount < AIO_STEP_MAX_BLOCKS ? prop.multiProcessorCount
                                                                   : AIO_STEP_MAX_BLOCKS;
  const char* sl = getenv("AIO_STEP_LAUNCH");
  m->mega_coop = !(sl && strcmp(sl, "plain") == 0);

  // RoPE table: cos/sin of pos * base^(-2i/hd), angles in double, stored fp32.
  const int half = cfg->head_dim / 2;
  const size_t n = (size_t)cfg->max_ctx * (size_t)half;
  float2* host = (float2*)malloc(n * sizeof(float2));
  if (!host) { delete m; return AIO_ENOMEM; }
  for (int i = 0; i < half; ++i) {
    const double theta = pow((double)cfg->rope_base, -2.0 * (double)i / (double)cfg->head_dim);
    for (int p = 0; p < cfg->max_ctx; ++p) {
      const double phi = (double)p * theta;
      host[(size_t)p * half + i] = make_float2((float)cos(phi), (float)sin(phi));
    }
  }
  e = hipMalloc((void**)&m->rope, n * sizeof(float2));
  if (e == hipSuccess) e = hipMemcpy(m->rope, host, n * sizeof(float2), hipMemcpyHostToDevice);
  free(host);
  if (e == hipSuccess && m->use_mega) {
    std::vector<MegaLayer> tab((size_t)cfg->n_layers);
    for (int l = 0; l < cfg->n_layers; ++l) {
      const aio_layer_weights& L = w->layers[l];
      MegaLayer& t = tab[(size_t)l];
      const void* mats[7] = {L.wq, L.wk, L.wv, L.wo, L.w_gate, L.w_up, L.w_down};
      const void* scs[7] = {L.sq, L.sk, L.sv, L.so, L.s_gate, L.s_up, L.s_down};
      for (int i = 0; i < 7; ++i) {
        t.w[i] = mats[i];
        t.s[i] = (const uint16_t*)scs[i];
      }
      t.attn_norm = (const uint16_t*)L.attn_norm;
      t.ffn_norm = (const uint16_t*)L.ffn_norm;
      t.kc = m->kv_layer(l, 0);
      t.vc = m->kv_layer(l, 1);
    }
    e = hipMalloc((void**)&m->mega_layers, tab.size() * sizeof(MegaLayer));
    if (e == hipSuccess)
      e = hipMemcpy(m->mega_layers, tab.data(), tab.size() * sizeof(MegaLayer),
                    hipMemcpyHostToDevice);
    if (e == hipSuccess) {
      // gate/up rows start evenly split; aio_tune_step recalibrates them
      const int nb = m->mega_blocks;
      m->gu_bounds.resize((size_t)nb + 1);
      for (int b = 0; b <= nb; ++b) m->gu_bounds[b] = (int)((long long)b * m->cfg.ffn_dim / nb);
      e = hipMalloc((void**)&m->gu_bounds_dev, m->gu_bounds.size() * sizeof(int));
      if (e == hipSuccess)
        e = hipMemcpy(m->gu_bounds_dev, m->gu_bounds.data(), m->gu_bounds.size() * sizeof(int),
                      hipMemcpyHostToDevice);
    }
    if (e == hipSuccess) e = hipMemset(m->ws + m->lay.sync, 0, (size_t)kSyncWords * 4);
    if (e == hipSuccess) e = hipMemset(m->ws + m->lay.vcnt, 0, (size_t)(cfg->d_model / 64) * 4);
    if (e == hipSuccess) e = hipMemset(m->ws + m->lay.skcnt, 0, m->lay.sk_tiles * 4);
    if (e == hipSuccess) e = hipMemset(m->ws + m->lay.pcnt, 0, m->lay.pcnt_n * 4);
    if (e == hipSuccess) e = hipMemset(m->ws + m->lay.vacnt, 0, (size_t)cfg->n_heads * 4);
    if (e == hipSuccess)
      e = hipMemset(m->ws + m->lay.mega_xa, 0, m->lay.mega_end - m->lay.mega_xa);
  }
  if (e != hipSuccess) {
    if (m->rope) (void)hipFree(m->rope);
    if (m->mega_layers) (void)hipFree(m->mega_layers);
    if (m->gu_bounds_dev) (void)hipFree(m->gu_bounds_dev);
    delete m;
    return hip_fail(e);
  }
  *out = m;
  return AIO_OK;
}

void aio_model_free(aio_model* m) {
  if (!m) return;
  if (m->prof_ev) {
    for (int i = 0; i < m->prof_cap + 1; ++i) (void)hipEventDestroy(m->prof_ev[i]);
    free(m->prof_ev);
  }
  if (m->greedy_exec) (void)hipGraphExecDestroy(m->greedy_exec);
  if (m->rope) (void)hipFree(m->rope);
  if (m->mega_layers) (void)hipFree(m->mega_layers);
  if (m->gu_bounds_dev) (void)hipFree(m->gu_bounds_dev);
  if (m->mega_trace) (void)hipFree(m->mega_trace);
  if (m->pf_scratch) (void)hipFree(m->pf_scratch);
  delete m;
}

static hipError_t enqueue_step_body(aio_model* m, float* logits) {
  if (m->use_mega) return aio_launch_step_kernel(*m, logits, nullptr, nullptr);
  hipError_t e;
  for (int l = 0; l < m->cfg.n_layers; ++l)
    if ((e = aio_launch_decode_layer(*m, l)) != hipSuccess) return e;
  return aio_launch_lm_head(*m, logits);
}

int aio_decode_step(aio_model* m, int32_t token, int32_t pos, float* logits_dev) {
  if (!m || !logits_dev || !aligned16(logits_dev)) return AIO_EINVAL;
  int rc = aio_check_decode(&m->cfg, token, pos);
  if (rc) return rc;
  hipError_t e = aio_launch_set_state(*m, token, pos);
  if (e == hipSuccess) e = enqueue_step_body(m, logits_dev);
  return e == hipSuccess ? AIO_OK : hip_fail(e);
}

int aio_verify(aio_model* m, int32_t token, const int32_t* drafts, int32_t k, int32_t pos,
               float* logits_dev) {
  if (!m || !logits_dev || !aligned16(logits_dev)) return AIO_EINVAL;
  int rc = aio_check_verify(&m->cfg, token, drafts, k, pos);
  if (rc) return rc;
  int32_t rows[AIO_MAX_VERIFY_ROWS];
  rows[0] = token;
  for (int i = 0; i < k; ++i) rows[i + 1] = drafts[i];
  hipError_t e = aio_launch_set_rows(*m, rows, k + 1, pos);
  if (e == hipSuccess) e = aio_launch_verify(*m, k + 1, pos, logits_dev);
  return e == hipSuccess ? AIO_OK : hip_fail(e);
}

int aio_argmax(aio_model* m, const float* logits_dev, int32_t rows, int32_t n, int32_t* out_dev) {
  if (!m || !logits_dev || !out_dev) return AIO_EINVAL;
  if (((uintptr_t)logits_dev & 3u) || ((uintptr_t)out_dev & 3u)) return AIO_EINVAL;
  if (rows < 1 || rows > 65535 || n < 1 || n > (1 << 30)) return AIO_ERANGE;
  hipError_t e = aio_launch_argmax(*m, logits_dev, rows, n, out_dev, false);
  return e == hipSuccess ? AIO_OK : hip_fail(e);
}

static hipError_t enqueue_greedy_body(aio_model* m, float* logits, int32_t* tokens) {
  if (m->use_mega) return aio_launch_step_kernel(*m, logits, tokens, nullptr);
  hipError_t e = enqueue_step_body(m, logits);
  if (e != hipSuccess) return e;
  return aio_launch_argmax(*m, logits, 1, m->cfg.vocab, tokens, true);
}

static hipError_t ensure_greedy_graph(aio_model* m, float* logits, int32_t* tokens) {
  if (m->greedy_exec && m->greedy_logits == logits && m->greedy_tokens == tokens)
    return hipSuccess;
  if (m->greedy_exec) {
    (void)hipGraphExecDestroy(m->greedy_exec);
    m->greedy_exec = nullptr;
  }
  hipGraph_t graph = nullptr;
  hipError_t e = hipStreamBeginCapture(m->stream, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) return e;
  hipError_t body = enqueue_greedy_body(m, logits, tokens);
  e = hipStreamEndCapture(m->stream, &graph);
  if (body != hipSuccess) e = body;
  if (e == hipSuccess) e = hipGraphInstantiate(&m->greedy_exec, graph, nullptr, nullptr, 0);
  if (graph) (void)hipGraphDestroy(graph);
  if (e != hipSuccess) {
    m->greedy_exec = nullptr;
    return e;
  }
  m->greedy_logits = logits;
  m->greedy_tokens = tokens;
  return hipSuccess;
}

int aio_decode_greedy(aio_model* m, int32_t token, int32_t pos, int32_t n_steps,
                      int32_t* tokens_dev, float* logits_dev) {
  if (!m || !tokens_dev || !logits_dev || !aligned16(logits_dev) || ((uintptr_t)tokens_dev & 3u))
    return AIO_EINVAL;
  int rc = aio_check_decode(&m->cfg, token, pos);
  if (rc) return rc;
  if (n_steps < 1 || (int64_t)pos + n_steps > (int64_t)m->cfg.max_ctx) return AIO_ERANGE;
  hipError_t e = aio_launch_set_state(*m, token, pos);
  if (e != hipSuccess) return hip_fail(e);
  if (m->use_graph && !m->use_mega) {
    if ((e = ensure_greedy_graph(m, logits_dev, tokens_dev)) != hipSuccess) return hip_fail(e);
    for (int s = 0; s < n_steps; ++s)
      if ((e = hipGraphLaunch(m->greedy_exec, m->stream)) != hipSuccess) return hip_fail(e);
    return AIO_OK;
  }
  for (int s = 0; s < n_steps; ++s)
    if ((e = enqueue_greedy_body(m, logits_dev, tokens_dev)) != hipSuccess) return hip_fail(e);
  return AIO_OK;
}

int aio_profile_step(aio_model* m, int32_t token, int32_t pos, float* logits_dev,
                     float* kernel_ms, int32_t max_kernels, int32_t* n_kernels) {
  if (!m || !logits_dev || !aligned16(logits_dev) || !kernel_ms || !n_kernels || max_kernels < 1)
    return AIO_EINVAL;
  int rc = aio_check_decode(&m->cfg, token, pos);
  if (rc) return rc;
  const int need = m->use_mega ? 1 : 6 * m->cfg.n_layers + 1;
  if (!m->prof_ev) {
    m->prof_ev = (hipEvent_t*)calloc((size_t)need + 1, sizeof(hipEvent_t));
    if (!m->prof_ev) return AIO_ENOMEM;
    for (int i = 0; i < need + 1; ++i) {
      hipError_t e = hipEventCreate(&m->prof_ev[i]);
      if (e != hipSuccess) return hip_fail(e);
    }
    m->prof_cap = need;
  }
  hipError_t e = aio_launch_set_state(*m, token, pos);
  if (e == hipSuccess) e = hipEventRecord(m->prof_ev[0], m->stream);
  if (e != hipSuccess) return hip_fail(e);
  hipEvent_t* saved = m->prof_ev;
  m->prof_ev = saved + 1;  // events 1..need follow the kernels
  m->prof_n = 0;
  e = enqueue_step_body(m, logits_dev);
  const int n = m->prof_n;
  m->prof_ev = saved;
  m->prof_n = 0;
  if (e != hipSuccess) return hip_fail(e);
  if ((e = hipEventSynchronize(saved[n])) != hipSuccess) return hip_fail(e);
  const int out = n < max_kernels ? n : max_kernels;
  for (int i = 0; i < out; ++i) {
    float ms = 0.f;
    if ((e = hipEventElapsedTime(&ms, saved[i], saved[i + 1])) != hipSuccess) return hip_fail(e);
    kernel_ms[i] = ms;
  }
  *n_kernels = out;
  return AIO_OK;
}

int aio_trace_step(aio_model* m, int32_t token, int32_t pos, float* logits_dev, double* phase_us,
                   int32_t max_phases, int32_t* n_phases) {
  if (!m || !logits_dev || !aligned16(logits_dev) || !phase_us || !n_phases || max_phases < 1)
    return AIO_EINVAL;
  int rc = aio_check_decode(&m->cfg, token, pos);
  if (rc) return rc;
  if (!m->use_mega) return AIO_EUNSUPPORTED;
  const int nb = 5 * m->cfg.n_layers + 1;  // barrier slots 1..5L, slot 0 unused
  hipError_t e = hipSuccess;
  if (!m->mega_trace) e = hipMalloc((void**)&m->mega_trace, (size_t)(nb + 1) * 8);
  if (e == hipSuccess) e = hipMemsetAsync(m->mega_trace, 0, (size_t)(nb + 1) * 8, m->stream);
  if (e == hipSuccess) e = aio_launch_set_state(*m, token, pos);
  if (e == hipSuccess) e = aio_launch_step_kernel(*m, logits_dev, nullptr, m->mega_trace);
  if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
  if (e != hipSuccess) return hip_fail(e);
  std::vector<unsigned long long> t((size_t)nb + 1);
  e = hipMemcpy(t.data(), m->mega_trace, t.size() * 8, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e);
  int clk_khz = 0;
  int dev = 0;
  (void)hipGetDevice(&dev);
  if (hipDeviceGetAttribute(&clk_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      clk_khz <= 0)
    clk_khz = 100000;
  // barrier exits 1..5L bound 5L - 1 phases (the first QKV and the LM head
  // lie outside them)
  const int out = (nb - 2) < max_phases ? (nb - 2) : max_phases;
  for (int i = 0; i < out; ++i)
    phase_us[i] = (double)(t[(size_t)i + 2] - t[(size_t)i + 1]) * 1e3 / (double)clk_khz;
  *n_phases = out;
  return AIO_OK;
}

int aio_trace_barriers(aio_model* m, int32_t token, int32_t pos, float* logits_dev,
                       uint64_t* arrive, uint64_t* leave, int32_t max_entries,
                       int32_t* n_barriers, int32_t* n_blocks) {
  if (!m || !logits_dev || !aligned16(logits_dev) || !arrive || !leave || !n_barriers ||
      !n_blocks)
    return AIO_EINVAL;
  int rc = aio_check_decode(&m->cfg, token, pos);
  if (rc) return rc;
  if (!m->use_mega) return AIO_EUNSUPPORTED;
  const int nbar = 5 * m->cfg.n_layers + 1, nblk = m->mega_blocks;
  const size_t n = (size_t)nbar * (size_t)nblk;
  if ((size_t)max_entries < n) return AIO_ERANGE;
  unsigned long long* dev = nullptr;  // arrive [n], leave [n], detail [n][2]
  hipError_t e = hipMalloc((void**)&dev, 4 * n * 8);
  if (e == hipSuccess) e = hipMemsetAsync(dev, 0, 4 * n * 8, m->stream);
  if (e == hipSuccess) e = aio_launch_set_state(*m, token, pos);
  if (e == hipSuccess) e = aio_launch_step_kernel(*m, logits_dev, nullptr, nullptr, dev, dev + n);
  if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
  if (e == hipSuccess) e = hipMemcpy(arrive, dev, n * 8, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(leave, dev + n, n * 8, hipMemcpyDeviceToHost);
  if (e == hipSuccess && (size_t)max_entries >= 4 * n)  // room for the detail times too
    e = hipMemcpy(arrive + n, dev + 2 * n, 2 * n * 8, hipMemcpyDeviceToHost);
  if (dev) (void)hipFree(dev);
  if (e != hipSuccess) return hip_fail(e);
  *n_barriers = nbar;
  *n_blocks = nblk;
  return AIO_OK;
}

// New gate/up split from measured loop times: each workgroup's share moves
// halfway towards its streaming rate (units per unit of loop time), capped
// at the LDS sizing; integer counts keep the sum.
static void rebalance_gu(std::vector<int>& bounds, const std::vector<double>& loop_ticks,
                         int total, int cap) {
  const int nb = (int)bounds.size() - 1;
  std::vector<double> units(nb), rate(nb);
  double rsum = 0.0, usum = 0.0, tsum = 0.0;
  for (int b = 0; b < nb; ++b) {
    units[b] = bounds[b + 1] - bounds[b];
    usum += units[b];
    tsum += loop_ticks[b];
  }
  const double mean_rate = usum / std::max(tsum, 1.0);
  for (int b = 0; b < nb; ++b) {
    rate[b] = units[b] > 0 && loop_ticks[b] > 0 ? units[b] / loop_ticks[b] : mean_rate;
    rsum += rate[b];
  }
  std::vector<double> want(nb);
  double wsum = 0.0;
  for (int b = 0; b < nb; ++b) {
    const double target = total * rate[b] / rsum;
    want[b] = std::min((double)cap, std::max(1.0, 0.5 * units[b] + 0.5 * target));
    wsum += want[b];
  }
  std::vector<int> cnt(nb);
  std::vector<std::pair<double, int>> frac;
  int used = 0;
  for (int b = 0; b < nb; ++b) {
    const double x = want[b] * total / wsum;
    cnt[b] = std::min(cap, (int)x);
    used += cnt[b];
    frac.push_back({x - (int)x, b});
  }
  std::sort(frac.begin(), frac.end(), [](const auto& p, const auto& q) { return p.first > q.first; });
  for (int pass = 0; used < total && pass < 4; ++pass)
    for (size_t i = 0; i < frac.size() && used < total; ++i)
      if (cnt[frac[i].second] < cap) {
        cnt[frac[i].second] += 1;
        used += 1;
      }
  if (used != total) return;  // cannot happen while nb * cap >= total; keep the old split
  bounds[0] = 0;
  for (int b = 0; b < nb; ++b) bounds[b + 1] = bounds[b] + cnt[b];
}

int aio_tune_step(aio_model* m, int32_t token, int32_t pos, float* logits_dev, int32_t rounds) {
  if (!m || !logits_dev || !aligned16(logits_dev)) return AIO_EINVAL;
  int rc = aio_check_decode(&m->cfg, token, pos);
  if (rc) return rc;
  if (rounds < 1 || rounds > 64) return AIO_ERANGE;
  if (!m->use_mega) return AIO_EUNSUPPORTED;
  const int L = m->cfg.n_layers, nbar = 5 * L + 1, nblk = m->mega_blocks;
  const size_t n = (size_t)nbar * (size_t)nblk;
  const int cap = aio_step_kernel_gu_cap(m->cfg, nblk);
  std::vector<unsigned long long> det(2 * n);
  unsigned long long* dev = nullptr;  // arrive [n], leave [n], loop start/end [n][2]
  hipError_t e = hipMalloc((void**)&dev, 4 * n * 8);
  for (int r = 0; r < rounds && e == hipSuccess; ++r) {
    e = hipMemsetAsync(dev, 0, 4 * n * 8, m->stream);
    if (e == hipSuccess) e = aio_launch_set_state(*m, token, pos);
    if (e == hipSuccess) e = aio_launch_step_kernel(*m, logits_dev, nullptr, nullptr, dev, dev + n);
    if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
    if (e == hipSuccess) e = hipMemcpy(det.data(), dev + 2 * n, 2 * n * 8, hipMemcpyDeviceToHost);
    if (e != hipSuccess) break;
    // gate/up loop time of each workgroup over the layers (phase 5 l + 4)
    std::vector<double> ticks(nblk, 0.0);
    for (int l = 0; l < L; ++l) {
      const size_t k = (size_t)(5 * l + 4);
      for (int b = 0; b < nblk; ++b) {
        const unsigned long long t0 = det[(k * nblk + b) * 2], t1 = det[(k * nblk + b) * 2 + 1];
        if (t1 > t0) ticks[b] += (double)(t1 - t0);
      }
    }
    rebalance_gu(m->gu_bounds, ticks, m->cfg.ffn_dim, cap);
    e = hipMemcpy(m->gu_bounds_dev, m->gu_bounds.data(), m->gu_bounds.size() * sizeof(int),
                  hipMemcpyHostToDevice);
  }
  if (dev) (void)hipFree(dev);
  return e == hipSuccess ? AIO_OK : hip_fail(e);
}

int aio_device_status(aio_model* m, int32_t* status) {
  if (!m || !status) return AIO_EINVAL;
  *status = 0;
  if (!m->use_mega) return AIO_OK;
  hipError_t e = hipStreamSynchronize(m->stream);
  unsigned err = 0;
  if (e == hipSuccess)
    e = hipMemcpy(&err, m->ws + m->lay.sync + (size_t)kSyncErr * 4, 4, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e);
  *status = (int32_t)err;
  return AIO_OK;
}

int aio_uses_step_kernel(const aio_model* m) { return m && m->use_mega ? 1 : 0; }

// Enqueues a copy of the persistent kernel's status word into *word (0 for
// handles that do not use that kernel); valid after the stream's next
// synchronisation, which the generation loops make every round anyway.
static hipError_t enqueue_status_copy(const aio_model* m, unsigned* word) {
  *word = 0;
  if (!m->use_mega) return hipSuccess;
  return hipMemcpyAsync(word, m->ws + m->lay.sync + (size_t)kSyncErr * 4, 4,
                        hipMemcpyDeviceToHost, m->stream);
}

// ---------------------------------------------------- the probe's front end

// Rows of one prefill chunk when the library sizes the scratch: the whole
// prompt up to this many rows, in multiples of the GEMM's 64-row tiles.
constexpr int kPrefillChunk = 2048;

// Checks shared by the prefill entry points.
static int check_prefill(const aio_model* m, const int32_t* tokens, int32_t n, int32_t pos,
                         const float* logits_dev) {
  if (!m || !tokens || !logits_dev || !aligned16(logits_dev)) return AIO_EINVAL;
  const aio_config& c = m->cfg;
  if (n < 1 || pos < 0 || (int64_t)pos + n > c.max_ctx) return AIO_ERANGE;
  for (int32_t i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= c.vocab) return AIO_ERANGE;
  return AIO_OK;
}

// Enqueues the prompt in chunks of at most b.rcap rows, then the last row's
// final RMSNorm and LM head into logits_dev.
static hipError_t enqueue_prefill(aio_model* m, const PfBuffers& b, const int32_t* tokens,
                                  int32_t n, int32_t pos, float* logits_dev) {
  const int d = m->cfg.d_model;
  int32_t done = 0, rows = 0;
  hipError_t e = hipSuccess;
  while (done < n && e == hipSuccess) {
    rows = std::min(n - done, b.rcap);
    e = hipMemcpyAsync(b.tokens, tokens + done, (size_t)rows * sizeof(int32_t),
                       hipMemcpyHostToDevice, m->stream);
    if (e == hipSuccess) e = aio_launch_prefill_chunk(*m, b, rows, pos + done);
    done += rows;
  }
  if (e == hipSuccess)
    e = hipMemcpyAsync(m->at<float>(m->lay.x), b.x + (size_t)(rows - 1) * d,
                       (size_t)d * sizeof(float), hipMemcpyDeviceToDevice, m->stream);
  if (e == hipSuccess) e = aio_launch_lm_rows(*m, 1, logits_dev);
  return e;
}

// A prompt of at most max_verify tokens goes through the verify forward
// (skinny products over the weights once): at the 1B, 10 tokens take 1.5
// against 3.7 ms in prompt-length products, whose tiles are 64 rows.
static bool prefill_as_verify(const aio_model* m, int32_t n) { return n <= m->cfg.max_verify; }

// A single token is one decode step (the persistent kernel: 0.80 against
// 1.25 ms for the 1B in the verify forward).
static hipError_t enqueue_prefill_as_verify(aio_model* m, const int32_t* tokens, int32_t n,
                                            int32_t pos, float* logits_dev) {
  if (n == 1) {
    hipError_t e = aio_launch_set_state(*m, tokens[0], pos);
    if (e == hipSuccess) e = enqueue_step_body(m, logits_dev);
    return e;
  }
  hipError_t e = aio_launch_set_rows(*m, tokens, n, pos);
  if (e == hipSuccess) e = aio_launch_verify(*m, n, pos, logits_dev, true);
  return e;
}

int aio_prefill(aio_model* m, const int32_t* tokens, int32_t n, int32_t pos, float* logits_dev) {
  int rc = check_prefill(m, tokens, n, pos, logits_dev);
  if (rc) return rc;
  if (prefill_as_verify(m, n)) {
    const hipError_t e = enqueue_prefill_as_verify(m, tokens, n, pos, logits_dev);
    return e == hipSuccess ? AIO_OK : hip_fail(e);
  }
  const int want = std::min((n + 63) / 64 * 64, kPrefillChunk);
  if (m->pf_rcap < want) {
    // grow the library-owned scratch (synchronous; later calls reuse it)
    hipError_t e = hipSuccess;
    if (m->pf_scratch) e = hipStreamSynchronize(m->stream);
    if (e == hipSuccess && m->pf_scratch) e = hipFree(m->pf_scratch);
    m->pf_scratch = nullptr;
    m->pf_rcap = 0;
    if (e == hipSuccess)
      e = hipMalloc((void**)&m->pf_scratch, aio_prefill_buffers(m->cfg, nullptr, want).bytes);
    if (e != hipSuccess) {
      m->pf_scratch = nullptr;
      return e == hipErrorOutOfMemory ? AIO_ENOMEM : hip_fail(e);
    }
    m->pf_rcap = want;
  }
  const PfBuffers b = aio_prefill_buffers(m->cfg, m->pf_scratch, m->pf_rcap);
  const hipError_t e = enqueue_prefill(m, b, tokens, n, pos, logits_dev);
  return e == hipSuccess ? AIO_OK : hip_fail(e);
}

int aio_prefill_noalloc_rows(const aio_config* cfg) {
  if (aio_check_config(cfg) != AIO_OK) return 0;
  // as many rows as the array holds, padding of the regions included
  const size_t cap = AIO_PREFILL_NOALLOC_SCRATCH_BYTES;
  int rcap = (int)std::min<size_t>(cap / aio_prefill_row_bytes(*cfg), (size_t)kPrefillChunk);
  while (rcap > 0 && aio_prefill_buffers(*cfg, nullptr, rcap).bytes > cap) --rcap;
  return rcap;
}

int aio_prefill_noalloc(aio_model* m, const int32_t* tokens, int32_t n, int32_t pos,
                        float* logits_dev) {
  int rc = check_prefill(m, tokens, n, pos, logits_dev);
  if (rc) return rc;
  if (!m->static_scratch) return AIO_EINVAL;
  if (prefill_as_verify(m, n)) {  // no scratch beyond the workspace
    const hipError_t e = enqueue_prefill_as_verify(m, tokens, n, pos, logits_dev);
    return e == hipSuccess ? AIO_OK : hip_fail(e);
  }
  const int rcap = aio_prefill_noalloc_rows(&m->cfg);
  if (rcap < 1) return AIO_EUNSUPPORTED;  // one row's scratch exceeds the array
  const PfBuffers b = aio_prefill_buffers(m->cfg, m->static_scratch, rcap);
  const hipError_t e = enqueue_prefill(m, b, tokens, n, pos, logits_dev);
  return e == hipSuccess ? AIO_OK : hip_fail(e);
}

int aio_probe_route(const float* category_logits, int32_t n_categories, int32_t code_category,
                    int32_t ctx_len, int32_t ctx_limit, float tau, float* entropy,
                    int32_t* category) {
  if (!category_logits) return AIO_EINVAL;
  if (n_categories < 1 || code_category < 0 || code_category >= n_categories) return AIO_ERANGE;
  int best = 0;
  for (int i = 1; i < n_categories; ++i)
    if (category_logits[i] > category_logits[best]) best = i;
  // softmax entropy in double: H = log(Z) - sum p_i (x_i - max), Z = sum e^(x_i - max)
  const double mx = category_logits[best];
  double z = 0.0, ez = 0.0;
  for (int i = 0; i < n_categories; ++i) {
    const double d = (double)category_logits[i] - mx, w = exp(d);
    z += w;
    ez += w * d;
  }
  const float h = (float)(log(z) - ez / z);  // the value reported is the value compared
  if (entropy) *entropy = h;
  if (category) *category = best;
  return best == code_category && ctx_len <= ctx_limit && h <= tau ? 1 : 0;
}

int aio_category_entropy(aio_model* m, const float* logits_dev, const int32_t* label_ids,
                         int32_t n_labels, float* out_dev) {
  if (!m || !logits_dev || !label_ids || !out_dev) return AIO_EINVAL;
  if (((uintptr_t)logits_dev & 3u) || ((uintptr_t)out_dev & 3u)) return AIO_EINVAL;
  if (n_labels < 1 || n_labels > AIO_MAX_CATEGORIES) return AIO_ERANGE;
  for (int i = 0; i < n_labels; ++i)
    if (label_ids[i] < 0 || label_ids[i] >= m->cfg.vocab) return AIO_ERANGE;
  const hipError_t e = aio_launch_category_entropy(*m, logits_dev, label_ids, n_labels, out_dev);
  return e == hipSuccess ? AIO_OK : hip_fail(e);
}

// ------------------------------------------------ draft-model speculation

int aio_spec_generate(aio_model* target, aio_model* draft, int32_t pos, int32_t token,
                      int32_t n_new, int32_t k, float* target_logits_dev,
                      float* draft_logits_dev, int32_t* argmax_dev, int32_t* draft_tokens_dev,
                      int32_t* out, aio_spec_stats* stats) {
  if (!target || !draft || !target_logits_dev || !draft_logits_dev || !argmax_dev ||
      !draft_tokens_dev || !out)
    return AIO_EINVAL;
  if (!aligned16(target_logits_dev) || !aligned16(draft_logits_dev) ||
      ((uintptr_t)argmax_dev & 3u) || ((uintptr_t)draft_tokens_dev & 3u))
    return AIO_EINVAL;
  const aio_config& ct = target->cfg;
  const aio_config& cd = draft->cfg;
  if (ct.vocab != cd.vocab) return AIO_EINVAL;
  if (token < 0 || token >= ct.vocab || pos < 0 || n_new < 1 || k < 0 || k + 1 > ct.max_verify)
    return AIO_ERANGE;
  const int32_t ctx = std::min(ct.max_ctx, cd.max_ctx);
  if ((int64_t)pos + n_new > ctx) return AIO_ERANGE;
  aio_spec_stats st{};
  int32_t d[AIO_MAX_VERIFY_ROWS], y[AIO_MAX_VERIFY_ROWS];
  int32_t p = pos, t = token, made = 0;
  hipError_t e;
  while (made < n_new) {
    const int kk = std::min(std::min(k, n_new - made - 1), ctx - 1 - p);
    int rc;
    if (kk > 0) {
      // the draft consumes t, d1 .. d(kk-1) at p .. p+kk-1 and proposes d1 .. dkk
      if ((rc = aio_decode_greedy(draft, t, p, kk, draft_tokens_dev, draft_logits_dev))) return rc;
      e = hipMemcpyAsync(d, draft_tokens_dev, (size_t)kk * sizeof(int32_t), hipMemcpyDeviceToHost,
                         draft->stream);
      if (e == hipSuccess) e = hipStreamSynchronize(draft->stream);
      if (e != hipSuccess) return hip_fail(e);
      st.draft_steps += kk;
      rc = aio_verify(target, t, d, kk, p, target_logits_dev);
    } else {
      rc = aio_decode_step(target, t, p, target_logits_dev);
    }
    if (rc) return rc;
    if ((rc = aio_argmax(target, target_logits_dev, kk + 1, ct.vocab, argmax_dev))) return rc;
    unsigned bad_t = 0, bad_d = 0;
    e = hipMemcpyAsync(y, argmax_dev, (size_t)(kk + 1) * sizeof(int32_t), hipMemcpyDeviceToHost,
                       target->stream);
    if (e == hipSuccess) e = enqueue_status_copy(target, &bad_t);
    if (e == hipSuccess) e = enqueue_status_copy(draft, &bad_d);
    if (e == hipSuccess) e = hipStreamSynchronize(target->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(draft->stream);
    if (e != hipSuccess) return hip_fail(e);
    if (bad_t || bad_d) return AIO_EDEVICE;
    int a = 0;
    while (a < kk && d[a] == y[a]) ++a;  // row a's argmax follows d[0..a)
    st.rounds += 1;
    st.drafted += kk;
    st.accepted += a;
    for (int i = 0; i <= a && made < n_new; ++i) out[made++] = y[i];
    if (kk > 0 && a == kk && made < n_new) {
      // every draft accepted: the draft model has not consumed the last one
      if ((rc = aio_decode_step(draft, d[kk - 1], p + kk, draft_logits_dev))) return rc;
      st.draft_steps += 1;
    }
    p += a + 1;
    t = y[a];
  }
  if (stats) *stats = st;
  return AIO_OK;
}

// ------------------------------------------------- prompt-lookup decoding

int aio_pld_match(const int32_t* hist, int32_t n_hist, int32_t ngram_max, int32_t ngram_min,
                  int32_t k, int32_t* drafts, int32_t* n_drafts) {
  if (!n_drafts || (n_hist > 0 && !hist) || (k > 0 && !drafts)) return AIO_EINVAL;
  if (n_hist < 0 || k < 0 || ngram_min < 1 || ngram_max < ngram_min) return AIO_ERANGE;
  *n_drafts = 0;
  if (k == 0) return AIO_OK;
  // largest n-gram first; within one n, the earliest occurrence with a
  // continuation (the suffix itself starts at n_hist - n and has none)
  for (int n = std::min(ngram_max, n_hist - 1); n >= ngram_min; --n) {
    const int32_t* suffix = hist + (n_hist - n);
    for (int i = 0; i + n < n_hist; ++i) {
      if (!std::equal(suffix, suffix + n, hist + i)) continue;
      const int cnt = std::min(k, n_hist - (i + n));
      std::copy(hist + i + n, hist + i + n + cnt, drafts);
      *n_drafts = cnt;
      return AIO_OK;
    }
  }
  return AIO_OK;
}

int aio_pld_generate(aio_model* m, const int32_t* history, int32_t pos, int32_t token,
                     int32_t n_new, int32_t ngram_max, int32_t ngram_min, int32_t k,
                     float* logits_dev, int32_t* argmax_dev, int32_t* out, aio_pld_stats* stats) {
  if (!m || !logits_dev || !aligned16(logits_dev) || !argmax_dev || !out) return AIO_EINVAL;
  if (((uintptr_t)argmax_dev & 3u) || (pos > 0 && !history)) return AIO_EINVAL;
  const aio_config& c = m->cfg;
  if (token < 0 || token >= c.vocab || pos < 0 || n_new < 1 || k < 0 || k + 1 > c.max_verify ||
      ngram_min < 1 || ngram_max < ngram_min)
    return AIO_ERANGE;
  if ((int64_t)pos + n_new > c.max_ctx) return AIO_ERANGE;
  for (int32_t i = 0; i < pos; ++i)
    if (history[i] < 0 || history[i] >= c.vocab) return AIO_EINVAL;
  std::vector<int32_t> hist(history, history + pos);
  hist.reserve((size_t)pos + (size_t)n_new + 1);
  hist.push_back(token);
  aio_pld_stats st{};
  int32_t drafts[AIO_MAX_VERIFY_ROWS], y[AIO_MAX_VERIFY_ROWS];
  int32_t p = pos, t = token, made = 0;
  while (made < n_new) {
    const int kk = std::min(std::min(k, n_new - made - 1), c.max_ctx - 1 - p);
    int32_t nd = 0;
    if (kk > 0) {
      const int rc = aio_pld_match(hist.data(), (int32_t)hist.size(), ngram_max, ngram_min, kk,
                                   drafts, &nd);
      if (rc) return rc;
    }
    int rc = nd > 0 ? aio_verify(m, t, drafts, nd, p, logits_dev)
                    : aio_decode_step(m, t, p, logits_dev);
    if (rc) return rc;
    if ((rc = aio_argmax(m, logits_dev, nd + 1, c.vocab, argmax_dev))) return rc;
    unsigned bad = 0;
    hipError_t e = hipMemcpyAsync(y, argmax_dev, (size_t)(nd + 1) * sizeof(int32_t),
                                  hipMemcpyDeviceToHost, m->stream);
    if (e == hipSuccess) e = enqueue_status_copy(m, &bad);
    if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
    if (e != hipSuccess) return hip_fail(e);
    if (bad) return AIO_EDEVICE;
    int a = 0;
    while (a < nd && drafts[a] == y[a]) ++a;  // row a's argmax follows drafts[0..a)
    st.forwards += 1;
    st.verifies += nd > 0;
    st.drafted += nd;
    st.accepted += a;
    for (int i = 0; i <= a && made < n_new; ++i) {
      out[made++] = y[i];
      hist.push_back(y[i]);
    }
    p += a + 1;
    t = y[a];
  }
  if (stats) *stats = st;
  return AIO_OK;
}

}  // extern "C"
