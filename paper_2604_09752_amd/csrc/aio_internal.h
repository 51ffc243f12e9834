// Internal structures shared by the host side (api.cpp) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "aio.h"
#include "step_kernel.h"

// Device-resident decode state: the token(s) and position the next kernels
// consume.  aio_decode_step writes it with a one-thread kernel; in greedy mode
// the argmax kernel advances it, so a captured step graph can be replayed.
struct aio_state {
  int32_t token[16];
  int32_t pos;
  int32_t step;
  int32_t rows;
  int32_t pad[13];
};

// Offsets (bytes) of the workspace regions; every region is 256-byte aligned.
struct WsLayout {
  size_t state;    // aio_state
  size_t x;        // fp32 [MV][d]            residual stream
  size_t q;        // fp32 [MV][H*hd]         rotated queries
  size_t o;        // fp32 [MV][H*hd]         attention output
  size_t m;        // fp32 [F]                SwiGLU output (decode)
  size_t part_o;   // fp32 [MV][H][S][hd]     split-KV partial outputs
  size_t part_ml;  // fp32 [MV][H][S][2]      split-KV (max, sum) in log2 units
  size_t act;      // bf16 [2][32][KA]        split activations for the verify GEMM
  size_t vpart;    // fp32 [kVerifyMaxKs][MV][d] verify residual products split over K
  size_t vss;      // fp32 [MV][d/64]         verify rows' sums of squares per 64 columns
  size_t vcnt;     // int32 [d/64]            arrived K slices per column tile, zeroed at load
  size_t skpart;   // fp32 [sk_tiles][kVerifySkMaxC][AIO_MAX_VERIFY_ROWS*64] stream-K shared tile sums
  size_t skcnt;    // int32 [sk_tiles]        arrived workgroups per shared tile pair, zeroed at load
  size_t sk_tiles; // tile pairs of the stream-K gate/up product
  size_t pfix;     // fp32                    prefill K-slice partial tiles
  size_t pfix_bytes;
  size_t pcnt;     // int32 [pcnt_n]          arrived K slices per prefill tile, zeroed at load
  size_t pcnt_n;
  size_t vacnt;    // int32 [H]               finished attention splits per head, zeroed at load
  size_t amax;     // int32 [MV]              argmax scratch
  size_t sync;     // uint32 [kSyncWords]     step-kernel barriers and counters
  // step-kernel exchange buffers (tagged words), mega_xa .. mega_end zeroed at load
  size_t mega_xa;    // [d]
  size_t mega_xb;    // [d]
  size_t mega_q;     // [H*hd]
  size_t mega_kvn;   // [2][Hkv][hd]
  size_t mega_o;     // [H*hd]
  size_t mega_m;     // [F]
  size_t mega_part;  // [H][S_mega][hd+2] split partials
  size_t mega_end;
  size_t total;
  int splits;      // S, split-KV partitions per head
  int vsplits;     // most split-KV partitions of a verify attention (part_o holds max(S, this))
  int mega_splits; // S_mega, split-KV partitions per kv head in the step kernel
  int ka;          // KA = max(d, H*hd, F)
};

// Largest number of K slices a verify residual product (O, down) is split
// into; each slice's product goes to its own vpart slot.
constexpr int kVerifyMaxKs = 8;

// Most workgroups of the stream-K verify gate/up product that share one
// tile pair; each has its slot of partial sums in skpart.
constexpr int kVerifySkMaxC = 8;

WsLayout aio_ws_layout(const aio_config& c);

struct aio_model {
  aio_config cfg;
  std::vector<aio_layer_weights> layers;
  const void* embed;
  const void* final_norm;
  const void* lm_head;
  const void* s_lm_head;
  uint16_t* kv;          // caller-owned cache
  char* ws;              // caller-owned workspace
  hipStream_t stream;
  float2* rope;          // library-owned [max_ctx][hd/2] (cos, sin)
  WsLayout lay;
  int num_cus;
  hipGraphExec_t greedy_exec;  // one decode step reading aio_state, argmax feeding back
  float* greedy_logits;        // logits pointer baked into greedy_exec
  int32_t* greedy_tokens;      // token output pointer baked into greedy_exec
  bool use_graph;
  // persistent step kernel (one cooperative launch per decode step)
  bool use_mega;
  bool mega_coop;  // cooperative launch (default); plain launch when AIO_STEP_LAUNCH=plain
  int mega_blocks;
  MegaLayer* mega_layers;          // library-owned device table [n_layers]
  int* gu_bounds_dev;              // library-owned [mega_blocks + 1] gate/up unit bounds
  std::vector<int> gu_bounds;      // host copy
  unsigned long long* mega_trace;  // library-owned, allocated on first trace
  // prefill scratch (aio_prefill), library-owned, grown on demand
  char* pf_scratch;
  int pf_rcap;
  // device address of the static scratch array on this model's GPU
  // (aio_prefill_noalloc); not owned
  char* static_scratch;
  // profiling: when prof_ev is set, every launcher records one event after
  // each kernel it enqueues (aio_profile_step)
  mutable hipEvent_t* prof_ev;
  mutable int prof_n;
  int prof_cap;

  aio_state* state() const { return (aio_state*)(ws + lay.state); }
  template <class T>
  T* at(size_t off) const { return (T*)(ws + off); }
  uint16_t* kv_layer(int l, int kind) const {  // kind 0 = K, 1 = V
    size_t per = (size_t)cfg.n_kv_heads * (size_t)cfg.max_ctx * (size_t)cfg.head_dim;
    return kv + ((size_t)l * 2 + (size_t)kind) * per;
  }
};

// Records the next profiling event after a kernel launch (no-op unless
// aio_profile_step is running).
inline void aio_prof_mark(const aio_model& m) {
  if (m.prof_ev && m.prof_n < m.prof_cap) (void)hipEventRecord(m.prof_ev[m.prof_n++], m.stream);
}

// ---- launchers (decode_kernels.hip); each enqueues on m.stream ----
hipError_t aio_launch_set_state(const aio_model& m, int32_t token, int32_t pos);
hipError_t aio_launch_set_rows(const aio_model& m, const int32_t* toks, int rows, int32_t pos);
hipError_t aio_launch_decode_layer(const aio_model& m, int l);
hipError_t aio_launch_lm_head(const aio_model& m, float* logits);
hipError_t aio_launch_category_entropy(const aio_model& m, const float* logits,
                                       const int32_t* labels, int n, float* out);
hipError_t aio_launch_argmax(const aio_model& m, const float* logits, int rows, int n,
                             int32_t* out, bool greedy_feedback);

// ---- launchers (verify_kernels.hip) ----
// The verify forward of the rows set by aio_launch_set_rows at pos .. pos +
// rows - 1: their K/V in every layer and logits [rows][vocab], or with
// last_row_only the last row's logits [vocab] only.
hipError_t aio_launch_verify(const aio_model& m, int rows, int pos, float* logits,
                             bool last_row_only = false);
// Final RMSNorm and LM head of the first `rows` rows of the workspace's
// residual rows (lay.x): logits [rows][vocab].
hipError_t aio_launch_lm_rows(const aio_model& m, int rows, float* logits);

// ---- prefill (prefill_kernels.hip) ----
// Scratch of one prefill chunk of up to rcap prompt rows.
struct PfBuffers {
  int32_t* tokens;  // [rcap]
  float* x;         // [rcap][d] residual rows
  float* q;         // [rcap][H hd] rotated queries
  float* actA;      // [rcap][lda_a] activations: QKV input (x g), O input
  float* actN;      // [rcap][d] x g of the pre-FFN norm: the gate/up input
  float* actB;      // [rcap][lda_b] SwiGLU output: the down input
  float* ss;        // [rcap][d / 64] sums of squares of x over 64-column blocks
  int rcap, lda_a, lda_b;
  size_t bytes;     // total, every region 256-byte aligned
};
// Scratch bytes per prompt row (without alignment padding).
size_t aio_prefill_row_bytes(const aio_config& c);
// The chunk scratch laid out from `base` (null: only .bytes is meaningful).
PfBuffers aio_prefill_buffers(const aio_config& c, char* base, int rcap);
// One chunk of R <= b.rcap rows (tokens already in b.tokens) at positions
// pos0 .. pos0 + R - 1.
hipError_t aio_launch_prefill_chunk(const aio_model& m, const PfBuffers& b, int R, int pos0);
