// Interface between the host side and the persistent decode-step kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "aio.h"

struct aio_model;
struct aio_state;

// Per-layer pointers, kept in a small device table (too many for kernel
// arguments).  w: wq, wk, wv, wo, w_gate, w_up, w_down; s: their int8 scales.
struct MegaLayer {
  const void* w[7];
  const uint16_t* s[7];
  const uint16_t* attn_norm;
  const uint16_t* ffn_norm;
  uint16_t* kc;  // [Hkv][max_ctx][hd]
  uint16_t* vc;
};

// Words of the synchronisation region (uint32, zeroed at load).
enum {
  kSyncEpoch = 1040,     // epoch base carried from one launch to the next
  kSyncErr = 1056,       // set when a bounded wait gives up
  kSyncAmaxCount = 2112, // argmax arrival counter
  kSyncAmax = 2176,      // [1024][2] per-workgroup (value, index)
  kSyncWords = 4224
};

// Largest grid the step kernel uses (one workgroup per CU).
#define AIO_STEP_MAX_BLOCKS 256

struct MegaArgs {
  const MegaLayer* layers;
  const uint16_t* embed;
  const uint16_t* final_norm;
  const void* lm_head;
  const uint16_t* s_lm;
  const float2* rope;
  aio_state* st;
  // Buffers exchanged between workgroups, every word tagged with the version
  // of the phase that wrote it (zeroed at load: version 0, never expected).
  unsigned* xa;    // [d]            residual after the attention block
  unsigned* xb;    // [d]            residual after the MLP block
  unsigned* q;     // [H*hd]         rotated queries
  unsigned* kvn;   // [2][Hkv][hd]   new K and V rows, bf16 << 16 | version
  unsigned* o;     // [H*hd]         attention output
  unsigned* m;     // [F]            SwiGLU output
  unsigned* part;  // [H][S][hd + 2] split partials (output, max, sum)
  unsigned* sync;  // kSyncWords
  float* logits;   // [V]
  int32_t* tokens_out;
  unsigned long long* trace;       // optional: [5 L + 2] workgroup 0's publish time of each phase
  unsigned long long* bar_arrive;  // optional: [5 L + 1][blocks] publish time of phase k
  unsigned long long* bar_leave;   // optional: [5 L + 1][blocks] time the inputs of phase k + 1 were in
  unsigned long long* detail;      // optional: [5 L + 1][blocks][2] loop start and end of phase k
  const int* gu_bounds;            // [blocks + 1] gate/up units of each workgroup (null: even split)
  int L, d, H, Hkv, hd, F, V, max_ctx, S;
  int red_words;   // floats of one LDS buffer of matrix-phase partials
  float eps, scale_log2;
};

bool aio_step_kernel_supports(const aio_config& c);
// Most gate/up units (row pairs) one workgroup may own: the even share plus
// an eighth (at least 2), which the LDS partial buffers are sized for.
int aio_step_kernel_gu_cap(const aio_config& c, int blocks);
int aio_step_kernel_vpl(const aio_config& c, int K);
size_t aio_step_kernel_lds(const aio_config& c, int blocks);
hipError_t aio_launch_step_kernel(const aio_model& m, float* logits, int32_t* tokens_out,
                                  unsigned long long* trace,
                                  unsigned long long* bar_arrive = nullptr,
                                  unsigned long long* bar_leave = nullptr);
