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
  kSyncFlags = 0,        // [1024] barrier arrival epochs, one per workgroup
  kSyncRelease = 1024,   // barrier release epoch
  kSyncEpoch = 1040,     // epoch base carried from one launch to the next
  kSyncErr = 1056,       // set when a bounded wait gives up
  kSyncAttn = 1088,      // [1024] split counters per kv head
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
  float* x;        // [d]     residual
  float* q;        // [H*hd]  rotated queries
  float* o;        // [H*hd]  attention output
  float* m;        // [F]     SwiGLU output
  float* part;     // [H][S][hd + 2] split partials (output, max, sum)
  unsigned* sync;  // kSyncWords
  float* logits;   // [V]
  int32_t* tokens_out;
  unsigned long long* trace;  // optional: barrier exit times (workgroup 0), [5 L + 1]
  unsigned long long* bar_arrive;  // optional: [5 L + 1][blocks] arrival times
  unsigned long long* bar_leave;   // optional: [5 L + 1][blocks] exit times
  unsigned long long* detail;      // optional: [5 L + 1][blocks][2] input-ready, loop-done
  int L, d, H, Hkv, hd, F, V, max_ctx, S;
  float eps, scale_log2;
};

bool aio_step_kernel_supports(const aio_config& c);
int aio_step_kernel_vpl(const aio_config& c, int K);
size_t aio_step_kernel_lds(const aio_config& c, int blocks);
hipError_t aio_launch_step_kernel(const aio_model& m, float* logits, int32_t* tokens_out,
                                  unsigned long long* trace,
                                  unsigned long long* bar_arrive = nullptr,
                                  unsigned long long* bar_leave = nullptr);
