// Decode-step kernels (one token, M = 1) for gfx950.
//
// Per layer the step runs five launches:
//   qkv    RMSNorm prologue -> q/k/v GEMV -> RoPE epilogue, K/V appended (bf16)
//   attn   split-KV flash-decode: per (split, kv head) online-softmax partials
//   merge  log-sum-exp merge of the splits -> o
//   o      GEMV W_o o, residual add into x
//   gateup RMSNorm prologue -> gate and up GEMV -> SwiGLU epilogue -> m
//   down   GEMV W_down m, residual add into x
// then the final RMSNorm + LM head, and (greedy decoding) the argmax.
//
// Every GEMV streams its weight rows once with 16-byte loads (8 bf16 or 16
// int8 per lane, 1 KB per wave per load, fully coalesced), multiplies them by
// fp32 activations staged in LDS, and reduces each row across the wave.  Rows
// are split over waves, never K, so each output has exactly one writer and
// the result is run-to-run deterministic.  At M = 1 a GEMV does ~1 flop per
// weight byte, far below the VALU ridge, so there is no MFMA here.
#include <math.h>

#include "aio_internal.h"
#include "common.h"

namespace {

constexpr int kBlock = 256;  // 4 waves
constexpr int kWaves = kBlock / AIO_WAVE;

enum Epi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_STORE = 3 };

struct GemvArgs {
  const float* in;          // fp32 activations (x when NORM, else o or m)
  const uint16_t* embed;    // NORM and layer 0: embedding table (token from state)
  float* x_copy;            // layer 0: block 0 stores the embedding row here
  const uint16_t* gain;     // NORM: bf16 gain
  const void* w0;           // QKV: wq, SWIGLU: w_gate, else the matrix
  const void* w1;           // QKV: wk, SWIGLU: w_up
  const void* w2;           // QKV: wv
  const uint16_t* s0;       // int8 scales matching w0..w2
  const uint16_t* s1;
  const uint16_t* s2;
  float* out;               // QKV: q, RESID: x (+=), SWIGLU: m, STORE: logits
  uint16_t* kc;             // QKV: K cache of this layer [Hkv][max_ctx][hd]
  uint16_t* vc;             // QKV: V cache of this layer
  const float2* rope;       // QKV: [max_ctx][hd/2] (cos, sin)
  const aio_state* st;
  int N;                    // output rows (QKV: (H + 2 Hkv) * hd)
  int K;                    // input length
  int H, Hkv, hd, max_ctx;
  float eps;
};

// Activation staging in LDS.  A lane consumes one 16-byte weight vector
// (EPV elements) per step; its EPV activations are stored as EPV/4 float4
// planes so that the 64 lanes of a wave read consecutive float4s (no bank
// conflicts): element e -> plane (e % EPV) / 4, vector e / EPV, slot e % 4.
template <int EPV>
AIO_DEV int stage_index(int e, int nv) {
  return (((e % EPV) >> 2) * nv + e / EPV) * 4 + (e & 3);
}

// acc[r] += row_r . h over the whole row, for R rows held by this wave.
template <int WFMT, int R, int U>
AIO_DEV void gemv_rows(const uint4* const (&rowp)[R], int nv, const float* __restrict__ hs,
                       float (&acc)[R]) {
  const int lane = threadIdx.x & (AIO_WAVE - 1);
  const float4* h4 = (const float4*)hs;
  for (int base = 0; base < nv; base += AIO_WAVE * U) {
    uint4 w[U][R];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int idx = base + u * AIO_WAVE + lane;
#pragma unroll
      for (int r = 0; r < R; ++r)
        w[u][r] = idx < nv ? ld_stream(rowp[r] + idx) : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int idx = base + u * AIO_WAVE + lane;
      if (idx < nv) {
        if constexpr (WFMT == AIO_WFMT_BF16) {
          const float4 a = h4[idx], b = h4[nv + idx];
#pragma unroll
          for (int r = 0; r < R; ++r) acc[r] = dot8_bf16(w[u][r], a, b, acc[r]);
        } else {
          const float4 a0 = h4[idx], a1 = h4[nv + idx], a2 = h4[2 * nv + idx],
                       a3 = h4[3 * nv + idx];
#pragma unroll
          for (int r = 0; r < R; ++r) {
            acc[r] = dot4_i8(w[u][r].x, a0, acc[r]);
            acc[r] = dot4_i8(w[u][r].y, a1, acc[r]);
            acc[r] = dot4_i8(w[u][r].z, a2, acc[r]);
            acc[r] = dot4_i8(w[u][r].w, a3, acc[r]);
          }
        }
      }
    }
  }
}

// Block-wide sum for 256 threads; `red` holds kWaves floats.
AIO_DEV float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int wid = threadIdx.x / AIO_WAVE;
  __syncthreads();
  if ((threadIdx.x & (AIO_WAVE - 1)) == 0) red[wid] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) t += red[i];
  return t;
}

// Row n of a projection: returns its 16-byte-vector pointer and scale array.
template <int WFMT>
AIO_DEV const uint4* row_ptr(const void* w, int n, int K) {
  const size_t bytes = (size_t)n * (size_t)K * (WFMT == AIO_WFMT_BF16 ? 2u : 1u);
  return (const uint4*)((const char*)w + bytes);
}

template <int WFMT, int EPI, int R, int U, bool NORM>
__global__ __launch_bounds__(kBlock) void k_gemv(GemvArgs a) {
  extern __shared__ float hs[];
  __shared__ float red[kWaves];
  constexpr int EPV = WFMT == AIO_WFMT_BF16 ? 8 : 16;
  const int tid = threadIdx.x, lane = tid & (AIO_WAVE - 1), wid = tid / AIO_WAVE;
  const int K = a.K, nv = K / EPV;

  // ---- which rows this wave owns ----
  // QKV: R/2 rotation pairs (i, i + hd/2) of one head section; SWIGLU: R/2
  // rows of gate and the same R/2 rows of up; otherwise R consecutive rows.
  const uint4* rowp[R];
  int base_row;
  if constexpr (EPI == EPI_QKV) {
    const int half = a.hd / 2;
    const int n_pairs = a.N / 2;
    base_row = (blockIdx.x * kWaves + wid) * (R / 2);  // first pair
#pragma unroll
    for (int j = 0; j < R / 2; ++j) {
      const int p = min(base_row + j, n_pairs - 1);
      const int head = p / half, i = p % half;
      const int qrows = a.H * a.hd, krows = a.Hkv * a.hd;
      int n_lo = head * a.hd + i;
      const void* w = a.w0;
      if (n_lo >= qrows + krows) { w = a.w2; n_lo -= qrows + krows; }
      else if (n_lo >= qrows) { w = a.w1; n_lo -= qrows; }
      rowp[j] = row_ptr<WFMT>(w, n_lo, K);
      rowp[j + R / 2] = row_ptr<WFMT>(w, n_lo + half, K);
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    base_row = (blockIdx.x * kWaves + wid) * (R / 2);
#pragma unroll
    for (int j = 0; j < R / 2; ++j) {
      const int n = min(base_row + j, a.N - 1);
      rowp[j] = row_ptr<WFMT>(a.w0, n, K);
      rowp[j + R / 2] = row_ptr<WFMT>(a.w1, n, K);
    }
  } else {
    base_row = (blockIdx.x * kWaves + wid) * R;
#pragma unroll
    for (int j = 0; j < R; ++j) rowp[j] = row_ptr<WFMT>(a.w0, min(base_row + j, a.N - 1), K);
  }

  // ---- prologue: stage the activation vector in LDS ----
  if constexpr (NORM) {
    const uint16_t* emb = nullptr;
    if (a.embed) emb = a.embed + (size_t)a.st->token[0] * (size_t)K;
    float ss = 0.f;
    for (int e = tid; e < K; e += kBlock) {
      const float v = emb ? bf16_to_f32(emb[e]) : a.in[e];
      ss = fmaf(v, v, ss);
    }
    ss = block_sum(ss, red);
    const float inv = rsqrtf(ss / (float)K + a.eps);
    for (int e = tid; e < K; e += kBlock) {
      const float v = emb ? bf16_to_f32(emb[e]) : a.in[e];
      if (emb && blockIdx.x == 0) a.x_copy[e] = v;
      hs[stage_index<EPV>(e, nv)] = v * inv * bf16_to_f32(a.gain[e]);
    }
  } else {
    for (int e = tid; e < K; e += kBlock) hs[stage_index<EPV>(e, nv)] = a.in[e];
  }
  __syncthreads();

  float acc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) acc[r] = 0.f;
  gemv_rows<WFMT, R, U>(rowp, nv, hs, acc);
#pragma unroll
  for (int r = 0; r < R; ++r) acc[r] = wave_sum(acc[r]);
  if (lane != 0) return;

  // ---- epilogues (one lane per wave writes) ----
  if constexpr (EPI == EPI_QKV) {
    const int half = a.hd / 2, n_pairs = a.N / 2;
    const int pos = a.st->pos;
    const int qrows = a.H * a.hd, krows = a.Hkv * a.hd;
#pragma unroll
    for (int j = 0; j < R / 2; ++j) {
      const int p = base_row + j;
      if (p >= n_pairs) break;
      const int head = p / half, i = p % half;
      const int n_lo = head * a.hd + i;
      float lo = acc[j], hi = acc[j + R / 2];
      if constexpr (WFMT == AIO_WFMT_INT8) {
        const uint16_t* sc = a.s0;
        int m_lo = n_lo;
        if (n_lo >= qrows + krows) { sc = a.s2; m_lo -= qrows + krows; }
        else if (n_lo >= qrows) { sc = a.s1; m_lo -= qrows; }
        lo *= fp16_to_f32(sc[m_lo]);
        hi *= fp16_to_f32(sc[m_lo + half]);
      }
      if (n_lo < qrows + krows) {  // rotate q and k
        const float2 cs = a.rope[(size_t)pos * half + i];
        const float r0 = lo * cs.x - hi * cs.y;
        const float r1 = hi * cs.x + lo * cs.y;
        lo = r0;
        hi = r1;
      }
      if (n_lo < qrows) {
        a.out[n_lo] = lo;
        a.out[n_lo + half] = hi;
      } else {
        const bool is_k = n_lo < qrows + krows;
        const int g = (n_lo - (is_k ? qrows : qrows + krows)) / a.hd;
        uint16_t* c = (is_k ? a.kc : a.vc) + ((size_t)g * a.max_ctx + pos) * a.hd;
        c[i] = f32_to_bf16(lo);
        c[i + half] = f32_to_bf16(hi);
      }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int j = 0; j < R / 2; ++j) {
      const int n = base_row + j;
      if (n >= a.N) break;
      float g = acc[j], u = acc[j + R / 2];
      if constexpr (WFMT == AIO_WFMT_INT8) {
        g *= fp16_to_f32(a.s0[n]);
        u *= fp16_to_f32(a.s1[n]);
      }
      a.out[n] = g / (1.f + expf(-g)) * u;
    }
  } else {
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const int n = base_row + j;
      if (n >= a.N) break;
      float y = acc[j];
      if constexpr (WFMT == AIO_WFMT_INT8) y *= fp16_to_f32(a.s0[n]);
      if constexpr (EPI == EPI_RESID) a.out[n] += y;
      else a.out[n] = y;
    }
  }
}

// ---------------------------------------------------------------- attention

struct AttnArgs {
  const float* q;        // [H*hd] rotated queries
  const uint16_t* kc;    // [Hkv][max_ctx][hd]
  const uint16_t* vc;
  float* part_o;         // [H][S][hd]  unnormalised partial outputs
  float* part_ml;        // [H][S][2]   (running max, sum) in log2 units
  const aio_state* st;
  int H, Hkv, max_ctx, S;
  float scale_log2;      // log2(e) / sqrt(hd)
};

// One workgroup per (split s, kv head g) covers the keys of split s for the
// G query heads sharing kv head g, so each K/V row is fetched once.  HD/8
// lanes hold one key row (16 bytes each); the 256 threads form 2048/HD such
// groups, and every group runs an online softmax over its keys before the
// groups are combined in LDS.  Split s of n = pos + 1 keys covers
// [s*c, min(n, (s+1)*c)) with c = ceil(n / S).
template <int HD, int G>
__global__ __launch_bounds__(kBlock) void k_attn(AttnArgs a) {
  constexpr int LPK = HD / 8;          // lanes per key row
  constexpr int NG = kBlock / LPK;     // key groups per workgroup
  __shared__ float sm_m[NG][G], sm_l[NG][G];
  __shared__ float sm_o[NG][G][HD];
  const int tid = threadIdx.x, gi = tid / LPK, li = tid % LPK;
  const int s = blockIdx.x, kvh = blockIdx.y;
  const int n_keys = a.st->pos + 1;
  const int chunk = (n_keys + a.S - 1) / a.S;
  const int j0 = s * chunk, j1 = min(n_keys, j0 + chunk);

  float q[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float* qp = a.q + (size_t)(kvh * G + g) * HD + li * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) q[g][i] = qp[i] * a.scale_log2;
  }
  float m[G], l[G], o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[g][i] = 0.f;
  }
  const uint16_t* kbase = a.kc + (size_t)kvh * a.max_ctx * HD + li * 8;
  const uint16_t* vbase = a.vc + (size_t)kvh * a.max_ctx * HD + li * 8;

  for (int j = j0 + gi; j < j1; j += NG) {
    const uint4 kk = *(const uint4*)(kbase + (size_t)j * HD);
    const uint4 vv = *(const uint4*)(vbase + (size_t)j * HD);
    const float vf[8] = {bf16_lo(vv.x), bf16_hi(vv.x), bf16_lo(vv.y), bf16_hi(vv.y),
                         bf16_lo(vv.z), bf16_hi(vv.z), bf16_lo(vv.w), bf16_hi(vv.w)};
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float sc = dot8_bf16(kk, make_float4(q[g][0], q[g][1], q[g][2], q[g][3]),
                           make_float4(q[g][4], q[g][5], q[g][6], q[g][7]), 0.f);
      sc = group_sum<LPK>(sc);
      const float mn = fmaxf(m[g], sc);
      const float c = exp2f(m[g] - mn);
      const float p = exp2f(sc - mn);
      l[g] = l[g] * c + p;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] = fmaf(p, vf[i], o[g][i] * c);
      m[g] = mn;
    }
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (li == 0) {
      sm_m[gi][g] = m[g];
      sm_l[gi][g] = l[g];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) sm_o[gi][g][li * 8 + i] = o[g][i];
  }
  __syncthreads();
  for (int t = tid; t < G * HD; t += kBlock) {
    const int g = t / HD, dim = t % HD;
    float M = -INFINITY;
    for (int k = 0; k < NG; ++k) M = fmaxf(M, sm_m[k][g]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
      for (int k = 0; k < NG; ++k) {
        const float mk = sm_m[k][g];
        if (mk == -INFINITY) continue;
        const float w = exp2f(mk - M);
        L = fmaf(w, sm_l[k][g], L);
        O = fmaf(w, sm_o[k][g][dim], O);
      }
    }
    const int h = kvh * G + g;
    const size_t slot = (size_t)h * a.S + s;
    a.part_o[slot * HD + dim] = O;
    if (dim == 0) {
      a.part_ml[slot * 2 + 0] = M;
      a.part_ml[slot * 2 + 1] = L;
    }
  }
}

struct MergeArgs {
  const float* part_o;
  const float* part_ml;
  float* o;  // [H*hd]
  int S, hd;
};

// o_h = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) L_s, M = max_s m_s.
__global__ __launch_bounds__(128) void k_merge(MergeArgs a) {
  const int h = blockIdx.x;
  const float* ml = a.part_ml + (size_t)h * a.S * 2;
  float M = -INFINITY;
  for (int s = 0; s < a.S; ++s) M = fmaxf(M, ml[2 * s]);
  for (int dim = threadIdx.x; dim < a.hd; dim += blockDim.x) {
    float L = 0.f, O = 0.f;
    for (int s = 0; s < a.S; ++s) {
      const float ms = ml[2 * s];
      if (ms == -INFINITY) continue;
      const float w = exp2f(ms - M);
      L = fmaf(w, ml[2 * s + 1], L);
      O = fmaf(w, a.part_o[((size_t)h * a.S + s) * a.hd + dim], O);
    }
    a.o[(size_t)h * a.hd + dim] = O / L;
  }
}

// ------------------------------------------------------------------- argmax

// (value, index) order: NaN above everything, then larger value, then
// lower index.
AIO_DEV bool am_better(float v, int i, float bv, int bi) {
  const bool n = v != v, bn = bv != bv;
  if (n != bn) return n;
  if (!n && v != bv) return v > bv;
  return i < bi;
}

struct ArgmaxArgs {
  const float* x;
  int n;
  int32_t* out;
  aio_state* st;  // greedy feedback when non-null
  int32_t* tokens_out;
};

__global__ __launch_bounds__(1024) void k_argmax(ArgmaxArgs a) {
  __shared__ float sv[16];
  __shared__ int si[16];
  const float* x = a.x + (size_t)blockIdx.x * a.n;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int i = threadIdx.x; i < a.n; i += blockDim.x) {
    const float v = x[i];
    if (am_better(v, i, bv, bi)) { bv = v; bi = i; }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(bv, off, AIO_WAVE);
    const int oi = __shfl_xor(bi, off, AIO_WAVE);
    if (am_better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
  }
  const int wid = threadIdx.x / AIO_WAVE;
  if ((threadIdx.x & (AIO_WAVE - 1)) == 0) { sv[wid] = bv; si[wid] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int nw = blockDim.x / AIO_WAVE;
    for (int w = 1; w < nw; ++w)
      if (am_better(sv[w], si[w], bv, bi)) { bv = sv[w]; bi = si[w]; }
    if (bi == 0x7fffffff) bi = 0;  // only -inf values (or n == 0)
    if (a.out) a.out[blockIdx.x] = bi;
    if (a.st) {
      a.tokens_out[a.st->step] = bi;
      a.st->token[0] = bi;
      a.st->pos += 1;
      a.st->step += 1;
    }
  }
}

// The probe's category scores: the logits of up to kMaxCategories label
// tokens.  One wave: lane i takes label i; the argmax (lowest index on ties)
// and H = log Z - sum_i p_i (x_i - max), Z = sum_i e^(x_i - max), in double
// and in label order (lane 0 folds the lanes' terms one by one), so the
// value is the one the host routing rule computes from the same logits.
constexpr int kMaxCategories = 64;
struct CategoryArgs {
  const float* logits;
  int32_t label[kMaxCategories];
  int n;
  float* out;  // [0] = H in nats, [1] = category index (as a float)
};

__global__ __launch_bounds__(AIO_WAVE) void k_category_entropy(CategoryArgs a) {
  __shared__ float xs[kMaxCategories];
  const int i = threadIdx.x;
  if (i < a.n) xs[i] = a.logits[a.label[i]];
  __syncthreads();
  if (i != 0) return;
  int best = 0;
  for (int j = 1; j < a.n; ++j)
    if (xs[j] > xs[best]) best = j;
  const double mx = xs[best];
  double z = 0.0, ez = 0.0;
  for (int j = 0; j < a.n; ++j) {
    const double d = (double)xs[j] - mx, w = exp(d);
    z += w;
    ez += w * d;
  }
  a.out[0] = (float)(log(z) - ez / z);
  a.out[1] = (float)best;
}

__global__ void k_set_state(aio_state* st, int32_t token, int32_t pos) {
  st->token[0] = token;
  st->pos = pos;
  st->step = 0;
  st->rows = 1;
}

struct RowsArgs {
  int32_t tok[16];
};

__global__ void k_set_rows(aio_state* st, RowsArgs r, int rows, int32_t pos) {
  for (int i = 0; i < rows; ++i) st->token[i] = r.tok[i];
  st->pos = pos;
  st->step = 0;
  st->rows = rows;
}

// ---------------------------------------------------------------- launching

template <int WFMT, int EPI, int R, int U, bool NORM>
hipError_t launch_gemv(const aio_model& m, const GemvArgs& a, int rows_per_wave_units) {
  const int blocks = (rows_per_wave_units + kWaves - 1) / kWaves;
  const size_t lds = (size_t)a.K * sizeof(float);
  hipLaunchKernelGGL((k_gemv<WFMT, EPI, R, U, NORM>), dim3(blocks), dim3(kBlock), lds, m.stream,
                     a);
  aio_prof_mark(m);
  return hipGetLastError();
}

template <int EPI, int R, int U, bool NORM>
hipError_t launch_gemv_fmt(const aio_model& m, const GemvArgs& a, int units) {
  if (m.cfg.wfmt == AIO_WFMT_INT8) return launch_gemv<AIO_WFMT_INT8, EPI, R, U, NORM>(m, a, units);
  return launch_gemv<AIO_WFMT_BF16, EPI, R, U, NORM>(m, a, units);
}

template <int HD>
hipError_t launch_attn_hd(const aio_model& m, const AttnArgs& a, int G) {
  const dim3 grid(a.S, a.Hkv);
  switch (G) {
#define AIO_ATTN_CASE(g) \
  case g: hipLaunchKernelGGL((k_attn<HD, g>), grid, dim3(kBlock), 0, m.stream, a); break;
    AIO_ATTN_CASE(1)
    AIO_ATTN_CASE(2)
    AIO_ATTN_CASE(4)
    AIO_ATTN_CASE(8)
#undef AIO_ATTN_CASE
    default: return hipErrorInvalidValue;
  }
  aio_prof_mark(m);
  return hipGetLastError();
}

}  // namespace

// Rows per wave of each GEMV.  QKV and SwiGLU count rotation pairs / row
// pairs, each using R = 2 * pairs rows.
#define AIO_R 4
#define AIO_U 2

hipError_t aio_launch_set_state(const aio_model& m, int32_t token, int32_t pos) {
  hipLaunchKernelGGL(k_set_state, dim3(1), dim3(1), 0, m.stream, m.state(), token, pos);
  return hipGetLastError();
}

hipError_t aio_launch_set_rows(const aio_model& m, const int32_t* toks, int rows, int32_t pos) {
  RowsArgs r{};
  for (int i = 0; i < rows && i < 16; ++i) r.tok[i] = toks[i];
  hipLaunchKernelGGL(k_set_rows, dim3(1), dim3(1), 0, m.stream, m.state(), r, rows, pos);
  return hipGetLastError();
}

hipError_t aio_launch_decode_layer(const aio_model& m, int l) {
  const aio_config& c = m.cfg;
  const aio_layer_weights& L = m.layers[(size_t)l];
  const int d = c.d_model, H = c.n_heads, Hkv = c.n_kv_heads, hd = c.head_dim, F = c.ffn_dim;
  float* x = m.at<float>(m.lay.x);
  hipError_t e;

  // qkv
  GemvArgs a{};
  a.in = x;
  a.embed = l == 0 ? (const uint16_t*)m.embed : nullptr;
  a.x_copy = x;
  a.gain = (const uint16_t*)L.attn_norm;
  a.w0 = L.wq; a.w1 = L.wk; a.w2 = L.wv;
  a.s0 = (const uint16_t*)L.sq; a.s1 = (const uint16_t*)L.sk; a.s2 = (const uint16_t*)L.sv;
  a.out = m.at<float>(m.lay.q);
  a.kc = m.kv_layer(l, 0);
  a.vc = m.kv_layer(l, 1);
  a.rope = m.rope;
  a.st = m.state();
  a.N = (H + 2 * Hkv) * hd;
  a.K = d;
  a.H = H; a.Hkv = Hkv; a.hd = hd; a.max_ctx = c.max_ctx;
  a.eps = c.rms_eps;
  e = launch_gemv_fmt<EPI_QKV, AIO_R, AIO_U, true>(m, a, (a.N / 2 + AIO_R / 2 - 1) / (AIO_R / 2));
  if (e != hipSuccess) return e;

  // split-KV attention + merge
  AttnArgs t{};
  t.q = m.at<float>(m.lay.q);
  t.kc = m.kv_layer(l, 0);
  t.vc = m.kv_layer(l, 1);
  t.part_o = m.at<float>(m.lay.part_o);
  t.part_ml = m.at<float>(m.lay.part_ml);
  t.st = m.state();
  t.H = H; t.Hkv = Hkv; t.max_ctx = c.max_ctx; t.S = m.lay.splits;
  t.scale_log2 = (float)(1.4426950408889634 / sqrt((double)hd));
  e = hd == 128 ? launch_attn_hd<128>(m, t, H / Hkv) : launch_attn_hd<64>(m, t, H / Hkv);
  if (e != hipSuccess) return e;
  MergeArgs mg{t.part_o, t.part_ml, m.at<float>(m.lay.o), m.lay.splits, hd};
  hipLaunchKernelGGL(k_merge, dim3(H), dim3(128), 0, m.stream, mg);
  aio_prof_mark(m);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  // o projection + residual
  GemvArgs b{};
  b.in = m.at<float>(m.lay.o);
  b.w0 = L.wo; b.s0 = (const uint16_t*)L.so;
  b.out = x;
  b.N = d; b.K = H * hd;
  e = launch_gemv_fmt<EPI_RESID, AIO_R, AIO_U, false>(m, b, (d + AIO_R - 1) / AIO_R);
  if (e != hipSuccess) return e;

  // ffn norm + gate/up + SwiGLU
  GemvArgs g{};
  g.in = x;
  g.gain = (const uint16_t*)L.ffn_norm;
  g.w0 = L.w_gate; g.w1 = L.w_up;
  g.s0 = (const uint16_t*)L.s_gate; g.s1 = (const uint16_t*)L.s_up;
  g.out = m.at<float>(m.lay.m);
  g.st = m.state();
  g.N = F; g.K = d; g.eps = c.rms_eps;
  e = launch_gemv_fmt<EPI_SWIGLU, AIO_R, AIO_U, true>(m, g, (F + AIO_R / 2 - 1) / (AIO_R / 2));
  if (e != hipSuccess) return e;

  // down projection + residual
  GemvArgs dn{};
  dn.in = m.at<float>(m.lay.m);
  dn.w0 = L.w_down; dn.s0 = (const uint16_t*)L.s_down;
  dn.out = x;
  dn.N = d; dn.K = F;
  return launch_gemv_fmt<EPI_RESID, AIO_R, AIO_U, false>(m, dn, (d + AIO_R - 1) / AIO_R);
}

hipError_t aio_launch_lm_head(const aio_model& m, float* logits) {
  const aio_config& c = m.cfg;
  GemvArgs a{};
  a.in = m.at<float>(m.lay.x);
  a.gain = (const uint16_t*)m.final_norm;
  a.w0 = m.lm_head; a.s0 = (const uint16_t*)m.s_lm_head;
  a.out = logits;
  a.st = m.state();
  a.N = c.vocab; a.K = c.d_model; a.eps = c.rms_eps;
  return launch_gemv_fmt<EPI_STORE, AIO_R, AIO_U, true>(m, a, (c.vocab + AIO_R - 1) / AIO_R);
}

hipError_t aio_launch_category_entropy(const aio_model& m, const float* logits,
                                       const int32_t* labels, int n, float* out) {
  if (n < 1 || n > kMaxCategories) return hipErrorInvalidValue;
  CategoryArgs a{};
  a.logits = logits;
  for (int i = 0; i < n; ++i) a.label[i] = labels[i];
  a.n = n;
  a.out = out;
  hipLaunchKernelGGL(k_category_entropy, dim3(1), dim3(AIO_WAVE), 0, m.stream, a);
  return hipGetLastError();
}

hipError_t aio_launch_argmax(const aio_model& m, const float* logits, int rows, int n,
                             int32_t* out, bool greedy_feedback) {
  ArgmaxArgs a{logits, n, greedy_feedback ? nullptr : out,
               greedy_feedback ? m.state() : nullptr, greedy_feedback ? out : nullptr};
  hipLaunchKernelGGL(k_argmax, dim3(rows), dim3(1024), 0, m.stream, a);
  aio_prof_mark(m);
  return hipGetLastError();
}
