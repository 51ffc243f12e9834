// Verify forward (prompt-lookup verification): M = k + 1 <= 10 rows at
// positions pos .. pos + k in one pass over the weights, for gfx950.
//
// At M rows a projection does ~M flops per weight byte (8-16 flop/B), close
// to the fp32 VALU ridge, so the matrix products run on MFMA
// (v_mfma_f32_32x32x16_bf16).  MFMA inputs are bf16; to keep fp32-level
// accuracy each fp32 activation a is split exactly into three bf16 terms,
// a = t0 + t1 + t2 + O(2^-27 a) (t0 = bf16(a), t1 = bf16(a - t0),
// t2 = bf16(a - t0 - t1); each subtraction is exact in fp32), and the three
// terms of all M rows form the 3M <= 30 columns of one 32-column B operand.
// Weights are the A operand (32 output channels per tile); int8 weights
// convert to bf16 exactly (|q| <= 127) and their fp16 scale is applied in the
// epilogue.
//
// RMSNorm is folded into the products around it.  Its scale
// 1 / sqrt(mean(x_r^2) + eps) is one number per row, so it commutes with the
// product: the GEMM that consumes a normed row multiplies the split of x * g
// and scales its result by the row's factor, which it forms from the row's
// sums of squares over 64-column chunks (written by whoever completed those
// columns of x, summed in chunk order).
//
// Per layer: QKV GEMM (+norm scale, RoPE, K/V append) -> vattn_mma (causal
// split-KV on MFMA, row r sees positions [0, pos + r]; the last split of a
// head merges the head's splits and writes the split output) -> O GEMM
// (+residual, split of x * g_ffn, sums of squares) -> gate/up GEMM (+norm
// scale, SwiGLU, split) -> down GEMM (+residual, split of x * g for the next
// layer or the final norm); then the LM head GEMM (+norm scale) -> logits
// [M][V].  Layer 0's input (the embedding rows) goes through vnorm.
#include <math.h>
#include <algorithm>

#include "aio_internal.h"
#include "common.h"

namespace {

// The skinny GEMM runs 8 waves per workgroup: more weight loads in flight
// per CU, and the K range of a workgroup split eight ways.
constexpr int kGBlock = 512;
constexpr int kGWaves = kGBlock / AIO_WAVE;
constexpr int kMaxRows = AIO_MAX_VERIFY_ROWS;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(1))) const u32x4 gl_u32x4;

// 16-byte loads through a global-address-space pointer.  Selected from a
// table the pointer's address space is unknown, and a flat load also counts
// against the LDS wait counter: every LDS wait would then wait for the
// weights in flight as well.
AIO_DEV uint4 ldg_nt(const void* p) {
  const u32x4 v = __builtin_nontemporal_load((gl_u32x4*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}
AIO_DEV uint4 ldg(const void* p) {
  const u32x4 v = *(gl_u32x4*)p;
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Device-coherent access for the slices of a split residual product: the
// parts are written through to memory and read past the (per-XCD) L2, so
// handing them over needs no fence that writes back or drops a whole L2
// (with fences, the hand-over cost about 40 us per product).
AIO_DEV int atomic_add_agent(int* p, int v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
AIO_DEV void atomic_store_agent(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
AIO_DEV void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
AIO_DEV float ld_agent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

enum Epi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_STORE = 3 };

// Exact three-term bf16 split of an fp32 value.
AIO_DEV void split3(float a, uint16_t& t0, uint16_t& t1, uint16_t& t2) {
  t0 = f32_to_bf16(a);
  const float r1 = a - bf16_to_f32(t0);
  t1 = f32_to_bf16(r1);
  const float r2 = r1 - bf16_to_f32(t1);
  t2 = f32_to_bf16(r2);
}

AIO_DEV void store_split(uint16_t* act, int lda, int M, int r, int col, float v) {
  uint16_t t0, t1, t2;
  split3(v, t0, t1, t2);
  act[(size_t)r * lda + col] = t0;
  act[(size_t)(M + r) * lda + col] = t1;
  act[(size_t)(2 * M + r) * lda + col] = t2;
}

// ------------------------------------------------------------ RMSNorm rows

struct VNormArgs {
  float* x;                 // [M][d] residual rows
  const uint16_t* embed;    // layer 0: embedding table (tokens from state), else null
  const uint16_t* gain;
  uint16_t* act;            // [32][lda] split of x * g
  int lda, d, M;
  float* ss;                // [M][d / 64] sums of squares of x over 64-column chunks
  const aio_state* st;
};

// One workgroup of 1024 threads per row r (in layer 0 x_r is the embedding
// row of the row's token, written to x): the split of x_r * g and the sums of
// squares of x_r per 64-column chunk.  Wave w holds chunks w, w + 16, ...
constexpr int kNormBlock = 1024;

__global__ __launch_bounds__(kNormBlock) void k_vnorm(VNormArgs a) {
  const int r = blockIdx.x, tid = threadIdx.x;
  const uint16_t* emb = a.embed ? a.embed + (size_t)a.st->token[r] * a.d : nullptr;
  float* xr = a.x + (size_t)r * a.d;
  for (int e = tid; e < a.d; e += kNormBlock) {  // wave-uniform: d % 64 == 0
    float v;
    if (emb) {
      v = bf16_to_f32(emb[e]);
      xr[e] = v;
    } else {
      v = xr[e];
    }
    store_split(a.act, a.lda, a.M, r, e, v * bf16_to_f32(a.gain[e]));
    const float sq = wave_sum(v * v);
    if ((tid & (AIO_WAVE - 1)) == 0) a.ss[(size_t)r * (a.d / 64) + e / 64] = sq;
  }
}

// ------------------------------------------------------------- skinny GEMM

struct VGemmArgs {
  const uint16_t* act;      // [32][lda] bf16, columns j = term * M + row
  int lda;
  const void* w0;           // QKV: wq | SWIGLU: w_gate | else the matrix
  const void* w1;           // QKV: wk | SWIGLU: w_up
  const void* w2;           // QKV: wv
  const uint16_t* s0;
  const uint16_t* s1;
  const uint16_t* s2;
  int N, K, M;
  float* out;               // QKV: q [M][H*hd] | RESID: x [M][N] | STORE: logits [M][N]
  int ldo;
  uint16_t* act_out;        // SWIGLU: split m [32][lda_out]
  int lda_out;
  uint16_t* kc;
  uint16_t* vc;
  const float2* rope;
  const aio_state* st;
  int H, Hkv, hd, max_ctx;
  int ks;                   // K splits across workgroups (grid.y); > 1 only for EPI_RESID
  float* part;              // RESID with ks > 1: [ks][M][ldo], slice y's product
  // QKV, SWIGLU, STORE: the act columns are the split of x * g; each output
  // is scaled by 1 / sqrt(sum(ss_in[r][0 .. nt)) / K + eps)
  const float* ss_in;
  int nt;
  float eps;
  // RESID: completes x (ldo == N == d), then writes act_next = split of
  // x * g_next and ss_out [M][N / 64]; cnt [N / 64] counts arrived slices
  int* cnt;
  const uint16_t* g_next;
  uint16_t* act_next;
  float* ss_out;
  // stream-K form (SWIGLU): tile pairs of the product, and the
  // partial sums [tiles][kSkMaxC][kMaxRows * 64] and arrival counters
  // [tiles] of tile pairs that several workgroups share
  int tiles;
  float* skpart;
  int* skcnt;
};

// The k of the two MFMA fragments a lane holds in a block of 32 k (lane
// half kh = l / 32): for bf16, k .. k+7 and k+16 .. k+23 from block + 8 kh;
// for int8, the 16 consecutive k from block + 16 kh.  Weights (frag_lds)
// and activations use the same k, so the permutation cancels.
template <int WFMT>
AIO_DEV int vk_lo(int block, int kh) { return WFMT == AIO_WFMT_BF16 ? block + 8 * kh : block + 16 * kh; }
template <int WFMT>
AIO_DEV int vk_hi(int block, int kh) { return WFMT == AIO_WFMT_BF16 ? block + 16 + 8 * kh : block + 16 * kh + 8; }

// Weights reach the MFMA through LDS in stages of 256 k per row (64 rows:
// 32 KB of bf16, 16 KB of int8), two stages in flight per workgroup.  Read
// straight into the MFMA operand layout, every load instruction would span
// 32 rows at 16-32 bytes each; staged, consecutive lanes read consecutive
// 16-byte chunks of one row, and the 64 rows of a stage go to LDS with a
// 16-byte skew per row, so that the fragment reads (32 rows at one column)
// spread over the banks.  Stages of 1 KB per row (64 KB, one workgroup per
// CU) measured slower: 5.16 against 4.89 ms per 7B bf16 verify.
// Register sets of weight stages in flight per workgroup (three measured
// slower: 4.56 against 4.20 ms per 7B bf16 verify, the extra registers
// leaving one workgroup per CU).
constexpr int kVNB = 2;

template <int WFMT>
struct VStage {
  static constexpr int KC = 256;                                     // k per stage
  static constexpr int RB = KC * (WFMT == AIO_WFMT_BF16 ? 2 : 1);    // bytes of a row
  static constexpr int RS = RB + 16;                                 // LDS row stride
  static constexpr int CPR = RB / 16;                                // 16-byte chunks per row
  static constexpr int NLD = 64 * CPR / kGBlock;                     // loads per thread
  static constexpr int BPS = KC / 32;                                // 32-k blocks per stage
  static constexpr int BPW = BPS / kGWaves;                          // blocks per wave
  static constexpr int BYTES = 64 * RS;
};

// Two bf16x8 MFMA fragments of one staged row for the wave's block of 32 k
// (the same k as vk_lo / vk_hi give for the activations).
template <int WFMT>
AIO_DEV void frag_lds(const char* rowl, int wblock, int kh, bf16x8& lo, bf16x8& hi) {
  if constexpr (WFMT == AIO_WFMT_BF16) {
    const char* p = rowl + (size_t)(wblock * 32 + 8 * kh) * 2;
    lo = __builtin_bit_cast(bf16x8, *(const uint4*)p);
    hi = __builtin_bit_cast(bf16x8, *(const uint4*)(p + 32));
  } else {
    const uint4 u = *(const uint4*)(rowl + wblock * 32 + 16 * kh);
    uint32_t w[4] = {u.x, u.y, u.z, u.w};
    uint32_t o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      // two int8 -> two bf16 (exact: |q| <= 127 has <= 7 significant bits)
      const uint32_t src = w[i / 2];
      const int sh = (i & 1) * 16;
      const float f0 = (float)(int8_t)(src >> sh);
      const float f1 = (float)(int8_t)(src >> (sh + 8));
      o[i] = (__float_as_uint(f0) >> 16) | (__float_as_uint(f1) & 0xffff0000u);
    }
    lo = __builtin_bit_cast(bf16x8, make_uint4(o[0], o[1], o[2], o[3]));
    hi = __builtin_bit_cast(bf16x8, make_uint4(o[4], o[5], o[6], o[7]));
  }
}

// Each workgroup owns T = 2 tiles of 32 output channels and one of a.ks
// slices of K (grid.y).  Its weights pass through LDS in stages (VStage),
// two stages in flight in registers; wave w multiplies block w of every
// stage, and the 8 waves' partial 32x32 tiles are summed in LDS at the end.
// Lane l of a wave covers tile row (l % 32) and 16 of the 32 k of a block
// (vk_lo, vk_hi): MFMA "a" takes 8 of them and MFMA "b" the other 8; the B
// operand (activation column l % 32) is loaded with the same k, so the k
// permutation cancels.
template <int WFMT, int T>
struct VFrag {
  bf16x8 wa[T], wb[T], ba, bb;
};

template <int WFMT, int T>
AIO_DEV void vmma(const VFrag<WFMT, T>& f, bool col_live, f32x16 (&acc)[T]) {
  // dead columns (past the 3M split terms) multiply zeros
  const bf16x8 z = __builtin_bit_cast(bf16x8, make_uint4(0u, 0u, 0u, 0u));
  const bf16x8 ba = col_live ? f.ba : z, bb = col_live ? f.bb : z;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.wa[t], ba, acc[t], 0, 0, 0);
    acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.wb[t], bb, acc[t], 0, 0, 0);
  }
}

// LDS of a skinny-GEMM workgroup: the weight stage during the product, then
// the partial tiles of the waves and a residual tile [M][64].
constexpr int kVRedBytes = (int)sizeof(float) * (kGWaves / 2) * 2 * 32 * 33;
constexpr int kVFinBytes = (int)sizeof(float) * kMaxRows * 64;
template <int WFMT>
constexpr int vgemm_lds() {
  return VStage<WFMT>::BYTES > kVRedBytes + kVFinBytes ? VStage<WFMT>::BYTES
                                                       : kVRedBytes + kVFinBytes;
}

// Epilogue of one output element of a QKV or gate/up tile pair tp (tile
// row i, verify row r) from the pair's two norm-scaled sums y0, y1:
//   QKV: rows (n, n + hd/2) of a head section, rotated at position pos + r,
//     to q or to the K / V cache;
//   SWIGLU: the same row n of gate and up, silu(g) u split into act_out.
template <int WFMT, int EPI>
AIO_DEV void vgemm_epi(const VGemmArgs& a, int tp, int r, int i, float y0, float y1, int pos) {
  if constexpr (EPI == EPI_QKV) {
    const int qrows = a.H * a.hd, krows = a.Hkv * a.hd;
    const int per_head = a.hd / 64;
    const int head = tp / per_head, sub = tp % per_head;
    const int ii = sub * 32 + i;  // index within the first half of the head
    const int n_lo = head * a.hd + ii;
    const int half = a.hd / 2;
    float lo = y0, hi = y1;
    if constexpr (WFMT == AIO_WFMT_INT8) {
      // both rows of the pair lie in the same (q, k or v) section
      const uint16_t* sc = a.s0;
      int m_lo = n_lo;
      if (n_lo >= qrows + krows) { sc = a.s2; m_lo -= qrows + krows; }
      else if (n_lo >= qrows) { sc = a.s1; m_lo -= qrows; }
      lo *= fp16_to_f32(sc[m_lo]);
      hi *= fp16_to_f32(sc[m_lo + half]);
    }
    const int p = pos + r;
    if (n_lo < qrows + krows) {
      const float2 cs = a.rope[(size_t)p * half + ii];
      const float r0 = lo * cs.x - hi * cs.y;
      const float r1 = hi * cs.x + lo * cs.y;
      lo = r0;
      hi = r1;
    }
    if (n_lo < qrows) {
      a.out[(size_t)r * a.ldo + n_lo] = lo;
      a.out[(size_t)r * a.ldo + n_lo + half] = hi;
    } else {
      const bool is_k = n_lo < qrows + krows;
      const int g = (n_lo - (is_k ? qrows : qrows + krows)) / a.hd;
      uint16_t* c = (is_k ? a.kc : a.vc) + ((size_t)g * a.max_ctx + p) * a.hd;
      c[ii] = f32_to_bf16(lo);
      c[ii + half] = f32_to_bf16(hi);
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int n = tp * 32 + i;
    if (n < a.N) {
      float g = y0, u = y1;
      if constexpr (WFMT == AIO_WFMT_INT8) {
        g *= fp16_to_f32(a.s0[n]);
        u *= fp16_to_f32(a.s1[n]);
      }
      store_split(a.act_out, a.lda_out, a.M, r, n, g / (1.f + expf(-g)) * u);
    }
  }
}

template <int WFMT, int EPI>
__global__ __launch_bounds__(kGBlock) void k_vgemm(VGemmArgs a) {
  constexpr int T = 2;
  using St = VStage<WFMT>;
  extern __shared__ __align__(16) char smem[];
  float (*red)[T][32][33] = (float (*)[T][32][33])smem;
  float (*fin)[64] = (float (*)[64])(smem + kVRedBytes);
  __shared__ float inv_s[kMaxRows];
  __shared__ int last_s;
  const int tid = threadIdx.x, lane = tid & (AIO_WAVE - 1), wid = tid / AIO_WAVE;
  const int rl = lane & 31, kh = lane >> 5;
  const size_t wbytes = WFMT == AIO_WFMT_BF16 ? 2 : 1;

  // tile rows: QKV pairs (rows, rows + hd/2) of one head section, SWIGLU the
  // same rows of gate and up, otherwise two consecutive tiles.
  int tile_row[T];
  const void* tile_w[T];
  if constexpr (EPI == EPI_QKV) {
    const int per_head = a.hd / 64;  // tile pairs per head (hd/2 rows / 32)
    const int head = blockIdx.x / per_head, sub = blockIdx.x % per_head;
    const int qrows = a.H * a.hd, krows = a.Hkv * a.hd;
    int n0 = head * a.hd + sub * 32;
    const void* w = a.w0;
    if (n0 >= qrows + krows) { w = a.w2; n0 -= qrows + krows; }
    else if (n0 >= qrows) { w = a.w1; n0 -= qrows; }
    tile_row[0] = n0;
    tile_row[1] = n0 + a.hd / 2;
    tile_w[0] = tile_w[1] = w;
  } else if constexpr (EPI == EPI_SWIGLU) {
    tile_row[0] = tile_row[1] = blockIdx.x * 32;
    tile_w[0] = a.w0;
    tile_w[1] = a.w1;
  } else {
    tile_row[0] = blockIdx.x * 64;
    tile_row[1] = blockIdx.x * 64 + 32;
    tile_w[0] = tile_w[1] = a.w0;
  }
  const int n_rows_w = (EPI == EPI_QKV) ? 0 : a.N;  // clamp bound for plain tiles
  const bool col_live = rl < 3 * a.M;
  // Norm scales: wave w sums the chunk sums of rows w and w + 8, lane l
  // taking chunks l and l + 64 (written by an earlier kernel).  They are
  // requested here and added only in the epilogue, so no wait in the
  // product is spent on them.
  static_assert(kMaxRows <= 2 * kGWaves, "two rows per wave");
  float ssp[2][2] = {{0.f, 0.f}, {0.f, 0.f}};
  if (EPI != EPI_RESID) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = wid + kGWaves * h;
      if (r < a.M) {
        const float* ssr = a.ss_in + (size_t)r * a.nt;
        if (lane < a.nt) ssp[h][0] = ssr[lane];
        if (lane + 64 < a.nt) ssp[h][1] = ssr[lane + 64];
      }
    }
  }
  // dead columns read row 0 (in bounds) and are zeroed before the product
  const uint16_t* actp = a.act + (size_t)(col_live ? rl : 0) * a.lda;

  // This workgroup's K slice in stages of BPS blocks of 32 k; wave w
  // multiplies blocks w, w + 8, ... of every stage.
  constexpr int BPS = St::BPS, BPW = St::BPW;
  const int nkb = a.K / 32;
  const int ks = (int)blockIdx.y;
  const int kbA = ks * nkb / a.ks, kbB = (ks + 1) * nkb / a.ks;
  const int nst = (kbB - kbA + BPS - 1) / BPS;
  // Workgroup b takes its stages starting at stage b mod nst (and wraps).
  // Every row of W is K * wbytes apart, a multiple of the HBM channel
  // interleave, so the same k offset of all rows lies in the same few
  // channels: in step, every workgroup would read the same channels at
  // once.
  const int rot = nst > 0 ? (int)(blockIdx.x % (unsigned)nst) : 0;
  auto kb0 = [&](int st) {  // first 32-k block of stage st (st < 2 nst)
    const int p = st + rot;
    return kbA + (p >= nst ? p - nst : p) * BPS;
  };
  f32x16 acc[T];
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[t][i] = 0.f;

  // staging: load j of this thread is chunk c of stage row r (r < 64: tile
  // r / 32, tile row r % 32); chunks past the slice re-read its last chunk
  const char* lrow[St::NLD];
  int lds_off[St::NLD], lchunk[St::NLD];
#pragma unroll
  for (int j = 0; j < St::NLD; ++j) {
    const int f = j * kGBlock + tid, r = f / St::CPR, c = f % St::CPR;
    int n = tile_row[r / 32] + r % 32;
    if (n_rows_w && n >= n_rows_w) n = n_rows_w - 1;
    lrow[j] = (const char*)tile_w[r / 32] + (size_t)n * a.K * wbytes;
    lds_off[j] = r * St::RS + c * 16;
    lchunk[j] = c;
  }
  const int kend = kbB * 32 * (int)wbytes - 16;  // last 16-byte chunk of the slice
  // A stage's weight chunks and this wave's activation fragments of it are
  // requested together, so waiting for one stage never waits for the
  // other stage's loads (vector loads complete in order); a block past the
  // slice re-reads the slice's last block and is not multiplied.
  auto gload_w = [&](uint4 (&R)[St::NLD], int st) {
#pragma unroll
    for (int j = 0; j < St::NLD; ++j) {
      int off = kb0(st) * 32 * (int)wbytes + lchunk[j] * 16;
      off = off < kend ? off : kend;
      R[j] = ldg_nt(lrow[j] + off);
    }
  };
  auto gload_a = [&](uint4 (&A)[BPW][2], int st) {
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
      const int block = min(kb0(st) + wid + kGWaves * j, kbB - 1);
      A[j][0] = ldg(actp + vk_lo<WFMT>(block * 32, kh));
      A[j][1] = ldg(actp + vk_hi<WFMT>(block * 32, kh));
    }
  };
  auto stage = [&](const uint4 (&R)[St::NLD]) {
    __syncthreads();  // every wave is done with the previous stage
#pragma unroll
    for (int j = 0; j < St::NLD; ++j) {
      const u32x4 w = {R[j].x, R[j].y, R[j].z, R[j].w};
      *(u32x4*)(smem + lds_off[j]) = w;
    }
    __syncthreads();
  };
  // Branch-free: a block past the slice multiplies zeros, so every path
  // through the loop has the same loads in flight and each wait names only
  // the stage it needs.
  auto product = [&](int st, const uint4 (&A)[BPW][2]) {
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
      const int wb = wid + kGWaves * j;
      const bool live = col_live && kb0(st) + wb < kbB;
      VFrag<WFMT, T> f;
#pragma unroll
      for (int t = 0; t < T; ++t)
        frag_lds<WFMT>(smem + (t * 32 + rl) * St::RS, wb, kh, f.wa[t], f.wb[t]);
      f.ba = __builtin_bit_cast(bf16x8, A[j][0]);
      f.bb = __builtin_bit_cast(bf16x8, A[j][1]);
      vmma(f, live, acc);
    }
  };
  // One stage: its weights go to LDS, the register set is refilled with the
  // weights kVNB stages ahead before the product (so kVNB stages stay in
  // flight through it), and the activation fragments after it.  Loads past
  // the slice re-read its last chunk.
  auto step = [&](uint4 (&R)[St::NLD], uint4 (&A)[BPW][2], int st) {
    stage(R);
    __builtin_amdgcn_sched_barrier(0);
    gload_w(R, st + kVNB);
    __builtin_amdgcn_sched_barrier(0);
    product(st, A);
    __builtin_amdgcn_sched_barrier(0);
    gload_a(A, st + kVNB);
    __builtin_amdgcn_sched_barrier(0);
  };
  if (nst > 0) {
    uint4 R0[St::NLD], R1[St::NLD], R2[St::NLD];
    uint4 A0[BPW][2], A1[BPW][2], A2[BPW][2];
    gload_w(R0, 0);
    gload_a(A0, 0);
    gload_w(R1, 1);
    gload_a(A1, 1);
    if (kVNB > 2) {
      gload_w(R2, 2);
      gload_a(A2, 2);
    }
    int st = 0;
    for (; st + kVNB < nst; st += kVNB) {
      step(R0, A0, st);
      step(R1, A1, st + 1);
      if (kVNB > 2) step(R2, A2, st + 2);
    }
    stage(R0);
    product(st, A0);
    if (st + 1 < nst) {
      stage(R1);
      product(st + 1, A1);
    }
    if (kVNB > 2 && st + 2 < nst) {
      stage(R2);
      product(st + 2, A2);
    }
  }
  __syncthreads();  // the stage buffer becomes the partial-tile buffer
  // D layout: lane l, register v -> column j = l % 32,
  // row i = 8 * (v / 4) + 4 * (l / 32) + (v % 4).  The upper four waves
  // hand their tiles to the lower four, which then write the sums.
  if (wid >= kGWaves / 2) {
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        red[wid - kGWaves / 2][t][8 * (v / 4) + 4 * kh + (v % 4)][rl] = acc[t][v];
  }
  __syncthreads();
  if (wid < kGWaves / 2) {
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float& r = red[wid][t][8 * (v / 4) + 4 * kh + (v % 4)][rl];
        r += acc[t][v];
      }
  }
  if (EPI != EPI_RESID) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = wid + kGWaves * h;
      if (r < a.M) {
        float p = ssp[h][0] + ssp[h][1];
        for (int c = lane + 128; c < a.nt; c += 64) p += a.ss_in[(size_t)r * a.nt + c];
        const float sum = wave_sum(p);
        if (lane == 0) inv_s[r] = rsqrtf(sum / (float)a.K + a.eps);
      }
    }
  }
  __syncthreads();

  // Sum the four wave pairs and the three split terms: y[r][i] for the tile.
  const int M = a.M;
  const int pos = a.st->pos;
  for (int e = tid; e < 32 * M; e += kGBlock) {
    const int i = e % 32, r = e / 32;
    float y[T];
#pragma unroll
    for (int t = 0; t < T; ++t) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kGWaves / 2; ++w)
        s += red[w][t][i][r] + red[w][t][i][M + r] + red[w][t][i][2 * M + r];
      y[t] = EPI == EPI_RESID ? s : s * inv_s[r];
    }
    if constexpr (EPI == EPI_QKV || EPI == EPI_SWIGLU) {
      vgemm_epi<WFMT, EPI>(a, (int)blockIdx.x, r, i, y[0], y[1], pos);
    } else {
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const int n = tile_row[t] + i;
        if (n >= a.N) continue;
        float v = y[t];
        if constexpr (WFMT == AIO_WFMT_INT8) v *= fp16_to_f32(a.s0[n]);
        if constexpr (EPI == EPI_RESID) {
          // K split over workgroups: each slice stores its part of the
          // product; the slice that arrives last adds them in slice order
          if (a.ks > 1) st_agent(a.part + ((size_t)blockIdx.y * M + r) * a.ldo + n, v);
          else fin[r][t * 32 + i] = v;
        } else {
          a.out[(size_t)r * a.ldo + n] = v;
        }
      }
    }
  }
  if constexpr (EPI == EPI_RESID) {
    if (a.ks > 1) {
      // every wave's part stores have completed (written through) before
      // the slice is counted; the last slice to arrive (in whatever order)
      // then reads the others' parts, which the count shows are in memory
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (tid == 0) last_s = atomic_add_agent(a.cnt + blockIdx.x, 1) == a.ks - 1;
      __syncthreads();
      if (!last_s) return;
      if (tid == 0) atomic_store_agent(a.cnt + blockIdx.x, 0);  // ready for the next product
    } else {
      __syncthreads();
    }
    // columns c0 .. c0 + 63 of the M rows, one row per wave pass; every
    // slot is requested before the first is added (slots past ks read
    // slot 0 and add nothing)
    const int c0 = blockIdx.x * 64, nt = a.N / 64;
    for (int e = tid; e < 64 * M; e += kGBlock) {
      const int r = e / 64, c = e % 64, n = c0 + c;
      float* xp = a.out + (size_t)r * a.ldo + n;
      float xn = *xp;
      if (a.ks > 1) {
        float pv[kVerifyMaxKs];
#pragma unroll
        for (int k = 0; k < kVerifyMaxKs; ++k)
          pv[k] = ld_agent(a.part + ((size_t)(k < a.ks ? k : 0) * M + r) * a.ldo + n);
#pragma unroll
        for (int k = 0; k < kVerifyMaxKs; ++k)
          if (k < a.ks) xn += pv[k];
      } else {
        xn += fin[r][c];
      }
      *xp = xn;
      store_split(a.act_next, a.lda, M, r, n, xn * bf16_to_f32(a.g_next[n]));
      const float sq = wave_sum(xn * xn);
      if (lane == 0) a.ss_out[(size_t)r * nt + blockIdx.x] = sq;
    }
  }
}

// Stream-K form of the gate/up product.  The product's units, a
// tile pair (64 weight rows) times a stage of 256 k, are dealt out in equal
// contiguous ranges in (tile pair, stage) order, one range per workgroup and
// one workgroup per CU: every CU streams the same number of bytes, and its
// register pipeline (two stages in flight, as in k_vgemm) runs on across
// tile-pair boundaries.  (With one whole tile pair per workgroup the gate /
// up product has 344 workgroups for 256 CUs, and the CUs that hold two of
// them set its length.)  A tile pair inside the range gets its epilogue as
// soon as its last stage is multiplied; a pair the range shares with its
// neighbours (at most one at each end) keeps its sums in registers until
// the range is done, then writes them through to skpart at its slot (its
// rank among the pair's workgroups) and counts itself in skcnt; the last to
// arrive adds the slots in slot order, so the result does not depend on the
// arrival order, and runs the epilogue.  (The QKV product keeps one tile
// pair per workgroup: its 192 pairs on 256 CUs are all shared in this form,
// and the end-of-range hand-over made it slower.)
constexpr int kSkMaxC = kVerifySkMaxC;  // most workgroups sharing one tile pair

template <int WFMT, int EPI>
__global__ __launch_bounds__(kGBlock, 1) void k_vgemm_sk(VGemmArgs a) {
  static_assert(EPI == EPI_SWIGLU, "the stream-K form serves the gate/up product");
  constexpr int T = 2;
  using St = VStage<WFMT>;
  extern __shared__ __align__(16) char smem[];
  float (*red)[T][32][33] = (float (*)[T][32][33])smem;
  __shared__ float inv_s[kMaxRows];
  __shared__ int last_s[2];
  const int tid = threadIdx.x, lane = tid & (AIO_WAVE - 1), wid = tid / AIO_WAVE;
  const int rl = lane & 31, kh = lane >> 5;
  const size_t wbytes = WFMT == AIO_WFMT_BF16 ? 2 : 1;
  const int M = a.M;
  const bool col_live = rl < 3 * M;
  constexpr int BPS = St::BPS, BPW = St::BPW;
  const int nkb = a.K / 32;
  const int nst = (nkb + BPS - 1) / BPS;
  const long long U = (long long)a.tiles * nst, G = gridDim.x, gb = blockIdx.x;
  const int u0 = (int)(gb * U / G), u1 = (int)((gb + 1) * U / G);
  // workgroup whose range holds unit u
  auto owner = [&](long long u) { return (int)(((u + 1) * G - 1) / U); };

  // norm scales: requested first, reduced once the first stages are in flight
  static_assert(kMaxRows <= 2 * kGWaves, "two rows per wave");
  float ssp[2][2] = {{0.f, 0.f}, {0.f, 0.f}};
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int r = wid + kGWaves * h;
    if (r < M) {
      const float* ssr = a.ss_in + (size_t)r * a.nt;
      if (lane < a.nt) ssp[h][0] = ssr[lane];
      if (lane + 64 < a.nt) ssp[h][1] = ssr[lane + 64];
    }
  }
  const uint16_t* actp = a.act + (size_t)(col_live ? rl : 0) * a.lda;

  // staging: load j of this thread is chunk lchunk[j] of stage row lrow[j]
  // (row < 32: tile 0, else tile 1, of whichever pair the unit belongs to)
  int lrow[St::NLD], lds_off[St::NLD], lchunk[St::NLD];
#pragma unroll
  for (int j = 0; j < St::NLD; ++j) {
    const int f = j * kGBlock + tid;
    lrow[j] = f / St::CPR;
    lchunk[j] = f % St::CPR;
    lds_off[j] = lrow[j] * St::RS + lchunk[j] * 16;
  }
  const int kend = nkb * 32 * (int)wbytes - 16;  // last 16-byte chunk of a row
  // first byte of weight row rr (0..63) of tile pair tp: rows tp 32 ..
  // tp 32 + 31 of gate (rr < 32), then the same rows of up
  auto row_ptr = [&](int tp, int rr) -> const char* {
    const void* w = rr >= 32 ? a.w1 : a.w0;
    int n = tp * 32 + (rr & 31);
    if (n >= a.N) n = a.N - 1;
    return (const char*)w + (size_t)n * a.K * wbytes;
  };
  // loads past the range re-read its last unit (and are not multiplied)
  auto gload_w = [&](uint4 (&R)[St::NLD], int u) {
    const int uu = u < u1 ? u : u1 - 1;
    const int tp = uu / nst, s = uu - tp * nst;
#pragma unroll
    for (int j = 0; j < St::NLD; ++j) {
      int off = s * St::KC * (int)wbytes + lchunk[j] * 16;
      off = off < kend ? off : kend;
      R[j] = ldg_nt(row_ptr(tp, lrow[j]) + off);
    }
  };
  auto gload_a = [&](uint4 (&A)[BPW][2], int u) {
    const int uu = u < u1 ? u : u1 - 1;
    const int s = uu % nst;
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
      const int block = min(s * BPS + wid + kGWaves * j, nkb - 1);
      A[j][0] = ldg(actp + vk_lo<WFMT>(block * 32, kh));
      A[j][1] = ldg(actp + vk_hi<WFMT>(block * 32, kh));
    }
  };
  auto stage = [&](const uint4 (&R)[St::NLD]) {
    __syncthreads();  // every wave is done with the previous stage
#pragma unroll
    for (int j = 0; j < St::NLD; ++j) {
      const u32x4 w = {R[j].x, R[j].y, R[j].z, R[j].w};
      *(u32x4*)(smem + lds_off[j]) = w;
    }
    __syncthreads();
  };
  f32x16 acc[T];
  auto product = [&](int u, const uint4 (&A)[BPW][2]) {
    const int s = u % nst;
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
      const int wb = wid + kGWaves * j;
      const bool live = col_live && s * BPS + wb < nkb;
      VFrag<WFMT, T> f;
#pragma unroll
      for (int t = 0; t < T; ++t)
        frag_lds<WFMT>(smem + (t * 32 + rl) * St::RS, wb, kh, f.wa[t], f.wb[t]);
      f.ba = __builtin_bit_cast(bf16x8, A[j][0]);
      f.bb = __builtin_bit_cast(bf16x8, A[j][1]);
      vmma(f, live, acc);
    }
  };
  auto zero_acc = [&]() {
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[t][i] = 0.f;
  };
  // The eight waves' sums of the current tile pair: element e = 32 r + i of
  // this thread (e < 32 M), both tiles, three split terms added; raw (the
  // norm scale comes later).
  auto reduce = [&](float (&y)[T]) {
    __syncthreads();  // the stage buffer becomes the partial-tile buffer
    if (wid >= kGWaves / 2) {
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          red[wid - kGWaves / 2][t][8 * (v / 4) + 4 * kh + (v % 4)][rl] = acc[t][v];
    }
    __syncthreads();
    if (wid < kGWaves / 2) {
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float& r = red[wid][t][8 * (v / 4) + 4 * kh + (v % 4)][rl];
          r += acc[t][v];
        }
    }
    __syncthreads();
    const int i = tid % 32, r = tid / 32;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      float s = 0.f;
      if (tid < 32 * M) {
#pragma unroll
        for (int w = 0; w < kGWaves / 2; ++w)
          s += red[w][t][i][r] + red[w][t][i][M + r] + red[w][t][i][2 * M + r];
      }
      y[t] = s;
    }
    // the next stage() starts with a barrier: every read of red is done
    // before the buffer is written again
  };

  uint4 R0[St::NLD], R1[St::NLD];
  uint4 A0[BPW][2], A1[BPW][2];
  gload_w(R0, u0);
  gload_a(A0, u0);
  gload_w(R1, u0 + 1);
  gload_a(A1, u0 + 1);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int r = wid + kGWaves * h;
    if (r < M) {
      float p = ssp[h][0] + ssp[h][1];
      for (int c = lane + 128; c < a.nt; c += 64) p += a.ss_in[(size_t)r * a.nt + c];
      const float sum = wave_sum(p);
      if (lane == 0) inv_s[r] = rsqrtf(sum / (float)a.K + a.eps);
    }
  }
  const int pos = a.st->pos;
  const int er = tid / 32, ei = tid % 32;  // this thread's epilogue element
  // the range's shared tile pairs: [0] the one it starts in, [1] the one it
  // ends in (-1: none)
  int ptp[2] = {-1, -1};
  float py[2][T] = {{0.f, 0.f}, {0.f, 0.f}};
  zero_acc();
  // After the product of unit u: if u ends a segment (the last unit of a
  // tile pair or of the range), reduce it and finish or keep it.
  auto seg_end = [&](int u) {
    const int tp = u / nst;
    if (u + 1 != u1 && u + 1 != (tp + 1) * nst) return;
    float y[T];
    reduce(y);
    zero_acc();
    const int sa = u0 > tp * nst ? u0 : tp * nst;  // first unit of the segment
    const bool whole = sa == tp * nst && u + 1 == (tp + 1) * nst;
    if (whole) {
      if (tid < 32 * M)
        vgemm_epi<WFMT, EPI>(a, tp, er, ei, y[0] * inv_s[er], y[1] * inv_s[er], pos);
    } else if (sa == u0) {
      ptp[0] = tp;
      py[0][0] = y[0];
      py[0][1] = y[1];
    } else {
      ptp[1] = tp;
      py[1][0] = y[0];
      py[1][1] = y[1];
    }
  };
  auto step = [&](uint4 (&R)[St::NLD], uint4 (&A)[BPW][2], int u) {
    stage(R);
    __builtin_amdgcn_sched_barrier(0);
    gload_w(R, u + 2);
    __builtin_amdgcn_sched_barrier(0);
    product(u, A);
    __builtin_amdgcn_sched_barrier(0);
    gload_a(A, u + 2);
    __builtin_amdgcn_sched_barrier(0);
    seg_end(u);
  };
  int u = u0;
  for (; u + 2 <= u1; u += 2) {
    step(R0, A0, u);
    step(R1, A1, u + 1);
  }
  if (u < u1) {
    stage(R0);
    product(u, A0);
    seg_end(u);
  }

  // shared tile pairs: write the sums through, count, and the last of the
  // pair's workgroups adds the slots in order and finishes it
  int slot[2], ncon[2];
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    slot[p] = ncon[p] = 0;
    if (ptp[p] < 0) continue;
    const long long first = (long long)ptp[p] * nst;
    const int g0 = owner(first), g1 = owner(first + nst - 1);
    slot[p] = (int)gb - g0;
    ncon[p] = g1 - g0 + 1;
    if (tid < 32 * M) {
      float* dst = a.skpart + ((size_t)ptp[p] * kSkMaxC + slot[p]) * (kMaxRows * 64) + er * 64 + ei;
      st_agent(dst, py[p][0]);
      st_agent(dst + 32, py[p][1]);
    }
  }
  if (ptp[0] < 0 && ptp[1] < 0) return;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid < 2) {
    last_s[tid] = 0;
    if (ptp[tid] >= 0) last_s[tid] = atomic_add_agent(a.skcnt + ptp[tid], 1) == ncon[tid] - 1;
  }
  __syncthreads();
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    if (!last_s[p]) continue;
    if (tid == 0) atomic_store_agent(a.skcnt + ptp[p], 0);  // ready for the next product
    if (tid < 32 * M) {
      const float* src = a.skpart + (size_t)ptp[p] * kSkMaxC * (kMaxRows * 64) + er * 64 + ei;
      float v0[kSkMaxC], v1[kSkMaxC];
#pragma unroll
      for (int k = 0; k < kSkMaxC; ++k) {
        const int kk = k < ncon[p] ? k : 0;
        v0[k] = ld_agent(src + (size_t)kk * (kMaxRows * 64));
        v1[k] = ld_agent(src + (size_t)kk * (kMaxRows * 64) + 32);
      }
      float y0 = 0.f, y1 = 0.f;
#pragma unroll
      for (int k = 0; k < kSkMaxC; ++k)
        if (k < ncon[p]) {
          y0 += v0[k];
          y1 += v1[k];
        }
      vgemm_epi<WFMT, EPI>(a, ptp[p], er, ei, y0 * inv_s[er], y1 * inv_s[er], pos);
    }
  }
}

// ------------------------------------------------------- causal attention

struct VAttnArgs {
  const float* q;       // [M][H*hd]
  const uint16_t* kc;   // [Hkv][max_ctx][hd]
  const uint16_t* vc;
  float* part_o;        // [M][H][S][hd]
  float* part_ml;       // [M][H][S][2]
  const aio_state* st;
  int H, Hkv, max_ctx, S, M;
  float scale_log2;
  // k_vattn_mma: the last split of head h to finish merges the head's
  // splits into act (split o [32][lda]); cnt [H] counts finished splits
  int* cnt;
  uint16_t* act;
  int lda;
};

// Causal attention of the M verify rows on MFMA.  One workgroup of kVAW
// waves per (split s, query head h); the split takes key blocks [kbA, kbB)
// of 32 keys, and wave w the blocks kbA + w, kbA + w + kVAW, ...  The
// products are 16 x 16 x 32 MFMAs (lane l: row or column l % 16 of a tile,
// k = 8 (l / 16) .. + 7 of the operands, rows 4 (l / 16) .. + 3 of the
// result): 16 query columns cover the M <= 10 rows with half the dead work
// of a 32-column tile.  Per block:
//   S^T = K Q^T, two tiles of 16 keys: A = key rows straight from the cache
//     (exact bf16), B = the M queries' three bf16 terms (log2-scaled) from
//     LDS; columns past M multiply zeros.  The three terms accumulate into
//     one tile, so column r of S^T is row r's scores in fp32-level
//     precision.  Lane l holds keys 4 (l / 16) .. + 3 of both tiles;
//   online softmax per query column (causal mask j <= pos + r), the max
//     over a column's four lane groups by two exchanges;
//   O^T += V^T P^T: B = the softmax weights' three bf16 terms straight from
//     registers (k slots 8 g .. 8 g + 7 of lane group g are its own keys of
//     tile 0 then tile 1), A = the value tile (staged in LDS row by row,
//     read back one bf16 per key and dimension in that key order).
//     (Transposing on the way in, with one 16-bit store per element, put
//     16 lanes on one bank and tripled the kernel's time.)
// The next block's keys and values are requested before the current one is
// multiplied.  Every wave then leaves its (max, sum, output) state of the
// live rows in LDS, and one pass combines the waves in wave order into the
// split's unnormalized state, written to part_o / part_ml; the head's last
// split to finish merges all of them (vattn_merge).
//
// Eight waves of two blocks each: the blocks a wave streams one after the
// other are the kernel's critical path (about 2 us each at 2K context), so
// a split of 16 blocks is spread over as many waves as fit one workgroup
// per CU with a block in flight per wave.
constexpr int kVAW = 8;
constexpr int kVattnBlocksPerSplit = 2 * kVAW;

template <int HD>
struct VAttnLds {
  static constexpr int QROW = HD * 2 + 16;                 // bytes per query row of one term
  static constexpr int QR = kMaxRows + 1;                   // query rows per term (+ a zero row)
  static constexpr int QBYTES = 3 * QR * QROW;              // three terms of the M queries
  static constexpr int VROW = HD * 2 + 16;                  // bytes per key row of a value tile
  static constexpr int VBYTES = 32 * VROW;                  // one wave's value tile
  static constexpr int OROW = HD + 1;                       // floats per wave output row
  static constexpr int OBYTES = kVAW * kMaxRows * OROW * 4 + 2 * kVAW * kMaxRows * 4;
  static constexpr int TAIL = kVAW * VBYTES > OBYTES ? kVAW * VBYTES : OBYTES;
  static constexpr int BYTES = QBYTES + TAIL;
};

// Key (within the block) of k slot 8 g + j of the P V product: the softmax
// weight register j of lane group g, keys 4 g .. + 3 of tile 0, then of tile 1.
AIO_DEV int vattn_key(int g, int j) { return 16 * (j >> 2) + 4 * g + (j & 3); }

typedef float f32x4 __attribute__((ext_vector_type(4)));

AIO_DEV bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// Wait for this wave's LDS operations (also a compiler barrier for LDS).
AIO_DEV void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Block kb's key fragments (A operand of tile tt: key row 16 tt + l % 16,
// dims 32 c + 8 (l / 16) ..) and value chunks (16 bytes each, row-major);
// keys past n_keys read key 0.
template <int HD>
AIO_DEV void vattn_load(const uint16_t* kbase, const uint16_t* vbase, int kb, int n_keys,
                        int lane, uint4 (&kr)[HD / 16], uint4 (&vr)[32 * HD / 8 / AIO_WAVE]) {
  const int r16 = lane & 15, g = lane >> 4, j0 = kb * 32;
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    const int key = j0 + 16 * tt + r16 < n_keys ? j0 + 16 * tt + r16 : 0;
    const uint16_t* krow = kbase + (size_t)key * HD;
#pragma unroll
    for (int c = 0; c < HD / 32; ++c) kr[tt * (HD / 32) + c] = *(const uint4*)(krow + c * 32 + 8 * g);
  }
#pragma unroll
  for (int it = 0; it < 32 * HD / 8 / AIO_WAVE; ++it) {
    const int f = it * AIO_WAVE + lane, kk = f / (HD / 8), d0 = (f % (HD / 8)) * 8;
    const int vkey = j0 + kk < n_keys ? j0 + kk : 0;
    vr[it] = *(const uint4*)(vbase + (size_t)vkey * HD + d0);
  }
}

// Online combination of one more (max m2, sum l2, output o2) state into
// (m, l, o), all in log2 units; a state with max -inf holds no key.
AIO_DEV void attn_fold(float& m, float& l, float& o, float m2, float l2, float o2) {
  const float mn = fmaxf(m, m2);
  const float c1 = m == -INFINITY ? 0.f : exp2f(m - mn);
  const float c2 = m2 == -INFINITY ? 0.f : exp2f(m2 - mn);
  o = o * c1 + o2 * c2;
  l = l * c1 + l2 * c2;
  m = mn;
}

// Merge of head h's S splits for the M rows (by the split that finished
// last; the others' states are in memory, read past the caches): per output
// element, the splits' states are folded in split order (attn_fold) and the
// result o / l is split into act.  Eight splits' states are requested
// together, so at up to 8 splits the merge is one round trip.
template <int HD>
AIO_DEV void vattn_merge(const VAttnArgs& a, int h) {
  constexpr int NT = kVAW * AIO_WAVE;
  const int M = a.M, S = a.S;
  for (int e = threadIdx.x; e < M * HD; e += NT) {
    const int r = e / HD, dim = e % HD;
    const float* po = a.part_o + ((size_t)r * a.H + h) * S * HD + dim;
    const float* ml = a.part_ml + ((size_t)r * a.H + h) * S * 2;
    float m = -INFINITY, l = 0.f, o = 0.f;
    for (int s0 = 0; s0 < S; s0 += 8) {
      float mv[8], lv[8], ov[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int sp = s0 + j < S ? s0 + j : S - 1;
        mv[j] = ld_agent(ml + 2 * sp);
        lv[j] = ld_agent(ml + 2 * sp + 1);
        ov[j] = ld_agent(po + (size_t)sp * HD);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (s0 + j < S) attn_fold(m, l, o, mv[j], lv[j], ov[j]);
    }
    store_split(a.act, a.lda, M, r, h * HD + dim, l > 0.f ? o / l : 0.f);
  }
}

template <int HD>
__global__ __launch_bounds__(kVAW * AIO_WAVE, 1) void k_vattn_mma(VAttnArgs a) {
  using Lds = VAttnLds<HD>;
  extern __shared__ __align__(16) char smem[];
  char* qs = smem;                  // [3][QR][QROW]; row kMaxRows of each term is zero
  char* tail = smem + Lds::QBYTES;  // per wave: value tile; at the end: the waves' states
  const int tid = threadIdx.x, lane = tid & (AIO_WAVE - 1), wid = tid / AIO_WAVE;
  const int col = lane & 15, g = lane >> 4;  // query column, lane group
  const int s = blockIdx.x, h = blockIdx.y, M = a.M;
  const int kvh = h / (a.H / a.Hkv);
  const int pos = a.st->pos;
  const int n_keys = pos + M;  // the last row sees keys [0, pos + M - 1]
  const int nkb = (n_keys + 31) / 32;
  const int kbA = (int)((long long)s * nkb / a.S), kbB = (int)((long long)(s + 1) * nkb / a.S);

  const uint16_t* kbase = a.kc + (size_t)kvh * a.max_ctx * HD;
  const uint16_t* vbase = a.vc + (size_t)kvh * a.max_ctx * HD;
  constexpr int NDT = HD / 16;           // 16-dim tiles of the output
  constexpr int NCH = HD / 32;           // 32-dim chunks of a key row
  constexpr int NVL = 32 * HD / 8 / AIO_WAVE;  // 16-byte value chunks per lane
  // The queries are requested first, then the wave's first key block:
  // loads complete in order, so waiting for the queries leaves the block in
  // flight.
  constexpr int NT = kVAW * AIO_WAVE;
  constexpr int NQ = (kMaxRows * HD + NT - 1) / NT;
  float qv[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const int e = tid + i * NT, qq = e / HD, dim = e % HD;
    qv[i] = e < M * HD ? a.q[(size_t)qq * a.H * HD + (size_t)h * HD + dim] : 0.f;
  }
  uint4 kr[2 * NCH], vr[NVL];
  int kb = kbA + wid;
  vattn_load<HD>(kbase, vbase, max(min(kb, kbB - 1), 0), n_keys, lane, kr, vr);

  // queries, scaled to log2 units and split into three bf16 terms
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const int e = tid + i * NT, qq = e / HD, dim = e % HD;
    if (e < M * HD) {
      uint16_t t0, t1, t2;
      split3(qv[i] * a.scale_log2, t0, t1, t2);
      *(uint16_t*)(qs + (0 * Lds::QR + qq) * Lds::QROW + dim * 2) = t0;
      *(uint16_t*)(qs + (1 * Lds::QR + qq) * Lds::QROW + dim * 2) = t1;
      *(uint16_t*)(qs + (2 * Lds::QR + qq) * Lds::QROW + dim * 2) = t2;
    }
  }
  for (int e = tid; e < 3 * HD; e += NT)
    *(uint16_t*)(qs + ((e / HD) * Lds::QR + kMaxRows) * Lds::QROW + (e % HD) * 2) = 0;
  __syncthreads();

  // this lane's query column col: row col sees keys [0, lim]
  const bool live = col < M;
  const int lim = pos + (live ? col : M - 1);
  // columns past the M rows read the zero row: their columns of S^T are zero
  const char* qrow = qs + (live ? col : kMaxRows) * Lds::QROW;
  char* vt = tail + wid * Lds::VBYTES;
  f32x4 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) o[dt][i] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  for (; kb < kbB; kb += kVAW) {
    const int j0 = kb * 32;
    // value rows -> LDS (a vector store: a uint4 struct copy is a memcpy,
    // which keeps vr in scratch memory)
#pragma unroll
    for (int it = 0; it < NVL; ++it) {
      const int f = it * AIO_WAVE + lane, kk = f / (HD / 8), d0 = (f % (HD / 8)) * 8;
      const u32x4 w = {vr[it].x, vr[it].y, vr[it].z, vr[it].w};
      *(u32x4*)(vt + kk * Lds::VROW + d0 * 2) = w;
    }
    // scores S^T[key][query] over the HD dims, three query terms, two
    // tiles of 16 keys.  The query fragments of chunk c + 1 are requested
    // before the products of chunk c.
    f32x4 sc[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) sc[tt][i] = 0.f;
    bf16x8 qf[2][3];
#pragma unroll
    for (int t = 0; t < 3; ++t)
      qf[0][t] = as_bf16x8(*(const uint4*)(qrow + t * Lds::QR * Lds::QROW + 8 * g * 2));
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      if (c + 1 < NCH) {
#pragma unroll
        for (int t = 0; t < 3; ++t)
          qf[(c + 1) & 1][t] = as_bf16x8(
              *(const uint4*)(qrow + t * Lds::QR * Lds::QROW + ((c + 1) * 32 + 8 * g) * 2));
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        const bf16x8 ak = as_bf16x8(kr[tt * NCH + c]);
#pragma unroll
        for (int t = 0; t < 3; ++t)
          sc[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ak, qf[c & 1][t], sc[tt], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // the next block's keys and values are in flight during the softmax and
    // the P V product (the last block re-reads itself: no branch, so the
    // fragments stay in registers)
    vattn_load<HD>(kbase, vbase, kb + kVAW < kbB ? kb + kVAW : kb, n_keys, lane, kr, vr);
    // causal mask (only a block holding keys past pos needs it; the test is
    // the same for the whole wave) and online softmax for this lane's query
    // column; register j = 4 tt + v holds key j0 + vattn_key(g, j)
    float sv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) sv[j] = sc[j >> 2][j & 3];
    if (j0 + 31 > pos) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j0 + vattn_key(g, j) > lim) sv[j] = -INFINITY;
    }
    float mx = sv[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) mx = fmaxf(mx, sv[j]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, AIO_WAVE));
    mx = fmaxf(mx, __shfl_xor(mx, 32, AIO_WAVE));
    const float mnew = fmaxf(m, mx);
    // while every key so far is masked, mnew is -inf: subtract 0 instead, so
    // exp2(-inf - 0) = 0 gives the zero weights (and o, lsum stay 0)
    const float mref = mnew == -INFINITY ? 0.f : mnew;
    const float cf = __builtin_amdgcn_exp2f(m - mref);
    float p[8];
    float ps = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      p[j] = __builtin_amdgcn_exp2f(sv[j] - mref);
      ps += p[j];
    }
    lsum = lsum * cf + ps;
    m = mnew;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) o[dt][i] *= cf;
    // the weights split by truncation: t0 = the top 16 bits of p, t1 those
    // of p - t0, t2 = p - t0 - t1 (exact: 8 significant bits each, 24 in
    // all), without the rounding's branches
    bf16x8 bp[3];
    {
      uint32_t tt[3][8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t u0 = __float_as_uint(p[e]) & 0xffff0000u;
        const float r1 = p[e] - __uint_as_float(u0);
        const uint32_t u1 = __float_as_uint(r1) & 0xffff0000u;
        const float r2 = r1 - __uint_as_float(u1);
        tt[0][e] = u0;
        tt[1][e] = u1;
        tt[2][e] = __float_as_uint(r2);
      }
#pragma unroll
      for (int t = 0; t < 3; ++t)
        bp[t] = as_bf16x8(make_uint4((tt[t][0] >> 16) | (tt[t][1] & 0xffff0000u),
                                     (tt[t][2] >> 16) | (tt[t][3] & 0xffff0000u),
                                     (tt[t][4] >> 16) | (tt[t][5] & 0xffff0000u),
                                     (tt[t][6] >> 16) | (tt[t][7] & 0xffff0000u)));
    }
    wave_lds_sync();  // the value tile is in LDS
    // O^T += V^T P^T per 16-dim tile, three terms of the weights
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      // V^T fragment: dimension 16 dt + col at this lane group's eight keys
      const char* vcol = vt + (dt * 16 + col) * 2;
      uint32_t w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = (uint32_t)*(const uint16_t*)(vcol + vattn_key(g, 2 * j) * Lds::VROW) |
               ((uint32_t)*(const uint16_t*)(vcol + vattn_key(g, 2 * j + 1) * Lds::VROW) << 16);
      const bf16x8 av = as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
#pragma unroll
      for (int t = 0; t < 3; ++t)
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bp[t], o[dt], 0, 0, 0);
    }
    wave_lds_sync();  // every read of the value tile is done before the next block's writes
  }
  lsum += __shfl_xor(lsum, 16, AIO_WAVE);
  lsum += __shfl_xor(lsum, 32, AIO_WAVE);

  // every wave's state of the live rows -> LDS (over the value tiles)
  __syncthreads();
  float* om = (float*)tail;                    // [kVAW][kMaxRows][OROW] outputs
  float* mm = om + kVAW * kMaxRows * Lds::OROW;  // [kVAW][kMaxRows] max
  float* ll = mm + kVAW * kMaxRows;            // [kVAW][kMaxRows] sum
  if (live) {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        om[(wid * kMaxRows + col) * Lds::OROW + dt * 16 + 4 * g + v] = o[dt][v];
    if (g == 0) {
      mm[wid * kMaxRows + col] = m;
      ll[wid * kMaxRows + col] = lsum;
    }
  }
  __syncthreads();

  // The split's state of its M rows: the waves folded in wave order
  // (unnormalized output, (max, sum) in log2 units), written through to
  // memory.
  for (int e = tid; e < M * HD; e += NT) {
    const int r = e / HD, dim = e % HD;
    float ms = -INFINITY, ls = 0.f, os = 0.f;
#pragma unroll
    for (int w = 0; w < kVAW; ++w)
      attn_fold(ms, ls, os, mm[w * kMaxRows + r], ll[w * kMaxRows + r],
                om[(w * kMaxRows + r) * Lds::OROW + dim]);
    st_agent(a.part_o + (((size_t)r * a.H + h) * a.S + s) * HD + dim, os);
    if (dim == 0) {
      float* ml = a.part_ml + (((size_t)r * a.H + h) * a.S + s) * 2;
      st_agent(ml, ms);
      st_agent(ml + 1, ls);
    }
  }
  // count the split; the last of head h's splits to arrive merges them
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  __shared__ int last_s;
  if (tid == 0) last_s = atomic_add_agent(a.cnt + h, 1) == a.S - 1;
  __syncthreads();
  if (!last_s) return;
  if (tid == 0) atomic_store_agent(a.cnt + h, 0);  // ready for the next layer
  vattn_merge<HD>(a, h);
}

// Launch with `blocks` tile pairs.  A residual-add product with fewer tile
// pairs than CUs also splits K over workgroups, as far as every wave keeps
// at least two blocks of 32 k (at most kVerifyMaxKs slices); the others run
// one K slice per workgroup.  Split slices store their products in the vpart
// region and count themselves in vcnt.
template <int EPI>
hipError_t launch_vgemm(const aio_model& m, const VGemmArgs& g, int blocks) {
  VGemmArgs a = g;
  a.ks = 1;
  a.nt = m.cfg.d_model / 64;
  a.eps = m.cfg.rms_eps;
  if (EPI == EPI_RESID) {
    const int nkb = a.K / 32;
    while (blocks * a.ks < m.num_cus && 2 * a.ks <= kVerifyMaxKs &&
           nkb / (2 * a.ks * kGWaves) >= 2)
      a.ks *= 2;
    a.part = m.at<float>(m.lay.vpart);
    a.cnt = m.at<int>(m.lay.vcnt);
    a.ss_out = m.at<float>(m.lay.vss);
  } else {
    a.ss_in = m.at<float>(m.lay.vss);
  }
  const dim3 grid(blocks, a.ks);
  if (m.cfg.wfmt == AIO_WFMT_INT8) {
    constexpr int lds = vgemm_lds<AIO_WFMT_INT8>();
    const hipError_t e = hipFuncSetAttribute((const void*)k_vgemm<AIO_WFMT_INT8, EPI>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_vgemm<AIO_WFMT_INT8, EPI>), grid, dim3(kGBlock), lds, m.stream, a);
  } else {
    constexpr int lds = vgemm_lds<AIO_WFMT_BF16>();
    const hipError_t e = hipFuncSetAttribute((const void*)k_vgemm<AIO_WFMT_BF16, EPI>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_vgemm<AIO_WFMT_BF16, EPI>), grid, dim3(kGBlock), lds, m.stream, a);
  }
  return hipGetLastError();
}

// Stream-K launch of the gate/up product of `tiles` tile pairs: one
// workgroup per CU, but every range at least `per` units long, so that at
// most kSkMaxC - 1 ranges meet in one tile pair (a pair of nst units spans
// at most 1 + ceil((nst - 1) / per) ranges).
template <int EPI>
hipError_t launch_vgemm_sk(const aio_model& m, const VGemmArgs& g, int tiles) {
  VGemmArgs a = g;
  a.ks = 1;
  a.nt = m.cfg.d_model / 64;
  a.eps = m.cfg.rms_eps;
  a.ss_in = m.at<float>(m.lay.vss);
  a.tiles = tiles;
  a.skpart = m.at<float>(m.lay.skpart);
  a.skcnt = m.at<int>(m.lay.skcnt);
  if ((size_t)tiles > m.lay.sk_tiles) return hipErrorInvalidValue;
  const int nst = (a.K / 32 + 7) / 8;  // stages of 256 k
  const long long U = (long long)tiles * nst;
  const int per = std::max(2, (nst - 1 + kSkMaxC - 3) / (kSkMaxC - 2));
  const long long G = std::max<long long>(1, std::min<long long>(m.num_cus, U / per));
  if (m.cfg.wfmt == AIO_WFMT_INT8) {
    constexpr int lds = vgemm_lds<AIO_WFMT_INT8>();
    const hipError_t e = hipFuncSetAttribute((const void*)k_vgemm_sk<AIO_WFMT_INT8, EPI>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_vgemm_sk<AIO_WFMT_INT8, EPI>), dim3((unsigned)G), dim3(kGBlock), lds,
                       m.stream, a);
  } else {
    constexpr int lds = vgemm_lds<AIO_WFMT_BF16>();
    const hipError_t e = hipFuncSetAttribute((const void*)k_vgemm_sk<AIO_WFMT_BF16, EPI>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_vgemm_sk<AIO_WFMT_BF16, EPI>), dim3((unsigned)G), dim3(kGBlock), lds,
                       m.stream, a);
  }
  return hipGetLastError();
}

// Split of x * g and chunk sums of squares for the M rows of x (layer 0:
// x is first set to the embedding rows).
hipError_t launch_vnorm(const aio_model& m, float* x, const uint16_t* embed, const void* gain,
                        uint16_t* act, int M) {
  VNormArgs n{};
  n.x = x;
  n.embed = embed;
  n.gain = (const uint16_t*)gain;
  n.act = act;
  n.lda = m.lay.ka;
  n.d = m.cfg.d_model;
  n.M = M;
  n.ss = m.at<float>(m.lay.vss);
  n.st = m.state();
  hipLaunchKernelGGL(k_vnorm, dim3(M), dim3(kNormBlock), 0, m.stream, n);
  return hipGetLastError();
}

template <int HD>
hipError_t launch_vattn_mma(const aio_model& m, const VAttnArgs& t) {
  constexpr int lds = VAttnLds<HD>::BYTES;
  const hipError_t e = hipFuncSetAttribute((const void*)k_vattn_mma<HD>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_vattn_mma<HD>, dim3(t.S, t.H), dim3(kVAW * AIO_WAVE), lds, m.stream, t);
  return hipGetLastError();
}

}  // namespace

hipError_t aio_launch_verify(const aio_model& m, int M, int pos, float* logits,
                             bool last_row_only) {
  const aio_config& c = m.cfg;
  const int d = c.d_model, H = c.n_heads, Hkv = c.n_kv_heads, hd = c.head_dim, F = c.ffn_dim;
  const int ka = m.lay.ka;
  // two split-activation buffers: A feeds the QKV / gate-up / LM-head GEMMs,
  // B feeds the O / down GEMMs.
  uint16_t* actA = m.at<uint16_t>(m.lay.act);
  uint16_t* actB = actA + (size_t)32 * ka;
  float* x = m.at<float>(m.lay.x);
  float* q = m.at<float>(m.lay.q);
  hipError_t e = launch_vnorm(m, x, (const uint16_t*)m.embed, m.layers[0].attn_norm, actA, M);
  if (e != hipSuccess) return e;
  for (int l = 0; l < c.n_layers; ++l) {
    const aio_layer_weights& L = m.layers[(size_t)l];
    const void* g_after = l + 1 < c.n_layers ? m.layers[(size_t)l + 1].attn_norm : m.final_norm;

    VGemmArgs g{};
    g.act = actA; g.lda = ka; g.M = M;
    g.w0 = L.wq; g.w1 = L.wk; g.w2 = L.wv;
    g.s0 = (const uint16_t*)L.sq; g.s1 = (const uint16_t*)L.sk; g.s2 = (const uint16_t*)L.sv;
    g.N = (H + 2 * Hkv) * hd; g.K = d;
    g.out = q; g.ldo = H * hd;
    g.kc = m.kv_layer(l, 0); g.vc = m.kv_layer(l, 1);
    g.rope = m.rope; g.st = m.state();
    g.H = H; g.Hkv = Hkv; g.hd = hd; g.max_ctx = c.max_ctx;
    if ((e = launch_vgemm<EPI_QKV>(m, g, (H + 2 * Hkv) * (hd / 64))) != hipSuccess) return e;

    VAttnArgs t{};
    t.q = q; t.kc = g.kc; t.vc = g.vc;
    t.part_o = m.at<float>(m.lay.part_o);
    t.part_ml = m.at<float>(m.lay.part_ml);
    t.st = m.state();
    t.H = H; t.Hkv = Hkv; t.max_ctx = c.max_ctx; t.S = m.lay.splits; t.M = M;
    t.scale_log2 = (float)(1.4426950408889634 / sqrt((double)hd));
    // splits of kVattnBlocksPerSplit key blocks, but no more workgroups than
    // CUs: a workgroup takes a whole CU, and a second round of workgroups
    // pays the queries' prologue and the merges again (at 32K, 64 splits per
    // head cost 9.2 ms per 7B verify).  The host's pos sizes the grid; the
    // kernel takes its key range from the device state.
    const int nkb = (pos + M + 31) / 32;
    const int s_cap = std::max(1, std::min(m.lay.vsplits, m.num_cus / H));
    t.S = std::max(1, std::min(s_cap, (nkb + kVattnBlocksPerSplit - 1) / kVattnBlocksPerSplit));
    t.cnt = m.at<int>(m.lay.vacnt);
    t.act = actB;
    t.lda = ka;
    if ((e = hd == 128 ? launch_vattn_mma<128>(m, t) : launch_vattn_mma<64>(m, t)) != hipSuccess)
      return e;

    VGemmArgs o{};
    o.act = actB; o.lda = ka; o.M = M;
    o.w0 = L.wo; o.s0 = (const uint16_t*)L.so;
    o.N = d; o.K = H * hd; o.out = x; o.ldo = d; o.st = m.state();
    o.g_next = (const uint16_t*)L.ffn_norm; o.act_next = actA;
    if ((e = launch_vgemm<EPI_RESID>(m, o, d / 64)) != hipSuccess) return e;

    VGemmArgs gu{};
    gu.act = actA; gu.lda = ka; gu.M = M;
    gu.w0 = L.w_gate; gu.w1 = L.w_up;
    gu.s0 = (const uint16_t*)L.s_gate; gu.s1 = (const uint16_t*)L.s_up;
    gu.N = F; gu.K = d; gu.act_out = actB; gu.lda_out = ka; gu.st = m.state();
    if ((e = launch_vgemm_sk<EPI_SWIGLU>(m, gu, (F + 31) / 32)) != hipSuccess) return e;

    VGemmArgs dn{};
    dn.act = actB; dn.lda = ka; dn.M = M;
    dn.w0 = L.w_down; dn.s0 = (const uint16_t*)L.s_down;
    dn.N = d; dn.K = F; dn.out = x; dn.ldo = d; dn.st = m.state();
    dn.g_next = (const uint16_t*)g_after; dn.act_next = actA;
    if ((e = launch_vgemm<EPI_RESID>(m, dn, d / 64)) != hipSuccess) return e;
  }
  if (last_row_only) {
    // the last row's final RMSNorm and LM head only (a prefill of M tokens)
    if (M > 1 && (e = hipMemcpyAsync(x, x + (size_t)(M - 1) * d, (size_t)d * sizeof(float),
                                     hipMemcpyDeviceToDevice, m.stream)) != hipSuccess)
      return e;
    return aio_launch_lm_rows(m, 1, logits);
  }
  VGemmArgs lm{};
  lm.act = actA; lm.lda = ka; lm.M = M;
  lm.w0 = m.lm_head; lm.s0 = (const uint16_t*)m.s_lm_head;
  lm.N = c.vocab; lm.K = d; lm.out = logits; lm.ldo = c.vocab; lm.st = m.state();
  return launch_vgemm<EPI_STORE>(m, lm, (c.vocab + 63) / 64);
}

hipError_t aio_launch_lm_rows(const aio_model& m, int rows, float* logits) {
  const aio_config& c = m.cfg;
  uint16_t* actA = m.at<uint16_t>(m.lay.act);
  float* x = m.at<float>(m.lay.x);
  hipError_t e = launch_vnorm(m, x, nullptr, m.final_norm, actA, rows);
  if (e != hipSuccess) return e;
  VGemmArgs lm{};
  lm.act = actA; lm.lda = m.lay.ka; lm.M = rows;
  lm.w0 = m.lm_head; lm.s0 = (const uint16_t*)m.s_lm_head;
  lm.N = c.vocab; lm.K = c.d_model; lm.out = logits; lm.ldo = c.vocab; lm.st = m.state();
  return launch_vgemm<EPI_STORE>(m, lm, (c.vocab + 63) / 64);
}
