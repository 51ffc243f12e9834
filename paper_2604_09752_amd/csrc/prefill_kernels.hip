// Prefill: a prompt of R rows at positions pos0 .. pos0 + R - 1 in one pass
// of prompt-length matrix products (M = R), for gfx950.  This is the probe's
// single forward over its templated request: every row's K and V go to the
// cache, and the last row's logits come out.
//
// Per layer: QKV GEMM (+norm scale, RoPE, K/V append) -> pattn (causal
// flash attention; row r sees positions [0, pos0 + r]) -> O GEMM
// (+residual, x g for the next norm) -> gate/up GEMM (+norm scale, SwiGLU)
// -> down GEMM (+residual, x g).  The RMSNorm is folded into the products:
// its factor 1 / sqrt(mean(x^2) + eps) is one number per row, so a residual
// product writes x g (not yet normalised) and the sums of squares of x over
// 64-column blocks, and the consuming product scales its outputs by the
// row's factor.  Only layer 0's embedding rows go through pnorm.  The last
// row then goes through the final RMSNorm and the LM head of the verify
// path.
//
// Precision.  Activations stay fp32 between kernels.  The GEMMs run on MFMA
// (v_mfma_f32_32x32x16_bf16) with every activation split exactly into three
// bf16 terms as it is staged in LDS (a = t0 + t1 + t2), so the products keep
// fp32 accuracy (two terms leave 2^-18, which measurably loosens the cache
// rows of deeper layers).  Weights are exact in bf16 (int8 weights
// convert exactly; their fp16 per-output-channel scale applies in the
// epilogue).  Attention splits the queries and the softmax weights into
// three terms as well.
#include <math.h>

#include "aio_internal.h"
#include "common.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

AIO_DEV f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

AIO_DEV bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// Terms of the activation split.
constexpr int kNT = 3;

// Three-term bf16 split by truncation, for fp32 bits `a`: t0 = the top 16
// bits of a, t1 those of r1 = a - t0, t2 those of r1 - t1.  Both
// subtractions are exact and r1 - t1 has at most 8 significant bits, so a =
// t0 + t1 + t2 exactly (for a normal, as every activation here is).
// Returned as fp32 bit patterns with the low 16 bits clear (the bf16 in the
// high half); branch-free.  (Rounding to nearest instead costs several
// times the operations, and in the stage loader its registers spilled.)
AIO_DEV void split3t(uint32_t a, uint32_t (&t)[kNT]) {
  t[0] = a & 0xffff0000u;
  const float r1 = __uint_as_float(a) - __uint_as_float(t[0]);
  t[1] = __float_as_uint(r1) & 0xffff0000u;
  t[2] = __float_as_uint(r1 - __uint_as_float(t[1])) & 0xffff0000u;
}

// Two floats as bf16 (round to nearest even) in one word, the first low.
AIO_DEV uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// Device-coherent access for the K slices of a split product: the partials
// are written through to memory and read past the (per-XCD) L2, and the
// slice counters are vector atomics at device scope.
AIO_DEV void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
AIO_DEV float ld_agent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
AIO_DEV int atomic_add_agent(int* p, int v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
AIO_DEV void atomic_store_agent(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wait for this wave's LDS operations; also a compiler barrier, so no LDS
// access moves across it.  Lanes of one wave exchange data through LDS
// without a workgroup barrier (the waves of a workgroup run different
// numbers of iterations).
AIO_DEV void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// ------------------------------------------------------------- RMSNorm rows

struct PNormArgs {
  float* x;                // [R][d] residual rows (layer 0: written from the embedding)
  const uint16_t* embed;   // layer 0: embedding table, else null
  const int32_t* tokens;   // [R] (layer 0)
  const uint16_t* gain;
  float* act;              // [R][lda]: x g
  int lda;
  int d;
  float* ss;               // [R][d / 64] sums of squares of x over 64-column blocks
};

constexpr int kNormThreads = 256;

// One workgroup per row (layer 0): x from the embedding table, x g, and the
// row's sums of squares of x per 64-column block.
__global__ __launch_bounds__(kNormThreads) void k_pnorm(PNormArgs a) {
  const int r = blockIdx.x, tid = threadIdx.x;
  float* xr = a.x + (size_t)r * a.d;
  const uint16_t* emb = a.embed ? a.embed + (size_t)a.tokens[r] * a.d : nullptr;
  float* out = a.act + (size_t)r * a.lda;
  // a wave covers one 64-column block per pass (d is a multiple of 64)
  for (int e0 = 0; e0 < a.d; e0 += kNormThreads) {
    const int e = e0 + tid;
    float v = 0.f;
    if (e < a.d) {
      if (emb) {
        v = bf16_to_f32(emb[e]);
        xr[e] = v;
      } else {
        v = xr[e];
      }
      out[e] = v * bf16_to_f32(a.gain[e]);
    }
    const float sq = wave_sum(v * v);
    if ((tid & (AIO_WAVE - 1)) == 0 && e < a.d) a.ss[(size_t)r * (a.d / 64) + e / 64] = sq;
  }
}

// --------------------------------------------------------------------- GEMM

// A workgroup of 2 WN waves computes a tile of 64 WN weight rows (2 WN
// blocks of 32, in "units" of 128 rows, the granule of the row mapping
// below) by 64 prompt rows, every term of each.  Wave (wn, wr) owns row
// blocks 2 wn ("lo") and 2 wn + 1 ("hi") and prompt rows [32 wr, 32 wr +
// 32), so the two rows an epilogue combines (a RoPE pair, gate and up) sit
// in one lane.  Long prompts take WN = 4 (256 rows): the loads, not the
// MFMAs, set the rate, and the larger tile does twice the products for 1.4x
// the bytes per stage (prefill of 2048 tokens 32.2 -> 28.5 ms); short ones
// WN = 2, which gives twice the workgroups.
// Weights and activations pass through LDS in stages of 32 k, double
// buffered: the next stage's global loads are in flight in registers while
// the current one is multiplied.  Rows in LDS are 80 bytes apart (64 + a
// 16-byte skew), so the 32 rows a fragment read touches spread over the
// banks.
constexpr int kPfMaxKs = 8;  // most K slices of a prefill product
constexpr int kUnit = 128;   // weight rows per unit of the row mapping (block_src)
constexpr int kBR = 64;   // prompt rows per tile
constexpr int kKT = 32;   // k per stage
constexpr int kRowB = kKT * 2 + 16;
constexpr int kBCols = kNT * kBR;                  // activation columns: term-major per wave half
constexpr int kBChunks = kBR * (kKT / 4);         // 16-byte (4 x fp32) activation chunks per stage

// The tile shape of WN waves across the weight rows.
template <int WN>
struct PTile {
  static constexpr int GT = 2 * WN * AIO_WAVE;              // threads
  static constexpr int BM = 64 * WN;                        // weight rows
  static constexpr int UPT = BM / kUnit;                    // units per tile
  static constexpr int BLd = (kBChunks + GT - 1) / GT;      // activation loads per thread
  static constexpr int StageB = (BM + kBCols) * kRowB;      // weight rows + activation columns
  static constexpr int Lds = 2 * StageB;
};

enum PEpi { PE_QKV = 0, PE_RESID = 1, PE_SWIGLU = 2 };

struct PGemmArgs {
  const float* act;     // [R][lda] activations (split into terms on the way to LDS)
  int lda;
  int R;
  const void* w0;       // QKV: wq | SWIGLU: w_gate | RESID: the matrix
  const void* w1;       // QKV: wk | SWIGLU: w_up
  const void* w2;       // QKV: wv
  const uint16_t* s0;
  const uint16_t* s1;
  const uint16_t* s2;
  int N, K;             // QKV: N = (H + 2 Hkv) hd virtual rows; SWIGLU: F; RESID: rows
  float* out;           // QKV: q [R][H hd] | RESID: x [R][N]
  int ldo;
  float* act_out;       // SWIGLU: [R][lda_out]
  int lda_out;
  uint16_t* kc;         // QKV: cache of the layer, [Hkv][max_ctx][hd]
  uint16_t* vc;
  const float2* rope;   // [max_ctx][hd / 2] (cos, sin)
  int pos0, H, Hkv, hd, max_ctx;
  // K split over workgroups (grid.z) when the tiles alone are too few: each
  // slice writes its partial tile through to fix and counts itself in
  // tcnt[tile]; the last slice to arrive adds the partials in slice order
  // and runs the epilogue
  int ks;
  float* fix;           // [tiles][ks][32][threads]
  int* tcnt;            // [tiles], zero between products
  // the folded RMSNorm: QKV and SWIGLU scale output row r by 1 / sqrt(sum
  // of ss_in[r][0 .. nss) / K + eps); RESID (with act_next) writes x g_next
  // to act_next and ss_out[r][n / 64] for its columns
  const float* ss_in;
  float* ss_out;
  int nss;
  float eps;
  float* act_next;
  int lda_next;
  const uint16_t* g_next;
};

// Where block `blk` (0..3) of unit `bx` reads its 32 rows: matrix index
// (0, 1, 2 = w0, w1, w2), first row in that matrix, and the number of valid
// rows (0 for a block past the end).
struct BlockSrc {
  int mat, row0, valid;
  int vrow0;  // QKV: virtual row of the block's first row
};

template <int EPI>
AIO_DEV BlockSrc block_src(const PGemmArgs& a, int bx, int blk) {
  BlockSrc b{0, 0, 0, 0};
  if constexpr (EPI == PE_QKV) {
    const int nheads = a.H + 2 * a.Hkv;
    int head, off;
    if (a.hd == 128) {
      head = bx;
      off = (blk & 1) * 64 + (blk >> 1) * 32;  // blocks 0..3 -> 0, 64, 32, 96
    } else {
      head = 2 * bx + (blk >> 1);
      off = (blk & 1) * 32;
    }
    if (head >= nheads) return b;
    const int vr = head * a.hd + off;
    const int qrows = a.H * a.hd, krows = a.Hkv * a.hd;
    b.vrow0 = vr;
    b.valid = 32;
    if (vr >= qrows + krows) { b.mat = 2; b.row0 = vr - qrows - krows; }
    else if (vr >= qrows) { b.mat = 1; b.row0 = vr - qrows; }
    else { b.mat = 0; b.row0 = vr; }
  } else if constexpr (EPI == PE_SWIGLU) {
    // blocks: gate f0, up f0, gate f0 + 32, up f0 + 32
    const int f = bx * 64 + (blk >> 1) * 32;
    b.mat = blk & 1;
    b.row0 = f;
    b.valid = f < a.N ? min(32, a.N - f) : 0;
  } else {
    const int n = bx * kUnit + blk * 32;
    b.row0 = n;
    b.valid = n < a.N ? min(32, a.N - n) : 0;
  }
  return b;
}

// One of the three weight matrices, selected arithmetically (an indexed
// local array would live in scratch memory).
AIO_DEV const char* pick_mat(const PGemmArgs& a, int mat) {
  const uint64_t b0 = (uint64_t)a.w0;
  const uint64_t d1 = (uint64_t)a.w1 - b0, d2 = (uint64_t)a.w2 - b0;
  return (const char*)(b0 + (uint64_t)(mat == 1) * d1 + (uint64_t)(mat == 2) * d2);
}

// Global loads of stage st: A_LD 16-byte weight chunks and BLD activation
// chunks per thread.
template <int WFMT, int WN, int A_LD, int BLD = PTile<WN>::BLd>
AIO_DEV void gload_stage(const char* const (&aptr)[A_LD], const float* const (&bptr)[BLD],
                         int st, uint4 (&ra)[A_LD], uint4 (&rb)[BLD]) {
  constexpr int GT = PTile<WN>::GT;
  constexpr int wbytes = WFMT == AIO_WFMT_BF16 ? 2 : 1;
  const size_t ko = (size_t)st * kKT;
#pragma unroll
  for (int j = 0; j < A_LD; ++j) ra[j] = ld_stream((const uint4*)(aptr[j] + ko * wbytes));
#pragma unroll
  for (int j = 0; j < BLD; ++j)
    if (j + 1 < BLD || kBChunks % GT == 0 || (int)threadIdx.x < kBChunks % GT)
      rb[j] = *(const uint4*)(bptr[j] + ko);
}

// The same chunks into an LDS stage buffer: int8 widened to bf16 (exact:
// |q| <= 127); each activation value split into its three bf16 terms, one
// 8-byte store per term column (4 consecutive k).
template <int WFMT, int WN, int A_LD, int BLD = PTile<WN>::BLd>
AIO_DEV void lstore_stage(char* buf, const int (&alds)[A_LD], const int (&blds)[BLD],
                          const uint4 (&ra)[A_LD], const uint4 (&rb)[BLD]) {
  constexpr int GT = PTile<WN>::GT;
  // (vector stores: a uint4 struct copy is a memcpy, which keeps the
  // register sets in scratch memory)
#pragma unroll
  for (int j = 0; j < A_LD; ++j) {
    if constexpr (WFMT == AIO_WFMT_BF16) {
      const u32x4 w = {ra[j].x, ra[j].y, ra[j].z, ra[j].w};
      *(u32x4*)(buf + alds[j]) = w;
    } else {
      const uint32_t w[4] = {ra[j].x, ra[j].y, ra[j].z, ra[j].w};
      uint32_t o[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t sw = w[i / 2];
        const int sh = (i & 1) * 16;
        const float f0 = (float)(int8_t)(sw >> sh), f1 = (float)(int8_t)(sw >> (sh + 8));
        o[i] = (__float_as_uint(f0) >> 16) | (__float_as_uint(f1) & 0xffff0000u);
      }
      const u32x4 w0 = {o[0], o[1], o[2], o[3]}, w1 = {o[4], o[5], o[6], o[7]};
      *(u32x4*)(buf + alds[j]) = w0;
      *(u32x4*)(buf + alds[j] + 16) = w1;
    }
  }
#pragma unroll
  for (int j = 0; j < BLD; ++j)
    if (j + 1 < BLD || kBChunks % GT == 0 || (int)threadIdx.x < kBChunks % GT) {
      uint32_t t[4][kNT];
      split3t(rb[j].x, t[0]);
      split3t(rb[j].y, t[1]);
      split3t(rb[j].z, t[2]);
      split3t(rb[j].w, t[3]);
#pragma unroll
      for (int k = 0; k < kNT; ++k) {
        const u32x2 w = {(t[0][k] >> 16) | t[1][k], (t[2][k] >> 16) | t[3][k]};
        *(u32x2*)(buf + blds[j] + k * 32 * kRowB) = w;
      }
    }
}

// The MFMA products of one LDS stage: 16-k chunks, the wave's two row blocks
// by the terms of its 32 prompt rows.  Activation columns of the stage are
// ordered [wave half wr][term][row].
template <int WN>
AIO_DEV void stage_product(const char* cur, int wn, int wr, int rl, int kh,
                           f32x16 (&acc)[2][kNT]) {
  constexpr int kBM = PTile<WN>::BM;
#pragma unroll
  for (int c16 = 0; c16 < kKT / 16; ++c16) {
    const int koff = (c16 * 16 + 8 * kh) * 2;
    bf16x8 af[2], bfr[kNT];
#pragma unroll
    for (int b = 0; b < 2; ++b)
      af[b] = as_bf16x8(*(const uint4*)(cur + ((2 * wn + b) * 32 + rl) * kRowB + koff));
#pragma unroll
    for (int t = 0; t < kNT; ++t)
      bfr[t] = as_bf16x8(
          *(const uint4*)(cur + (kBM + (wr * kNT + t) * 32 + rl) * kRowB + koff));
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int t = 0; t < kNT; ++t) acc[b][t] = mfma(af[b], bfr[t], acc[b][t]);
  }
}

// The logical (weight tile, prompt-row tile, K slice) of this workgroup.
// Workgroups go to the 8 XCDs round-robin by linear id, and each XCD has its
// own L2; so the linear ids are renumbered to give every XCD a contiguous
// run of the logical order, in which the tiles go down bands of up to 8
// prompt-row tiles per weight tile.  The workgroups that run at once on one
// XCD then share a few weight tiles and a few activation tiles in its L2,
// instead of each bringing its own from memory (2048 tokens 20.8 -> 18.9
// ms).  A product split over K keeps the hardware order: its workgroups
// all run in one round, and renumbered, the workgroups of one XCD would
// all read one K slice, whose rows' equal k offsets share a few HBM
// channels (128 tokens 3.31 -> 3.49 ms).
struct PTileId {
  int bx, by, kz;
};
AIO_DEV PTileId ptile_id() {
  PTileId t;
  if (gridDim.z > 1) {
    t.bx = (int)blockIdx.x;
    t.by = (int)blockIdx.y;
    t.kz = (int)blockIdx.z;
    return t;
  }
  const int nx = (int)gridDim.x, ny = (int)gridDim.y, g = nx * ny;
  const int lin = (int)(blockIdx.x + gridDim.x * blockIdx.y);
  const int rem = g % 8 == 0 ? (lin % 8) * (g / 8) + lin / 8 : lin;
  t.kz = 0;
  constexpr int kBand = 8;
  const int by0 = rem / (kBand * nx) * kBand;
  const int nb = min(kBand, ny - by0);
  const int in = rem - by0 * nx;
  t.bx = in / nb;
  t.by = by0 + in % nb;
  return t;
}

template <int WFMT, int EPI, int WN>
__global__ __launch_bounds__(PTile<WN>::GT) void k_pgemm(PGemmArgs a) {
  using Tl = PTile<WN>;
  constexpr int kGT = Tl::GT, kBM = Tl::BM, kBLd = Tl::BLd, kStageB = Tl::StageB;
  extern __shared__ __align__(16) char smem[];
  const int tid = threadIdx.x, lane = tid & (AIO_WAVE - 1), wid = tid / AIO_WAVE;
  const int wn = wid % WN, wr = wid / WN;
  const int rl = lane & 31, kh = lane >> 5;
  const PTileId tid3 = ptile_id();
  const int bx = tid3.bx, r0 = tid3.by * kBR;
  constexpr int wbytes = WFMT == AIO_WFMT_BF16 ? 2 : 1;

  // Staging assignments.  A: row ra of the tile (block ra / 32), 16-byte
  // chunk ca of the stage's 32 k (bf16: 4 chunks of 8 weights; int8: 2
  // chunks of 16 weights, widened to 32 bytes in LDS).  B: prompt row r0 +
  // p (p = 32 wr' + j), 8 chunks of 4 fp32 k; its terms t go to the LDS
  // activation columns (wr' kNT + t) 32 + j.
  constexpr int A_CPR = WFMT == AIO_WFMT_BF16 ? 4 : 2;
  constexpr int A_LD = kBM * A_CPR / kGT;
  const char* aptr[A_LD];
  int alds[A_LD];
#pragma unroll
  for (int j = 0; j < A_LD; ++j) {
    const int f = j * kGT + tid, ra = f / A_CPR, ca = f % A_CPR;
    const int blk = ra >> 5;  // block of the tile: unit UPT bx + blk / 4, block blk % 4 of it
    const BlockSrc s = block_src<EPI>(a, Tl::UPT * bx + (blk >> 2), blk & 3);
    int row = s.row0 + ((ra & 31) < s.valid ? (ra & 31) : 0);
    if (s.valid == 0) row = 0;  // a block past the end reads row 0 of w0 (discarded)
    const char* w = s.valid ? pick_mat(a, s.mat) : (const char*)a.w0;
    aptr[j] = w + ((size_t)row * a.K + (size_t)ca * (16 / wbytes)) * wbytes;
    alds[j] = ra * kRowB + ca * 16 * (2 / wbytes);
  }
  const float* bptr[kBLd];
  int blds[kBLd];
#pragma unroll
  for (int j = 0; j < kBLd; ++j) {
    const int f = min(j * kGT + tid, kBChunks - 1), p = f / 8, c = f % 8;
    const int row = r0 + p;
    bptr[j] = a.act + (size_t)(row < a.R ? row : a.R - 1) * a.lda + c * 4;
    blds[j] = (kBM + (p / 32) * kNT * 32 + (p % 32)) * kRowB + c * 8;
  }
  uint4 ra_[A_LD], rb_[kBLd];
  f32x16 acc[2][kNT];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int t = 0; t < kNT; ++t)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[b][t][i] = 0.f;

  // this workgroup's stages [sA, sB) of K (all of them unless K is split).
  // Two register sets keep two stages' loads in flight (a stage's loads take
  // a memory round trip, its products a fraction of one): set 1 holds the
  // stages sA + 1, sA + 3, ..., set 0 the others; loads past sB re-read the
  // last stage and are not used.
  const int nst = a.K / kKT, kz = tid3.kz;
  const int sA = kz * nst / a.ks, sB = (kz + 1) * nst / a.ks;
  uint4 ra1[A_LD], rb1[kBLd];
  const int sL = sB - 1;
  gload_stage<WFMT, WN, A_LD>(aptr, bptr, sA, ra_, rb_);
  gload_stage<WFMT, WN, A_LD>(aptr, bptr, min(sA + 1, sL), ra1, rb1);
  // the folded norm's row factors of the tile's 64 prompt rows, Tl::GT / 64
  // threads per row (their loads queue behind the first stages'; the
  // barrier below publishes them)
  __shared__ float inv_rows[kBR];
  if constexpr (EPI != PE_RESID) {
    constexpr int TPR = Tl::GT / kBR;
    const int j = tid / TPR, part = tid % TPR;
    const float* ssr = a.ss_in + (size_t)min(r0 + j, a.R - 1) * a.nss;
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    int c = part;
    for (; c + 3 * TPR < a.nss; c += 4 * TPR) {
      s0 += ssr[c];
      s1 += ssr[c + TPR];
      s2 += ssr[c + 2 * TPR];
      s3 += ssr[c + 3 * TPR];
    }
    for (; c < a.nss; c += TPR) s0 += ssr[c];
    float sum = (s0 + s1) + (s2 + s3);
#pragma unroll
    for (int off = TPR / 2; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, AIO_WAVE);
    if (part == 0) inv_rows[j] = rsqrtf(sum / (float)a.K + a.eps);
  }
  lstore_stage<WFMT, WN, A_LD>(smem, alds, blds, ra_, rb_);
  __syncthreads();
  gload_stage<WFMT, WN, A_LD>(aptr, bptr, min(sA + 2, sL), ra_, rb_);
  // stage S from its LDS buffer; then stage S + 1 (in set RA, RB) to the
  // other buffer, and the set refilled with stage S + 3 (written out for
  // each set: a set chosen at run time would live in scratch memory)
#define AIO_PF_STEP(S, RA, RB)                                                          \
  do {                                                                                 \
    stage_product<WN>(smem + (((S) - sA) & 1) * kStageB, wn, wr, rl, kh, acc);             \
    lstore_stage<WFMT, WN, A_LD>(smem + (((S) + 1 - sA) & 1) * kStageB, alds, blds, RA, RB); \
    __syncthreads();                                                                   \
    gload_stage<WFMT, WN, A_LD>(aptr, bptr, min((S) + 3, sL), RA, RB);                     \
  } while (0)
  int st = sA;
  for (; st + 2 < sB; st += 2) {
    AIO_PF_STEP(st, ra1, rb1);
    AIO_PF_STEP(st + 1, ra_, rb_);
  }
  if (st + 1 < sB) {
    AIO_PF_STEP(st, ra1, rb1);
    ++st;
  }
#undef AIO_PF_STEP
  stage_product<WN>(smem + ((st - sA) & 1) * kStageB, wn, wr, rl, kh, acc);

  // the tile's sums over the three terms: lane l, register v -> column
  // (prompt row) l % 32, row i = 8 (v / 4) + 4 (l / 32) + v % 4 of the
  // 32-row blocks lo and hi
  float ylo[16], yhi[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    ylo[v] = acc[0][0][v];
    yhi[v] = acc[1][0][v];
#pragma unroll
    for (int t = 1; t < kNT; ++t) {
      ylo[v] += acc[0][t][v];
      yhi[v] += acc[1][t][v];
    }
  }
  if (a.ks > 1) {
    // K split: every slice's partial goes through memory (written through,
    // read past the caches); the last slice to arrive adds them in slice
    // order, so the sum is the same whatever the arrival order
    // (element-major, so that each store and load instruction of a wave
    // covers 256 contiguous bytes).  Lanes of prompt rows past R move
    // nothing: at a short prompt most of the tile's rows are (the last
    // slice's reads of 8 partial tiles were half of a 23-row O product).
    const int tile = tid3.by * (int)gridDim.x + bx;
    const bool row_live = r0 + wr * 32 + rl < a.R;
    float* mine = a.fix + ((size_t)tile * a.ks + kz) * 32 * kGT + tid;
    if (row_live) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        st_agent(mine + v * kGT, ylo[v]);
        st_agent(mine + (16 + v) * kGT, yhi[v]);
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    __shared__ int last_s;
    if (tid == 0) last_s = atomic_add_agent(a.tcnt + tile, 1) == a.ks - 1;
    __syncthreads();
    if (!last_s) return;
    if (tid == 0) atomic_store_agent(a.tcnt + tile, 0);  // ready for the next product
#pragma unroll
    for (int v = 0; v < 16; ++v) ylo[v] = yhi[v] = 0.f;
    for (int k = 0; k < (row_live ? a.ks : 0); ++k) {
      const float* pk = a.fix + ((size_t)tile * a.ks + k) * 32 * kGT + tid;
      float plo[16], phi[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        plo[v] = ld_agent(pk + v * kGT);
        phi[v] = ld_agent(pk + (16 + v) * kGT);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        ylo[v] += plo[v];
        yhi[v] += phi[v];
      }
    }
  }

  // Epilogue.
  const int r = r0 + wr * 32 + rl;
  if (r >= a.R) return;
  const BlockSrc slo = block_src<EPI>(a, Tl::UPT * bx + (wn >> 1), 2 * (wn & 1));
  const BlockSrc shi = block_src<EPI>(a, Tl::UPT * bx + (wn >> 1), 2 * (wn & 1) + 1);
  if constexpr (EPI == PE_RESID) {
    // N is a multiple of 64: the wave's two blocks (adjacent, from a
    // multiple of 64) are both whole or both past the end.  The lane's 16
    // values of a block are 4 runs of 4 columns, moved as float4.
    if (!slo.valid) return;
    float* xrow = a.out + (size_t)r * a.ldo;
    float sq = 0.f;  // the lane's sum of squares of the new x
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
      const int nb = (hb ? shi.row0 : slo.row0) + 4 * kh;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = nb + 8 * g;
        float y[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          y[e] = hb ? yhi[4 * g + e] : ylo[4 * g + e];
          if constexpr (WFMT == AIO_WFMT_INT8) y[e] *= fp16_to_f32(a.s0[n + e]);
        }
        float4* xp = (float4*)(xrow + n);
        float4 xn = *xp;
        xn.x += y[0];
        xn.y += y[1];
        xn.z += y[2];
        xn.w += y[3];
        *xp = xn;
        if (a.act_next) {
          const uint16_t* gn = a.g_next + n;
          *(float4*)(a.act_next + (size_t)r * a.lda_next + n) =
              make_float4(xn.x * bf16_to_f32(gn[0]), xn.y * bf16_to_f32(gn[1]),
                          xn.z * bf16_to_f32(gn[2]), xn.w * bf16_to_f32(gn[3]));
          sq = fmaf(xn.x, xn.x, sq);
          sq = fmaf(xn.y, xn.y, sq);
          sq = fmaf(xn.z, xn.z, sq);
          sq = fmaf(xn.w, xn.w, sq);
        }
      }
    }
    // the wave's 64 columns are one block of the sums for row r: this lane
    // holds 32 of them, the lane 32 away (same row) the other 32
    if (a.act_next) {
      sq += __shfl_xor(sq, 32, AIO_WAVE);
      if (kh == 0) a.ss_out[(size_t)r * a.nss + slo.row0 / 64] = sq;
    }
    return;
  }
  const float rs = inv_rows[wr * 32 + rl];
  if constexpr (EPI == PE_SWIGLU) {
    // F is a multiple of 64: the block is whole or past the end; the lane's
    // 16 values are 4 runs of 4 columns, one float4 store each
    if (!slo.valid) return;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int n = slo.row0 + 8 * g + 4 * kh;
      float h[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float gt = ylo[4 * g + e] * rs, up = yhi[4 * g + e] * rs;
        if constexpr (WFMT == AIO_WFMT_INT8) {
          gt *= fp16_to_f32(a.s0[n + e]);
          up *= fp16_to_f32(a.s1[n + e]);
        }
        h[e] = gt / (1.f + expf(-gt)) * up;
      }
      *(float4*)(a.act_out + (size_t)r * a.lda_out + n) = make_float4(h[0], h[1], h[2], h[3]);
    }
    return;
  }
  // QKV: the pair (row, row + hd/2) of a head section in blocks lo and hi;
  // the lane's rows come in runs of 4, stored as one vector each (q fp32,
  // the K / V cache bf16)
  if (slo.valid == 0) return;
  const int half = a.hd / 2, mat = slo.mat, p = a.pos0 + r;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int i0 = 8 * g + 4 * kh;
    const int row = slo.row0 + i0;           // first of 4 rows in its matrix
    const int ii = (slo.vrow0 + i0) % a.hd;  // its index in the head (< hd / 2)
    float lo[4], hi[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo[e] = ylo[4 * g + e] * rs;
      hi[e] = yhi[4 * g + e] * rs;
      if constexpr (WFMT == AIO_WFMT_INT8) {
        const uint16_t* sc = mat == 0 ? a.s0 : (mat == 1 ? a.s1 : a.s2);
        lo[e] *= fp16_to_f32(sc[row + e]);
        hi[e] *= fp16_to_f32(sc[row + e + half]);
      }
      if (mat < 2) {
        const float2 cs = a.rope[(size_t)p * half + ii + e];
        const float r0v = lo[e] * cs.x - hi[e] * cs.y;
        const float r1v = hi[e] * cs.x + lo[e] * cs.y;
        lo[e] = r0v;
        hi[e] = r1v;
      }
    }
    if (mat == 0) {
      float* q = a.out + (size_t)r * a.ldo + row;
      *(float4*)q = make_float4(lo[0], lo[1], lo[2], lo[3]);
      *(float4*)(q + half) = make_float4(hi[0], hi[1], hi[2], hi[3]);
    } else {
      uint16_t* c = (mat == 1 ? a.kc : a.vc) + ((size_t)(row / a.hd) * a.max_ctx + p) * a.hd + ii;
      *(uint2*)c = make_uint2(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]));
      *(uint2*)(c + half) = make_uint2(pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3]));
    }
  }
}

// ------------------------------------------------------ causal attention

struct PAttnArgs {
  const float* q;       // [R][H hd] rotated queries
  int ldq;
  const uint16_t* kc;   // [Hkv][max_ctx][hd]
  const uint16_t* vc;
  float* act;           // [R][lda]: the output, at columns h hd ..
  int lda;
  int R, pos0, H, Hkv, max_ctx;
  float scale_log2;     // log2(e) / sqrt(hd)
};

constexpr int kAW = 4;  // waves per workgroup: they split the key blocks

template <int HD>
struct AttnLds {
  static constexpr int QROW = HD * 2 + 16;        // bytes per query row of one term
  static constexpr int QBYTES = 3 * 32 * QROW;     // three terms of 32 queries
  static constexpr int VROW = HD * 2 + 16;         // bytes per key row of a value tile
  static constexpr int VBYTES = 32 * VROW;         // one wave's value tile (32 keys)
  static constexpr int OROW = HD + 1;              // floats per combined output row (padded)
  static constexpr int OBYTES = 2 * 32 * OROW * 4 + 2 * 2 * 32 * 4;  // combine: 2 waves' O, m, l
  static constexpr int TAIL = kAW * VBYTES > OBYTES ? kAW * VBYTES : OBYTES;
  static constexpr int BYTES = QBYTES + TAIL;
};

// Key of element e (0..7) of lane half kh's softmax weights in 16-key chunk
// c2.  The weights reach the P V product as the B operand straight from the
// score tile's registers: score register v = 8 c2 + e holds key
// 8 (v / 4) + 4 kh + v % 4, so the A fragment (V^T) gathers the value rows
// of those keys.
AIO_DEV int pkey(int c2, int kh, int e) { return 16 * c2 + 8 * (e >> 2) + 4 * kh + (e & 3); }

// One workgroup per (32 query rows, head): wave w takes key blocks w, w + 4,
// ... of 32 keys.  Per block: S^T = K Q^T on MFMA (A = 32 key rows from the
// cache, B = the queries' three bf16 terms from LDS), the online softmax per
// query (one query per lane pair), then O^T += V^T P^T (A = the value tile,
// staged in LDS row by row and read back one bf16 per key and dimension; B =
// the softmax weights' three terms from registers).  Transposing the value
// tile on its way into LDS, one 16-bit store per element, put 16 lanes on
// one bank.  The waves' (max, sum, output) states are merged through LDS at
// the end.
template <int HD>
__global__ __launch_bounds__(kAW * AIO_WAVE, 2) void k_pattn(PAttnArgs a) {
  using Lds = AttnLds<HD>;
  extern __shared__ __align__(16) char smem[];
  char* qs = smem;                  // [3][32][QROW]
  char* tail = smem + Lds::QBYTES;  // per wave: value tile; at the end: the merge
  const int tid = threadIdx.x, lane = tid & (AIO_WAVE - 1), wid = tid / AIO_WAVE;
  const int rl = lane & 31, kh = lane >> 5;
  // Query tiles in reverse: a causal tile's work grows with its position,
  // and workgroups start in index order, so the longest start first.  With
  // a multiple of 8 heads, each XCD (workgroups go to the 8 XCDs
  // round-robin by linear id) takes H / 8 consecutive heads, whose keys and
  // values (shared through G) then stay in its own L2 instead of being
  // read by all eight; its heads' tiles interleave, longest first.
  int qt = (int)blockIdx.x, h = (int)blockIdx.y;
  if (gridDim.y % 8 == 0) {
    const int lin = (int)(blockIdx.x + gridDim.x * blockIdx.y);
    const int hpx = (int)gridDim.y / 8, j = lin / 8;
    h = (lin % 8) * hpx + j % hpx;
    qt = j / hpx;
  }
  const int q0 = ((int)gridDim.x - 1 - qt) * 32;
  const int G = a.H / a.Hkv, kvh = h / G;
  const int rows = min(32, a.R - q0);
  const int n_keys = a.pos0 + q0 + rows;  // keys the block's last row sees
  const int nkb = (n_keys + 31) / 32;

  // queries, scaled to log2 units and split into three bf16 terms
  for (int e = tid; e < 32 * HD; e += kAW * AIO_WAVE) {
    const int qq = e / HD, dim = e % HD;
    const float v = qq < rows ? a.q[(size_t)(q0 + qq) * a.ldq + (size_t)h * HD + dim] * a.scale_log2
                              : 0.f;
    const uint16_t t0 = f32_to_bf16(v);
    const float r1 = v - bf16_to_f32(t0);
    const uint16_t t1 = f32_to_bf16(r1);
    const uint16_t t2 = f32_to_bf16(r1 - bf16_to_f32(t1));
    *(uint16_t*)(qs + (0 * 32 + qq) * Lds::QROW + dim * 2) = t0;
    *(uint16_t*)(qs + (1 * 32 + qq) * Lds::QROW + dim * 2) = t1;
    *(uint16_t*)(qs + (2 * 32 + qq) * Lds::QROW + dim * 2) = t2;
  }
  __syncthreads();

  // this lane's query: row q0 + rl sees keys [0, lim]
  const int lim = a.pos0 + q0 + (rl < rows ? rl : rows - 1);
  char* vt = tail + wid * Lds::VBYTES;
  const uint16_t* kbase = a.kc + (size_t)kvh * a.max_ctx * HD;
  const uint16_t* vbase = a.vc + (size_t)kvh * a.max_ctx * HD;
  constexpr int NHB = HD / 32;
  f32x16 o[NHB];
#pragma unroll
  for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[hb][i] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  // Block kb's key fragments (A operand: key row rl, dims 16 c + 8 kh ..) and
  // value chunks (16 bytes of 8 dims, row-major) into registers; keys past
  // n_keys read key 0.  The next block of the wave is requested while the
  // current one is multiplied.
  constexpr int NKC = HD / 16, VCH = 32 * HD / 8, NVL = VCH / AIO_WAVE;
  uint4 kr[NKC], vr[NVL];
  auto load_block = [&](int kb) {
    const int j0 = kb * 32;
    const int key = j0 + rl < n_keys ? j0 + rl : 0;
    const uint16_t* krow = kbase + (size_t)key * HD;
#pragma unroll
    for (int c = 0; c < NKC; ++c) kr[c] = *(const uint4*)(krow + c * 16 + 8 * kh);
#pragma unroll
    for (int it = 0; it < NVL; ++it) {
      const int f = it * AIO_WAVE + lane, kk = f / (HD / 8), d0 = (f % (HD / 8)) * 8;
      const int vkey = j0 + kk < n_keys ? j0 + kk : 0;
      vr[it] = *(const uint4*)(vbase + (size_t)vkey * HD + d0);
    }
  };
  if (wid < nkb) load_block(wid);

  for (int kb = wid; kb < nkb; kb += kAW) {
    const int j0 = kb * 32;
    // value rows -> LDS, row by row (a vector store: a uint4 struct copy
    // would go through scratch memory)
#pragma unroll
    for (int it = 0; it < NVL; ++it) {
      const int f = it * AIO_WAVE + lane, kk = f / (HD / 8), d0 = (f % (HD / 8)) * 8;
      const u32x4 wv = {vr[it].x, vr[it].y, vr[it].z, vr[it].w};
      *(u32x4*)(vt + kk * Lds::VROW + d0 * 2) = wv;
    }
    // scores: S^T[key i][query j] over the HD dims, three query terms
    f32x16 s;
#pragma unroll
    for (int i = 0; i < 16; ++i) s[i] = 0.f;
#pragma unroll
    for (int c = 0; c < NKC; ++c) {
      const bf16x8 ak = as_bf16x8(kr[c]);
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const bf16x8 bq =
            as_bf16x8(*(const uint4*)(qs + (t * 32 + rl) * Lds::QROW + (c * 16 + 8 * kh) * 2));
        s = mfma(ak, bq, s);
      }
    }
    // the wave's next block (the last one re-reads itself: no branch, so
    // the fragments stay in registers)
    load_block(kb + kAW < nkb ? kb + kAW : kb);
    // causal mask and online softmax for this lane's query (column rl)
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int key = j0 + 8 * (v / 4) + 4 * kh + (v % 4);
      if (key > lim) s[v] = -INFINITY;
      mx = fmaxf(mx, s[v]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, AIO_WAVE));
    const float mnew = fmaxf(m, mx);
    // (the hardware exp2: every argument is <= 0, and exp2(-inf) = 0)
    const float c =
        (m == -INFINITY) ? (mnew == -INFINITY ? 1.f : 0.f) : __builtin_amdgcn_exp2f(m - mnew);
    const float mref = mnew == -INFINITY ? 0.f : mnew;
    float p[16];
    float ps = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      p[v] = __builtin_amdgcn_exp2f(s[v] - mref);
      ps += p[v];
    }
    lsum = lsum * c + ps;
    m = mnew;
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[hb][i] *= c;
    wave_lds_sync();  // the value tile is in LDS
    // O^T += V^T P^T, two chunks of 16 keys, three terms of the weights
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      // the weights split by truncation: t0 = the top 16 bits of p, t1 those
      // of p - t0, t2 = p - t0 - t1 (exact: 8 significant bits each)
      uint32_t tt[3][8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t u0 = __float_as_uint(p[8 * c2 + e]) & 0xffff0000u;
        const float r1 = p[8 * c2 + e] - __uint_as_float(u0);
        const uint32_t u1 = __float_as_uint(r1) & 0xffff0000u;
        tt[0][e] = u0;
        tt[1][e] = u1;
        tt[2][e] = __float_as_uint(r1 - __uint_as_float(u1));
      }
      bf16x8 bp[3];
#pragma unroll
      for (int t = 0; t < 3; ++t)
        bp[t] = as_bf16x8(make_uint4((tt[t][0] >> 16) | (tt[t][1] & 0xffff0000u),
                                     (tt[t][2] >> 16) | (tt[t][3] & 0xffff0000u),
                                     (tt[t][4] >> 16) | (tt[t][5] & 0xffff0000u),
                                     (tt[t][6] >> 16) | (tt[t][7] & 0xffff0000u)));
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb) {
        // V^T fragment: dimension hb 32 + rl at this lane's eight keys
        const char* vcol = vt + (hb * 32 + rl) * 2;
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          w[j] = (uint32_t)*(const uint16_t*)(vcol + pkey(c2, kh, 2 * j) * Lds::VROW) |
                 ((uint32_t)*(const uint16_t*)(vcol + pkey(c2, kh, 2 * j + 1) * Lds::VROW) << 16);
        const bf16x8 av = as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
#pragma unroll
        for (int t = 0; t < 3; ++t) o[hb] = mfma(av, bp[t], o[hb]);
      }
    }
    wave_lds_sync();  // every read of the value tile is done before the next block's writes
  }
  lsum += __shfl_xor(lsum, 32, AIO_WAVE);

  // merge the waves' states: 2, 3 into 0, 1, then 1 into 0
  __syncthreads();
  float* om = (float*)tail;                 // [2][32][OROW] outputs (rows padded: no bank conflicts)
  float* mm = om + 2 * 32 * Lds::OROW;      // [2][32] max
  float* ll = mm + 2 * 32;                  // [2][32] sum
  auto put = [&](int slot) {
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        om[((size_t)slot * 32 + rl) * Lds::OROW + hb * 32 + 8 * (v / 4) + 4 * kh + (v % 4)] = o[hb][v];
    if (kh == 0) {
      mm[slot * 32 + rl] = m;
      ll[slot * 32 + rl] = lsum;
    }
  };
  auto take = [&](int slot) {
    const float m2 = mm[slot * 32 + rl], l2 = ll[slot * 32 + rl];
    const float M = fmaxf(m, m2);
    const float c1 = m == -INFINITY ? 0.f : exp2f(m - M);
    const float c2 = m2 == -INFINITY ? 0.f : exp2f(m2 - M);
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        o[hb][v] = o[hb][v] * c1 +
                   om[((size_t)slot * 32 + rl) * Lds::OROW + hb * 32 + 8 * (v / 4) + 4 * kh + (v % 4)] * c2;
    lsum = lsum * c1 + l2 * c2;
    m = M;
  };
  if (wid >= 2) put(wid - 2);
  __syncthreads();
  if (wid < 2) take(wid);
  __syncthreads();
  if (wid == 1) put(0);
  __syncthreads();
  if (wid != 0) return;
  take(0);
  if (rl >= rows) return;
  const int r = q0 + rl;
  const float inv = 1.f / lsum;
  float* out = a.act + (size_t)r * a.lda + (size_t)h * HD;
  // the lane's dimensions come in runs of 4: one float4 store each
#pragma unroll
  for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
    for (int g = 0; g < 4; ++g)
      *(float4*)(out + hb * 32 + 8 * g + 4 * kh) =
          make_float4(o[hb][4 * g] * inv, o[hb][4 * g + 1] * inv, o[hb][4 * g + 2] * inv,
                      o[hb][4 * g + 3] * inv);
}

// ----------------------------------------------------------------- launchers

hipError_t launch_pnorm(const aio_model& m, const PfBuffers& b, int R, const uint16_t* embed,
                        const void* gain) {
  PNormArgs n{};
  n.x = b.x;
  n.embed = embed;
  n.tokens = b.tokens;
  n.gain = (const uint16_t*)gain;
  n.act = b.actA;
  n.lda = b.lda_a;
  n.d = m.cfg.d_model;
  n.ss = b.ss;
  hipLaunchKernelGGL(k_pnorm, dim3(R), dim3(kNormThreads), 0, m.stream, n);
  return hipGetLastError();
}

// Launch over `units` (of 128 weight rows) x (R / 64) prompt-row tiles,
// in tiles of WN / 2 units.  A product also splits K over workgroups (up
// to kPfMaxKs slices of at least 8 stages, within the fix-up buffer's
// room) as far as the workgroups still fit one round of the CUs: a
// workgroup streams its stages one latency apart, so at a short prompt the
// 1B's QKV product (32 tiles of 64 stages) took 57 us unsplit, and a split
// past one round (the 1B's gate/up at 128 rows: 704 workgroups) leaves a
// second, partial round.
template <int WFMT, int EPI, int WN>
hipError_t launch_pgemm_t(const aio_model& m, const PGemmArgs& g0, int units) {
  using Tl = PTile<WN>;
  PGemmArgs g = g0;
  const int tiles = (units + Tl::UPT - 1) / Tl::UPT;
  const int rt = (g.R + kBR - 1) / kBR, nst = g.K / kKT;
  // workgroups one round of the CUs holds: two of 4 waves, one of 8
  const int slots = (WN == 2 ? 2 : 1) * m.num_cus;
  g.ks = 1;
  while (tiles * rt * 2 * g.ks <= slots && 2 * g.ks <= kPfMaxKs &&
         nst / (2 * g.ks) >= 8 &&
         (size_t)tiles * rt * 2 * g.ks * Tl::GT * 32 * 4 <= m.lay.pfix_bytes &&
         (size_t)tiles * rt <= m.lay.pcnt_n)
    g.ks *= 2;
  g.fix = m.at<float>(m.lay.pfix);
  g.tcnt = m.at<int>(m.lay.pcnt);
  const void* fn = (const void*)k_pgemm<WFMT, EPI, WN>;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, Tl::Lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_pgemm<WFMT, EPI, WN>), dim3(tiles, rt, g.ks), dim3(Tl::GT), Tl::Lds,
                     m.stream, g);
  return hipGetLastError();
}

// 256-row tiles from 16 prompt-row tiles (1024 rows) on, 128-row tiles
// below (at 512 rows the smaller tiles were still ahead: 8.76 against
// 8.99 ms for the 1B).
template <int WFMT, int EPI>
hipError_t launch_pgemm_w(const aio_model& m, const PGemmArgs& g, int units) {
  if ((g.R + kBR - 1) / kBR >= 16) return launch_pgemm_t<WFMT, EPI, 4>(m, g, units);
  return launch_pgemm_t<WFMT, EPI, 2>(m, g, units);
}

template <int EPI>
hipError_t launch_pgemm(const aio_model& m, const PGemmArgs& g, int units) {
  if (m.cfg.wfmt == AIO_WFMT_INT8) return launch_pgemm_w<AIO_WFMT_INT8, EPI>(m, g, units);
  return launch_pgemm_w<AIO_WFMT_BF16, EPI>(m, g, units);
}

template <int HD>
hipError_t launch_pattn_t(const aio_model& m, const PAttnArgs& t) {
  const void* fn = (const void*)k_pattn<HD>;
  hipError_t e =
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, AttnLds<HD>::BYTES);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_pattn<HD>, dim3((t.R + 31) / 32, t.H), dim3(kAW * AIO_WAVE),
                     AttnLds<HD>::BYTES, m.stream, t);
  return hipGetLastError();
}

}  // namespace

size_t aio_prefill_row_bytes(const aio_config& c) {
  const size_t d = (size_t)c.d_model, Hd = (size_t)c.n_heads * c.head_dim, F = (size_t)c.ffn_dim;
  const size_t ka = d > Hd ? d : Hd;
  return 4 + 4 * d + 4 * Hd + 4 * ka + 4 * d + 4 * F + 4 * (d / 64);
}

PfBuffers aio_prefill_buffers(const aio_config& c, char* base, int rcap) {
  PfBuffers b{};
  const size_t d = (size_t)c.d_model, Hd = (size_t)c.n_heads * c.head_dim, F = (size_t)c.ffn_dim;
  auto al = [](size_t v) { return (v + 255u) & ~(size_t)255u; };
  size_t off = 0;
  b.rcap = rcap;
  b.lda_a = (int)(d > Hd ? d : Hd);
  b.lda_b = (int)F;
  b.tokens = (int32_t*)(base + off); off = al(off + 4 * (size_t)rcap);
  b.x = (float*)(base + off); off = al(off + 4 * d * rcap);
  b.q = (float*)(base + off); off = al(off + 4 * Hd * rcap);
  b.actA = (float*)(base + off); off = al(off + 4 * (size_t)b.lda_a * rcap);
  b.actN = (float*)(base + off); off = al(off + 4 * d * rcap);
  b.actB = (float*)(base + off); off = al(off + 4 * (size_t)b.lda_b * rcap);
  b.ss = (float*)(base + off); off = al(off + 4 * (d / 64) * rcap);
  b.bytes = off;
  return b;
}

// One chunk of R <= b.rcap prompt rows at positions pos0 .. pos0 + R - 1;
// their tokens are in b.tokens.  On return (enqueued) the cache holds their
// K/V rows in every layer and b.x row R - 1 the last row's final residual.
hipError_t aio_launch_prefill_chunk(const aio_model& m, const PfBuffers& b, int R, int pos0) {
  const aio_config& c = m.cfg;
  const int d = c.d_model, H = c.n_heads, Hkv = c.n_kv_heads, hd = c.head_dim, F = c.ffn_dim;
  const int nss = d / 64;
  hipError_t e;
  // layer 0's input rows: the embeddings, with x g and the sums of squares
  // for its attention norm; every later norm input comes from the residual
  // product before it
  if ((e = launch_pnorm(m, b, R, (const uint16_t*)m.embed, m.layers[0].attn_norm)) != hipSuccess)
    return e;
  for (int l = 0; l < c.n_layers; ++l) {
    const aio_layer_weights& L = m.layers[(size_t)l];
    const bool last = l + 1 == c.n_layers;

    PGemmArgs g{};
    g.act = b.actA; g.lda = b.lda_a; g.R = R;
    g.ss_in = b.ss; g.nss = nss; g.eps = c.rms_eps;
    g.w0 = L.wq; g.w1 = L.wk; g.w2 = L.wv;
    g.s0 = (const uint16_t*)L.sq; g.s1 = (const uint16_t*)L.sk; g.s2 = (const uint16_t*)L.sv;
    g.N = (H + 2 * Hkv) * hd; g.K = d;
    g.out = b.q; g.ldo = H * hd;
    g.kc = m.kv_layer(l, 0); g.vc = m.kv_layer(l, 1);
    g.rope = m.rope; g.pos0 = pos0;
    g.H = H; g.Hkv = Hkv; g.hd = hd; g.max_ctx = c.max_ctx;
    const int qkv_tiles = hd == 128 ? H + 2 * Hkv : (H + 2 * Hkv + 1) / 2;
    if ((e = launch_pgemm<PE_QKV>(m, g, qkv_tiles)) != hipSuccess) return e;

    PAttnArgs t{};
    t.q = b.q; t.ldq = H * hd;
    t.kc = g.kc; t.vc = g.vc;
    t.act = b.actA; t.lda = b.lda_a;
    t.R = R; t.pos0 = pos0; t.H = H; t.Hkv = Hkv; t.max_ctx = c.max_ctx;
    t.scale_log2 = (float)(1.4426950408889634 / sqrt((double)hd));
    e = hd == 128 ? launch_pattn_t<128>(m, t) : launch_pattn_t<64>(m, t);
    if (e != hipSuccess) return e;

    PGemmArgs o{};
    o.act = b.actA; o.lda = b.lda_a; o.R = R;
    o.w0 = L.wo; o.s0 = (const uint16_t*)L.so;
    o.N = d; o.K = H * hd; o.out = b.x; o.ldo = d;
    o.act_next = b.actN; o.lda_next = d;
    o.g_next = (const uint16_t*)L.ffn_norm; o.ss_out = b.ss; o.nss = nss;
    if ((e = launch_pgemm<PE_RESID>(m, o, (d + kUnit - 1) / kUnit)) != hipSuccess) return e;

    PGemmArgs gu{};
    gu.act = b.actN; gu.lda = d; gu.R = R;
    gu.ss_in = b.ss; gu.nss = nss; gu.eps = c.rms_eps;
    gu.w0 = L.w_gate; gu.w1 = L.w_up;
    gu.s0 = (const uint16_t*)L.s_gate; gu.s1 = (const uint16_t*)L.s_up;
    gu.N = F; gu.K = d;
    gu.act_out = b.actB; gu.lda_out = b.lda_b;
    if ((e = launch_pgemm<PE_SWIGLU>(m, gu, (F + 63) / 64)) != hipSuccess) return e;

    PGemmArgs dn{};
    dn.act = b.actB; dn.lda = b.lda_b; dn.R = R;
    dn.w0 = L.w_down; dn.s0 = (const uint16_t*)L.s_down;
    dn.N = d; dn.K = F; dn.out = b.x; dn.ldo = d;
    if (!last) {
      dn.act_next = b.actA; dn.lda_next = b.lda_a;
      dn.g_next = (const uint16_t*)m.layers[(size_t)l + 1].attn_norm;
      dn.ss_out = b.ss; dn.nss = nss;
    }
    if ((e = launch_pgemm<PE_RESID>(m, dn, (d + kUnit - 1) / kUnit)) != hipSuccess) return e;
  }
  return hipSuccess;
}
