// The whole decode step as one persistent, cooperatively launched kernel.
//
// Why: at batch 1 every token streams all weights once (the paper's
// Section 2.1 / Section 3.1 bandwidth argument), and a layer is a chain of
// five dependent matrix-vector products and an attention.  Launched as
// separate kernels, each link pays a dispatch ramp, a prologue and a tail
// (several microseconds each, ~190 links per 7B token).  Here one workgroup
// per CU (512 threads, 8 waves) walks all phases of all layers, separated by
// grid barriers, and issues the first weight loads of the next phase before
// each barrier so HBM keeps streaming while the grid synchronises.
//
// Phases per layer, each followed by a grid barrier:
//   QKV   RMSNorm(x) -> q, k, v rows -> RoPE; q stored, k/v appended (bf16)
//   ATTN  split-KV flash-decode per (kv head, split); the last split to
//         finish for a kv head merges all splits (log-sum-exp) into o
//   O     x += W_o o
//   GU    RMSNorm(x) -> m = silu(W_gate h) * (W_up h)
//   DOWN  x += W_down m
// then LM head (RMSNorm(x) -> logits) with the greedy argmax fused: each
// workgroup reduces its rows and the last one to finish reduces the
// workgroup results, writes the token and advances the position.
//
// Matrix phases: the rows of a matrix are split evenly over workgroups; the
// 8 waves of a workgroup split K, so each lane keeps only its slice of the
// activation in registers; per-wave partial sums meet in LDS.  Weights are
// double-buffered in registers, 8 loads of 16 bytes per lane per batch, and
// every wait for a buffer names only the loads issued before it (the loops
// are branch-free and nothing else is loaded inside them).
//
// Coherence: the 8 XCDs have separate L2 caches that are not kept coherent
// with each other, and a device-scope fence (L2 write-back + invalidate)
// costs 15-20 us.  So every value one workgroup produces for another (x, q,
// o, m, split partials, the new K/V row, barrier flags) is written with
// device-scope stores and read with device-scope loads (both bypass the
// non-coherent L2); a workgroup-scope fence then only has to wait for its own
// stores to complete.  Weights and older KV rows are read-only in the step
// and use ordinary loads.
//
// Every wait is a bounded spin: if a barrier never completes the kernel sets
// an error word and runs to its end instead of hanging.
#include <math.h>

#include <algorithm>

#include "aio_internal.h"
#include "common.h"
#include "step_kernel.h"

namespace {

constexpr int kT = 512;          // threads per workgroup
constexpr int kW = kT / AIO_WAVE; // waves per workgroup
constexpr int kNLD = 8;          // 16-byte weight loads per lane per batch
// Batches in flight per wave (register buffers).  Three stream the loops
// faster but lose overall: the barrier's polling loads are queued behind the
// prefetched weight loads (vector memory returns in order), so a deeper
// prefetch delays every workgroup's view of the release.
constexpr int kNBUF = 2;
constexpr unsigned kSpinLimit = 1u << 17;  // ~0.1-0.2 s of polling

// s_waitcnt immediate for vmcnt(0) with expcnt and lgkmcnt left at their
// maximum (no wait): vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8].
constexpr int kVmcnt0 = 0x0F70;

enum Kind { K_QKV = 0, K_O = 1, K_GU = 2, K_DOWN = 3, K_LM = 4 };

template <int KIND>
constexpr int rpu_of() { return KIND == K_QKV ? 4 : (KIND == K_GU ? 2 : 1); }

// ---------------------------------------------------------- coherent access

AIO_DEV unsigned ld_dev(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
AIO_DEV void st_dev(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
AIO_DEV unsigned add_dev(unsigned* p, unsigned v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
AIO_DEV float ldf_dev(const float* p) { return __uint_as_float(ld_dev((const unsigned*)p)); }
AIO_DEV void stf_dev(float* p, float v) { st_dev((unsigned*)p, __float_as_uint(v)); }

// Wait until this thread's stores have completed, then for the whole
// workgroup; a flag or counter written after this is seen by other
// workgroups only after the data.  The device-scope stores are acknowledged
// once they are visible at device scope; the wait is explicit because a
// workgroup-scope fence does not wait for global stores (the workgroup
// shares one CU).
AIO_DEV void wg_publish() {
  __builtin_amdgcn_s_waitcnt(kVmcnt0);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
}

// Bounded wait.  Once any wait has given up (the error word is set), every
// later wait returns at its next check, so a broken barrier costs well under
// a second instead of hanging the device.
AIO_DEV void spin_ge(const MegaArgs& a, const unsigned* p, unsigned target) {
  unsigned spins = 0;
  while ((int)(ld_dev(p) - target) < 0) {
    __builtin_amdgcn_s_sleep(1);
    if ((++spins & 255u) == 0) {
      if (ld_dev(a.sync + kSyncErr) != 0u) break;
      if (spins > kSpinLimit) {
        st_dev(a.sync + kSyncErr, 1u);
        break;
      }
    }
  }
}

// Grid barrier: every workgroup raises its flag to `epoch`; workgroup 0
// gathers all flags and raises the release word; everyone waits for it.
// The release fence before the flag is an s_waitcnt on every outstanding
// vector memory operation (loads included), so `prefetch` -- the first
// weight loads of the next phase -- is issued only after the flag is up; it
// then proceeds while the workgroup waits for the release.
template <class F>
AIO_DEV void grid_sync(const MegaArgs& a, unsigned ep0, unsigned k, F&& prefetch) {
  const unsigned epoch = ep0 + k;
  wg_publish();
  const int tid = threadIdx.x;
  if (a.bar_arrive && tid == 0) a.bar_arrive[(size_t)k * gridDim.x + blockIdx.x] = wall_clock64();
  if (tid == 0) st_dev(a.sync + kSyncFlags + blockIdx.x, epoch);
  prefetch();
  if (blockIdx.x == 0) {
    for (int i = tid; i < (int)gridDim.x; i += kT) spin_ge(a, a.sync + kSyncFlags + i, epoch);
    __syncthreads();
    if (tid == 0) st_dev(a.sync + kSyncRelease, epoch);
  }
  if (tid == 0) spin_ge(a, a.sync + kSyncRelease, epoch);
  __syncthreads();
  if (a.trace && blockIdx.x == 0 && tid == 0) a.trace[k] = wall_clock64();
  if (a.bar_leave && tid == 0) a.bar_leave[(size_t)k * gridDim.x + blockIdx.x] = wall_clock64();
}

// ------------------------------------------------------------- matrix phase

// The per-layer pointer table is read-only during the step; reading it
// through the constant address space gives scalar loads, which complete on
// their own counter.  A vector load here would be queued behind the weight
// loads already in flight, and the first use of the pointer inside a weight
// loop would then wait for all of them.
typedef __attribute__((address_space(4))) const MegaLayer CMegaLayer;
AIO_DEV const CMegaLayer* layer_at(const MegaArgs& a, int layer) {
  return (const CMegaLayer*)(a.layers + layer);
}


typedef __attribute__((address_space(1))) const u32x4 gl_u32x4;

// Streaming 16-byte weight load through a global-address-space pointer.
AIO_DEV uint4 ldg_stream(const void* p) {
  const u32x4 v = __builtin_nontemporal_load((gl_u32x4*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

struct GPhase {
  const char* w0;          // QKV: q, k, v matrices; GU: gate, up; else w0
  const char* w1;
  const char* w2;
  const uint16_t* s0;      // int8 per-output-channel scales of w0..w2
  const uint16_t* s1;
  const uint16_t* s2;
  int K;                   // input length
  int nvw;                 // 16-byte vectors in one wave's K-slice
  int u0, u1;              // this workgroup's units
  int nu;                  // units of the whole phase
};

template <int WFMT>
constexpr int epv() { return WFMT == AIO_WFMT_BF16 ? 8 : 16; }

// Units of a matrix phase: QKV unit u = rotation pairs 2u, 2u+1 (rows lo
// and hi of each); GU unit = row n of gate and of up; else one row.
template <int KIND>
AIO_DEV int n_units(const MegaArgs& a) {
  if (KIND == K_QKV) return (a.H + 2 * a.Hkv) * a.hd / 4;
  if (KIND == K_O || KIND == K_DOWN) return a.d;
  if (KIND == K_GU) return a.F;
  return a.V;
}

template <int WFMT, int KIND>
AIO_DEV GPhase make_phase(const MegaArgs& a, int layer) {
  GPhase P;
  const CMegaLayer* L = layer_at(a, layer < a.L ? layer : 0);
  P.w1 = P.w2 = nullptr;
  P.s1 = P.s2 = nullptr;
  if (KIND == K_QKV) {
    P.w0 = (const char*)L->w[0]; P.s0 = L->s[0];
    P.w1 = (const char*)L->w[1]; P.s1 = L->s[1];
    P.w2 = (const char*)L->w[2]; P.s2 = L->s[2];
    P.K = a.d;
  } else if (KIND == K_O) {
    P.w0 = (const char*)L->w[3]; P.s0 = L->s[3]; P.K = a.H * a.hd;
  } else if (KIND == K_GU) {
    P.w0 = (const char*)L->w[4]; P.s0 = L->s[4];
    P.w1 = (const char*)L->w[5]; P.s1 = L->s[5];
    P.K = a.d;
  } else if (KIND == K_DOWN) {
    P.w0 = (const char*)L->w[6]; P.s0 = L->s[6]; P.K = a.F;
  } else {
    P.w0 = (const char*)a.lm_head; P.s0 = a.s_lm; P.K = a.d;
  }
  P.nvw = P.K / (kW * epv<WFMT>());
  const int nu = n_units<KIND>(a);
  P.nu = nu;
  const int b = blockIdx.x, nbk = gridDim.x;
  P.u0 = (int)((long long)b * nu / nbk);
  P.u1 = (int)((long long)(b + 1) * nu / nbk);
  return P;
}

// One of three pointers, blended arithmetically: written as a select among
// fields of a struct the compiler builds a lookup table in scratch memory,
// and the scratch load then waits behind every weight load in flight.
template <class T>
AIO_DEV T* pick3(int i, T* p0, T* p1, T* p2) {
  const uint64_t b0 = (uint64_t)p0;
  const uint64_t d1 = (uint64_t)p1 - b0, d2 = (uint64_t)p2 - b0;
  return (T*)(b0 + (uint64_t)(i == 1) * d1 + (uint64_t)(i == 2) * d2);
}

// Row r of unit u as (matrix base, row index in it, scale array).
template <int WFMT, int KIND, int HD>
AIO_DEV const char* row_base(const MegaArgs& a, const GPhase& P, int u, int r) {
  constexpr size_t wb = WFMT == AIO_WFMT_BF16 ? 2 : 1;
  int mat = 0, row = u;
  if (KIND == K_QKV) {
    constexpr int half = HD / 2;
    const int p = 2 * u + (r & 1);
    int v = (p / half) * HD + (p % half) + (r >> 1) * half;  // virtual row
    const int qrows = a.H * a.hd, krows = a.Hkv * a.hd;
    if (v >= qrows + krows) { mat = 2; v -= qrows + krows; }
    else if (v >= qrows) { mat = 1; v -= qrows; }
    row = v;
  } else if (KIND == K_GU) {
    mat = r;
  }
  return pick3(mat, P.w0, P.w1, P.w2) + (size_t)row * (size_t)P.K * wb;
}

// The row base is the same for every lane of a wave; say so, so that the
// address arithmetic runs on the scalar unit.
AIO_DEV const char* wave_uniform(const char* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const char*)(((uint64_t)hi << 32) | lo);
}

// This thread's position.  Each phase takes a fresh copy that the compiler
// cannot see through, so values derived from it (per-lane offsets, shuffle
// addresses) are recomputed in the phase that uses them instead of being
// hoisted out of the layer loop and kept live -- and spilled -- across the
// whole kernel.
struct Thr {
  int tid, lane, wave;
};
AIO_DEV Thr thr() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return Thr{t, t & (AIO_WAVE - 1), t / AIO_WAVE};
}

// Whether load slot (unit u, vector vi) of a batch carries data.
AIO_DEV bool slot_ok(const GPhase& P, int u, int vi) { return u < P.u1 && vi < P.nvw; }

// Issue one batch.  Every slot is loaded unconditionally (an empty slot reads
// the first vector of a row the workgroup streams anyway, a cache hit) and
// masked when consumed: loads under branches would leave the compiler unable
// to count the loads in flight, and it would then wait for all of them --
// both buffers -- before every batch.
template <int WFMT, int KIND, int VPL, int HD>
AIO_DEV void issue(const MegaArgs& a, const GPhase& P, int batch, uint4 (&buf)[kNLD], const Thr& T) {
  constexpr int RPU = rpu_of<KIND>();
  constexpr int UB = kNLD / (RPU * VPL);
  const int lane = T.lane, wave = T.wave;
  const int ulast = P.nu - 1;
#pragma unroll
  for (int j = 0; j < UB * RPU * VPL; ++j) {
    const int ul = j / (RPU * VPL), r = (j / VPL) % RPU, v = j % VPL;
    const int u = P.u0 + batch * UB + ul;
    const int vi = v * AIO_WAVE + lane;
    const bool ok = slot_ok(P, u, vi);
    const char* rb = wave_uniform(row_base<WFMT, KIND, HD>(a, P, u < ulast ? u : ulast, r));
    const uint4* p = (const uint4*)rb + (size_t)wave * P.nvw + (ok ? vi : 0);
    buf[j] = ldg_stream(p);
  }
}

// Reduce kNLD per-lane values over the 64 lanes of a wave.  Each halving
// exchange (offsets 32, 16, 8) keeps half of the values, so lane l ends with
// value (l >> 3) & 7 summed over 8 lanes; three plain exchanges finish the
// sum (10 shuffles for 8 values instead of 48).
AIO_DEV float reduce_rows(float (&v)[kNLD], int lane) {
  static_assert(kNLD == 8, "reduce_rows assumes 8 values");
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bool up = lane & 32;
    const float send = up ? v[i] : v[i + 4], keep = up ? v[i + 4] : v[i];
    v[i] = keep + __shfl_xor(send, 32, AIO_WAVE);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const bool up = lane & 16;
    const float send = up ? v[i] : v[i + 2], keep = up ? v[i + 2] : v[i];
    v[i] = keep + __shfl_xor(send, 16, AIO_WAVE);
  }
  {
    const bool up = lane & 8;
    const float send = up ? v[0] : v[1], keep = up ? v[1] : v[0];
    v[0] = keep + __shfl_xor(send, 8, AIO_WAVE);
  }
  float s = v[0];
  s += __shfl_xor(s, 4, AIO_WAVE);
  s += __shfl_xor(s, 2, AIO_WAVE);
  s += __shfl_xor(s, 1, AIO_WAVE);
  return s;
}

// Multiply-accumulate one batch and leave each wave's row partials in LDS
// red[(local unit * RPU + r) * kW + wave].  Slots are not masked here: a
// lane past the end of its K-slice holds h = 0 (load_input) and reads a
// vector of the same row, so it adds an exact zero for finite weights; a
// unit past the workgroup's range is dropped at the LDS write.
template <int WFMT, int KIND, int VPL>
AIO_DEV void compute(const GPhase& P, int batch, const uint4 (&buf)[kNLD],
                     const float (&h)[VPL][epv<WFMT>()], float* red, const Thr& T) {
  constexpr int RPU = rpu_of<KIND>();
  constexpr int UB = kNLD / (RPU * VPL);
  const int lane = T.lane, wave = T.wave;
  float acc[kNLD];
#pragma unroll
  for (int i = 0; i < kNLD; ++i) acc[i] = 0.f;
#pragma unroll
  for (int j = 0; j < UB * RPU * VPL; ++j) {
    const int ul = j / (RPU * VPL), r = (j / VPL) % RPU, v = j % VPL;
    float& t = acc[ul * RPU + r];
    const uint4 w = buf[j];
    if constexpr (WFMT == AIO_WFMT_BF16) {
      t = dot8_bf16(w, make_float4(h[v][0], h[v][1], h[v][2], h[v][3]),
                    make_float4(h[v][4], h[v][5], h[v][6], h[v][7]), t);
    } else {
      t = dot4_i8(w.x, make_float4(h[v][0], h[v][1], h[v][2], h[v][3]), t);
      t = dot4_i8(w.y, make_float4(h[v][4], h[v][5], h[v][6], h[v][7]), t);
      t = dot4_i8(w.z, make_float4(h[v][8], h[v][9], h[v][10], h[v][11]), t);
      t = dot4_i8(w.w, make_float4(h[v][12], h[v][13], h[v][14], h[v][15]), t);
    }
  }
  const float s = reduce_rows(acc, lane);
  const int idx = (lane >> 3) & 7;
  if ((lane & 7) == 0 && idx < UB * RPU) {
    const int ul = idx / RPU, r = idx % RPU;
    const int lu = batch * UB + ul;
    if (P.u0 + lu < P.u1) red[(lu * RPU + r) * kW + wave] = s;
  }
}

// This lane's slice of the phase input, normalised when the phase starts
// with an RMSNorm.  The slice of wave w, vector v is elements
// [(w * nvw + v * 64 + lane) * EPV, +EPV).
template <int WFMT, int KIND, int VPL>
AIO_DEV void load_input(const MegaArgs& a, const GPhase& P, int layer, int token,
                        float (&h)[VPL][epv<WFMT>()], float* red8, const Thr& T) {
  constexpr int E = epv<WFMT>();
  const int lane = T.lane, wave = T.wave;
  const float* src = KIND == K_O ? a.o : (KIND == K_DOWN ? a.m : a.x);
  const bool emb = KIND == K_QKV && layer == 0;
  float ss = 0.f;
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    const int vi = v * AIO_WAVE + lane;
    const int e0 = (wave * P.nvw + vi) * E;
#pragma unroll
    for (int i = 0; i < E; ++i) h[v][i] = 0.f;
    if (vi < P.nvw) {
      if (emb) {
        const uint16_t* er = a.embed + (size_t)token * a.d + e0;
#pragma unroll
        for (int i = 0; i < E; ++i) h[v][i] = bf16_to_f32(er[i]);
        if (blockIdx.x == 0) {
#pragma unroll
          for (int i = 0; i < E; ++i) stf_dev(a.x + e0 + i, h[v][i]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < E; ++i) h[v][i] = ldf_dev(src + e0 + i);
      }
#pragma unroll
      for (int i = 0; i < E; ++i) ss = fmaf(h[v][i], h[v][i], ss);
    }
  }
  if (KIND == K_QKV || KIND == K_GU || KIND == K_LM) {
    ss = wave_sum(ss);
    if (lane == 0) red8[wave] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kW; ++w) tot += red8[w];
    __syncthreads();  // red8 is reused by the next phase
    const float inv = rsqrtf(tot / (float)P.K + a.eps);
    const CMegaLayer* L = layer_at(a, layer < a.L ? layer : 0);
    const uint16_t* g = KIND == K_QKV ? L->attn_norm : (KIND == K_GU ? L->ffn_norm : a.final_norm);
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const int vi = v * AIO_WAVE + lane;
      if (vi < P.nvw) {
        const int e0 = (wave * P.nvw + vi) * E;
#pragma unroll
        for (int i = 0; i < E; ++i) h[v][i] = h[v][i] * inv * bf16_to_f32(g[e0 + i]);
      }
    }
  }
}

// (value, index) order of the argmax: NaN first, then larger, then lower index.
AIO_DEV bool am_better(float v, int i, float bv, int bi) {
  const bool n = v != v, bn = bv != bv;
  if (n != bn) return n;
  if (!n && v != bv) return v > bv;
  return i < bi;
}

AIO_DEV void block_argmax(float& bv, int& bi, float* sv, int* si) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(bv, off, AIO_WAVE);
    const int oi = __shfl_xor(bi, off, AIO_WAVE);
    if (am_better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
  }
  const int wave = threadIdx.x / AIO_WAVE;
  if ((threadIdx.x & (AIO_WAVE - 1)) == 0) { sv[wave] = bv; si[wave] = bi; }
  __syncthreads();
  bv = sv[0];
  bi = si[0];
  for (int w = 1; w < kW; ++w)
    if (am_better(sv[w], si[w], bv, bi)) { bv = sv[w]; bi = si[w]; }
  __syncthreads();
}

struct Smem {
  float red8[kW];
  float sv[kW];
  int si[kW];
  unsigned flag;
};

// Epilogue of a matrix phase: sum the kW wave partials of each row, then the
// phase-specific output.
template <int WFMT, int KIND>
AIO_DEV void epilogue(const MegaArgs& a, const GPhase& P, int layer, int pos, const float* red,
                      Smem& sm, float xpre, const Thr& T) {
  constexpr int RPU = rpu_of<KIND>();
  const int nu = P.u1 - P.u0;
  const int tid = T.tid;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int t = tid; t < nu; t += kT) {
    float y[RPU];
#pragma unroll
    for (int r = 0; r < RPU; ++r) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kW; ++w) s += red[(t * RPU + r) * kW + w];
      y[r] = s;
    }
    const int u = P.u0 + t;
    if constexpr (KIND == K_QKV) {
      const int half = a.hd / 2, qrows = a.H * a.hd, krows = a.Hkv * a.hd;
      const int p = 2 * u, head = p / half, i = p % half;  // pairs p, p+1 -> dims i, i+1
      const int vlo = head * a.hd + i;                        // virtual row of dim i
      int sec = 0, rlo = vlo;
      if (vlo >= qrows + krows) { sec = 2; rlo -= qrows + krows; }
      else if (vlo >= qrows) { sec = 1; rlo -= qrows; }
      // y[0] = dim i, y[1] = dim i+1, y[2] = dim i+half, y[3] = dim i+1+half
      if constexpr (WFMT == AIO_WFMT_INT8) {
        const uint16_t* sc = pick3(sec, P.s0, P.s1, P.s2);
        y[0] *= fp16_to_f32(sc[rlo]);
        y[1] *= fp16_to_f32(sc[rlo + 1]);
        y[2] *= fp16_to_f32(sc[rlo + half]);
        y[3] *= fp16_to_f32(sc[rlo + 1 + half]);
      }
      if (sec < 2) {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const float2 cs = a.rope[(size_t)pos * half + i + k];
          const float lo = y[k], hi = y[k + 2];
          y[k] = lo * cs.x - hi * cs.y;
          y[k + 2] = hi * cs.x + lo * cs.y;
        }
      }
      if (sec == 0) {
        stf_dev(a.q + rlo, y[0]);
        stf_dev(a.q + rlo + 1, y[1]);
        stf_dev(a.q + rlo + half, y[2]);
        stf_dev(a.q + rlo + half + 1, y[3]);
      } else {
        const int g = rlo / a.hd, ii = rlo % a.hd;
        const CMegaLayer* L = layer_at(a, layer);
        uint16_t* c = (sec == 1 ? L->kc : L->vc) + ((size_t)g * a.max_ctx + pos) * a.hd;
        st_dev((unsigned*)(c + ii), (unsigned)f32_to_bf16(y[0]) | ((unsigned)f32_to_bf16(y[1]) << 16));
        st_dev((unsigned*)(c + ii + half),
               (unsigned)f32_to_bf16(y[2]) | ((unsigned)f32_to_bf16(y[3]) << 16));
      }
    } else if constexpr (KIND == K_GU) {
      float g = y[0], up = y[1];
      if constexpr (WFMT == AIO_WFMT_INT8) {
        g *= fp16_to_f32(P.s0[u]);
        up *= fp16_to_f32(P.s1[u]);
      }
      stf_dev(a.m + u, g / (1.f + expf(-g)) * up);
    } else {
      float yy = y[0];
      if constexpr (WFMT == AIO_WFMT_INT8) yy *= fp16_to_f32(P.s0[u]);
      if constexpr (KIND == K_LM) {
        a.logits[u] = yy;
        if (am_better(yy, u, bv, bi)) { bv = yy; bi = u; }
      } else {
        const float xo = t == tid ? xpre : ldf_dev(a.x + u);
        stf_dev(a.x + u, xo + yy);
      }
    }
  }
  if constexpr (KIND == K_LM) {
    // fused greedy argmax: workgroup result, then the last workgroup reduces
    block_argmax(bv, bi, sm.sv, sm.si);
    if (tid == 0) {
      stf_dev((float*)(a.sync + kSyncAmax + 2 * blockIdx.x), bv);
      st_dev(a.sync + kSyncAmax + 2 * blockIdx.x + 1, (unsigned)bi);
    }
    wg_publish();
    if (tid == 0) sm.flag = add_dev(a.sync + kSyncAmaxCount, 1u) == gridDim.x - 1;
    __syncthreads();
    if (sm.flag) {
      float gv = -INFINITY;
      int gi = 0x7fffffff;
      for (int b = tid; b < (int)gridDim.x; b += kT) {
        const float v = ldf_dev((const float*)(a.sync + kSyncAmax + 2 * b));
        const int i = (int)ld_dev(a.sync + kSyncAmax + 2 * b + 1);
        if (am_better(v, i, gv, gi)) { gv = v; gi = i; }
      }
      block_argmax(gv, gi, sm.sv, sm.si);
      if (tid == 0) {
        if (gi == 0x7fffffff) gi = 0;
        aio_state* st = a.st;
        if (a.tokens_out) a.tokens_out[st->step] = gi;
        st->token[0] = gi;
        st->pos = pos + 1;
        st->step += 1;
        st_dev(a.sync + kSyncAmaxCount, 0u);
      }
    }
  }
}

// The register buffers of a wave: kNBUF batches of kNLD 16-byte loads.
struct Bufs {
  uint4 b[kNBUF][kNLD];
};

// One matrix phase.  On entry buffer j holds (in flight) batch j of this
// phase; each buffer is refilled with the phase's batch kNBUF further on as
// soon as it is consumed.
template <int WFMT, int HD, int KIND, int VPL>
AIO_DEV void gemv_phase(const MegaArgs& a, const GPhase& P, int layer, int pos, int token,
                        Bufs& W, float* red, Smem& sm, unsigned kb) {
  constexpr int RPU = rpu_of<KIND>();
  constexpr int UB = kNLD / (RPU * VPL);
  const int nb = (P.u1 - P.u0 + UB - 1) / UB;
  const Thr T = thr();
  // residual rows this workgroup will update, fetched now to hide the trip
  float xpre = 0.f;
  if (KIND == K_O || KIND == K_DOWN) {
    if (T.tid < P.u1 - P.u0) xpre = ldf_dev(a.x + P.u0 + T.tid);
  }
  float h[VPL][epv<WFMT>()];
  load_input<WFMT, KIND, VPL>(a, P, layer, token, h, sm.red8, T);
  if (a.detail && T.tid == 0) a.detail[((size_t)kb * gridDim.x + blockIdx.x) * 2] = wall_clock64();
  // The input loads above were issued after this phase's first batches,
  // so waiting for them has waited for everything; say so explicitly
  // (vmcnt(0)), so that the loop below starts from a state in which only
  // its own loads are in flight and waits only for the buffer it consumes.
  __builtin_amdgcn_s_waitcnt(kVmcnt0);
  // Branch-free body: a batch past the end is computed fully masked and its
  // refill is a masked dummy (cache-hit) load, so the compiler sees the same
  // loads in flight behind each buffer on every path.
  int b = 0;
  for (; b + kNBUF < nb; b += kNBUF) {
#pragma unroll
    for (int j = 0; j < kNBUF; ++j) {
      compute<WFMT, KIND, VPL>(P, b + j, W.b[j], h, red, T);
      issue<WFMT, KIND, VPL, HD>(a, P, b + j + kNBUF, W.b[j], T);
    }
  }
  // last round: no refills, so that nothing is in flight when the phase's
  // outputs are published (the release waits for every outstanding load)
#pragma unroll
  for (int j = 0; j < kNBUF; ++j) compute<WFMT, KIND, VPL>(P, b + j, W.b[j], h, red, T);
  __syncthreads();
  if (a.detail && T.tid == 0) a.detail[((size_t)kb * gridDim.x + blockIdx.x) * 2 + 1] = wall_clock64();
  epilogue<WFMT, KIND>(a, P, layer, pos, red, sm, xpre, T);
}

// Issue the first kNBUF batches of a matrix phase into the buffers.
template <int WFMT, int HD, int KIND, int VPL>
AIO_DEV void prefetch(const MegaArgs& a, int layer, Bufs& W) {
  const GPhase N = make_phase<WFMT, KIND>(a, layer);
  const Thr T = thr();
#pragma unroll
  for (int j = 0; j < kNBUF; ++j) issue<WFMT, KIND, VPL, HD>(a, N, j, W.b[j], T);
}

// ---------------------------------------------------------------- attention

// 16-byte load through a global-address-space pointer (the KV base comes
// from a table in memory, so the compiler cannot infer the address space).
AIO_DEV uint4 ldg16(const uint16_t* p) {
  const u32x4 v = *(gl_u32x4*)p;
  return make_uint4(v.x, v.y, v.z, v.w);
}

// One DPP lane move of a float (a VALU operation: no LDS round trip).
template <int CTRL>
AIO_DEV float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over aligned groups of 8 or 16 lanes; every lane of a group receives
// the same total.  Each step adds a lane's value to that of a partner in the
// other half of its current group: lane ^ 1, lane ^ 2 (quad permutations),
// then the mirror lane of the other quad (row_half_mirror) and, for 16, of
// the other half row (row_mirror).
template <int WIDTH>
AIO_DEV float group_sum_dpp(float v) {
  static_assert(WIDTH == 8 || WIDTH == 16, "DPP sums cover 8 or 16 lanes");
  v += dpp_mov<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_mov<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_mov<0x141>(v);  // row_half_mirror
  if (WIDTH == 16) v += dpp_mov<0x140>(v);  // row_mirror
  return v;
}

// Online-softmax update of one group with one key row (already loaded).  A
// key past the group's range (valid false) leaves the state unchanged; the
// masking is done with selects so that the loop has no divergent branches.
template <int HD, int G>
AIO_DEV void attend_key(const uint4 kk, const uint4 vv, bool valid, const float (&q)[G][8],
                        float (&o)[G][8], float (&m)[G], float (&l)[G]) {
  constexpr int LPK = HD / 8;
  const float vf[8] = {bf16_lo(vv.x), bf16_hi(vv.x), bf16_lo(vv.y), bf16_hi(vv.y),
                       bf16_lo(vv.z), bf16_hi(vv.z), bf16_lo(vv.w), bf16_hi(vv.w)};
#pragma unroll
  for (int gg = 0; gg < G; ++gg) {
    float sc = dot8_bf16(kk, make_float4(q[gg][0], q[gg][1], q[gg][2], q[gg][3]),
                         make_float4(q[gg][4], q[gg][5], q[gg][6], q[gg][7]), 0.f);
    sc = group_sum_dpp<LPK>(sc);
    const float mn = valid ? fmaxf(m[gg], sc) : m[gg];
    const float c = valid ? exp2f(m[gg] - mn) : 1.f;
    const float p = valid ? exp2f(sc - mn) : 0.f;
    l[gg] = l[gg] * c + p;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[gg][i] = fmaf(p, vf[i], o[gg][i] * c);
    m[gg] = mn;
  }
}

// Four keys of a group: their K and V rows.
struct KV4 {
  uint4 k[4], v[4];
};

// Workgroup unit = (kv head g, split s) of the keys [0, pos].  HD/8 lanes
// hold one key row; each group of lanes runs an online softmax over its keys,
// the groups combine in LDS, and the split's (max, sum, unnormalised output)
// goes out as a partial.  The last split of a kv head to finish merges the S
// partials into o.  Keys stream through two sets of registers in turn (four
// keys each): one set is in flight while the other is consumed, with no
// copies between them, so the loads of the next keys are never waited for
// early.  The first keys are requested before q, the group combine is split
// four ways, and the merge loads all partials before reducing them.
template <int HD, int G>
AIO_DEV void attn_phase(const MegaArgs& a, int layer, int pos, float* lds, Smem& sm) {
  constexpr int LPK = HD / 8, NGR = kT / LPK;
  constexpr int NOUT = G * HD;            // outputs of a unit
  constexpr int R = kT / NOUT > 0 ? kT / NOUT : 1;  // threads per output
  static_assert(NGR % R == 0, "groups must split evenly");
  float* sm_m = lds;                      // [NGR][G]
  float* sm_l = lds + NGR * G;            // [NGR][G]
  float* sm_o = lds + 2 * NGR * G;        // [NGR][G][HD]
  float* sm_r = sm_o + NGR * G * HD;      // [R][NOUT] partial sums, then merge scratch
  const int tid = thr().tid, gi = tid / LPK, li = tid % LPK;
  const CMegaLayer* L = layer_at(a, layer);
  const int S = a.S, units = a.Hkv * S;
  const int n_keys = pos + 1;
  const int chunk = (n_keys + S - 1) / S;
  for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
    const int g = unit / S, s = unit % S;
    const int j0 = s * chunk, j1 = min(n_keys, j0 + chunk);
    // keys of this group: j = j0 + gi + t * NGR for t < nk.  Loads are
    // unconditional: key t >= nk reads the last valid key of the split (a
    // cache hit) and is masked when consumed.
    const int nk = j1 - j0 > gi ? (j1 - j0 - gi + NGR - 1) / NGR : 0;
    const int jlast = j1 > j0 ? j1 - 1 : (n_keys - 1);  // a key row of this kv head
    const uint16_t* kb = L->kc + (size_t)g * a.max_ctx * HD + li * 8;
    const uint16_t* vb = L->vc + (size_t)g * a.max_ctx * HD + li * 8;
    auto load4 = [&](KV4& d, int t0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + i;
        const size_t off = (size_t)(t < nk ? j0 + gi + t * NGR : jlast) * HD;
        d.k[i] = ldg16(kb + off);
        d.v[i] = ldg16(vb + off);
      }
    };
    KV4 X, Y;
    load4(X, 0);
    float q[G][8], o[G][8], m[G], l[G];
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
      const float* qp = a.q + (size_t)(g * G + gg) * HD + li * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) q[gg][i] = ldf_dev(qp + i);
    }
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        q[gg][i] *= a.scale_log2;
        o[gg][i] = 0.f;
      }
      m[gg] = -INFINITY;
      l[gg] = 0.f;
    }
    // The scheduling barriers keep each set's loads where they are written:
    // hoisted together, both sets would be waited for at the top of the loop.
    for (int t = 0; t < nk; t += 8) {
      load4(Y, t + 4);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 4; ++i) attend_key<HD, G>(X.k[i], X.v[i], t + i < nk, q, o, m, l);
      __builtin_amdgcn_sched_barrier(0);
      load4(X, t + 8);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 4; ++i) attend_key<HD, G>(Y.k[i], Y.v[i], t + 4 + i < nk, q, o, m, l);
      __builtin_amdgcn_sched_barrier(0);
    }
    // combine the NGR groups: R threads per output, NGR / R groups each
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
      if (li == 0) {
        sm_m[gi * G + gg] = m[gg];
        sm_l[gi * G + gg] = l[gg];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) sm_o[(gi * G + gg) * HD + li * 8 + i] = o[gg][i];
    }
    __syncthreads();
    float* part = a.part + (size_t)g * G * S * (HD + 2);
    {
      const int c = tid % NOUT, r = tid / NOUT;  // output c, part r
      const int gg = c / HD, dim = c % HD;
      float M = -INFINITY;
      for (int k = 0; k < NGR; ++k) M = fmaxf(M, sm_m[k * G + gg]);
      float Ls = 0.f, Os = 0.f;
      if (r < R && M != -INFINITY) {
        for (int k = r * (NGR / R); k < (r + 1) * (NGR / R); ++k) {
          const float mk = sm_m[k * G + gg];
          const float w = mk == -INFINITY ? 0.f : exp2f(mk - M);
          Ls = fmaf(w, sm_l[k * G + gg], Ls);
          Os = fmaf(w, sm_o[(k * G + gg) * HD + dim], Os);
        }
      }
      __syncthreads();
      if (r < R) {
        sm_r[r * NOUT + c] = Os;
        if (dim == 0) sm_r[R * NOUT + r * G + gg] = Ls;
      }
      __syncthreads();
      if (tid < NOUT) {
        float Ot = 0.f, Lt = 0.f;
#pragma unroll
        for (int k = 0; k < R; ++k) {
          Ot += sm_r[k * NOUT + c];
          Lt += sm_r[R * NOUT + k * G + gg];
        }
        float* slot = part + ((size_t)gg * S + s) * (HD + 2);
        stf_dev(slot + dim, Ot);
        if (dim == 0) {
          stf_dev(slot + HD, M);
          stf_dev(slot + HD + 1, Lt);
        }
      }
    }
    wg_publish();
    if (tid == 0) sm.flag = add_dev(a.sync + kSyncAttn + g, 1u) == (unsigned)(S - 1);
    __syncthreads();
    if (sm.flag) {
      // last split of kv head g: merge the S partials of its G query heads.
      // 1) all (max, sum) pairs at once
      float* mm = sm_r;             // [G][S]
      float* ww = sm_r + G * S;     // [G][S] weights, then [G] totals
      for (int e = tid; e < G * S; e += kT) {
        const int gg = e / S, k = e % S;
        const float* sl = part + ((size_t)gg * S + k) * (HD + 2);
        mm[e] = ldf_dev(sl + HD);
        ww[e] = ldf_dev(sl + HD + 1);
      }
      __syncthreads();
      if (tid < G) {
        float M = -INFINITY;
        for (int k = 0; k < S; ++k) M = fmaxf(M, mm[tid * S + k]);
        float Lt = 0.f;
        for (int k = 0; k < S; ++k) {
          const float w = mm[tid * S + k] == -INFINITY ? 0.f : exp2f(mm[tid * S + k] - M);
          Lt = fmaf(w, ww[tid * S + k], Lt);
          mm[tid * S + k] = w;  // reuse as the weight of split k
        }
        ww[G * S + tid] = Lt;
      }
      __syncthreads();
      // 2) R threads per output, each over every R-th split, loads first
      const int c = tid % NOUT, r = tid / NOUT;
      const int gg = c / HD, dim = c % HD;
      float acc = 0.f;
      if (r < R) {
        const float* base = part + (size_t)gg * S * (HD + 2) + dim;
        int k = r;
        for (; k + 3 * R < S; k += 4 * R) {
          const float x0 = ldf_dev(base + (size_t)k * (HD + 2));
          const float x1 = ldf_dev(base + (size_t)(k + R) * (HD + 2));
          const float x2 = ldf_dev(base + (size_t)(k + 2 * R) * (HD + 2));
          const float x3 = ldf_dev(base + (size_t)(k + 3 * R) * (HD + 2));
          acc = fmaf(mm[gg * S + k], x0, acc);
          acc = fmaf(mm[gg * S + k + R], x1, acc);
          acc = fmaf(mm[gg * S + k + 2 * R], x2, acc);
          acc = fmaf(mm[gg * S + k + 3 * R], x3, acc);
        }
        for (; k < S; k += R) acc = fmaf(mm[gg * S + k], ldf_dev(base + (size_t)k * (HD + 2)), acc);
      }
      float* red = sm_o;  // [R][NOUT]; the group outputs are no longer needed
      if (r < R) red[r * NOUT + c] = acc;
      __syncthreads();
      if (tid < NOUT) {
        float ot = 0.f;
#pragma unroll
        for (int k = 0; k < R; ++k) ot += red[k * NOUT + c];
        stf_dev(a.o + (size_t)(g * G + gg) * HD + dim, ot / ww[G * S + gg]);
      }
      if (tid == 0) st_dev(a.sync + kSyncAttn + g, 0u);
    }
    __syncthreads();
  }
}

template <int WFMT, int HD, int G, int VQ, int VD>
__global__ __launch_bounds__(kT, 1) void k_step(MegaArgs a) {
  extern __shared__ float lds[];
  __shared__ Smem sm;
  const int pos = a.st->pos, token = a.st->token[0];
  // every thread reads the epoch base before the first barrier; workgroup 0
  // advances it for the next launch once that barrier has passed
  const unsigned ep0 = ld_dev(a.sync + kSyncEpoch);
  unsigned k = 0;
  Bufs W;
  prefetch<WFMT, HD, K_QKV, VQ>(a, 0, W);
  auto none = [] {};
  for (int l = 0; l < a.L; ++l) {
    {
      const GPhase P = make_phase<WFMT, K_QKV>(a, l);
      gemv_phase<WFMT, HD, K_QKV, VQ>(a, P, l, pos, token, W, lds, sm, k + 1);
    }
    grid_sync(a, ep0, ++k, none);
    if (l == 0 && blockIdx.x == 0 && threadIdx.x == 0)
      st_dev(a.sync + kSyncEpoch, ep0 + 5u * (unsigned)a.L);
    attn_phase<HD, G>(a, l, pos, lds, sm);
    grid_sync(a, ep0, ++k, [&] { prefetch<WFMT, HD, K_O, VQ>(a, l, W); });
    {
      const GPhase P = make_phase<WFMT, K_O>(a, l);
      gemv_phase<WFMT, HD, K_O, VQ>(a, P, l, pos, token, W, lds, sm, k + 1);
    }
    grid_sync(a, ep0, ++k, [&] { prefetch<WFMT, HD, K_GU, VQ>(a, l, W); });
    {
      const GPhase P = make_phase<WFMT, K_GU>(a, l);
      gemv_phase<WFMT, HD, K_GU, VQ>(a, P, l, pos, token, W, lds, sm, k + 1);
    }
    grid_sync(a, ep0, ++k, [&] { prefetch<WFMT, HD, K_DOWN, VD>(a, l, W); });
    {
      const GPhase P = make_phase<WFMT, K_DOWN>(a, l);
      gemv_phase<WFMT, HD, K_DOWN, VD>(a, P, l, pos, token, W, lds, sm, k + 1);
    }
    if (l + 1 < a.L)
      grid_sync(a, ep0, ++k, [&] { prefetch<WFMT, HD, K_QKV, VQ>(a, l + 1, W); });
    else
      grid_sync(a, ep0, ++k, [&] { prefetch<WFMT, HD, K_LM, VQ>(a, l + 1, W); });
  }
  const GPhase P = make_phase<WFMT, K_LM>(a, a.L);
  gemv_phase<WFMT, HD, K_LM, VQ>(a, P, a.L, pos, token, W, lds, sm, 0u);
}

// The grid is one workgroup per CU and a CU holds at most one (registers
// and LDS), so all workgroups are resident together.  The cooperative
// launch states that requirement to the runtime, which refuses the launch
// if it cannot be met; a plain launch of the same grid relies on the GPU
// running nothing else (every barrier wait is bounded either way).
template <int WFMT, int HD, int G, int VQ, int VD>
hipError_t launch_t(const MegaArgs& a, int blocks, size_t lds, hipStream_t s, bool coop) {
  void* args[] = {(void*)&a};
  const void* fn = (const void*)k_step<WFMT, HD, G, VQ, VD>;
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  if (coop) return hipLaunchCooperativeKernel(fn, dim3(blocks), dim3(kT), args, (unsigned)lds, s);
  return hipLaunchKernel(fn, dim3(blocks), dim3(kT), args, lds, s);
}

template <int WFMT, int HD, int G>
hipError_t launch_vd(const MegaArgs& a, int blocks, size_t lds, hipStream_t s, int vd, bool coop) {
  switch (vd) {
    case 1: return launch_t<WFMT, HD, G, 1, 1>(a, blocks, lds, s, coop);
    case 2: return launch_t<WFMT, HD, G, 1, 2>(a, blocks, lds, s, coop);
    case 3: return launch_t<WFMT, HD, G, 1, 3>(a, blocks, lds, s, coop);
    default: return hipErrorInvalidValue;
  }
}

template <int WFMT, int HD>
hipError_t launch_g(const MegaArgs& a, int blocks, size_t lds, hipStream_t s, int G, int vd,
                    bool coop) {
  switch (G) {
    case 1: return launch_vd<WFMT, HD, 1>(a, blocks, lds, s, vd, coop);
    case 2: return launch_vd<WFMT, HD, 2>(a, blocks, lds, s, vd, coop);
    case 4: return launch_vd<WFMT, HD, 4>(a, blocks, lds, s, vd, coop);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int aio_step_kernel_vpl(const aio_config& c, int K) {
  const int epv_ = c.wfmt == AIO_WFMT_BF16 ? 8 : 16;
  if (K % (kW * epv_)) return 0;
  const int nvw = K / (kW * epv_);
  return (nvw + AIO_WAVE - 1) / AIO_WAVE;
}

bool aio_step_kernel_supports(const aio_config& c) {
  const int G = c.n_heads / c.n_kv_heads;
  if (G != 1 && G != 2 && G != 4) return false;
  if (c.head_dim != 64 && c.head_dim != 128) return false;
  // the QKV, O, gate/up and LM-head inputs must fit one 16-byte vector per lane
  if (aio_step_kernel_vpl(c, c.d_model) != 1) return false;
  if (aio_step_kernel_vpl(c, c.n_heads * c.head_dim) != 1) return false;
  const int vd = aio_step_kernel_vpl(c, c.ffn_dim);
  if (vd < 1 || vd > 3) return false;
  if ((c.n_heads + 2 * c.n_kv_heads) * c.head_dim % 4) return false;
  return true;
}

size_t aio_step_kernel_lds(const aio_config& c, int blocks) {
  const int G = c.n_heads / c.n_kv_heads;
  const int ngr = kT / (c.head_dim / 8);
  const int nout = G * c.head_dim;
  const int r = kT / nout > 0 ? kT / nout : 1;
  const int S = AIO_STEP_MAX_BLOCKS / c.n_kv_heads > 0 ? AIO_STEP_MAX_BLOCKS / c.n_kv_heads : 1;
  // group state + [R][NOUT] partials (+ R * G sums) or the merge's 2 G S + G
  const size_t scratch = std::max((size_t)r * nout + (size_t)r * G, (size_t)2 * G * S + G);
  const size_t attn = ((size_t)ngr * G * (c.head_dim + 2) + scratch) * 4;
  auto red = [&](int units, int rpu) { return (size_t)((units + blocks - 1) / blocks) * rpu * kW * 4; };
  size_t gemv = red((c.n_heads + 2 * c.n_kv_heads) * c.head_dim / 4, 4);
  gemv = std::max(gemv, red(c.d_model, 1));
  gemv = std::max(gemv, red(c.ffn_dim, 2));
  gemv = std::max(gemv, red(c.vocab, 1));
  return std::max(attn, gemv);
}

hipError_t aio_launch_step_kernel(const aio_model& m, float* logits, int32_t* tokens_out,
                                  unsigned long long* trace, unsigned long long* bar_arrive,
                                  unsigned long long* bar_leave) {
  const aio_config& c = m.cfg;
  MegaArgs a{};
  a.layers = m.mega_layers;
  a.embed = (const uint16_t*)m.embed;
  a.final_norm = (const uint16_t*)m.final_norm;
  a.lm_head = m.lm_head;
  a.s_lm = (const uint16_t*)m.s_lm_head;
  a.rope = m.rope;
  a.st = m.state();
  a.x = m.at<float>(m.lay.x);
  a.q = m.at<float>(m.lay.q);
  a.o = m.at<float>(m.lay.o);
  a.m = m.at<float>(m.lay.m);
  a.part = m.at<float>(m.lay.mega_part);
  a.sync = m.at<unsigned>(m.lay.sync);
  a.logits = logits;
  a.tokens_out = tokens_out;
  a.trace = trace;
  a.bar_arrive = bar_arrive;
  a.bar_leave = bar_leave;
  a.detail = bar_leave ? bar_leave + (size_t)(5 * c.n_layers + 1) * m.mega_blocks : nullptr;
  a.L = c.n_layers;
  a.d = c.d_model;
  a.H = c.n_heads;
  a.Hkv = c.n_kv_heads;
  a.hd = c.head_dim;
  a.F = c.ffn_dim;
  a.V = c.vocab;
  a.max_ctx = c.max_ctx;
  a.S = m.lay.mega_splits;
  a.eps = c.rms_eps;
  a.scale_log2 = (float)(1.4426950408889634 / sqrt((double)c.head_dim));
  const int blocks = m.mega_blocks;
  const size_t lds = aio_step_kernel_lds(c, blocks);
  const int G = c.n_heads / c.n_kv_heads;
  const int vd = aio_step_kernel_vpl(c, c.ffn_dim);
  hipError_t e;
  if (c.wfmt == AIO_WFMT_INT8)
    e = c.head_dim == 128 ? launch_g<AIO_WFMT_INT8, 128>(a, blocks, lds, m.stream, G, vd, m.mega_coop)
                          : launch_g<AIO_WFMT_INT8, 64>(a, blocks, lds, m.stream, G, vd, m.mega_coop);
  else
    e = c.head_dim == 128 ? launch_g<AIO_WFMT_BF16, 128>(a, blocks, lds, m.stream, G, vd, m.mega_coop)
                          : launch_g<AIO_WFMT_BF16, 64>(a, blocks, lds, m.stream, G, vd, m.mega_coop);
  aio_prof_mark(m);
  return e;
}
