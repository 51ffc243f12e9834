// The whole decode step as one persistent, cooperatively launched kernel.
//
// Why: at batch 1 every token streams all weights once (the paper's
// Section 2.1 / Section 3.1 bandwidth argument), and a layer is a chain of
// five dependent matrix-vector products and an attention.  Launched as
// separate kernels, each link pays a dispatch ramp, a prologue and a tail
// (several microseconds each, ~190 links per 7B token).  Here one workgroup
// per CU (512 threads, 8 waves) walks all phases of all layers, and issues
// the first weight loads of each phase as soon as it has finished the one
// before, so HBM keeps streaming while the workgroup waits for its inputs.
//
// Phases per layer (phase index k = 5 l + 1 .. 5 l + 5):
//   QKV   RMSNorm(x) -> q, k, v rows -> RoPE; q stored, k/v appended (bf16)
//   ATTN  split-KV flash-decode per (kv head, split) over the cached keys;
//         the last split of a kv head also takes the new key, and then
//         merges the S partials of its head (log-sum-exp) into o
//   O     x' = x + W_o o
//   GU    RMSNorm(x') -> m = silu(W_gate h) * (W_up h)
//   DOWN  x = x' + W_down m
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
// Synchronisation without grid barriers: every value one workgroup produces
// for another carries its own readiness.  An fp32 value is stored with the
// 3-bit version (epoch base + phase index) mod 8 in its lowest mantissa bits
// (the value truncated to 20 mantissa bits: a relative change below 2^-20);
// the new K/V row goes out as bf16 in the high half of a word whose low bits
// hold the version.  A consumer loads its slice of a buffer and reloads each
// word whose version is not the one it expects.  A stale word holds the
// buffer's previous use, five phases earlier, whose version differs mod 8.
// A phase therefore starts one memory round trip after the words it needs
// are stored, instead of after a flag store, a gather, a release and a
// second load; and its first poll is issued right behind the phase's
// prefetched weights, so it usually returns together with them.
//
// Reuse of a buffer needs no barrier either: every phase waits for all the
// outputs of the phase before it (attention: every q row of its head, the
// merge: every split of its head, O: all of o), so a producer reaches its
// next write of a buffer, five phases on, only after every reader of the
// previous contents has consumed them.  A workgroup with no rows in a phase
// reads nothing in it.
//
// Coherence: the 8 XCDs have separate L2 caches that are not kept coherent
// with each other, so every value exchanged between workgroups is written
// with device-scope stores and read with device-scope loads, which bypass
// the non-coherent L2.  Weights, norm gains and older KV rows are read-only
// in the step and use ordinary loads.
//
// Every wait is a bounded spin: if a value never arrives the kernel sets an
// error word and runs to its end instead of hanging.
#include <math.h>

#include <algorithm>

#include "aio_internal.h"
#include "common.h"
#include "step_kernel.h"

namespace {

constexpr int kT = 512;          // threads per workgroup
constexpr int kW = kT / AIO_WAVE; // waves per workgroup
#ifndef AIO_STEP_NLD
#define AIO_STEP_NLD 8
#endif
constexpr int kNLD = AIO_STEP_NLD;  // 16-byte weight loads per lane per batch
// Batches in flight per wave (register buffers).  A deeper prefetch streams
// the loops a little faster but delays the input poll queued behind it
// (vector memory returns in order).
#ifndef AIO_STEP_NBUF
#define AIO_STEP_NBUF 2
#endif
constexpr int kNBUF = AIO_STEP_NBUF;
constexpr unsigned kSpinLimit = 1u << 17;  // ~0.1-0.2 s of polling

// s_waitcnt immediate for vmcnt(0) with expcnt and lgkmcnt left at their
// maximum (no wait): vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8].
constexpr int kVmcnt0 = 0x0F70;
// Cache-policy operand of a buffer load: device scope (sc1).
constexpr int kSC1 = 16;

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

// 16-byte device-scope load of words base[off .. off + 3].  `base` must be
// the same for the whole wave (it becomes a buffer descriptor).
AIO_DEV u32x4 ld16_dev(const unsigned* base, int off) {
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, 0x7ffffff0, 0x00020000);
  return __builtin_amdgcn_raw_buffer_load_b128(r, off * 4, 0, kSC1);
}

typedef __attribute__((address_space(1))) const u32x4 gl_u32x4;

// 16-byte ordinary load through a global-address-space pointer (weights,
// gains and K/V rows come from a table in memory, so the compiler cannot
// infer the address space).
AIO_DEV uint4 ldg16(const uint16_t* p) {
  const u32x4 v = *(gl_u32x4*)p;
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Wait until this thread's stores have completed, then for the whole
// workgroup; a counter raised after this is seen by other workgroups only
// after the data.  The wait is explicit because a workgroup-scope fence does
// not wait for global stores (the workgroup shares one CU).
AIO_DEV void wg_publish() {
  __builtin_amdgcn_s_waitcnt(kVmcnt0);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
}

// ----------------------------------------------------------------- versions

AIO_DEV unsigned ver_of(unsigned ep0, unsigned k) { return (ep0 + k) & 7u; }
AIO_DEV unsigned tagf(float v, unsigned ver) { return (__float_as_uint(v) & ~7u) | ver; }
AIO_DEV float untagf(unsigned w) { return __uint_as_float(w & ~7u); }
AIO_DEV void st_tag(unsigned* p, float v, unsigned ver) { st_dev(p, tagf(v, ver)); }
AIO_DEV bool tags_ok(const u32x4 v, unsigned ver) {
  return ((v.x & 7u) == ver) & ((v.y & 7u) == ver) & ((v.z & 7u) == ver) & ((v.w & 7u) == ver);
}

// One step of a bounded wait.  Once any wait has given up (the error word is
// set), every later wait stops at its next check, so a value that never
// arrives costs well under a second instead of hanging the device.
AIO_DEV bool spin_on(const MegaArgs& a, unsigned& spins) {
  __builtin_amdgcn_s_sleep(2);
  if ((++spins & 63u) == 0) {
    if (ld_dev(a.sync + kSyncErr) != 0u) return false;
    if (spins > kSpinLimit) {
      st_dev(a.sync + kSyncErr, 1u);
      return false;
    }
  }
  return true;
}

// Calls f(0) .. f(N - 1) with constant indices.  A plain unrolled loop is
// not unrolled by the compiler once it sits inside a wait loop, and the
// arrays it indexes then move to scratch memory.
template <int I, int N>
struct Unroll {
  template <class F>
  AIO_DEV static void run(F&& f) {
    f(I);
    Unroll<I + 1, N>::run(f);
  }
};
template <int N>
struct Unroll<N, N> {
  template <class F>
  AIO_DEV static void run(F&&) {}
};

// Wait until the loaded 16-byte words this thread needs carry version `ver`,
// reloading only the stale ones.  The first check sits outside the retry
// loop: there the compiler knows which loads were issued after the words
// (the next weight batch) and waits only for the words themselves.
template <int N>
AIO_DEV bool stale16(const bool (&need)[N], const u32x4 (&v)[N], unsigned ver) {
  bool stale = false;
  Unroll<0, N>::run([&](int i) __attribute__((always_inline)) {
    stale |= need[i] && !tags_ok(v[i], ver);
  });
  return stale;
}
template <int N>
AIO_DEV void await16(const MegaArgs& a, const unsigned* base, const int (&off)[N],
                     const bool (&need)[N], u32x4 (&v)[N], unsigned ver) {
  if (!stale16(need, v, ver)) return;
  unsigned spins = 0;
  do {
    if (!spin_on(a, spins)) break;
    Unroll<0, N>::run([&](int i) __attribute__((always_inline)) {
      if (need[i] && !tags_ok(v[i], ver)) v[i] = ld16_dev(base, off[i]);
    });
  } while (stale16(need, v, ver));
}

// The same for single words.
template <int N>
AIO_DEV bool stale4(const bool (&need)[N], const unsigned (&v)[N], unsigned ver) {
  bool stale = false;
  Unroll<0, N>::run([&](int i) __attribute__((always_inline)) {
    stale |= need[i] && (v[i] & 7u) != ver;
  });
  return stale;
}
template <int N>
AIO_DEV void await4(const MegaArgs& a, const unsigned* base, const int (&off)[N],
                    const bool (&need)[N], unsigned (&v)[N], unsigned ver) {
  if (!stale4(need, v, ver)) return;
  unsigned spins = 0;
  do {
    if (!spin_on(a, spins)) break;
    Unroll<0, N>::run([&](int i) __attribute__((always_inline)) {
      if (need[i] && (v[i] & 7u) != ver) v[i] = ld_dev(base + off[i]);
    });
  } while (stale4(need, v, ver));
}

// Optional timing records (profiling aids; null in normal runs).
AIO_DEV void stamp(unsigned long long* arr, unsigned k) {
  if (arr && threadIdx.x == 0) arr[(size_t)k * gridDim.x + blockIdx.x] = wall_clock64();
}
AIO_DEV void stamp_detail(const MegaArgs& a, unsigned k, int col) {
  if (a.detail && threadIdx.x == 0)
    a.detail[((size_t)k * gridDim.x + blockIdx.x) * 2 + col] = wall_clock64();
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

// Lanes that share one weight row in a load: the whole wave for bf16; a half
// wave for int8, whose two halves take two rows.  A wave's K-slice of 4096
// int8 inputs is 32 vectors of 16: spread over the wave it would leave half
// the lanes multiplying zeros (the int8 loops were bound by that waste),
// and 8-byte loads instead would double the load instructions per byte.
template <int WFMT>
constexpr int lpr() { return WFMT == AIO_WFMT_INT8 ? AIO_WAVE / 2 : AIO_WAVE; }

// The K-slice vector of a lane's load v.
template <int WFMT>
AIO_DEV int lane_vec(int v, int lane) {
  if constexpr (lpr<WFMT>() == AIO_WAVE) return v * AIO_WAVE + lane;
  else return v * lpr<WFMT>() + (lane & (lpr<WFMT>() - 1));
}

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
  if (KIND == K_GU && a.gu_bounds) {
    // calibrated split (aio_tune_step), read as wave-uniform scalars
    typedef __attribute__((address_space(4))) const int cint;
    P.u0 = ((cint*)a.gu_bounds)[b];
    P.u1 = ((cint*)a.gu_bounds)[b + 1];
  } else {
    P.u0 = (int)((long long)b * nu / nbk);
    P.u1 = (int)((long long)(b + 1) * nu / nbk);
  }
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
  static_assert(UB >= 1, "a batch must hold at least one unit");
  constexpr bool HALF = lpr<WFMT>() < AIO_WAVE;
  const int lane = T.lane, wave = T.wave;
  const int ulast = P.nu - 1;
#pragma unroll
  for (int j = 0; j < UB * RPU * VPL; ++j) {
    const int ul = j / (RPU * VPL), r = (j / VPL) % RPU, v = j % VPL;
    if constexpr (HALF) {
      // units 2 ul and 2 ul + 1 of the batch in the lower and upper half
      const int vi = lane_vec<WFMT>(v, lane);
      const int ua = P.u0 + batch * 2 * UB + 2 * ul, ub = ua + 1;
      const char* r0;
      const char* r1;
      if constexpr (KIND == K_QKV) {
        // a QKV unit's four rows lie at virtual rows 0, 1, hd/2, hd/2 + 1
        // of its first, in one head and so in one matrix: one row base per
        // unit (recomputed for every row, the scalar address arithmetic
        // took as many instructions as the products)
        static_assert(WFMT == AIO_WFMT_INT8, "half-wave rows are int8 (one byte per weight)");
        const size_t ro = (size_t)((r & 1) + (r >> 1) * (HD / 2)) * (size_t)P.K;
        r0 = wave_uniform(row_base<WFMT, KIND, HD>(a, P, ua < ulast ? ua : ulast, 0)) + ro;
        r1 = wave_uniform(row_base<WFMT, KIND, HD>(a, P, ub < ulast ? ub : ulast, 0)) + ro;
      } else {
        r0 = wave_uniform(row_base<WFMT, KIND, HD>(a, P, ua < ulast ? ua : ulast, r));
        r1 = wave_uniform(row_base<WFMT, KIND, HD>(a, P, ub < ulast ? ub : ulast, r));
      }
      const bool hi = lane >= AIO_WAVE / 2;
      const bool ok = slot_ok(P, hi ? ub : ua, vi);
      const uint4* p = (const uint4*)(hi ? r1 : r0) + (size_t)wave * P.nvw + (ok ? vi : 0);
      buf[j] = ldg_stream(p);
    } else {
      const int u = P.u0 + batch * UB + ul;
      const int vi = v * AIO_WAVE + lane;
      const bool ok = slot_ok(P, u, vi);
      const char* rb;
      if constexpr (KIND == K_QKV) {  // one row base per unit, as above
        constexpr size_t wb = WFMT == AIO_WFMT_BF16 ? 2 : 1;
        const size_t ro = (size_t)((r & 1) + (r >> 1) * (HD / 2)) * (size_t)P.K * wb;
        rb = wave_uniform(row_base<WFMT, KIND, HD>(a, P, u < ulast ? u : ulast, 0)) + ro;
      } else {
        rb = wave_uniform(row_base<WFMT, KIND, HD>(a, P, u < ulast ? u : ulast, r));
      }
      const uint4* p = (const uint4*)rb + (size_t)wave * P.nvw + (ok ? vi : 0);
      buf[j] = ldg_stream(p);
    }
  }
}

// Reduce N per-lane values over the 64 lanes of a wave.  Each halving
// exchange (offsets 32, 16, ...) keeps half of the values, so after log2 N
// of them lane l holds value (l >> (6 - log2 N)) & (N - 1) summed over N
// lanes; plain exchanges finish the sum within groups of 64 / N lanes
// (10 shuffles for 8 values instead of 48).
template <int N>
constexpr int log2_of() { return N == 8 ? 3 : (N == 4 ? 2 : (N == 2 ? 1 : 0)); }

// One halving exchange over lane bit OFF: values [0, HALF) keep the lower
// or upper half of [0, 2 HALF) and add the partner's other half.
template <int OFF, int HALF, int N>
AIO_DEV void halve(float (&v)[N], int lane) {
  const bool up = lane & OFF;
#pragma unroll
  for (int i = 0; i < HALF; ++i) {
    const float send = up ? v[i] : v[i + HALF], keep = up ? v[i + HALF] : v[i];
    v[i] = keep + __shfl_xor(send, OFF, AIO_WAVE);
  }
}

template <int N>
AIO_DEV float reduce_rows(float (&v)[N], int lane) {
  static_assert(N == 2 || N == 4 || N == 8, "reduce_rows takes 2, 4 or 8 values");
  constexpr int LOG = log2_of<N>();
  halve<32, N / 2>(v, lane);
  if constexpr (N >= 4) halve<16, N / 4>(v, lane);
  if constexpr (N >= 8) halve<8, 1>(v, lane);
  float s = v[0];
#pragma unroll
  for (int off = 32 >> LOG; off >= 1; off >>= 1) s += __shfl_xor(s, off, AIO_WAVE);
  return s;
}

// The same over each half wave (lanes 0-31 and 32-63 separately): lane l
// then holds value ((l >> (5 - log2 N)) & (N - 1)) of half l / 32.
template <int N>
AIO_DEV float reduce_rows_half(float (&v)[N], int lane) {
  static_assert(N == 2 || N == 4 || N == 8, "reduce_rows_half takes 2, 4 or 8 values");
  constexpr int LOG = log2_of<N>();
  halve<16, N / 2>(v, lane);
  if constexpr (N >= 4) halve<8, N / 4>(v, lane);
  if constexpr (N >= 8) halve<4, 1>(v, lane);
  float s = v[0];
#pragma unroll
  for (int off = 16 >> LOG; off >= 1; off >>= 1) s += __shfl_xor(s, off, AIO_WAVE);
  return s;
}

// Multiply-accumulate one batch and leave each wave's row partials in LDS
// red[(local unit * RPU + r) * kW + wave].  Slots are not masked here: a
// lane past the end of its K-slice holds h = 0 (input_finish) and reads a
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
  constexpr int LOG = log2_of<kNLD>();
  if constexpr (lpr<WFMT>() < AIO_WAVE) {
    const float s = reduce_rows_half<kNLD>(acc, lane);
    const int idx = (lane >> (5 - LOG)) & (kNLD - 1), hf = lane >> 5;
    if ((lane & ((AIO_WAVE / 2 >> LOG) - 1)) == 0 && idx < UB * RPU) {
      const int ul = idx / RPU, r = idx % RPU;
      const int lu = batch * 2 * UB + 2 * ul + hf;
      if (P.u0 + lu < P.u1) red[(lu * RPU + r) * kW + wave] = s;
    }
  } else {
    const float s = reduce_rows<kNLD>(acc, lane);
    const int idx = (lane >> (6 - LOG)) & (kNLD - 1);
    if ((lane & ((AIO_WAVE >> LOG) - 1)) == 0 && idx < UB * RPU) {
      const int ul = idx / RPU, r = idx % RPU;
      const int lu = batch * UB + ul;
      if (P.u0 + lu < P.u1) red[(lu * RPU + r) * kW + wave] = s;
    }
  }
}

// This lane's slice of the phase input, normalised when the phase starts
// with an RMSNorm.  The slice of wave w, vector v is elements
// [(w * nvw + v * 64 + lane) * EPV, +EPV).  Issued in two steps so that the
// caller can put the phase's second weight batch between the input loads
// and the wait for them: vector memory returns in order, so a wait queued
// behind less prefetch sees the input sooner.
template <int WFMT, int KIND, int VPL>
struct Input {
  static constexpr int E = epv<WFMT>(), NQ = E / 4, NG = E / 8, N = VPL * NQ;
  uint4 gw[VPL][NG];  // norm gains (bf16)
  int off[N];         // word offsets of the input vectors
  bool need[N];
  u32x4 w[N];
};

// Step 1: request the norm gains (they do not depend on other workgroups)
// and the input words.
template <int WFMT, int KIND, int VPL>
AIO_DEV void input_issue(const MegaArgs& a, const GPhase& P, int layer, Input<WFMT, KIND, VPL>& I,
                         const Thr& T) {
  using In = Input<WFMT, KIND, VPL>;
  constexpr int E = In::E, NQ = In::NQ, NG = In::NG;
  constexpr bool NORM = KIND == K_QKV || KIND == K_GU || KIND == K_LM;
  const int lane = T.lane, wave = T.wave;
  const bool any = P.u1 > P.u0;  // a workgroup with no rows reads nothing
  if constexpr (NORM) {
    const CMegaLayer* L = layer_at(a, layer < a.L ? layer : 0);
    const uint16_t* g = KIND == K_QKV ? L->attn_norm : (KIND == K_GU ? L->ffn_norm : a.final_norm);
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const int vi = lane_vec<WFMT>(v, lane);
      const int e0 = (wave * P.nvw + (vi < P.nvw ? vi : 0)) * E;
#pragma unroll
      for (int j = 0; j < NG; ++j) I.gw[v][j] = ldg16(g + e0 + 8 * j);
    }
  }
  if (KIND == K_QKV && layer == 0) return;  // the embedding row: read in step 2
  const unsigned* src = KIND == K_O ? a.o : (KIND == K_DOWN ? a.m : (KIND == K_GU ? a.xa : a.xb));
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    const int vi = lane_vec<WFMT>(v, lane);
    const bool ok = vi < P.nvw;
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      I.off[v * NQ + j] = (wave * P.nvw + (ok ? vi : 0)) * E + 4 * j;
      I.need[v * NQ + j] = any && ok;
    }
  }
#pragma unroll
  for (int i = 0; i < In::N; ++i) I.w[i] = ld16_dev(src, I.off[i]);
}

// Step 2: wait until the input words carry version `ver` and unpack them.
// Nothing here waits for the other waves: each wave starts its loop as soon
// as its own slice is in.  The RMSNorm is applied in two parts: the gains
// here (h = g * x) and the scalar 1 / rms(x) in the epilogue, after the
// products (it is the same for every row); this wave's share of sum(x^2)
// goes to ss8[wave].
template <int WFMT, int KIND, int VPL>
AIO_DEV void input_finish(const MegaArgs& a, const GPhase& P, int layer, int token, unsigned ver,
                          Input<WFMT, KIND, VPL>& I, float (&h)[VPL][epv<WFMT>()], float* ss8,
                          const Thr& T) {
  using In = Input<WFMT, KIND, VPL>;
  constexpr int E = In::E, NQ = In::NQ, NG = In::NG;
  constexpr bool NORM = KIND == K_QKV || KIND == K_GU || KIND == K_LM;
  const int lane = T.lane, wave = T.wave;
  if (KIND == K_QKV && layer == 0) {
    const uint16_t* er = a.embed + (size_t)token * a.d;
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const int vi = lane_vec<WFMT>(v, lane);
      const bool ok = vi < P.nvw;
      const int e0 = (wave * P.nvw + (ok ? vi : 0)) * E;
#pragma unroll
      for (int j = 0; j < NG; ++j) {
        const uint4 b = ldg16(er + e0 + 8 * j);
        const uint32_t w[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          h[v][8 * j + 2 * i] = ok ? bf16_lo(w[i]) : 0.f;
          h[v][8 * j + 2 * i + 1] = ok ? bf16_hi(w[i]) : 0.f;
        }
      }
    }
  } else {
    const unsigned* src = KIND == K_O ? a.o : (KIND == K_DOWN ? a.m : (KIND == K_GU ? a.xa : a.xb));
    await16(a, src, I.off, I.need, I.w, ver);
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
#pragma unroll
      for (int j = 0; j < NQ; ++j) {
        const u32x4 x = I.w[v * NQ + j];
        const bool ok = I.need[v * NQ + j];
        h[v][4 * j + 0] = ok ? untagf(x.x) : 0.f;
        h[v][4 * j + 1] = ok ? untagf(x.y) : 0.f;
        h[v][4 * j + 2] = ok ? untagf(x.z) : 0.f;
        h[v][4 * j + 3] = ok ? untagf(x.w) : 0.f;
      }
    }
  }
  if constexpr (NORM) {
    float ss = 0.f;
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
#pragma unroll
      for (int i = 0; i < E; ++i) ss = fmaf(h[v][i], h[v][i], ss);
    }
    if (lpr<WFMT>() < AIO_WAVE && lane >= AIO_WAVE / 2) ss = 0.f;  // the halves hold the same slice
    ss = wave_sum(ss);
    if (lane == 0) ss8[wave] = ss;
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
#pragma unroll
      for (int j = 0; j < NG; ++j) {
        const uint32_t g4[4] = {I.gw[v][j].x, I.gw[v][j].y, I.gw[v][j].z, I.gw[v][j].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          h[v][8 * j + 2 * i] *= bf16_lo(g4[i]);
          h[v][8 * j + 2 * i + 1] *= bf16_hi(g4[i]);
        }
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
  float ss8[2][kW];  // per-wave sum(x^2) of a normed phase, by phase parity
  float sv[kW];
  int si[kW];
  unsigned flag;
};

// Residual row u (tagged word) before a phase that adds to it: this
// workgroup's own output of two phases back (O reads the DOWN output, or at
// the first layer the embedding row stored at the start of the step; DOWN
// reads the O output).  Same rows, same thread, so no wait.  Only rows past
// a thread's first (more rows per workgroup than threads) read it: the
// first row's exact value stays in the thread's register (k_step's xr).
template <int KIND>
AIO_DEV unsigned resid(const MegaArgs& a, int u) {
  return ld_dev((KIND == K_O ? a.xb : a.xa) + u);
}

// Epilogue inputs of this thread's first unit (u0 + tid) that do not depend
// on this step's data: the RoPE cos/sin pairs at `pos` and the int8
// per-channel scales.  They are requested when the phase starts, so the
// epilogue does not wait a memory round trip for them after the loop.
struct EpiPre {
  float4 cs;      // QKV: (cos, sin) of dims i and i + 1
  uint32_t s[2];  // int8 scales as fp16 bits: QKV two pairs, GU gate and up, else s[0]
};

// Position of QKV unit u: rotation dims i, i + 1 of a head, the matrix
// (0 q, 1 k, 2 v) and the row of dim i in it.
struct QkvRow {
  int i, sec, rlo;
};
AIO_DEV QkvRow qkv_row(const MegaArgs& a, int u) {
  const int half = a.hd / 2, qrows = a.H * a.hd, krows = a.Hkv * a.hd;
  const int p = 2 * u, head = p / half, i = p % half;  // pairs p, p+1 -> dims i, i+1
  int sec = 0, rlo = head * a.hd + i;                   // virtual row of dim i
  if (rlo >= qrows + krows) { sec = 2; rlo -= qrows + krows; }
  else if (rlo >= qrows) { sec = 1; rlo -= qrows; }
  return QkvRow{i, sec, rlo};
}

template <int WFMT, int KIND>
AIO_DEV EpiPre epi_fetch(const MegaArgs& a, const GPhase& P, int pos, int u) {
  EpiPre e;
  e.cs = make_float4(0.f, 0.f, 0.f, 0.f);
  e.s[0] = e.s[1] = 0u;
  if constexpr (KIND == K_QKV) {
    const QkvRow r = qkv_row(a, u);
    const int half = a.hd / 2;
    const u32x4 c = *(gl_u32x4*)(a.rope + (size_t)pos * half + r.i);
    e.cs = make_float4(__uint_as_float(c.x), __uint_as_float(c.y), __uint_as_float(c.z),
                       __uint_as_float(c.w));
    if constexpr (WFMT == AIO_WFMT_INT8) {
      const uint16_t* sc = pick3(r.sec, P.s0, P.s1, P.s2);
      e.s[0] = *(const __attribute__((address_space(1))) uint32_t*)(sc + r.rlo);
      e.s[1] = *(const __attribute__((address_space(1))) uint32_t*)(sc + r.rlo + half);
    }
  } else if constexpr (WFMT == AIO_WFMT_INT8) {
    e.s[0] = *(const __attribute__((address_space(1))) uint16_t*)(P.s0 + u);
    if constexpr (KIND == K_GU) e.s[1] = *(const __attribute__((address_space(1))) uint16_t*)(P.s1 + u);
  }
  return e;
}

AIO_DEV float fp16_lo(uint32_t w) { return fp16_to_f32((uint16_t)(w & 0xffffu)); }
AIO_DEV float fp16_hi(uint32_t w) { return fp16_to_f32((uint16_t)(w >> 16)); }

// Epilogue of a matrix phase: sum the kW wave partials of each row, then the
// phase-specific output, stored with version `vo`.
template <int WFMT, int KIND>
AIO_DEV void epilogue(const MegaArgs& a, const GPhase& P, int layer, int pos, const float* red,
                      Smem& sm, float& xr, const EpiPre& pre, float inv, const Thr& T,
                      unsigned vo, unsigned ep0) {
  constexpr int RPU = rpu_of<KIND>();
  const int nu = P.u1 - P.u0;
  const int tid = T.tid;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  // the layer's cache pointers, read as wave-uniform values: selected per
  // lane from the table, they would come back through a vector load that
  // waits behind every store and load in flight
  uint16_t* kc = nullptr;
  uint16_t* vc = nullptr;
  if constexpr (KIND == K_QKV) {
    const CMegaLayer* L = layer_at(a, layer);
    kc = (uint16_t*)wave_uniform((const char*)L->kc);
    vc = (uint16_t*)wave_uniform((const char*)L->vc);
  }
  for (int t = tid; t < nu; t += kT) {
    float y[RPU];
#pragma unroll
    for (int r = 0; r < RPU; ++r) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kW; ++w) s += red[(t * RPU + r) * kW + w];
      y[r] = KIND == K_O || KIND == K_DOWN ? s : s * inv;  // 1 / rms of a normed input
    }
    const int u = P.u0 + t;
    // the prefetched epilogue inputs serve the first unit; a later one loads its own
    const EpiPre e = t == tid ? pre : epi_fetch<WFMT, KIND>(a, P, pos, u);
    if constexpr (KIND == K_QKV) {
      const int half = a.hd / 2;
      const QkvRow qr = qkv_row(a, u);
      const int sec = qr.sec, rlo = qr.rlo;
      // y[0] = dim i, y[1] = dim i+1, y[2] = dim i+half, y[3] = dim i+1+half
      if constexpr (WFMT == AIO_WFMT_INT8) {
        y[0] *= fp16_lo(e.s[0]);
        y[1] *= fp16_hi(e.s[0]);
        y[2] *= fp16_lo(e.s[1]);
        y[3] *= fp16_hi(e.s[1]);
      }
      if (sec < 2) {
        const float c[2] = {e.cs.x, e.cs.z}, s[2] = {e.cs.y, e.cs.w};
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const float lo = y[k], hi = y[k + 2];
          y[k] = lo * c[k] - hi * s[k];
          y[k + 2] = hi * c[k] + lo * s[k];
        }
      }
      if (sec == 0) {
        st_tag(a.q + rlo, y[0], vo);
        st_tag(a.q + rlo + 1, y[1], vo);
        st_tag(a.q + rlo + half, y[2], vo);
        st_tag(a.q + rlo + half + 1, y[3], vo);
      } else {
        const int g = rlo / a.hd, ii = rlo % a.hd;
        uint16_t* c = (sec == 1 ? kc : vc) + ((size_t)g * a.max_ctx + pos) * a.hd;
        const unsigned b0 = f32_to_bf16(y[0]), b1 = f32_to_bf16(y[1]);
        const unsigned b2 = f32_to_bf16(y[2]), b3 = f32_to_bf16(y[3]);
        st_dev((unsigned*)(c + ii), b0 | (b1 << 16));
        st_dev((unsigned*)(c + ii + half), b2 | (b3 << 16));
        // the same bf16 values, tagged, for this step's attention
        unsigned* n = a.kvn + ((size_t)(sec - 1) * a.Hkv + g) * a.hd + ii;
        st_dev(n, (b0 << 16) | vo);
        st_dev(n + 1, (b1 << 16) | vo);
        st_dev(n + half, (b2 << 16) | vo);
        st_dev(n + half + 1, (b3 << 16) | vo);
      }
    } else if constexpr (KIND == K_GU) {
      float g = y[0], up = y[1];
      if constexpr (WFMT == AIO_WFMT_INT8) {
        g *= fp16_lo(e.s[0]);
        up *= fp16_lo(e.s[1]);
      }
      st_tag(a.m + u, g / (1.f + expf(-g)) * up, vo);
    } else {
      float yy = y[0];
      if constexpr (WFMT == AIO_WFMT_INT8) yy *= fp16_lo(e.s[0]);
      if constexpr (KIND == K_LM) {
        a.logits[u] = yy;
        if (am_better(yy, u, bv, bi)) { bv = yy; bi = u; }
      } else {
        // the thread's first row keeps its exact value in xr; only the
        // copy handed to other workgroups carries the version tag
        const float xo = t == tid ? xr : untagf(resid<KIND>(a, u));
        const float xn = xo + yy;
        if (t == tid) xr = xn;
        st_tag((KIND == K_O ? a.xa : a.xb) + u, xn, vo);
      }
    }
  }
  if constexpr (KIND == K_LM) {
    // fused greedy argmax: workgroup result, then the last workgroup reduces
    block_argmax(bv, bi, sm.sv, sm.si);
    if (tid == 0) {
      st_dev(a.sync + kSyncAmax + 2 * blockIdx.x, __float_as_uint(bv));
      st_dev(a.sync + kSyncAmax + 2 * blockIdx.x + 1, (unsigned)bi);
    }
    wg_publish();
    if (tid == 0) sm.flag = add_dev(a.sync + kSyncAmaxCount, 1u) == gridDim.x - 1;
    __syncthreads();
    if (sm.flag) {
      float gv = -INFINITY;
      int gi = 0x7fffffff;
      for (int b = tid; b < (int)gridDim.x; b += kT) {
        const float v = __uint_as_float(ld_dev(a.sync + kSyncAmax + 2 * b));
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
        // every workgroup has read the epoch base: advance it for the next step
        st_dev(a.sync + kSyncEpoch, ep0 + 5u * (unsigned)a.L);
      }
    }
  }
}

// The register buffers of a wave: kNBUF batches of kNLD 16-byte loads.
struct Bufs {
  uint4 b[kNBUF][kNLD];
};

// Matrix phase k.  On entry buffer 0 holds (in flight) batch 0 of this
// phase; each buffer is refilled with the phase's batch kNBUF further on as
// soon as it is consumed.
template <int WFMT, int HD, int KIND, int VPL>
AIO_DEV void gemv_phase(const MegaArgs& a, int layer, int pos, int token, Bufs& W, float* lds,
                        Smem& sm, unsigned ep0, unsigned k, float& xr) {
  constexpr int RPU = rpu_of<KIND>();
  // LDS partials and norm sums alternate between two buffers by phase
  // parity: a wave may start this phase while another still reads the
  // previous phase's partials in its epilogue
  float* red = lds + (k & 1u) * (unsigned)a.red_words;
  float* ss8 = sm.ss8[k & 1u];
  // units per batch (two halves of a wave take two units each slot for int8)
  constexpr int UB = kNLD / (RPU * VPL) * (AIO_WAVE / lpr<WFMT>());
  const GPhase P = make_phase<WFMT, KIND>(a, layer);
  const int nb = (P.u1 - P.u0 + UB - 1) / UB;
  const unsigned slot = KIND == K_LM ? 0u : k;  // timing slot
  const Thr T = thr();
  EpiPre pre;
  {
    const int t = T.tid < P.u1 - P.u0 ? T.tid : 0;
    pre = epi_fetch<WFMT, KIND>(a, P, pos, P.u0 + t < P.nu ? P.u0 + t : P.nu - 1);
  }
  // batch 0 is in flight (prefetch); then the input words, then the other
  // batches, so the wait for the input is queued behind one batch only
  // (the scheduling barriers keep the three groups of loads, and the first
  // check of the input, in this order)
  Input<WFMT, KIND, VPL> I;
  input_issue<WFMT, KIND, VPL>(a, P, layer, I, T);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int j = 1; j < kNBUF; ++j) issue<WFMT, KIND, VPL, HD>(a, P, j, W.b[j], T);
  __builtin_amdgcn_sched_barrier(0);
  float h[VPL][epv<WFMT>()];
  input_finish<WFMT, KIND, VPL>(a, P, layer, token, ver_of(ep0, k - 1), I, h, ss8, T);
  stamp(a.bar_leave, k - 1);
  stamp_detail(a, slot, 0);
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
  // last round: no refills, so that nothing is queued ahead of the next
  // phase's prefetch and input poll
#pragma unroll
  for (int j = 0; j < kNBUF; ++j) compute<WFMT, KIND, VPL>(P, b + j, W.b[j], h, red, T);
  __syncthreads();
  stamp_detail(a, slot, 1);
  float inv = 1.f;
  if (KIND == K_QKV || KIND == K_GU || KIND == K_LM) {
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kW; ++w) tot += ss8[w];
    inv = rsqrtf(tot / (float)P.K + a.eps);
  }
  epilogue<WFMT, KIND>(a, P, layer, pos, red, sm, xr, pre, inv, T, ver_of(ep0, k), ep0);
  if (KIND != K_LM) {
    // A workgroup's memory requests leave its CU in the order they were
    // issued, by whatever wave.  The outputs are stored by the first waves
    // only; without this barrier the other waves would already have queued
    // the next phase's prefetch (tens of KB) in front of those stores, and
    // every consumer would see them microseconds later.
    __syncthreads();
    stamp(a.bar_arrive, k);
    if (a.trace && blockIdx.x == 0 && threadIdx.x == 0) a.trace[k] = wall_clock64();
  }
}

// Issue the first batch of a matrix phase into buffer 0 (the phase itself
// issues the others once its input words are requested).
template <int WFMT, int HD, int KIND, int VPL>
AIO_DEV void prefetch(const MegaArgs& a, int layer, Bufs& W) {
  const GPhase N = make_phase<WFMT, KIND>(a, layer);
  issue<WFMT, KIND, VPL, HD>(a, N, 0, W.b[0], thr());
}

// ---------------------------------------------------------------- attention

// Online-softmax update of one group with one key row (already loaded).  A
// key past the group's range (valid false) leaves the state unchanged: its
// row (a dummy read, possibly of a position not yet written) is replaced by
// zeros, so no stray Inf or NaN can enter, and the masking is done with
// selects so that the loop has no divergent branches.
template <int HD, int G>
AIO_DEV void attend_key(uint4 kk, uint4 vv, bool valid, const float (&q)[G][8],
                        float (&o)[G][8], float (&m)[G], float (&l)[G]) {
  constexpr int LPK = HD / 8;
  // component-wise: a select of whole vectors is built as an indexed copy
  // in scratch memory
  kk = make_uint4(valid ? kk.x : 0u, valid ? kk.y : 0u, valid ? kk.z : 0u, valid ? kk.w : 0u);
  vv = make_uint4(valid ? vv.x : 0u, valid ? vv.y : 0u, valid ? vv.z : 0u, valid ? vv.w : 0u);
  const float vf[8] = {bf16_lo(vv.x), bf16_hi(vv.x), bf16_lo(vv.y), bf16_hi(vv.y),
                       bf16_lo(vv.z), bf16_hi(vv.z), bf16_lo(vv.w), bf16_hi(vv.w)};
#pragma unroll
  for (int gg = 0; gg < G; ++gg) {
    float sc = dot8_bf16(kk, make_float4(q[gg][0], q[gg][1], q[gg][2], q[gg][3]),
                         make_float4(q[gg][4], q[gg][5], q[gg][6], q[gg][7]), 0.f);
    sc = group_sum_dpp<LPK>(sc);
    // exponents are <= 0 (the score or the old maximum minus the new one);
    // the first valid key turns m = -inf into c = exp2(-inf) = 0
    const float mn = valid ? fmaxf(m[gg], sc) : m[gg];
    const float c = valid ? __builtin_amdgcn_exp2f(m[gg] - mn) : 1.f;
    const float p = valid ? __builtin_amdgcn_exp2f(sc - mn) : 0.f;
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

// Work unit = (kv head g, split s).  The cached keys [0, pos) are split into
// S even chunks; HD/8 lanes hold one key row, and group gi of a split takes
// keys j + t * NGR (t < nk).  nkw is nk of the first group of the wave, the
// largest in the wave, so the key loop has a wave-uniform trip count.
struct AUnit {
  const uint16_t* kb;  // K rows of kv head g, at this lane's 8 dims
  const uint16_t* vb;
  int g, s, j, nk, nkw, jd;  // jd: a row read by masked slots
};

template <int HD>
AIO_DEV AUnit attn_unit(const MegaArgs& a, int layer, int unit, int pos, const Thr& T) {
  constexpr int LPK = HD / 8, NGR = kT / LPK, GPW = AIO_WAVE / LPK;
  const int S = a.S;
  AUnit u;
  u.g = unit / S;
  u.s = unit % S;
  const int chunk = (pos + S - 1) / S;
  const int j0 = min(pos, u.s * chunk), j1 = min(pos, j0 + chunk);
  const int n = j1 - j0;
  const int gi = T.tid / LPK, li = T.tid % LPK, gw = T.wave * GPW;
  u.j = j0 + gi;
  u.nk = n > gi ? (n - gi + NGR - 1) / NGR : 0;
  u.nkw = __builtin_amdgcn_readfirstlane(n > gw ? (n - gw + NGR - 1) / NGR : 0);
  u.jd = j1 > j0 ? j1 - 1 : 0;
  const CMegaLayer* L = layer_at(a, layer);
  u.kb = L->kc + (size_t)u.g * a.max_ctx * HD + li * 8;
  u.vb = L->vc + (size_t)u.g * a.max_ctx * HD + li * 8;
  return u;
}

// Keys t0 .. t0+3 of this lane's group (unconditional loads; a slot past the
// group's keys reads row jd and is masked when consumed).
template <int HD>
AIO_DEV void load4(const AUnit& u, KV4& d, int t0) {
  constexpr int NGR = kT / (HD / 8);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = t0 + i;
    const size_t off = (size_t)(t < u.nk ? u.j + t * NGR : u.jd) * HD;
    d.k[i] = ldg16(u.kb + off);
    d.v[i] = ldg16(u.vb + off);
  }
}

// The first eight keys of each group of this workgroup's first unit (both
// register sets), requested as soon as its QKV rows are out: the cached keys
// do not depend on this step.  A workgroup's loads return in order and its
// poll for q waits behind them, but the keys are needed before q is of any
// use, so nothing is lost; requesting them earlier lets them arrive sooner.
template <int HD>
AIO_DEV void attn_prefetch(const MegaArgs& a, int layer, int pos, KV4& X, KV4& Y) {
  const int units = a.Hkv * a.S;
  const int unit = (int)blockIdx.x < units ? (int)blockIdx.x : units - 1;
  const AUnit u = attn_unit<HD>(a, layer, unit, pos, thr());
  load4<HD>(u, X, 0);
  load4<HD>(u, Y, 4);
}

// Merge the S split partials of kv head g (its G query heads) into o.
// Thread (r, c) folds splits r, r + R, ... of output c with a running
// log-sum-exp; the R partial folds then meet in LDS.  All loads of a thread
// are issued before its first wait.
template <int HD, int G, int MS>
AIO_DEV void attn_merge(const MegaArgs& a, int g, float* lds, unsigned ver) {
  constexpr int NOUT = G * HD, R = kT / NOUT;
  const Thr T = thr();
  const int tid = T.tid, c = tid % NOUT, r = tid / NOUT, gg = c / HD, dim = c % HD;
  const int S = a.S;
  const unsigned* base = a.part + (size_t)g * G * S * (HD + 2);
  float Mt = -INFINITY, Lt = 0.f, Ot = 0.f;
  for (int s0 = r; s0 < S; s0 += MS * R) {
    int off[3 * MS];
    bool need[3 * MS];
    unsigned v[3 * MS];
#pragma unroll
    for (int i = 0; i < MS; ++i) {
      const int s = s0 + i * R;
      const bool ok = s < S;
      const int so = (gg * S + (ok ? s : 0)) * (HD + 2);
      off[3 * i] = so + dim;
      off[3 * i + 1] = so + HD;
      off[3 * i + 2] = so + HD + 1;
      need[3 * i] = need[3 * i + 1] = need[3 * i + 2] = ok;
    }
#pragma unroll
    for (int i = 0; i < 3 * MS; ++i) v[i] = ld_dev(base + off[i]);
    await4(a, base, off, need, v, ver);
#pragma unroll
    for (int i = 0; i < MS; ++i) {
      const float ms = untagf(v[3 * i + 1]);
      if (need[3 * i] && ms != -INFINITY) {
        const float mn = fmaxf(Mt, ms);
        const float c0 = exp2f(Mt - mn), c1 = exp2f(ms - mn);
        Ot = Ot * c0 + c1 * untagf(v[3 * i]);
        Lt = Lt * c0 + c1 * untagf(v[3 * i + 2]);
        Mt = mn;
      }
    }
  }
  float* sm_M = lds;              // [R][G]
  float* sm_L = lds + R * G;      // [R][G]
  float* sm_O = lds + 2 * R * G;  // [R][NOUT]
  if (dim == 0) {
    sm_M[r * G + gg] = Mt;
    sm_L[r * G + gg] = Lt;
  }
  sm_O[r * NOUT + c] = Ot;
  __syncthreads();
  if (tid < NOUT) {
    float M = -INFINITY;
#pragma unroll
    for (int k = 0; k < R; ++k) M = fmaxf(M, sm_M[k * G + gg]);
    float Os = 0.f, Ls = 0.f;
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const float mk = sm_M[k * G + gg];
      const float w = mk == -INFINITY ? 0.f : exp2f(mk - M);
      Os = fmaf(w, sm_O[k * NOUT + c], Os);
      Ls = fmaf(w, sm_L[k * G + gg], Ls);
    }
    st_tag(a.o + (size_t)(g * G + gg) * HD + dim, Os / Ls, ver);
  }
  __syncthreads();
}

// Attention phase k.  Per unit: poll q of the kv head's G query heads
// (version of phase k - 1), run the online softmax over the split's keys
// (the first eight per group already in X and Y), add the new key in the
// last split, combine the NGR groups in LDS and store the split's (output,
// max, sum).  Keys stream through the two register sets in turn, one in
// flight while the other is consumed, with no copies between them.  Then
// the workgroup merges the heads whose last split it ran.
template <int HD, int G>
AIO_DEV void attn_phase(const MegaArgs& a, int layer, int pos, KV4& X, KV4& Y, float* lds,
                        Smem& sm, unsigned ep0, unsigned k) {
  constexpr int LPK = HD / 8, NGR = kT / LPK;
  constexpr int NOUT = G * HD;            // outputs of a unit
  constexpr int R = kT / NOUT > 0 ? kT / NOUT : 1;  // threads per output
  static_assert(NGR % R == 0, "groups must split evenly");
  float* sm_m = lds;                      // [kW][G] wave states
  float* sm_l = lds + NGR * G;            // [kW][G]
  float* sm_o = lds + 2 * NGR * G;        // [kW][G][HD]
  const Thr T = thr();
  const int tid = T.tid, gi = tid / LPK, li = tid % LPK;
  const int wv = __builtin_amdgcn_readfirstlane(T.wave);
  const int S = a.S, units = a.Hkv * S;
  const unsigned vq = ver_of(ep0, k - 1), vo = ver_of(ep0, k);
  for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
    const AUnit u = attn_unit<HD>(a, layer, unit, pos, T);
    const bool first = unit == (int)blockIdx.x;  // keys 0-7 already requested
    if (!first) load4<HD>(u, X, 0);
    // q at this lane's 8 dims; in wave 0 of the last split also the new K/V row
    const unsigned* qb = a.q + (size_t)u.g * G * HD;
    int qoff[2 * G];
    bool qneed[2 * G];
    u32x4 qw[2 * G];
#pragma unroll
    for (int i = 0; i < 2 * G; ++i) {
      qoff[i] = (i >> 1) * HD + li * 8 + 4 * (i & 1);
      qneed[i] = true;
      qw[i] = ld16_dev(qb, qoff[i]);
    }
    const bool nw = u.s == S - 1 && wv == 0;
    const unsigned* nb = a.kvn + (size_t)u.g * HD;  // K row; the V row is Hkv * HD further
    int noff[4];
    bool nneed[4];
    u32x4 nwd[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      noff[i] = (i >> 1) * a.Hkv * HD + li * 8 + 4 * (i & 1);
      nneed[i] = gi == 0;
    }
    if (nw) {
#pragma unroll
      for (int i = 0; i < 4; ++i) nwd[i] = ld16_dev(nb, noff[i]);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (!first) load4<HD>(u, Y, 4);
    __builtin_amdgcn_sched_barrier(0);
    await16(a, qb, qoff, qneed, qw, vq);
    if (unit == (int)blockIdx.x) stamp(a.bar_leave, k - 1);
    float q[G][8], o[G][8], m[G], l[G];
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
      const u32x4 q0 = qw[2 * gg], q1 = qw[2 * gg + 1];
      const unsigned qq[8] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        q[gg][i] = untagf(qq[i]) * a.scale_log2;
        o[gg][i] = 0.f;
      }
      m[gg] = -INFINITY;
      l[gg] = 0.f;
    }
    // The scheduling barriers keep each set's loads where they are written:
    // hoisted together, both sets would be waited for at the top of the loop.
    int t = 0;
    for (; t + 8 < u.nkw; t += 8) {
#pragma unroll
      for (int i = 0; i < 4; ++i) attend_key<HD, G>(X.k[i], X.v[i], t + i < u.nk, q, o, m, l);
      __builtin_amdgcn_sched_barrier(0);
      load4<HD>(u, X, t + 8);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 4; ++i) attend_key<HD, G>(Y.k[i], Y.v[i], t + 4 + i < u.nk, q, o, m, l);
      __builtin_amdgcn_sched_barrier(0);
      load4<HD>(u, Y, t + 12);
      __builtin_amdgcn_sched_barrier(0);
    }
    // the last eight keys: slots past the wave's largest key count are
    // skipped (a split of a few keys per group would otherwise spend most
    // of its time on masked slots)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (t + i < u.nkw) attend_key<HD, G>(X.k[i], X.v[i], t + i < u.nk, q, o, m, l);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (t + 4 + i < u.nkw) attend_key<HD, G>(Y.k[i], Y.v[i], t + 4 + i < u.nk, q, o, m, l);
    if (nw) {
      // the new key (position pos), taken by group 0 of the last split
      await16(a, nb, noff, nneed, nwd, vq);
      const u32x4 k0 = nwd[0], k1 = nwd[1], v0 = nwd[2], v1 = nwd[3];
      const uint4 kk = make_uint4((k0.x >> 16) | (k0.y & 0xffff0000u), (k0.z >> 16) | (k0.w & 0xffff0000u),
                                  (k1.x >> 16) | (k1.y & 0xffff0000u), (k1.z >> 16) | (k1.w & 0xffff0000u));
      const uint4 vv = make_uint4((v0.x >> 16) | (v0.y & 0xffff0000u), (v0.z >> 16) | (v0.w & 0xffff0000u),
                                  (v1.x >> 16) | (v1.y & 0xffff0000u), (v1.z >> 16) | (v1.w & 0xffff0000u));
      attend_key<HD, G>(kk, vv, gi == 0, q, o, m, l);
    }
    // combine the groups: the AIO_WAVE / LPK groups of each wave with lane
    // exchanges (every group of the wave ends with the wave's state), then
    // the kW wave states in LDS
#pragma unroll
    for (int off = LPK; off < AIO_WAVE; off <<= 1) {
#pragma unroll
      for (int gg = 0; gg < G; ++gg) {
        const float m2 = __shfl_xor(m[gg], off, AIO_WAVE);
        const float l2 = __shfl_xor(l[gg], off, AIO_WAVE);
        const float mx = fmaxf(m[gg], m2);
        const float c1 = m[gg] == -INFINITY ? 0.f : exp2f(m[gg] - mx);
        const float c2 = m2 == -INFINITY ? 0.f : exp2f(m2 - mx);
        l[gg] = l[gg] * c1 + l2 * c2;
#pragma unroll
        for (int i = 0; i < 8; ++i)
          o[gg][i] = o[gg][i] * c1 + __shfl_xor(o[gg][i], off, AIO_WAVE) * c2;
        m[gg] = mx;
      }
    }
    if (T.lane < LPK) {  // group 0 of each wave
#pragma unroll
      for (int gg = 0; gg < G; ++gg) {
        if (li == 0) {
          sm_m[wv * G + gg] = m[gg];
          sm_l[wv * G + gg] = l[gg];
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) sm_o[(wv * G + gg) * HD + li * 8 + i] = o[gg][i];
      }
    }
    __syncthreads();
    if (tid < NOUT) {
      const int gg = tid / HD, dim = tid % HD;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kW; ++w) M = fmaxf(M, sm_m[w * G + gg]);
      float Ot = 0.f, Lt = 0.f;
      if (M != -INFINITY) {
#pragma unroll
        for (int w = 0; w < kW; ++w) {
          const float mk = sm_m[w * G + gg];
          const float wt = mk == -INFINITY ? 0.f : exp2f(mk - M);
          Ot = fmaf(wt, sm_o[(w * G + gg) * HD + dim], Ot);
          Lt = fmaf(wt, sm_l[w * G + gg], Lt);
        }
      }
      unsigned* slot = a.part + ((size_t)(u.g * G + gg) * S + u.s) * (HD + 2);
      st_tag(slot + dim, Ot, vo);
      if (dim == 0) {
        st_tag(slot + HD, M, vo);
        st_tag(slot + HD + 1, Lt, vo);
      }
    }
    __syncthreads();  // the LDS is reused by the next unit or the merge
  }
  stamp_detail(a, k, 0);
  // splits per merging thread (R threads per output): as many loads as
  // there are splits to fold
  for (int g = 0; g < a.Hkv; ++g) {
    if ((g * S + S - 1) % (int)gridDim.x != (int)blockIdx.x) continue;
    if (S <= 2 * R) attn_merge<HD, G, 2>(a, g, lds, vo);
    else if (S <= 8 * R) attn_merge<HD, G, 8>(a, g, lds, vo);
    else attn_merge<HD, G, 16>(a, g, lds, vo);
  }
  stamp_detail(a, k, 1);
  stamp(a.bar_arrive, k);
  if (a.trace && blockIdx.x == 0 && threadIdx.x == 0) a.trace[k] = wall_clock64();
}

template <int WFMT, int HD, int G, int VQ, int VD>
__global__ __launch_bounds__(kT, 1) void k_step(MegaArgs a) {
  extern __shared__ float lds[];
  __shared__ Smem sm;
  const int pos = a.st->pos, token = a.st->token[0];
  // the epoch base of this step; the last workgroup of the argmax advances it
  const unsigned ep0 = ld_dev(a.sync + kSyncEpoch);
  Bufs W;
  KV4 X, Y;
  prefetch<WFMT, HD, K_QKV, VQ>(a, 0, W);
  // The residual stream of this thread's first row of the O and down
  // projections (both split the d rows the same way), kept exact in a
  // register for the whole step: handing it between workgroups costs its
  // 3 low mantissa bits (the version tag), which would otherwise accumulate
  // over the 2 L additions.
  float xr = 0.f;
  {
    // the residual before layer 0 (the embedding row) of the rows this
    // workgroup updates in the O projection
    const GPhase P = make_phase<WFMT, K_O>(a, 0);
    const int t = thr().tid;
    if (t < P.u1 - P.u0) {
      xr = bf16_to_f32(a.embed[(size_t)token * a.d + P.u0 + t]);
      st_tag(a.xb + P.u0 + t, xr, ver_of(ep0, 0));
    }
  }
  for (int l = 0; l < a.L; ++l) {
    const unsigned k = 5u * (unsigned)l;
    gemv_phase<WFMT, HD, K_QKV, VQ>(a, l, pos, token, W, lds, sm, ep0, k + 1, xr);
    attn_prefetch<HD>(a, l, pos, X, Y);
    attn_phase<HD, G>(a, l, pos, X, Y, lds + 2 * a.red_words, sm, ep0, k + 2);
    prefetch<WFMT, HD, K_O, VQ>(a, l, W);
    gemv_phase<WFMT, HD, K_O, VQ>(a, l, pos, token, W, lds, sm, ep0, k + 3, xr);
    prefetch<WFMT, HD, K_GU, VQ>(a, l, W);
    gemv_phase<WFMT, HD, K_GU, VQ>(a, l, pos, token, W, lds, sm, ep0, k + 4, xr);
    prefetch<WFMT, HD, K_DOWN, VD>(a, l, W);
    gemv_phase<WFMT, HD, K_DOWN, VD>(a, l, pos, token, W, lds, sm, ep0, k + 5, xr);
    if (l + 1 < a.L)
      prefetch<WFMT, HD, K_QKV, VQ>(a, l + 1, W);
    else
      prefetch<WFMT, HD, K_LM, VQ>(a, l + 1, W);
  }
  gemv_phase<WFMT, HD, K_LM, VQ>(a, a.L, pos, token, W, lds, sm, ep0, 5u * (unsigned)a.L + 1, xr);
}

// The grid is one workgroup per CU and a CU holds at most one (registers
// and LDS), so all workgroups are resident together.  The cooperative
// launch states that requirement to the runtime, which refuses the launch
// if it cannot be met; a plain launch of the same grid relies on the GPU
// running nothing else (every wait is bounded either way).
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
  const bool i8 = c.wfmt == AIO_WFMT_INT8;
  const int epv_ = i8 ? epv<AIO_WFMT_INT8>() : epv<AIO_WFMT_BF16>();
  const int lpr_ = i8 ? lpr<AIO_WFMT_INT8>() : lpr<AIO_WFMT_BF16>();
  if (K % (kW * epv_)) return 0;
  const int nvw = K / (kW * epv_);
  return (nvw + lpr_ - 1) / lpr_;
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

int aio_step_kernel_gu_cap(const aio_config& c, int blocks) {
  const int even = (c.ffn_dim + blocks - 1) / blocks;
  return even + std::max(2, even / 8);
}

// Floats of one buffer of matrix-phase partials: [units per workgroup][RPU][kW].
static int red_words(const aio_config& c, int blocks) {
  auto red = [&](int units, int rpu) { return ((units + blocks - 1) / blocks) * rpu * kW; };
  int w = red((c.n_heads + 2 * c.n_kv_heads) * c.head_dim / 4, 4);
  w = std::max(w, red(c.d_model, 1));
  w = std::max(w, aio_step_kernel_gu_cap(c, blocks) * 2 * kW);
  w = std::max(w, red(c.vocab, 1));
  return (w + 63) & ~63;
}

size_t aio_step_kernel_lds(const aio_config& c, int blocks) {
  const int G = c.n_heads / c.n_kv_heads;
  const int ngr = kT / (c.head_dim / 8);
  const int nout = G * c.head_dim;
  const int r = kT / nout > 0 ? kT / nout : 1;
  // group state + [R][NOUT] partials + R * G sums; the merge needs
  // 2 R G + R NOUT, which fits in the same space
  const size_t attn = ((size_t)ngr * G * (c.head_dim + 2) + (size_t)r * nout + (size_t)r * G) * 4;
  // attention area after the two matrix-phase partial buffers
  return (size_t)2 * red_words(c, blocks) * 4 + attn;
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
  a.xa = m.at<unsigned>(m.lay.mega_xa);
  a.xb = m.at<unsigned>(m.lay.mega_xb);
  a.q = m.at<unsigned>(m.lay.mega_q);
  a.kvn = m.at<unsigned>(m.lay.mega_kvn);
  a.o = m.at<unsigned>(m.lay.mega_o);
  a.m = m.at<unsigned>(m.lay.mega_m);
  a.part = m.at<unsigned>(m.lay.mega_part);
  a.sync = m.at<unsigned>(m.lay.sync);
  a.logits = logits;
  a.tokens_out = tokens_out;
  a.trace = trace;
  a.bar_arrive = bar_arrive;
  a.bar_leave = bar_leave;
  a.detail = bar_leave ? bar_leave + (size_t)(5 * c.n_layers + 1) * m.mega_blocks : nullptr;
  a.gu_bounds = m.gu_bounds_dev;
  a.L = c.n_layers;
  a.d = c.d_model;
  a.H = c.n_heads;
  a.Hkv = c.n_kv_heads;
  a.hd = c.head_dim;
  a.F = c.ffn_dim;
  a.V = c.vocab;
  a.max_ctx = c.max_ctx;
  a.S = m.lay.mega_splits;
  a.red_words = red_words(c, m.mega_blocks);
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
