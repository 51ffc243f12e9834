// Device helpers shared by the decode and verify kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define AIO_WAVE 64
#define AIO_DEV __device__ __forceinline__

// bf16 -> fp32 is a 16-bit shift; both halves of a packed dword.
AIO_DEV float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
AIO_DEV float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
AIO_DEV float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
AIO_DEV uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

AIO_DEV float fp16_to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }

// Sum over the 64 lanes of a wave; every lane receives the total.
AIO_DEV float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, AIO_WAVE);
  return v;
}

// Sum over aligned groups of `width` lanes (a power of two <= 64).
template <int WIDTH>
AIO_DEV float group_sum(float v) {
#pragma unroll
  for (int off = WIDTH / 2; off >= 1; off >>= 1) v += __shfl_xor(v, off, AIO_WAVE);
  return v;
}

AIO_DEV float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, AIO_WAVE));
  return v;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16-byte streaming load of weights (read once per token: no reuse to keep).
AIO_DEV uint4 ld_stream(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// dot of 8 bf16 (one uint4) with 8 fp32 activations.
AIO_DEV float dot8_bf16(uint4 w, const float4 a, const float4 b, float acc) {
  acc = fmaf(bf16_lo(w.x), a.x, acc);
  acc = fmaf(bf16_hi(w.x), a.y, acc);
  acc = fmaf(bf16_lo(w.y), a.z, acc);
  acc = fmaf(bf16_hi(w.y), a.w, acc);
  acc = fmaf(bf16_lo(w.z), b.x, acc);
  acc = fmaf(bf16_hi(w.z), b.y, acc);
  acc = fmaf(bf16_lo(w.w), b.z, acc);
  acc = fmaf(bf16_hi(w.w), b.w, acc);
  return acc;
}

// int8 byte j of a dword, sign-extended, as fp32 (exact).
AIO_DEV float i8_at(uint32_t w, int j) { return (float)(int8_t)(w >> (8 * j)); }

// dot of 4 int8 (one dword) with 4 fp32 activations.
AIO_DEV float dot4_i8(uint32_t w, const float4 a, float acc) {
  acc = fmaf(i8_at(w, 0), a.x, acc);
  acc = fmaf(i8_at(w, 1), a.y, acc);
  acc = fmaf(i8_at(w, 2), a.z, acc);
  acc = fmaf(i8_at(w, 3), a.w, acc);
  return acc;
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
