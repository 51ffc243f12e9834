/*
 * Seeded synthetic inputs shared by the CPU oracle and the GPU path.
 *
 * This file draws random numbers and rounds them to storage formats; it
 * holds none of the decoder's arithmetic.  Every tensor gets its own stream
 * of a counter-based generator, Philox4x32-10 (Salmon, Moraes, Dror, Shaw,
 * "Parallel Random Numbers: As Easy as 1, 2, 3", SC'11), keyed by the root
 * seed and addressed by (element block, 64-bit stream id).  Any element can
 * therefore be regenerated without drawing the ones before it, and large
 * tensors are filled in parallel with OpenMP.
 *
 * Counter layout per Philox call: ctr = {block_lo, block_hi, stream_lo,
 * stream_hi}, key = {seed_lo, seed_hi}.  One call yields four 32-bit words.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static inline void philox_round(uint32_t c[4], const uint32_t k[2]) {
  uint64_t p0 = (uint64_t)PHILOX_M0 * c[0];
  uint64_t p1 = (uint64_t)PHILOX_M1 * c[2];
  uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
  uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
  uint32_t n0 = hi1 ^ c[1] ^ k[0];
  uint32_t n1 = lo1;
  uint32_t n2 = hi0 ^ c[3] ^ k[1];
  uint32_t n3 = lo0;
  c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
}

/* Philox4x32 with ten rounds; the key is bumped by the Weyl constants
 * between rounds. */
void synth_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
  uint32_t k[2] = {key[0], key[1]};
  for (int r = 0; r < 10; ++r) {
    if (r) { k[0] += PHILOX_W0; k[1] += PHILOX_W1; }
    philox_round(c, k);
  }
  memcpy(out, c, sizeof c);
}

static inline void draw(uint64_t seed, uint64_t stream, uint64_t block, uint32_t out[4]) {
  uint32_t ctr[4] = {(uint32_t)block, (uint32_t)(block >> 32), (uint32_t)stream,
                     (uint32_t)(stream >> 32)};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  synth_philox4x32_10(ctr, key, out);
}

/* FNV-1a 64-bit hash: maps a tensor name to its stream id. */
uint64_t synth_stream_id(const char* name) {
  uint64_t h = 0xcbf29ce484222325ull;
  for (const unsigned char* p = (const unsigned char*)name; *p; ++p) {
    h ^= *p;
    h *= 0x100000001b3ull;
  }
  return h;
}

/* float -> bfloat16 bits, round to nearest even (storage format only). */
static inline uint16_t to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* float -> IEEE binary16 bits, round to nearest even; inputs are finite
 * and within the normal range of binary16 here (scales in (0.001, 0.01)). */
static inline uint16_t to_fp16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  uint32_t sign = (u >> 16) & 0x8000u;
  int32_t e = (int32_t)((u >> 23) & 0xff) - 127 + 15;
  uint32_t m = u & 0x7fffffu;
  if (e <= 0) { /* subnormal half */
    if (e < -10) return (uint16_t)sign;
    m |= 0x800000u;
    uint32_t shift = (uint32_t)(14 - e);
    uint32_t half = m >> shift;
    uint32_t rem = m & ((1u << shift) - 1u);
    uint32_t mid = 1u << (shift - 1);
    if (rem > mid || (rem == mid && (half & 1u))) half++;
    return (uint16_t)(sign | half);
  }
  if (e >= 31) return (uint16_t)(sign | 0x7c00u);
  uint32_t half = ((uint32_t)e << 10) | (m >> 13);
  uint32_t rem = m & 0x1fffu;
  if (rem > 0x1000u || (rem == 0x1000u && (half & 1u))) half++;
  return (uint16_t)(sign | half);
}

/* Two standard normals from two 32-bit words by the Box-Muller transform,
 * evaluated in single precision: u1 in (0, 1], u2 in [0, 1). */
static inline void box_muller(uint32_t a, uint32_t b, double z[2]) {
  float u1 = ((float)(a >> 8) + 1.0f) * (1.0f / 16777216.0f);
  float u2 = (float)(b >> 8) * (1.0f / 16777216.0f);
  float r = sqrtf(-2.0f * logf(u1));
  float t = 6.2831853071795864769f * u2;
  z[0] = (double)(r * cosf(t));
  z[1] = (double)(r * sinf(t));
}

/* out[i] = bf16(mean + std * N(0,1)); elements 4b..4b+3 come from block b. */
void synth_normal_bf16(uint64_t seed, uint64_t stream, uint16_t* out, uint64_t n, double mean,
                       double std) {
  int64_t nb = (int64_t)((n + 3) / 4);
#pragma omp parallel for schedule(static)
  for (int64_t b = 0; b < nb; ++b) {
    uint32_t w[4];
    double z[4];
    draw(seed, stream, (uint64_t)b, w);
    box_muller(w[0], w[1], z);
    box_muller(w[2], w[3], z + 2);
    for (int j = 0; j < 4; ++j) {
      uint64_t i = (uint64_t)b * 4 + (uint64_t)j;
      if (i < n) out[i] = to_bf16((float)(mean + std * z[j]));
    }
  }
}

/* out[i] = float(mean + std * N(0,1)) (fp32, for activation-level tests). */
void synth_normal_f32(uint64_t seed, uint64_t stream, float* out, uint64_t n, double mean,
                       double std) {
  int64_t nb = (int64_t)((n + 3) / 4);
#pragma omp parallel for schedule(static)
  for (int64_t b = 0; b < nb; ++b) {
    uint32_t w[4];
    double z[4];
    draw(seed, stream, (uint64_t)b, w);
    box_muller(w[0], w[1], z);
    box_muller(w[2], w[3], z + 2);
    for (int j = 0; j < 4; ++j) {
      uint64_t i = (uint64_t)b * 4 + (uint64_t)j;
      if (i < n) out[i] = (float)(mean + std * z[j]);
    }
  }
}

/* Integers uniform on {-127, ..., 127}: floor(u * 255 / 2^32) - 127. */
void synth_int8_sym(uint64_t seed, uint64_t stream, int8_t* out, uint64_t n) {
  int64_t nb = (int64_t)((n + 3) / 4);
#pragma omp parallel for schedule(static)
  for (int64_t b = 0; b < nb; ++b) {
    uint32_t w[4];
    draw(seed, stream, (uint64_t)b, w);
    for (int j = 0; j < 4; ++j) {
      uint64_t i = (uint64_t)b * 4 + (uint64_t)j;
      if (i < n) out[i] = (int8_t)((int)(((uint64_t)w[j] * 255u) >> 32) - 127);
    }
  }
}

/* out[i] = fp16(lo + (hi - lo) * (u + 0.5) / 2^32). */
void synth_uniform_fp16(uint64_t seed, uint64_t stream, uint16_t* out, uint64_t n, double lo,
                        double hi) {
  int64_t nb = (int64_t)((n + 3) / 4);
#pragma omp parallel for schedule(static)
  for (int64_t b = 0; b < nb; ++b) {
    uint32_t w[4];
    draw(seed, stream, (uint64_t)b, w);
    for (int j = 0; j < 4; ++j) {
      uint64_t i = (uint64_t)b * 4 + (uint64_t)j;
      if (i < n) {
        double u = ((double)w[j] + 0.5) * (1.0 / 4294967296.0);
        out[i] = to_fp16((float)(lo + (hi - lo) * u));
      }
    }
  }
}

/* Token ids uniform on [0, vocab): floor(u * vocab / 2^32). */
void synth_tokens(uint64_t seed, uint64_t stream, int32_t* out, uint64_t n, uint32_t vocab) {
  for (uint64_t b = 0; b < (n + 3) / 4; ++b) {
    uint32_t w[4];
    draw(seed, stream, b, w);
    for (int j = 0; j < 4; ++j) {
      uint64_t i = b * 4 + (uint64_t)j;
      if (i < n) out[i] = (int32_t)(((uint64_t)w[j] * vocab) >> 32);
    }
  }
}

/* Uniform integers on [0, n) for picking positions (same rule as tokens). */
uint32_t synth_uniform_index(uint64_t seed, uint64_t stream, uint64_t which, uint32_t n) {
  uint32_t w[4];
  draw(seed, stream, which / 4, w);
  return (uint32_t)(((uint64_t)w[which % 4] * n) >> 32);
}
