/*
 * Seeded synthetic-input generator shared by the GPU path's harness and by the
 * oracle.  It holds none of the MoE method's arithmetic: it only turns
 * (seed, stream, element index) into a normally distributed number.
 *
 * Generator: Philox4x32-10, the counter-based generator of Salmon, Moraes,
 * Dror and Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3" (SC 2011),
 * written here from its published definition (two 32x32->64 multiplies per
 * round with multipliers 0xD2511F53 and 0xCD9E8D57, Weyl key increments
 * 0x9E3779B9 and 0xBB67AE85, ten rounds).
 * Normals: the Box-Muller transform (Box and Muller, 1958) on two uniforms.
 *
 * Element i of stream s under seed k comes from Philox block i/4 with
 * counter (i/4 low, i/4 high, s low, s high) and key (k low, k high);
 * words (0,1) give normals 0,1 and words (2,3) give normals 2,3.  The value
 * depends only on (k, s, i), so any split of the work over threads yields
 * the same bytes.
 *
 * bf16 outputs are the round-to-nearest-even truncation of the fp32 value to
 * its upper 16 bits (the bf16 format is the upper half of an IEEE-754
 * binary32).
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
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
  uint32_t n2 = hi0 ^ c[3] ^ k[1];
  c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
}

void synth_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
  uint32_t k[2] = {key[0], key[1]};
  for (int r = 0; r < 10; ++r) {
    if (r > 0) { k[0] += PHILOX_W0; k[1] += PHILOX_W1; }
    philox_round(c, k);
  }
  memcpy(out, c, sizeof(c));
}

static inline void normals4(uint64_t seed, uint64_t stream, uint64_t blk, float z[4]) {
  uint32_t ctr[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), (uint32_t)stream, (uint32_t)(stream >> 32)};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t x[4];
  synth_philox4x32_10(ctr, key, x);
  const float two_pi = 6.283185307179586f;
  const float inv32 = 2.3283064365386963e-10f; /* 2^-32 */
  for (int p = 0; p < 2; ++p) {
    /* u1 in (0,1], u2 in [0,1) */
    float u1 = ((float)x[2 * p] + 1.0f) * inv32;
    if (u1 > 1.0f) u1 = 1.0f;
    float u2 = (float)(x[2 * p + 1] >> 8) * (1.0f / 16777216.0f);
    float r = sqrtf(-2.0f * logf(u1));
    float t = two_pi * u2;
    z[2 * p] = r * cosf(t);
    z[2 * p + 1] = r * sinf(t);
  }
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* out[j] = mean + std * N(0,1)[offset + j], j < n.  fp32. */
void synth_normal_f32(uint64_t seed, uint64_t stream, uint64_t offset, size_t n, float mean, float std,
                      float* out) {
  #pragma omp parallel for schedule(static)
  for (int64_t b = (int64_t)(offset / 4); b < (int64_t)((offset + n + 3) / 4); ++b) {
    float z[4];
    normals4(seed, stream, (uint64_t)b, z);
    for (int q = 0; q < 4; ++q) {
      uint64_t i = (uint64_t)b * 4 + (uint64_t)q;
      if (i >= offset && i < offset + n) out[i - offset] = mean + std * z[q];
    }
  }
}

/* Same values as synth_normal_f32, rounded to bf16 (RNE); out holds raw bf16 bits. */
void synth_normal_bf16(uint64_t seed, uint64_t stream, uint64_t offset, size_t n, float mean, float std,
                       uint16_t* out) {
  #pragma omp parallel for schedule(static)
  for (int64_t b = (int64_t)(offset / 4); b < (int64_t)((offset + n + 3) / 4); ++b) {
    float z[4];
    normals4(seed, stream, (uint64_t)b, z);
    for (int q = 0; q < 4; ++q) {
      uint64_t i = (uint64_t)b * 4 + (uint64_t)q;
      if (i >= offset && i < offset + n) out[i - offset] = f32_to_bf16_rne(mean + std * z[q]);
    }
  }
}

/*
 * Symmetric round-to-nearest 4-bit storage of bf16 rows (data preparation of
 * the 4-bit synthetic models, not part of the method): for each group of
 * `group` consecutive values of a row, scale s = bf16(absmax / 7) and
 * code = clamp(rint(w / s), -8, 7) + 8 (0 when s == 0), computed in fp32 with
 * round-half-to-even; two codes per byte, even k in the low nibble.
 * codes: R x K/2 bytes; scales: R x K/group bf16 bits.
 */
void synth_quant_int4(const uint16_t* w, int64_t R, int64_t K, int64_t group, uint8_t* codes, uint16_t* scales) {
  #pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < R; ++r) {
    const uint16_t* row = w + r * K;
    for (int64_t g0 = 0; g0 < K; g0 += group) {
      float amax = 0.0f;
      for (int64_t k = g0; k < g0 + group; ++k) {
        uint32_t u = (uint32_t)row[k] << 16;
        float v;
        memcpy(&v, &u, 4);
        v = fabsf(v);
        if (v > amax) amax = v;
      }
      const uint16_t sb = f32_to_bf16_rne(amax / 7.0f);
      scales[r * (K / group) + g0 / group] = sb;
      uint32_t su = (uint32_t)sb << 16;
      float s;
      memcpy(&s, &su, 4);
      for (int64_t k = g0; k < g0 + group; k += 2) {
        int q[2];
        for (int j = 0; j < 2; ++j) {
          uint32_t u = (uint32_t)row[k + j] << 16;
          float v;
          memcpy(&v, &u, 4);
          float t = s > 0.0f ? rintf(v / s) : 0.0f;
          if (t < -8.0f) t = -8.0f;
          if (t > 7.0f) t = 7.0f;
          q[j] = (int)t + 8;
        }
        codes[r * (K / 2) + k / 2] = (uint8_t)(q[0] | (q[1] << 4));
      }
    }
  }
}
