/*
 * Seeded synthetic inputs for the convolution hot path.
 *
 * This file holds no arithmetic of the method under test: it only turns
 * (seed, stream id, element index) into numbers.  Both the fp64 oracle and the
 * HIP path receive the arrays written here.
 *
 * Generator: Philox-4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11), the counter-based generator the paper
 * adopts for its RNG (Sec. 3, reference-default semantics).  One call maps a
 * 128-bit counter and a 64-bit key to four 32-bit words:
 *   key    = (seed, stream)
 *   counter = (block lo 32 bits, block hi 32 bits, 0, 0), block = index / 4
 * Uniform:  u = (word >> 8) * 2^-24 in [0, 1)
 * Normal:   Box-Muller on word pairs (0,1) and (2,3) of a block.
 * Values are then rounded to bf16 with round-to-nearest-even (or kept fp32).
 */
#include <math.h>
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
  uint32_t n2 = hi0 ^ c[3] ^ k[1];
  c[0] = n0;
  c[1] = lo1;
  c[2] = n2;
  c[3] = lo0;
}

/* Philox-4x32 with 10 rounds; exported for known-answer tests. */
void synth_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
  uint32_t k[2] = {key_in[0], key_in[1]};
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k[0] += PHILOX_W0;
      k[1] += PHILOX_W1;
    }
    philox_round(c, k);
  }
  memcpy(out, c, sizeof c);
}

static inline void block_words(uint32_t seed, uint32_t stream, uint64_t block, uint32_t w[4]) {
  uint32_t ctr[4] = {(uint32_t)block, (uint32_t)(block >> 32), 0u, 0u};
  uint32_t key[2] = {seed, stream};
  synth_philox4x32_10(ctr, key, w);
}

/* float -> bf16 bits, round to nearest even, NaN kept quiet. */
static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x40u);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

enum { SYNTH_UNIFORM = 0, SYNTH_NORMAL = 1 };

static inline double word_uniform(uint32_t w) { return (double)(w >> 8) * (1.0 / 16777216.0); }

/* value of element i of the stream, as double */
static inline void block_values(int dist, double p0, double p1, uint32_t seed, uint32_t stream,
                                uint64_t block, double v[4]) {
  uint32_t w[4];
  block_words(seed, stream, block, w);
  if (dist == SYNTH_UNIFORM) {
    for (int j = 0; j < 4; ++j) v[j] = p0 + (p1 - p0) * word_uniform(w[j]);
  } else {
    for (int j = 0; j < 4; j += 2) {
      /* u1 in (0, 1] so that log is finite */
      double u1 = ((double)(w[j] >> 8) + 1.0) * (1.0 / 16777216.0);
      double u2 = word_uniform(w[j + 1]);
      double rad = sqrt(-2.0 * log(u1));
      double ang = 6.283185307179586476925 * u2;
      v[j] = p0 + p1 * rad * cos(ang);
      v[j + 1] = p0 + p1 * rad * sin(ang);
    }
  }
}

/* dist: 0 uniform [p0, p1), 1 normal (mean p0, std p1).  out: n bf16 bit patterns. */
void synth_fill_bf16(uint16_t* out, int64_t n, uint32_t seed, uint32_t stream, int dist, double p0,
                     double p1) {
  int64_t nblocks = (n + 3) / 4;
#pragma omp parallel for schedule(static)
  for (int64_t b = 0; b < nblocks; ++b) {
    double v[4];
    block_values(dist, p0, p1, seed, stream, (uint64_t)b, v);
    for (int j = 0; j < 4; ++j) {
      int64_t i = b * 4 + j;
      if (i < n) out[i] = f32_to_bf16_rne((float)v[j]);
    }
  }
}

void synth_fill_f32(float* out, int64_t n, uint32_t seed, uint32_t stream, int dist, double p0,
                    double p1) {
  int64_t nblocks = (n + 3) / 4;
#pragma omp parallel for schedule(static)
  for (int64_t b = 0; b < nblocks; ++b) {
    double v[4];
    block_values(dist, p0, p1, seed, stream, (uint64_t)b, v);
    for (int j = 0; j < 4; ++j) {
      int64_t i = b * 4 + j;
      if (i < n) out[i] = (float)v[j];
    }
  }
}

/* Draw `count` distinct-ish sample indices in [0, n) (with replacement). */
void synth_indices(int64_t* out, int64_t count, int64_t n, uint32_t seed, uint32_t stream) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) {
    uint32_t w[4];
    block_words(seed, stream, (uint64_t)i, w);
    uint64_t r = ((uint64_t)w[0] << 32) | w[1];
    out[i] = (int64_t)(r % (uint64_t)n);
  }
}
