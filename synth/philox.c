/*
 * Seeded synthetic tensors for the workloads: Philox4x32-10 counter-based
 * generator (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
 * 1, 2, 3", SC'11) feeding the Box-Muller transform (Box & Muller, 1958).
 *
 * This file holds no arithmetic of the transformer blocks: it only fills
 * buffers with pseudo-random values, so both the oracle and the GPU path can
 * be fed the same inputs and weights.  Element i of a stream with 64-bit seed
 * s is a pure function of (s, i): the four 32-bit words of block j = i / 4 are
 * philox(counter = {j_lo, j_hi, 0, 0}, key = {s_lo, s_hi}); words (0,1) give
 * normals 4j, 4j+1 and words (2,3) give normals 4j+2, 4j+3.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC philox.c -o libsynth.so -lm
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

void synth_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
  uint32_t k[2] = {key_in[0], key_in[1]};
  for (int r = 0; r < 10; ++r) {
    philox_round(c, k);
    k[0] += PHILOX_W0;
    k[1] += PHILOX_W1;
  }
  memcpy(out, c, sizeof(c));
}

/* uniform in (0, 1]: (x + 1) * 2^-32, exact in double */
static inline double u01(uint32_t x) { return ((double)x + 1.0) * (1.0 / 4294967296.0); }

static inline void block_normals(uint64_t seed, uint64_t j, double z[4]) {
  uint32_t ctr[4] = {(uint32_t)j, (uint32_t)(j >> 32), 0u, 0u};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t w[4];
  synth_philox4x32_10(ctr, key, w);
  const double two_pi = 6.283185307179586476925286766559;
  double r0 = sqrt(-2.0 * log(u01(w[0]))), t0 = two_pi * u01(w[1]);
  double r1 = sqrt(-2.0 * log(u01(w[2]))), t1 = two_pi * u01(w[3]);
  z[0] = r0 * cos(t0); z[1] = r0 * sin(t0);
  z[2] = r1 * cos(t1); z[3] = r1 * sin(t1);
}

/* float32 -> bfloat16 bits, round to nearest even (inputs are finite). */
static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7FFFu + lsb;
  return (uint16_t)(u >> 16);
}

/* out[i] = (float)(mean + std * z_{offset+i}) for i in [0, n). */
void synth_normal_f32(uint64_t seed, uint64_t offset, uint64_t n, float mean, float std, float *out) {
  if (n == 0) return;
  uint64_t first = offset / 4, last = (offset + n - 1) / 4;
  #pragma omp parallel for schedule(static)
  for (int64_t jj = (int64_t)first; jj <= (int64_t)last; ++jj) {
    double z[4];
    block_normals(seed, (uint64_t)jj, z);
    for (int q = 0; q < 4; ++q) {
      uint64_t e = (uint64_t)jj * 4 + q;
      if (e < offset || e >= offset + n) continue;
      out[e - offset] = (float)mean + std * (float)z[q];
    }
  }
}

/* Same values as synth_normal_f32, each rounded to bfloat16 (RNE); bits out. */
void synth_normal_bf16(uint64_t seed, uint64_t offset, uint64_t n, float mean, float std, uint16_t *out) {
  if (n == 0) return;
  uint64_t first = offset / 4, last = (offset + n - 1) / 4;
  #pragma omp parallel for schedule(static)
  for (int64_t jj = (int64_t)first; jj <= (int64_t)last; ++jj) {
    double z[4];
    block_normals(seed, (uint64_t)jj, z);
    for (int q = 0; q < 4; ++q) {
      uint64_t e = (uint64_t)jj * 4 + q;
      if (e < offset || e >= offset + n) continue;
      out[e - offset] = f32_to_bf16_rne((float)mean + std * (float)z[q]);
    }
  }
}

/* Uniform in [lo, hi) as float32, for perturbed norm gains; u in (0,1] maps to (lo, hi]. */
void synth_uniform_f32(uint64_t seed, uint64_t offset, uint64_t n, float lo, float hi, float *out) {
  if (n == 0) return;
  uint64_t first = offset / 4, last = (offset + n - 1) / 4;
  #pragma omp parallel for schedule(static)
  for (int64_t jj = (int64_t)first; jj <= (int64_t)last; ++jj) {
    uint32_t ctr[4] = {(uint32_t)jj, (uint32_t)((uint64_t)jj >> 32), 0u, 0u};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[4];
    synth_philox4x32_10(ctr, key, w);
    for (int q = 0; q < 4; ++q) {
      uint64_t e = (uint64_t)jj * 4 + q;
      if (e < offset || e >= offset + n) continue;
      out[e - offset] = (float)((double)lo + ((double)hi - (double)lo) * u01(w[q]));
    }
  }
}

/* bfloat16 bits -> float32 (exact). */
void synth_bf16_to_f32(const uint16_t *in, uint64_t n, float *out) {
  #pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)n; ++i) {
    uint32_t u = (uint32_t)in[i] << 16;
    memcpy(&out[i], &u, 4);
  }
}

void synth_f32_to_bf16(const float *in, uint64_t n, uint16_t *out) {
  #pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)n; ++i) out[i] = f32_to_bf16_rne(in[i]);
}
