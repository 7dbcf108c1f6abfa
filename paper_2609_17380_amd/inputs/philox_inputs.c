/*
 * Seeded synthetic inputs for the canonical training step.
 *
 * This file holds only the input generator; none of the method's arithmetic.
 * Both the CPU oracle and the GPU library receive buffers produced here, so
 * neither side generates its own inputs.
 *
 * Generator: Philox4x32-10, the counter-based generator of Salmon, Moraes,
 * Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC'11).
 * The paper's reproducibility rules ask for a counter-based stream: each value
 * is a pure function of (seed, tensor id, element index), independent of how
 * the work is split across threads.
 *
 *   key     = (seed, tensor_id)
 *   counter = (block_lo, block_hi, 0, 0) where block = element_index / 4
 *   lane    = element_index % 4 picks one of the four 32-bit outputs
 *
 * Normals use Box-Muller in double on the two output pairs of a block:
 *   (x0, x1) -> lanes 0, 1 and (x2, x3) -> lanes 2, 3,
 *   u1 = (x_even + 1) * 2^-32 in (0, 1], u2 = x_odd * 2^-32 in [0, 1),
 *   rad = sqrt(-2 ln u1), even lane = rad cos(2 pi u2), odd lane = rad sin(2 pi u2).
 * The value mean + std * z is rounded to fp32 (round-to-nearest-even) and, for
 * bf16 outputs, that fp32 value is rounded to bf16 with round-to-nearest-even.
 * Uniform integers in [0, V): (x_lane * V) >> 32.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static inline void mulhilo(uint32_t a, uint32_t b, uint32_t* hi, uint32_t* lo) {
  uint64_t p = (uint64_t)a * (uint64_t)b;
  *hi = (uint32_t)(p >> 32);
  *lo = (uint32_t)p;
}

/* Ten rounds of Philox4x32 on ctr with key k; result written to out. */
void canon_in_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    uint32_t hi0, lo0, hi1, lo1;
    mulhilo(PHILOX_M0, c0, &hi0, &lo0);
    mulhilo(PHILOX_M1, c2, &hi1, &lo1);
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    uint32_t n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += PHILOX_W0;
    k1 += PHILOX_W1;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

static inline void block_words(uint64_t seed, uint32_t tid, uint64_t block, uint32_t w[4]) {
  uint32_t ctr[4] = {(uint32_t)block, (uint32_t)(block >> 32), 0u, 0u};
  uint32_t key[2] = {(uint32_t)seed ^ (uint32_t)(seed >> 32), tid};
  canon_in_philox4x32_10(ctr, key, w);
}

static inline double normal_of(const uint32_t w[4], int lane) {
  const double two_pi = 6.283185307179586476925286766559;
  int pair = lane >> 1;
  double u1 = ((double)w[2 * pair] + 1.0) * 0x1p-32;
  double u2 = (double)w[2 * pair + 1] * 0x1p-32;
  double rad = sqrt(-2.0 * log(u1));
  return (lane & 1) ? rad * sin(two_pi * u2) : rad * cos(two_pi * u2);
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u = u + 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* Elements [start, start + n) of the stream, written to out[0 .. n). */
void canon_in_normal_f32(uint64_t seed, uint32_t tid, uint64_t start, int64_t n, double mean, double std,
                         float* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    uint64_t e = start + (uint64_t)i;
    uint32_t w[4];
    block_words(seed, tid, e >> 2, w);
    out[i] = (float)(mean + std * normal_of(w, (int)(e & 3)));
  }
}

void canon_in_normal_bf16(uint64_t seed, uint32_t tid, uint64_t start, int64_t n, double mean, double std,
                          uint16_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    uint64_t e = start + (uint64_t)i;
    uint32_t w[4];
    block_words(seed, tid, e >> 2, w);
    out[i] = f32_to_bf16_rne((float)(mean + std * normal_of(w, (int)(e & 3))));
  }
}

void canon_in_uniform_int(uint64_t seed, uint32_t tid, uint64_t start, int64_t n, uint32_t bound, int32_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    uint64_t e = start + (uint64_t)i;
    uint32_t w[4];
    block_words(seed, tid, e >> 2, w);
    out[i] = (int32_t)(((uint64_t)w[e & 3] * (uint64_t)bound) >> 32);
  }
}
