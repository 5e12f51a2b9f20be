/*
 * Seeded synthetic inputs shared by the oracle and the GPU tests/bench.
 *
 * This file holds no arithmetic of the decoding method: it only turns
 * (seed, stream, index) triples into random numbers and stores them in
 * the caller's buffers.  Every value is a pure function of its index,
 * so OpenMP chunking never changes the output.
 *
 * Generator: Philox4x32-10, the counter-based generator of Salmon,
 * Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3"
 * (SC'11).  One block (counter, key) yields four 32-bit words:
 *   counter = (j_lo, j_hi, stream, 0x5EED5EED), key = (seed_lo, seed_hi)
 * where j is the block index.  Element i of a stream uses word i % 4 of
 * block i / 4.  Normals use the Box-Muller transform on word pairs
 * (w0, w1) and (w2, w3), computed in double precision.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u
#define SYNTH_TAG 0x5EED5EEDu

static inline void mulhilo32(uint32_t a, uint32_t b, uint32_t* hi, uint32_t* lo) {
  uint64_t p = (uint64_t)a * (uint64_t)b;
  *hi = (uint32_t)(p >> 32);
  *lo = (uint32_t)p;
}

/* Philox4x32 with R rounds; exported for known-answer tests. */
void synth_philox4x32(const uint32_t ctr_in[4], const uint32_t key_in[2], int rounds,
                      uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int r = 0; r < rounds; ++r) {
    uint32_t hi0, lo0, hi1, lo1;
    mulhilo32(PHILOX_M0, c0, &hi0, &lo0);
    mulhilo32(PHILOX_M1, c2, &hi1, &lo1);
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

static inline void block4(uint64_t seed, uint32_t stream, uint64_t j, uint32_t w[4]) {
  uint32_t ctr[4] = {(uint32_t)j, (uint32_t)(j >> 32), stream, SYNTH_TAG};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  synth_philox4x32(ctr, key, 10, w);
}

/* uniform in the open interval (0, 1) from one 32-bit word */
static inline double u01(uint32_t w) { return ((double)w + 0.5) * (1.0 / 4294967296.0); }

static inline void box_muller(uint32_t a, uint32_t b, double* z0, double* z1) {
  double r = sqrt(-2.0 * log(u01(a)));
  double t = 6.283185307179586476925286766559 * u01(b);
  *z0 = r * cos(t);
  *z1 = r * sin(t);
}

/* round-to-nearest-even float -> bfloat16 bit pattern (storage conversion) */
static inline uint16_t f32_to_bf16_bits(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u); /* NaN */
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

static inline double normal_at(uint64_t seed, uint32_t stream, uint64_t i) {
  uint32_t w[4];
  block4(seed, stream, i >> 2, w);
  double z0, z1;
  unsigned q = (unsigned)(i & 3);
  if (q < 2) box_muller(w[0], w[1], &z0, &z1);
  else box_muller(w[2], w[3], &z0, &z1);
  return (q & 1) ? z1 : z0;
}

/* four consecutive normals of block j (elements 4j .. 4j+3) */
static inline void normal_block(uint64_t seed, uint32_t stream, uint64_t j, double z[4]) {
  uint32_t w[4];
  block4(seed, stream, j, w);
  box_muller(w[0], w[1], &z[0], &z[1]);
  box_muller(w[2], w[3], &z[2], &z[3]);
}

/* out[i] = mean + std * N(0,1)_{start+i}, i < n, stored as float32 */
void synth_normal_f32(uint64_t seed, uint32_t stream, uint64_t start, uint64_t n, double mean,
                      double std, float* out) {
  if (n == 0) return;
  int64_t j0 = (int64_t)(start >> 2), j1 = (int64_t)((start + n - 1) >> 2);
#pragma omp parallel for schedule(static)
  for (int64_t j = j0; j <= j1; ++j) {
    double z[4];
    normal_block(seed, stream, (uint64_t)j, z);
    for (int q = 0; q < 4; ++q) {
      uint64_t e = ((uint64_t)j << 2) + (uint64_t)q;
      if (e >= start && e < start + n) out[e - start] = (float)(mean + std * z[q]);
    }
  }
}

/* same values as synth_normal_f32, then rounded (RNE) to bfloat16 bits */
void synth_normal_bf16(uint64_t seed, uint32_t stream, uint64_t start, uint64_t n, double mean,
                       double std, uint16_t* out) {
  if (n == 0) return;
  int64_t j0 = (int64_t)(start >> 2), j1 = (int64_t)((start + n - 1) >> 2);
#pragma omp parallel for schedule(static)
  for (int64_t j = j0; j <= j1; ++j) {
    double z[4];
    normal_block(seed, stream, (uint64_t)j, z);
    for (int q = 0; q < 4; ++q) {
      uint64_t e = ((uint64_t)j << 2) + (uint64_t)q;
      if (e >= start && e < start + n)
        out[e - start] = f32_to_bf16_bits((float)(mean + std * z[q]));
    }
  }
}

/* out[i] uniform integer in [lo, lo + span) by 32x32 multiply-shift */
void synth_uniform_int(uint64_t seed, uint32_t stream, uint64_t n, int64_t lo, uint32_t span,
                       int32_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)n; ++i) {
    uint32_t w[4];
    block4(seed, stream, (uint64_t)i >> 2, w);
    uint32_t x = w[i & 3];
    out[i] = (int32_t)(lo + (int64_t)(((uint64_t)x * (uint64_t)span) >> 32));
  }
}

/* out[i] uniform double in (0, 1) */
void synth_uniform_f64(uint64_t seed, uint32_t stream, uint64_t n, double* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)n; ++i) {
    uint32_t w[4];
    block4(seed, stream, (uint64_t)i >> 2, w);
    out[i] = u01(w[i & 3]);
  }
}

/* single normal draw, for spot checks */
double synth_normal_at(uint64_t seed, uint32_t stream, uint64_t i) {
  return normal_at(seed, stream, i);
}
