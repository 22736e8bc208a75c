/*
 * Seeded synthetic-input generator: N(0,1) samples from a counter-based
 * generator, written as float32 or as bfloat16 bit patterns.
 *
 * Generator: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC 2011), followed by the Box-Muller
 * transform (Box and Muller, 1958). Element e of a stream is lane e%4 of the
 * Philox block with counter (e/4, stream); the key is the 64-bit seed. The
 * result therefore does not depend on how the work is split over threads.
 *
 * This file produces inputs only (weights, caches); it holds no step of the
 * decoding method. Build: gcc -O2 -fPIC -shared -pthread (no -ffast-math, no
 * FMA contraction, so the doubles below round the same way on every x86-64).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <string.h>

static inline void mulhilo32(uint32_t a, uint32_t b, uint32_t* hi, uint32_t* lo) {
  uint64_t p = (uint64_t)a * (uint64_t)b;
  *hi = (uint32_t)(p >> 32);
  *lo = (uint32_t)p;
}

/* Philox4x32 with 10 rounds; constants from the SC'11 paper. */
static void philox4x32_10(uint32_t ctr[4], uint32_t k0, uint32_t k1) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
  for (int r = 0; r < 10; ++r) {
    uint32_t hi0, lo0, hi1, lo1;
    mulhilo32(M0, ctr[0], &hi0, &lo0);
    mulhilo32(M1, ctr[2], &hi1, &lo1);
    uint32_t n0 = hi1 ^ ctr[1] ^ k0;
    uint32_t n2 = hi0 ^ ctr[3] ^ k1;
    ctr[0] = n0; ctr[1] = lo1; ctr[2] = n2; ctr[3] = lo0;
    k0 += W0; k1 += W1;
  }
}

/* Four N(0,1) doubles for block `blk` of stream `stream` under key `seed`. */
static void normal4(uint64_t seed, uint64_t stream, uint64_t blk, double out[4]) {
  uint32_t c[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), (uint32_t)stream, (uint32_t)(stream >> 32)};
  philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
  const double two_pi = 6.283185307179586476925286766559;
  const double inv32 = 1.0 / 4294967296.0;
  for (int j = 0; j < 2; ++j) {
    double u1 = ((double)c[2 * j] + 1.0) * inv32;  /* (0, 1] */
    double u2 = (double)c[2 * j + 1] * inv32;      /* [0, 1) */
    double rad = sqrt(-2.0 * log(u1));
    out[2 * j] = rad * cos(two_pi * u2);
    out[2 * j + 1] = rad * sin(two_pi * u2);
  }
}

/* float32 -> bfloat16 bit pattern, round to nearest even (inputs are finite). */
static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

typedef struct {
  uint64_t seed, stream;
  double scale;
  int64_t begin, end; /* element range */
  float* out_f32;
  uint16_t* out_bf16;
} job_t;

static void* run_job(void* arg) {
  job_t* j = (job_t*)arg;
  double z[4];
  int64_t e = j->begin;
  while (e < j->end) {
    int64_t blk = e >> 2;
    normal4(j->seed, j->stream, (uint64_t)blk, z);
    for (int lane = (int)(e & 3); lane < 4 && e < j->end; ++lane, ++e) {
      float v = (float)(z[lane] * j->scale);
      if (j->out_f32) j->out_f32[e] = v;
      else j->out_bf16[e] = f32_to_bf16_rne(v);
    }
  }
  return 0;
}

static void run(uint64_t seed, uint64_t stream, double scale, int64_t n, float* of, uint16_t* ob,
                int nthreads) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if (n < (int64_t)1 << 16) nthreads = 1;
  pthread_t th[256];
  job_t jobs[256];
  int64_t chunk = ((n + nthreads - 1) / nthreads + 3) & ~(int64_t)3;
  int started = 0;
  for (int t = 0; t < nthreads; ++t) {
    int64_t b = (int64_t)t * chunk, e = b + chunk;
    if (b >= n) break;
    if (e > n) e = n;
    jobs[t] = (job_t){seed, stream, scale, b, e, of, ob};
    if (t == nthreads - 1 || pthread_create(&th[t], 0, run_job, &jobs[t]) != 0) {
      run_job(&jobs[t]);
      th[t] = 0;
    }
    started = t + 1;
  }
  for (int t = 0; t < started; ++t)
    if (th[t]) pthread_join(th[t], 0);
}

void synth_normal_f32(uint64_t seed, uint64_t stream, double scale, float* out, int64_t n, int nthreads) {
  run(seed, stream, scale, n, out, 0, nthreads);
}

void synth_normal_bf16(uint64_t seed, uint64_t stream, double scale, uint16_t* out, int64_t n,
                       int nthreads) {
  run(seed, stream, scale, n, 0, out, nthreads);
}
