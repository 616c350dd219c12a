/*
 * Seeded synthetic inputs shared by the CPU oracle's tests and the GPU path.
 *
 * This module holds no part of the stage's arithmetic: it only turns
 * (seed, config, stream, layer, kind, element index) into numbers.  Every
 * element is a pure function of its coordinates (a counter-based generator),
 * so any slice of any tensor can be regenerated alone, in any order and on
 * any number of threads, with identical bits.
 *
 *   word(key, i)  = splitmix64_mix(key + (i + 1) * 0x9E3779B97F4A7C15)
 *     (the SplitMix64 output function of Steele, Lea and Flood,
 *      "Fast splittable pseudorandom number generators", OOPSLA 2014)
 *   key           = chain of splitmix64_mix over the five coordinates
 *   normal pair   = Box-Muller (1958) on the top two 24-bit fields of word:
 *                   u1 = (w >> 40 + 0.5) 2^-24, u2 = ((w >> 16) & 0xFFFFFF + 0.5) 2^-24
 *                   z0 = sqrt(-2 ln u1) cos(2 pi u2), z1 = sqrt(-2 ln u1) sin(2 pi u2)
 *                   element 2j takes z0 of word j, element 2j+1 takes z1
 *   uniform int   = (word >> 11) mod n   (for token ids; bias < 2^-40 for n < 2^13..2^17)
 *
 * Normals are evaluated in double precision and stored either as fp32 or as
 * bf16 bit patterns (mean + std * z, rounded to nearest even).
 */
#define _GNU_SOURCE
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t synth_key(uint64_t seed, int64_t a, int64_t b, int64_t c, int64_t d) {
  uint64_t k = mix64(seed + GOLDEN);
  k = mix64(k + GOLDEN * (uint64_t)(a + 1));
  k = mix64(k + GOLDEN * (uint64_t)(b + 1));
  k = mix64(k + GOLDEN * (uint64_t)(c + 2)); /* layer may be -1 for head tensors */
  k = mix64(k + GOLDEN * (uint64_t)(d + 1));
  return k;
}

static inline uint64_t word(uint64_t key, uint64_t j) { return mix64(key + (j + 1) * GOLDEN); }

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFF) ? 0x40 : 0));
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

typedef struct {
  uint64_t key, i0, i1;
  double mean, std;
  void* out;
  int kind; /* 0 bf16, 1 f32, 2 int32 uniform */
  int64_t modulus;
} job_t;

static inline void normal_pair(uint64_t key, uint64_t j, double* z0, double* z1) {
  uint64_t w = word(key, j);
  double u1 = ((double)(w >> 40) + 0.5) * (1.0 / 16777216.0);
  double u2 = ((double)((w >> 16) & 0xFFFFFFULL) + 0.5) * (1.0 / 16777216.0);
  double r = sqrt(-2.0 * log(u1));
  double t = 6.283185307179586476925286766559 * u2;
  double s, c;
  sincos(t, &s, &c);
  *z0 = r * c;
  *z1 = r * s;
}

static void* run_job(void* p) {
  job_t* j = (job_t*)p;
  if (j->kind == 2) {
    int32_t* o = (int32_t*)j->out;
    for (uint64_t i = j->i0; i < j->i1; ++i) o[i] = (int32_t)((word(j->key, i) >> 11) % (uint64_t)j->modulus);
    return 0;
  }
  for (uint64_t i = j->i0 & ~1ULL; i < j->i1; i += 2) {
    double z[2];
    normal_pair(j->key, i >> 1, &z[0], &z[1]);
    for (int h = 0; h < 2; ++h) {
      uint64_t e = i + h;
      if (e < j->i0 || e >= j->i1) continue;
      double v = j->mean + j->std * z[h];
      if (j->kind == 0) ((uint16_t*)j->out)[e] = f32_to_bf16_rne((float)v);
      else ((float*)j->out)[e] = (float)v;
    }
  }
  return 0;
}

static void run(uint64_t key, int64_t n, double mean, double std, void* out, int kind, int64_t modulus, int threads) {
  if (n <= 0) return;
  if (threads < 1) threads = 1;
  if (threads > 64) threads = 64;
  if (n < (int64_t)1 << 16) threads = 1;
  job_t jobs[64];
  pthread_t th[64];
  uint64_t chunk = ((uint64_t)n + threads - 1) / threads;
  chunk = (chunk + 1) & ~1ULL; /* keep normal pairs inside one job */
  int used = 0;
  for (int t = 0; t < threads; ++t) {
    uint64_t a = (uint64_t)t * chunk, b = a + chunk;
    if (a >= (uint64_t)n) break;
    if (b > (uint64_t)n) b = (uint64_t)n;
    jobs[t] = (job_t){key, a, b, mean, std, out, kind, modulus};
    used++;
  }
  for (int t = 1; t < used; ++t) pthread_create(&th[t], 0, run_job, &jobs[t]);
  run_job(&jobs[0]);
  for (int t = 1; t < used; ++t) pthread_join(th[t], 0);
}

/* out[i] = bf16(mean + std * N_i) for i in [0, n) */
void synth_normal_bf16(uint64_t key, int64_t n, double mean, double std, uint16_t* out, int threads) {
  run(key, n, mean, std, out, 0, 0, threads);
}

/* out[i] = float(mean + std * N_i) */
void synth_normal_f32(uint64_t key, int64_t n, double mean, double std, float* out, int threads) {
  run(key, n, mean, std, out, 1, 0, threads);
}

/* out[i] = uniform integer in [0, modulus) */
void synth_uniform_i32(uint64_t key, int64_t n, int64_t modulus, int32_t* out, int threads) {
  run(key, n, 0.0, 0.0, out, 2, modulus, threads);
}
