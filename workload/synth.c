/*
 * Seeded synthetic inputs shared by the oracle and the GPU path.
 *
 * Holds no arithmetic of the decoding method: it only turns (key, index)
 * into reproducible pseudo-random numbers.  Every value is a pure function
 * of (key, index), so the output does not depend on the thread count.
 *
 * Generator: the SplitMix64 output function (Steele, Lea and Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA 2014) applied
 * to a Weyl sequence key + c*i, i.e. a counter-based stream.  Normal
 * deviates use the Box-Muller transform (Box and Muller, 1958) in double
 * precision.
 */
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

/* Round a float to the nearest bfloat16 value (ties to even); NaN is not
 * produced by this generator. Returns the 16 high bits. */
static inline uint16_t f32_to_bf16_bits(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* Normal pair number p of stream `key`. */
static inline void normal_pair(uint64_t key, uint64_t p, double* z0, double* z1) {
  uint64_t r = mix64(key + GOLDEN * (p + 1));
  double u1 = ((double)(r >> 32) + 0.5) * (1.0 / 4294967296.0); /* (0,1) */
  double u2 = (double)(r & 0xFFFFFFFFu) * (1.0 / 4294967296.0); /* [0,1) */
  double rad = sqrt(-2.0 * log(u1));
  double th = 6.283185307179586476925286766559 * u2;
  *z0 = rad * cos(th);
  *z1 = rad * sin(th);
}

typedef struct {
  uint64_t key;
  double std;
  int mode; /* 0: float32, 1: float32 rounded to bf16 values, 2: bf16 bits */
  void* out;
  int64_t begin, end; /* element range, begin even */
} job_t;

static void emit(const job_t* j, int64_t i, double z) {
  float f = (float)(z * j->std);
  if (j->mode == 0) {
    ((float*)j->out)[i] = f;
  } else {
    uint16_t b = f32_to_bf16_bits(f);
    if (j->mode == 1) {
      uint32_t u = (uint32_t)b << 16;
      memcpy(&((float*)j->out)[i], &u, 4);
    } else {
      ((uint16_t*)j->out)[i] = b;
    }
  }
}

static void* run_normal(void* arg) {
  const job_t* j = (const job_t*)arg;
  for (int64_t i = j->begin; i < j->end; i += 2) {
    double z0, z1;
    normal_pair(j->key, (uint64_t)(i >> 1), &z0, &z1);
    emit(j, i, z0);
    if (i + 1 < j->end) emit(j, i + 1, z1);
  }
  return 0;
}

/* Fill out[0..n) with N(0, std^2) deviates of stream `key`. */
int synth_normal(uint64_t key, double std, int mode, void* out, int64_t n, int nthreads) {
  if (n <= 0) return 0;
  if (mode < 0 || mode > 2) return -1;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 64) nthreads = 64;
  if (n < (1 << 20)) nthreads = 1;
  pthread_t th[64];
  int made[64];
  job_t jobs[64];
  int64_t per = ((n + nthreads - 1) / nthreads + 1) & ~(int64_t)1; /* even */
  for (int t = 0; t < nthreads; ++t) {
    int64_t b = (int64_t)t * per, e = b + per;
    if (b > n) b = n;
    if (e > n) e = n;
    jobs[t] = (job_t){key, std, mode, out, b, e};
    made[t] = pthread_create(&th[t], 0, run_normal, &jobs[t]) == 0;
    if (!made[t]) run_normal(&jobs[t]);
  }
  for (int t = 0; t < nthreads; ++t)
    if (made[t]) pthread_join(th[t], 0);
  return 0;
}

/* Uniform integers in [0, hi) of stream `key` (plain modulo reduction
 * of a 64-bit draw; the bias is below 2^-40 for hi < 2^24). */
int synth_uniform_int(uint64_t key, int64_t hi, int32_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i)
    out[i] = (int32_t)(mix64(key + GOLDEN * (uint64_t)(i + 1)) % (uint64_t)hi);
  return 0;
}

/* Uniform doubles in [0, 1) of stream `key`. */
int synth_uniform_f64(uint64_t key, double* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i)
    out[i] = (double)(mix64(key + GOLDEN * (uint64_t)(i + 1)) >> 11) * (1.0 / 9007199254740992.0);
  return 0;
}
