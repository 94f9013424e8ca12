/*
 * Seeded synthetic-input generator shared by the CPU oracle and the GPU path.
 *
 * It produces random numbers only: normal and uniform variates addressed by a
 * (seed, stream, index) counter, so any element of any tensor can be
 * regenerated independently and in parallel.  It holds none of the decoding
 * method's arithmetic (no forward pass, no selection rule): the callers turn
 * these numbers into weights, prompts and planted drafts.
 *
 * Counter-based source: SplitMix64 (Steele, Lea & Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014).  Output n (1-based) of the
 * SplitMix64 stream seeded with s is mix(s + n * 0x9E3779B97F4A7C15).  Here a
 * (seed, stream) pair selects the stream s = mix(seed ^ mix(stream)) and the
 * element index selects n.
 *
 * Normal variates: Box-Muller transform on two 53-bit uniforms.
 * bf16 output: round-to-nearest-even of the fp32 value.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC gen.c -o libsynth.so -lm
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
  return sm_mix(seed ^ sm_mix(stream + GOLDEN));
}

/* n-th (0-based) 64-bit output of the stream. */
static inline uint64_t draw(uint64_t key, uint64_t n) {
  return sm_mix(key + (n + 1) * GOLDEN);
}

static inline double u53(uint64_t r) { /* (0, 1] */
  return ((double)(r >> 11) + 1.0) * (1.0 / 9007199254740992.0);
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static inline double normal_at(uint64_t key, uint64_t i) {
  /* pair index i/2 -> two uniforms -> (cos, sin) branch by parity */
  uint64_t pr = i >> 1;
  double a = u53(draw(key, 2 * pr));
  double b = u53(draw(key, 2 * pr + 1));
  double rad = sqrt(-2.0 * log(a));
  double th = 6.283185307179586476925 * b;
  return (i & 1) ? rad * sin(th) : rad * cos(th);
}

/* raw 64-bit draws: out[i] = draw(stream, i0 + i) */
void synth_u64(uint64_t seed, uint64_t stream, uint64_t i0, int64_t n, uint64_t* out) {
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = draw(key, i0 + (uint64_t)i);
}

/* mean + std * N(0,1), written as fp32 */
void synth_normal_f32(uint64_t seed, uint64_t stream, double mean, double std, int64_t n, float* out) {
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = (float)(mean + std * normal_at(key, (uint64_t)i));
}

/* mean + std * N(0,1), rounded to fp32 then to bf16 (RNE), written as raw bits */
void synth_normal_bf16(uint64_t seed, uint64_t stream, double mean, double std, int64_t n, uint16_t* out) {
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = f32_to_bf16_rne((float)(mean + std * normal_at(key, (uint64_t)i)));
}

/* uniform integers in [lo, hi) (multiply-shift on the top 32 bits; hi-lo < 2^31) */
void synth_randint(uint64_t seed, uint64_t stream, int32_t lo, int32_t hi, int64_t n, int32_t* out) {
  uint64_t key = stream_key(seed, stream);
  uint64_t span = (uint64_t)(hi - lo);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = lo + (int32_t)(((draw(key, (uint64_t)i) >> 32) * span) >> 32);
}

/* uniform doubles in [0, 1) with 53 bits */
void synth_uniform(uint64_t seed, uint64_t stream, int64_t n, double* out) {
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = (double)(draw(key, (uint64_t)i) >> 11) * (1.0 / 9007199254740992.0);
}
