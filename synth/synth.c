/*
 * Seeded synthetic inputs shared by the CPU oracle and the HIP path.
 *
 * This file holds no arithmetic of the decoding method: it only turns
 * (seed, tensor id, element index) into numbers, using one splitmix64 output
 * (Steele, Lea & Flood, "Fast splittable pseudorandom number generators",
 * OOPSLA 2014) of the counter  (seed << 48) | (tid << 36) | j , so any element
 * can be produced on its own and in parallel.
 *   - normal: elements 2j and 2j+1 share the output for counter j: two 24-bit
 *     uniforms feed Box-Muller in float64 (cosine branch for the even element,
 *     sine branch for the odd one); sigma * n is rounded to float32, then to
 *     bfloat16 (round to nearest even).
 *   - ids: element j is the output for counter j, mod V.
 * Limits: seed < 2^16, tid < 2^12, i < 2^36.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static inline uint64_t sm64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t counter(uint32_t seed, uint32_t tid, uint64_t i) {
  return ((uint64_t)seed << 48) | ((uint64_t)tid << 36) | i;
}

static inline void std_normal_pair(uint64_t x, double* c, double* s) {
  const double two24 = 16777216.0;
  double u1 = ((double)(x >> 40) + 0.5) / two24;
  double u2 = ((double)((x >> 16) & 0xFFFFFFULL) + 0.5) / two24;
  double r = sqrt(-2.0 * log(u1));
  double a = 6.283185307179586 * u2;
  *c = r * cos(a);
  *s = r * sin(a);
}

static inline double std_normal_at(uint32_t seed, uint32_t tid, uint64_t i) {
  double c, s;
  std_normal_pair(sm64(counter(seed, tid, i >> 1)), &c, &s);
  return (i & 1) ? s : c;
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* Elements [i0, i0 + n) of the tensor; pairs sharing a counter are drawn once. */
void synth_normal_bf16(uint16_t* out, uint64_t n, uint64_t i0, uint32_t seed,
                       uint32_t tid, double sigma) {
  uint64_t j0 = i0 >> 1, j1 = (i0 + n + 1) >> 1;
#pragma omp parallel for schedule(static)
  for (int64_t j = (int64_t)j0; j < (int64_t)j1; ++j) {
    double c, s;
    std_normal_pair(sm64(counter(seed, tid, (uint64_t)j)), &c, &s);
    uint64_t e = 2 * (uint64_t)j;
    if (e >= i0 && e < i0 + n) out[e - i0] = f32_to_bf16_rne((float)(sigma * c));
    if (e + 1 >= i0 && e + 1 < i0 + n) out[e + 1 - i0] = f32_to_bf16_rne((float)(sigma * s));
  }
}

void synth_normal_f32(float* out, uint64_t n, uint64_t i0, uint32_t seed,
                      uint32_t tid, double sigma) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)n; ++i)
    out[i] = (float)(sigma * std_normal_at(seed, tid, i0 + (uint64_t)i));
}

void synth_ids(int32_t* out, uint64_t n, uint64_t i0, uint32_t seed,
               uint32_t tid, uint32_t vocab) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)n; ++i)
    out[i] = (int32_t)(sm64(counter(seed, tid, i0 + (uint64_t)i)) % vocab);
}

/* Copy helper so Python can build weight buffers without extra passes. */
void synth_fill_bf16(uint16_t* out, uint64_t n, uint16_t bits) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)n; ++i) out[i] = bits;
}
