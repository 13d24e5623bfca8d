/*
 * synth.c -- seeded, counter-based synthetic inputs (gradients and word streams).
 *
 * This module holds no arithmetic of the compression method: it only draws random
 * numbers. Both the CPU oracle and the GPU library are fed from the buffers it fills,
 * so they see bit-identical inputs.
 *
 * Generator: SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014), used counter-style:
 *   key  K = mix(mix(mix(seed ^ tag) ^ step) ^ worker)
 *   word w(K, n) = mix(K + (n + 1) * GOLDEN)
 *   uniform U = ((w >> 11) + 0.5) * 2^-53, in (0, 1)
 * Every transform runs in double precision and is rounded once to float.
 * Element n of a stream depends only on (K, n), so OpenMP threads can fill any range
 * in any order and produce the same bytes.
 */
#include <math.h>
#include <stdint.h>

#define SYN_GOLDEN 0x9E3779B97F4A7C15ULL
#define SYN_TWO_PI 6.283185307179586476925286766559

uint64_t synth_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t synth_key(uint64_t seed, uint64_t tag, uint64_t step, uint64_t worker) {
  return synth_mix(synth_mix(synth_mix(seed ^ tag) ^ step) ^ worker);
}

static inline uint64_t word_at(uint64_t key, uint64_t n) { return synth_mix(key + (n + 1) * SYN_GOLDEN); }

static inline double unif(uint64_t w) { return ((double)(w >> 11) + 0.5) * 0x1.0p-53; }

/* Box-Muller pair from words (2m, 2m+1); returns the cosine branch in *z0, sine in *z1. */
static inline void normal_pair(uint64_t key, uint64_t m, double* z0, double* z1) {
  double u1 = unif(word_at(key, 2 * m)), u2 = unif(word_at(key, 2 * m + 1));
  double rad = sqrt(-2.0 * log(u1));
  *z0 = rad * cos(SYN_TWO_PI * u2);
  *z1 = rad * sin(SYN_TWO_PI * u2);
}

/* Student-t with 3 degrees of freedom for element n: Z / sqrt((Z1^2 + Z2^2 + Z3^2) / 3),
 * the four normals taken from words 4n .. 4n+3. */
static inline double student_t3(uint64_t key, uint64_t n) {
  double z, z1, z2, z3;
  normal_pair(key, 2 * n, &z, &z1);
  normal_pair(key, 2 * n + 1, &z2, &z3);
  return z / sqrt((z1 * z1 + z2 * z2 + z3 * z3) / 3.0);
}

/* Laplace(0, 1) for element n from word n: -sgn(U - 1/2) * ln(1 - 2 |U - 1/2|). */
static inline double laplace1(uint64_t key, uint64_t n) {
  double x = unif(word_at(key, n)) - 0.5;
  double s = x < 0 ? -1.0 : 1.0;
  return -s * log(1.0 - 2.0 * fabs(x));
}

/* Standard normal for element n from words (2n, 2n+1), cosine branch. */
static inline double normal1(uint64_t key, uint64_t n) {
  double z0, z1;
  normal_pair(key, n, &z0, &z1);
  return z0;
}

enum { SYN_STUDENT_T3 = 0, SYN_LAPLACE = 1, SYN_NORMAL = 2 };

static inline double draw(int kind, uint64_t key, uint64_t n) {
  if (kind == SYN_STUDENT_T3) return student_t3(key, n);
  if (kind == SYN_LAPLACE) return laplace1(key, n);
  return normal1(key, n);
}

/*
 * Fill out[0 .. n) with scale_s * X_n for the piecewise-constant scale given by segments:
 * elements [seg_start[s], seg_start[s+1]) use seg_scale[s]; seg_start[0] == 0 and
 * seg_start[nseg] == n. A segment with scale 0 is filled with exact zeros (no draw).
 * X_n is drawn with counter n (the element's own index), so a sub-range is reproducible.
 */
int synth_fill(int kind, uint64_t key, int64_t n, int64_t nseg, const int64_t* seg_start,
               const double* seg_scale, float* out) {
  if (n < 0 || nseg < 1 || seg_start[0] != 0 || seg_start[nseg] != n) return 1;
  for (int64_t s = 0; s < nseg; ++s) {
    if (seg_start[s + 1] < seg_start[s]) return 1;
  }
  for (int64_t s = 0; s < nseg; ++s) {
    const int64_t lo = seg_start[s], hi = seg_start[s + 1];
    const double sc = seg_scale[s];
    if (sc == 0.0) {
#pragma omp parallel for schedule(static)
      for (int64_t t = lo; t < hi; ++t) out[t] = 0.0f;
      continue;
    }
#pragma omp parallel for schedule(static)
    for (int64_t t = lo; t < hi; ++t) out[t] = (float)(sc * draw(kind, key, (uint64_t)t));
  }
  return 0;
}

/* Double-precision draws at chosen element indices (used to re-draw a few coordinates
 * with a different scale before the single rounding). */
void synth_draw_at(int kind, uint64_t key, int64_t count, const int64_t* idx, double* out) {
  for (int64_t t = 0; t < count; ++t) out[t] = draw(kind, key, (uint64_t)idx[t]);
}

/* Raw 64-bit words n0 .. n0+count-1 of stream key. */
void synth_words(uint64_t key, int64_t n0, int64_t count, uint64_t* out) {
  for (int64_t t = 0; t < count; ++t) out[t] = word_at(key, (uint64_t)(n0 + t));
}
