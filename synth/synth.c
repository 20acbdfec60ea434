/*
 * Seeded synthetic inputs for batched monotonic alignment search.
 *
 * This module holds no arithmetic of the alignment method itself: it only
 * produces the log-likelihood matrices and lengths that both the HIP library
 * and the CPU oracle consume.
 *
 * Random numbers: SplitMix64 (Steele, Lea, Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), the 64-bit variant with the
 * golden-gamma increment and the published 30/27/31 mixer.  Uniform doubles
 * take the top 53 bits.  Normals use the Box-Muller transform in double, the
 * cosine output first and the sine output second.
 *
 * Gaussian log-likelihood (the quantity MAS aligns, a diagonal unit-variance
 * Gaussian per text token evaluated at every speech frame):
 *   value[i][j] = -0.5 * sum_{d ascending} (x[j][d] - mu[i][d])^2 - (D/2) ln(2 pi)
 * evaluated in double with no contraction, then rounded once to fp32.
 *
 * Build: gcc -O3 -ffp-contract=off -fno-fast-math -fopenmp; results do not
 * depend on the thread count (each cell is summed by one thread, in order).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>

static uint64_t splitmix64_next(uint64_t* s) {
  uint64_t z = (*s += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* Uniform in [0, 1) from the top 53 bits. */
static double uniform01(uint64_t* s) { return (double)(splitmix64_next(s) >> 11) * 0x1.0p-53; }

/* n raw 64-bit draws (for tests of the generator itself). */
void synth_raw(uint64_t* state, uint64_t* out, size_t n) {
  for (size_t k = 0; k < n; ++k) out[k] = splitmix64_next(state);
}

/* Inclusive integer draw a + (x mod (b - a + 1)); the modulo bias is below
 * 2^-40 for the ranges used here. */
void synth_randint(uint64_t* state, int32_t lo, int32_t hi, int32_t* out, size_t n) {
  uint64_t span = (uint64_t)((int64_t)hi - (int64_t)lo + 1);
  for (size_t k = 0; k < n; ++k) out[k] = (int32_t)((int64_t)lo + (int64_t)(splitmix64_next(state) % span));
}

/* n standard normals (double).  Pairs come from one Box-Muller step; for odd
 * n the sine half of the last pair is discarded. */
void synth_normal(uint64_t* state, double* out, size_t n) {
  const double two_pi = 6.283185307179586476925286766559;
  size_t k = 0;
  while (k < n) {
    double u1 = 1.0 - uniform01(state); /* (0, 1] so the log is finite */
    double u2 = uniform01(state);
    double r = sqrt(-2.0 * log(u1));
    double a = two_pi * u2;
    out[k++] = r * cos(a);
    if (k < n) out[k++] = r * sin(a);
  }
}

/* Round doubles to fp32 (round to nearest even). */
void synth_to_f32(const double* in, float* out, size_t n) {
  for (size_t k = 0; k < n; ++k) out[k] = (float)in[k];
}

/*
 * Gaussian log-likelihood slab: mu [T, D], x [S, D] (double, row-major),
 * out [T, S] fp32 with row stride S.  For every (i, j) the D squared
 * differences are accumulated in double with d ascending; x is first copied
 * to a [D, S] layout so the inner loop runs over contiguous frames (the order
 * of the additions per cell is unchanged).  Returns -1 on allocation failure.
 */
int synth_gauss_loglik(const double* mu, const double* x, int32_t T, int32_t S, int32_t D, float* out) {
  const double half_log_two_pi = 0.91893853320467274178032973640562; /* ln(2 pi) / 2 */
  const double c = (double)D * half_log_two_pi;
  double* xt = (double*)malloc((size_t)D * (size_t)S * sizeof(double));
  if (!xt) return -1;
  for (int32_t j = 0; j < S; ++j)
    for (int32_t d = 0; d < D; ++d) xt[(size_t)d * (size_t)S + (size_t)j] = x[(size_t)j * (size_t)D + (size_t)d];
#pragma omp parallel
  {
    double acc[512];
#pragma omp for schedule(static)
    for (int32_t i = 0; i < T; ++i) {
      const double* m = mu + (size_t)i * (size_t)D;
      for (int32_t j0 = 0; j0 < S; j0 += 512) {
        int32_t nj = S - j0 < 512 ? S - j0 : 512;
        for (int32_t jj = 0; jj < nj; ++jj) acc[jj] = 0.0;
        for (int32_t d = 0; d < D; ++d) {
          const double md = m[d];
          const double* xr = xt + (size_t)d * (size_t)S + (size_t)j0;
          for (int32_t jj = 0; jj < nj; ++jj) {
            double t = xr[jj] - md;
            acc[jj] = acc[jj] + t * t;
          }
        }
        float* o = out + (size_t)i * (size_t)S + (size_t)j0;
        for (int32_t jj = 0; jj < nj; ++jj) o[jj] = (float)(-0.5 * acc[jj] - c);
      }
    }
  }
  free(xt);
  return 0;
}
