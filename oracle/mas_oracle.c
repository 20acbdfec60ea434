/*
 * CPU oracle for batched Monotonic Alignment Search (MAS).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file: only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header, table or helper with
 * the HIP library; both sides only consume the same seeded inputs.
 *
 * What it computes (Super-MAS paper, Sec. 2 "Monotonic Alignment Search",
 * Algorithm 1 "Original Monotonic Alignment Search"):
 *   - a cache Q of maximum cumulative log-likelihoods, initialised to -inf;
 *   - the first text row of Q as the left-to-right running sum of q;
 *   - for every later speech column j and every text row i that a monotonic
 *     path can reach by column j (i <= j), Q[i][j] = max(Q[i-1][j-1],
 *     Q[i][j-1]) + q[i][j];
 *   - a backtrack that starts in the last text row at the last speech column
 *     and, column by column, keeps the row or moves one row up (towards row
 *     0), whichever of the two candidates holds the larger Q in the previous
 *     column;
 *   - the alignment A* as a 0/1 matrix of the input's size with exactly one 1
 *     per speech column (Sec. 2: the output has the input's size).
 *
 * Readings of points the paper leaves open (each is a decision of this
 * oracle, shared by the GPU path through the specification, not code):
 *   R1 backtrack tie: the paper's argmax over {A*(j+1)-1, A*(j+1)} does not
 *      say what happens on a tie.  We keep the row (stay) on ties and step
 *      up only when Q[i][j-1] is strictly below Q[i-1][j-1] (in the order of
 *      R2), or when i == j (the stay candidate is outside the reachable
 *      triangle).
 *   R2 max and argmax order values as IEEE 754-2019 maximum() does: the
 *      numeric order, with -0 below +0 (the paper's max leaves signed zeros
 *      open; this order defines the score's bits).  The forward max is
 *      (stay below diag) ? diag : stay.  NaN is outside the method's domain.
 *   R3 masked cells are IEEE -inf (the paper names -inf in Algorithm 1 and
 *      discusses finite stand-ins -1e9 / -1e32 in Sec. 2); a finite sentinel
 *      is kept only as a test knob to reproduce the -1e9 failure the paper
 *      describes.
 *   R4 the first-row formula in Algorithm 1 carries a garbled index; it is
 *      the prefix sum of text row 1 (0-based row 0), accumulated left to
 *      right in fp32.
 *   R5 Q[0][0] = q[0][0] with no "+0" (keeps a -0.0 input bit-exact).
 *   R6 0-based indices; lengths are per item, t_x text rows and t_y speech
 *      columns inside a [T, S] padded slab; padding is never read.
 *   R7 invalid lengths give an all-zero slab, score -inf and a status code.
 *
 * Arithmetic: fp32 adds in the stated order, round to nearest even.  Build
 * with -O2 -ffp-contract=off -fno-fast-math on x86-64 (SSE2, no x87).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* R2: a strictly below b (numeric order, -0 below +0). */
static int below(float a, float b) {
  return a < b || (a == 0.0f && b == 0.0f && signbit(a) && !signbit(b));
}

/* Per-item status codes (R7). */
#define ORACLE_ITEM_OK 0
#define ORACLE_ITEM_EMPTY 1
#define ORACLE_ITEM_INFEASIBLE 2
#define ORACLE_ITEM_OUT_OF_RANGE 3

static int item_status(int32_t tx, int32_t ty, int32_t T, int32_t S) {
  if (tx < 0 || ty < 0 || tx > T || ty > S) return ORACLE_ITEM_OUT_OF_RANGE;
  if (tx == 0 || ty == 0) return ORACLE_ITEM_EMPTY;
  if (ty < tx) return ORACLE_ITEM_INFEASIBLE;
  return ORACLE_ITEM_OK;
}

/*
 * One item.  q points at the item's [T, S] slab (row stride S); path at its
 * [T, S] output slab.  Q is scratch of tx*ty floats, stored column by
 * column.  neg is the value of masked cells (-INFINITY for the method; a
 * finite number only for the legacy-sentinel test).
 */
static void mas_one(const float* q, int32_t S, int32_t tx, int32_t ty, float neg,
                    float* Q, uint8_t* path, float* score) {
#define QC(i, j) Q[(size_t)(j) * (size_t)tx + (size_t)(i)] /* column-major: the inner loop runs over i */
#define QV(i, j) q[(size_t)(i) * (size_t)S + (size_t)(j)]
  /* Algorithm 1: initialise the cache to -inf (R3). */
  for (size_t k = 0; k < (size_t)tx * (size_t)ty; ++k) Q[k] = neg;

  /* Algorithm 1: first row, running sum over speech columns (R4, R5). */
  QC(0, 0) = QV(0, 0);
  for (int32_t j = 1; j < ty; ++j) QC(0, j) = QC(0, j - 1) + QV(0, j);

  /* Algorithm 1: forward loop, speech column outer, text row inner; the
   * inner bound min(j, T) keeps the cells a monotonic path can reach. */
  for (int32_t j = 1; j < ty; ++j) {
    int32_t imax = j < tx - 1 ? j : tx - 1;
    for (int32_t i = 1; i <= imax; ++i) {
      float stay = QC(i, j - 1);     /* neg when i == j: outside the triangle */
      float diag = QC(i - 1, j - 1);
      int take_diag = below(stay, diag); /* R2 */
      QC(i, j) = (take_diag ? diag : stay) + QV(i, j);
    }
  }

  /* Algorithm 1: backtrack from the last text row at the last speech column.
   * At column j the path sits in row idx; the row for column j-1 is idx-1
   * when that candidate's Q is strictly above (R2 order), or when idx == j (R1). */
  int32_t idx = tx - 1;
  for (int32_t j = ty - 1; j >= 0; --j) {
    path[(size_t)idx * (size_t)S + (size_t)j] = 1;
    if (j > 0 && idx > 0 && (idx == j || below(QC(idx, j - 1), QC(idx - 1, j - 1)))) idx -= 1;
  }
  *score = QC(tx - 1, ty - 1);
#undef QC
#undef QV
}

/*
 * Batched entry: value [B, T, S] fp32 row-major, t_x / t_y [B] int32,
 * path [B, T, S] u8 (fully overwritten), score [B] fp32 (nullable),
 * status [B] int32 (nullable).  neg: masked value.
 * Returns 0, or -1 on allocation failure.
 */
int oracle_mas_batch_neg(const float* value, int32_t B, int32_t T, int32_t S,
                         const int32_t* t_x, const int32_t* t_y, float neg,
                         uint8_t* path, float* score, int32_t* status) {
  size_t slab = (size_t)T * (size_t)S;
  memset(path, 0, (size_t)B * slab);
  for (int32_t b = 0; b < B; ++b) {
    int32_t tx = t_x[b], ty = t_y[b];
    int st = item_status(tx, ty, T, S);
    if (status) status[b] = st;
    if (st != ORACLE_ITEM_OK) {
      if (score) score[b] = -INFINITY;
      continue;
    }
    float* Q = (float*)malloc((size_t)tx * (size_t)ty * sizeof(float));
    if (!Q) return -1;
    float sc;
    mas_one(value + (size_t)b * slab, S, tx, ty, neg, Q, path + (size_t)b * slab, &sc);
    if (score) score[b] = sc;
    free(Q);
  }
  return 0;
}

int oracle_mas_batch(const float* value, int32_t B, int32_t T, int32_t S,
                     const int32_t* t_x, const int32_t* t_y,
                     uint8_t* path, float* score, int32_t* status) {
  return oracle_mas_batch_neg(value, B, T, S, t_x, t_y, -INFINITY, path, score, status);
}

/* Durations (frames per text token) of a path slab: the row sums of A*, the
 * quantity a duration predictor is trained on (Sec. 2). */
void oracle_durations(const uint8_t* path, int32_t B, int32_t T, int32_t S, int32_t* dur) {
  for (int32_t b = 0; b < B; ++b)
    for (int32_t i = 0; i < T; ++i) {
      const uint8_t* row = path + ((size_t)b * (size_t)T + (size_t)i) * (size_t)S;
      int32_t s = 0;
      for (int32_t j = 0; j < S; ++j) s += row[j];
      dur[(size_t)b * (size_t)T + (size_t)i] = s;
    }
}

/* Aligned text grid (Sec. 5, Conclusion: the MAS path multiplied with the
 * text representation).  For every item, out[b][j] = sum over i of
 * path[b][i][j] * h[b][i]: the frame-rate copy of the text features, of shape
 * [S, C] per item, with h of shape [T, C].  A MAS path has at most one 1 per
 * speech column, so that sum is the row of h the column is aligned to (taken
 * as it is, element bytes copied) or all zeros for a column no row covers
 * (the padding j >= t_y, and invalid items).  Elements are elem_bytes wide,
 * whatever their type.  Returns -1, leaving the item's output unspecified,
 * when a column holds more than one 1 (not a MAS path), else 0. */
int oracle_expand_text(const uint8_t* path, const uint8_t* h, int32_t B, int32_t T, int32_t S, int32_t C,
                       int32_t elem_bytes, uint8_t* out) {
  const size_t row = (size_t)C * (size_t)elem_bytes;
  int rc = 0;
  for (int32_t b = 0; b < B; ++b) {
    const uint8_t* pb = path + (size_t)b * (size_t)T * (size_t)S;
    for (int32_t j = 0; j < S; ++j) {
      uint8_t* dst = out + ((size_t)b * (size_t)S + (size_t)j) * row;
      int32_t src = -1, ones = 0;
      for (int32_t i = 0; i < T; ++i)
        if (pb[(size_t)i * (size_t)S + (size_t)j]) {
          src = i;
          ++ones;
        }
      if (ones > 1) rc = -1;
      if (src < 0)
        memset(dst, 0, row);
      else
        memcpy(dst, h + ((size_t)b * (size_t)T + (size_t)src) * row, row);
    }
  }
  return rc;
}

/* Gaussian log-likelihood of speech frames under text-token Gaussians, the
 * input MAS maximises (Sec. 2: q[i][j] is log N(z_j; mu_i, sigma_i), here
 * with a diagonal covariance over D channels):
 *   q[i][j] = sum over d of ( -ln(2 pi)/2 - log_sigma[i][d]
 *                             - (z[j][d] - mu[i][d])^2 / (2 sigma[i][d]^2) ),
 * sigma = exp(log_sigma).  Evaluated in double, d ascending, for n cells
 * (cells[3k], cells[3k+1], cells[3k+2]) = (b, i, j); mu and log_sigma are
 * [B][T][D] fp32, z is [B][S][D] fp32, log_sigma NULL means sigma = 1.
 * Returns -1 for a cell outside [B, T, S] (out left unspecified), else 0. */
int oracle_gauss_loglik_cells(const float* mu, const float* log_sigma, const float* z, int32_t B, int32_t T,
                              int32_t S, int32_t D, const int32_t* cells, int64_t n, double* out) {
  const double half_log_two_pi = 0.91893853320467274178032973640562; /* ln(2 pi) / 2 */
  for (int64_t k = 0; k < n; ++k) {
    const int32_t b = cells[3 * k], i = cells[3 * k + 1], j = cells[3 * k + 2];
    if (b < 0 || b >= B || i < 0 || i >= T || j < 0 || j >= S) return -1;
    const float* m = mu + ((size_t)b * (size_t)T + (size_t)i) * (size_t)D;
    const float* ls = log_sigma ? log_sigma + ((size_t)b * (size_t)T + (size_t)i) * (size_t)D : NULL;
    const float* x = z + ((size_t)b * (size_t)S + (size_t)j) * (size_t)D;
    double q = 0.0;
    for (int32_t d = 0; d < D; ++d) {
      const double lsd = ls ? (double)ls[d] : 0.0;
      const double sigma = exp(lsd);
      const double t = (double)x[d] - (double)m[d];
      q += -half_log_two_pi - lsd - t * t / (2.0 * sigma * sigma);
    }
    out[k] = q;
  }
  return 0;
}

int oracle_version(void) { return 2; }
