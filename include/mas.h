/*
 * libmas — batched Monotonic Alignment Search (MAS) on AMD Instinct MI355X
 * (gfx950).
 *
 * MAS (Super-MAS paper, Sec. 2, Algorithm 1; parallel form in Algorithm 2)
 * finds, for every item b of a batch, the monotonic alignment between t_x[b]
 * text tokens and t_y[b] speech frames that maximises the summed
 * log-likelihood value[b, i, j]:
 *   - forward pass: Q[i][j] = max(Q[i-1][j-1], Q[i][j-1]) + value[i][j] over
 *     0 <= i < t_x, 0 <= j < t_y, with Q[0][0] = value[0][0] and every cell
 *     a path cannot reach by column j (i > j) at -inf; each speech column
 *     depends only on the previous one and is parallel over text rows
 *     (Algorithm 2);
 *   - backtrack from (t_x-1, t_y-1): at column j in row i the path continues
 *     in row i-1 at column j-1 when Q[i][j-1] is strictly below
 *     Q[i-1][j-1] in the order defined next, or when i == j; it stays in row
 *     i otherwise (ties stay);
 *   - output: the 0/1 alignment A* of the input's [T, S] size per item, with
 *     exactly one 1 per speech column j < t_y (Sec. 2).
 * Order of the max and of the backtrack's comparison: the numeric order of
 * IEEE 754-2019 maximum(), in which -0 is below +0.  Algorithm 1's max is a
 * real-valued max and does not say how signed zeros compare; this order
 * answers it.  It differs from the plain IEEE `<` only when the two
 * candidates are zeros of opposite sign: for stay = -0, diag = +0 the
 * forward max is +0 and the path steps to row i-1 (with `<` it would keep
 * -0 and stay).  Every add is one fp32 round-to-nearest-even operation in
 * column order, with subnormals kept, so paths and scores are bit-for-bit
 * reproducible and equal to a sequential CPU evaluation in this order.
 *
 * Conventions for every entry point:
 *   - value is [B, T, S] fp32, t_x / t_y are [B] int32, path_out is
 *     [B, T, S] uint8, row_start is [B, T+1] int32, all contiguous row-major
 *     and all DEVICE pointers (memory of the current HIP device).
 *   - T and S are the padded extents; each item uses its own t_x <= T text
 *     rows and t_y <= S speech columns.  Padding of value and the cells no
 *     path can reach (i > j) never influence any result: they are either not
 *     loaded or loaded and discarded (loads never leave the [B, T, S] tensor).
 *     Padding of path_out is written as 0.
 *   - Shape limits: B, T, S >= 1, T <= 8192 (the backtrack keeps an item's
 *     row_start table in on-chip memory), T * S * 4 < 2^31 (one item's value
 *     slab is addressed with 32-bit byte offsets) and B * T * S <= 2^46.
 *     Other shapes return MAS_ERR_BAD_SHAPE.
 *   - Every call only enqueues work on `stream` (0 = the null stream) and
 *     returns; results are valid once the stream reaches that point.  No call
 *     synchronises the host or copies device data to the host.
 *   - The caller owns every buffer; the library never frees or retains
 *     caller memory.  value, t_x and t_y are read-only.
 *   - Errors detectable on the host return a non-zero mas_status and enqueue
 *     nothing.  Per-item length errors can only be seen on the device (the
 *     lengths live there); they give the item an all-zero slab, score -inf
 *     and a code in item_status_out.
 *   - Alignment: when S is a multiple of 4 and value is 16-byte aligned the
 *     forward pass uses 16-byte loads; other shapes take a general path with
 *     the same results.  Likewise the path writer uses 16-byte stores when S
 *     is a multiple of 16 and path_out is 16-byte aligned.
 */
#ifndef LIBMAS_MAS_H_
#define LIBMAS_MAS_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MAS_VERSION 2

typedef enum mas_status {
  MAS_OK = 0,
  MAS_ERR_NULL_POINTER = 1, /* a required pointer is NULL */
  MAS_ERR_BAD_SHAPE = 2,    /* B, T or S < 1, or past the shape limits above */
  MAS_ERR_WORKSPACE = 3,    /* workspace NULL, misaligned or too small */
  MAS_ERR_HIP = 4,          /* a HIP runtime call or kernel launch failed */
  MAS_ERR_SCRATCH = 5,      /* mas_forward_static: the batch needs more than MAS_STATIC_SCRATCH_BYTES */
  MAS_ERR_BAD_VALUE = 6     /* mas_forward_sentinel: the sentinel is not a finite negative number */
} mas_status;

/* Per-item status codes written to item_status_out[b]. */
#define MAS_ITEM_OK 0
#define MAS_ITEM_EMPTY 1        /* t_x == 0 or t_y == 0 */
#define MAS_ITEM_INFEASIBLE 2   /* t_y < t_x: no monotonic alignment exists */
#define MAS_ITEM_OUT_OF_RANGE 3 /* t_x or t_y negative, t_x > T or t_y > S */
#define MAS_ITEM_SYNC_TIMEOUT 4 /* an internal device-side wait hit its bound; the item's outputs are invalid */
#define MAS_ITEM_BAD_WORKSPACE 5 /* the workspace was never initialised by mas_workspace_init; nothing was computed */

/*
 * Every device-side wait is bounded: a wave gives up after a number of polls
 * without progress (about 2^20 by default, far beyond any real wait) and its
 * item is reported as MAS_ITEM_SYNC_TIMEOUT; the kernel still ends normally.
 * Diagnostics: the environment variable MAS_WAIT_BOUND, read at every call,
 * replaces that bound with a positive integer of at most 2^30 (tests use a
 * small one to exercise the timeout path).
 */

/*
 * Bytes of device workspace that mas_search / mas_forward_ex need for a
 * batch of this shape (decision bits, row hand-off slots, progress flags
 * and, for mas_forward_ex, the row_start table).  Returns 0 for invalid
 * shapes.  The workspace must be 256-byte aligned.
 */
size_t mas_workspace_bytes(int32_t B, int32_t T, int32_t S);

/*
 * Prepare a workspace for first use: zero-fills it on `stream` and marks it
 * initialised.  Required once per workspace allocation before the first
 * mas_search / mas_forward_ex that uses it; every later call leaves the
 * workspace ready for the next one.  A call on a workspace without that mark
 * computes nothing and sets every item_status_out entry to
 * MAS_ITEM_BAD_WORKSPACE (other outputs are left as they were).  A workspace serves one call at a time: calls that share
 * a workspace must be ordered (same stream or synchronised).
 */
mas_status mas_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Forward pass and backtrack without the dense path (Sec. 2 and Algorithm 1
 * up to A*(j); Algorithm 2 for the column-parallel forward loop).
 *
 * row_start_out [B, T+1] int32 (required): for a valid item, row_start[b][i]
 * is the first speech column whose alignment is text row i (i < t_x), so row
 * i covers columns [row_start[b][i], row_start[b][i+1]); entries i >= t_x
 * equal t_y.  Invalid items get all zeros.
 * durations_out [B, T] int32 (nullable): the number of speech frames aligned
 * to each text row (Sec. 2: the durations a duration predictor is trained
 * on), row_start[b][i+1] - row_start[b][i]; 0 for rows i >= t_x and for
 * invalid items.  Equal to the row sums of the dense path.
 * score_out [B] fp32 (nullable): Q[t_x-1][t_y-1], the log-likelihood of the
 * chosen alignment, -inf for invalid items.
 * item_status_out [B] int32 (nullable): MAS_ITEM_* per item.
 * workspace: at least mas_workspace_bytes(B, T, S) bytes, initialised once by
 * mas_workspace_init.
 */
mas_status mas_search(const float* value, const int32_t* t_x, const int32_t* t_y,
                      int32_t B, int32_t T, int32_t S,
                      int32_t* row_start_out, int32_t* durations_out, float* score_out, int32_t* item_status_out,
                      void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Dense alignment from a row_start table (Sec. 2: the path is a zero matrix
 * of the input's size with the alignment marked in it).  Writes every byte of
 * path_out [B, T, S]: path[b][i][j] = 1 iff row_start[b][i] <= j <
 * row_start[b][i+1], else 0.  row_start [B, T+1] must satisfy
 * 0 <= row_start[b][i] <= row_start[b][i+1] <= S (as mas_search produces).
 */
mas_status mas_expand_path(const int32_t* row_start, int32_t B, int32_t T, int32_t S,
                           uint8_t* path_out, hipStream_t stream);

/*
 * Aligned text grid (Sec. 5, Conclusion: the MAS path multiplied with the
 * text to give the text features at the speech frame rate).  For every item,
 * out[b][j] = sum over i of path[b][i][j] * text[b][i], with the path that
 * mas_expand_path would write from row_start: frame j < t_y takes the text
 * row whose segment [row_start[b][i], row_start[b][i+1]) holds it, copied as
 * it is (bit for bit, any element type, -0 / inf / NaN included); frames no
 * segment holds (j >= t_y, every frame of an invalid item) are all zero
 * bytes.  Computed as a gather; no path is formed.
 *   text [B, T, C] and out [B, S, C]: elements of elem_bytes (1, 2, 4 or 8)
 *   bytes, contiguous row-major, device pointers; out is fully overwritten.
 *   row_start [B, T+1] int32 as mas_search writes it (monotone, within
 *   [0, S]).  A table that is not monotone cannot make the kernel access
 *   memory outside these tensors, but its frames are then unspecified.
 *   Shape limits: B, T, S, C >= 1, T <= 2^30, C * elem_bytes <= 2^24, each
 *   tensor at most 2^48 bytes; else MAS_ERR_BAD_SHAPE (also for another
 *   elem_bytes).  16-byte words when text, out and the row size allow, else
 *   the widest that does.
 */
mas_status mas_expand_text(const void* text, const int32_t* row_start, int32_t B, int32_t T, int32_t S, int32_t C,
                           int32_t elem_bytes, void* out, hipStream_t stream);

/*
 * Gaussian log-likelihood, the quantity MAS maximises (Sec. 2: q[i][j] =
 * log N(z_j; mu_i, sigma_i), here with a diagonal covariance over D channels;
 * Sec. 5, Conclusion, names its calculation as the step to fuse with MAS):
 *   value[b][i][j] = sum over d of ( -ln(2 pi)/2 - log_sigma[b][i][d]
 *                    - (z[b][j][d] - mu[b][i][d])^2 / (2 exp(2 log_sigma[b][i][d])) )
 * for exactly the cells MAS reads: 0 <= i < t_x[b], i <= j < t_y[b],
 * j - i <= t_y[b] - t_x[b] (the feasible band).  Every other cell of
 * value_out, and every cell of an item with invalid lengths, is left as it
 * was; mas_search / mas_forward_ex on value_out never read those.
 *   mu, log_sigma [B, T, D] and z [B, S, D] fp32, contiguous row-major,
 *   device pointers; log_sigma may be NULL (sigma = 1).  t_x, t_y [B] int32.
 *   Precision: fp32-level, not bit-reproducible against a CPU: the sum is
 *   formed as a matrix product on fp16 matrix cores with each operand split
 *   into two fp16 parts after an exact power-of-2 scaling (about 22
 *   significant bits per product) and fp32 accumulation.  The error of a
 *   cell is within a few units of 2^-24 times the sum of the absolute values
 *   of its terms; repeated calls give identical bits.
 *   Shape limits: those of mas_forward_ex, and 1 <= D <= 192; else
 *   MAS_ERR_BAD_SHAPE.
 */
mas_status mas_loglik(const float* mu, const float* log_sigma, const float* z, const int32_t* t_x, const int32_t* t_y,
                      int32_t B, int32_t T, int32_t S, int32_t D, float* value_out, hipStream_t stream);

/*
 * Full alignment: mas_search into the workspace's row_start table followed by
 * mas_expand_path.  score_out and item_status_out are nullable as above.
 * No allocation; workspace as for mas_search.
 */
mas_status mas_forward_ex(const float* value, const int32_t* t_x, const int32_t* t_y,
                          uint8_t* path_out, int32_t B, int32_t T, int32_t S,
                          float* score_out, int32_t* item_status_out,
                          void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Legacy-sentinel mode (Sec. 2, issue 4 of the list of problems with the
 * original MAS, and the max_neg_val paragraph): the same call as
 * mas_forward_ex, except that every cell Algorithm 1 sets to -inf (the cache's
 * initial value: the cells i > j no path reaches by column j) holds the
 * finite `sentinel` instead, as in implementations that use max_neg_val
 * (-1e9 in the original, -1e32 in the paper's).  The forward max and the
 * backtrack are otherwise unchanged: the first text row is still the running
 * sum of its values, and the backtrack still steps up where i == j.  Results
 * equal Algorithm 1 run with that sentinel, including the alignments such a
 * sentinel spoils once cumulative log-likelihoods fall below it (Sec. 2: -1e9
 * is not small enough); for inputs whose partial sums stay far above it they
 * equal mas_forward_ex's.
 * sentinel: finite and negative, else MAS_ERR_BAD_VALUE (nothing enqueued).
 * Other arguments as for mas_forward_ex (same workspace).
 */
mas_status mas_forward_sentinel(const float* value, const int32_t* t_x, const int32_t* t_y,
                                uint8_t* path_out, int32_t B, int32_t T, int32_t S, float sentinel,
                                float* score_out, int32_t* item_status_out,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Full alignment with a stream-ordered workspace: allocates it with
 * hipMallocAsync on `stream`, initialises it, runs mas_forward_ex and frees
 * it with hipFreeAsync on the same stream.
 */
mas_status mas_forward(const float* value, const int32_t* t_x, const int32_t* t_y,
                       uint8_t* path_out, int32_t B, int32_t T, int32_t S, hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * call as mas_forward_ex, with the workspace taken from a static device array
 * of MAS_STATIC_SCRATCH_BYTES that the library holds on every device it runs
 * on until the process ends.  No allocation, ever.
 *   - Limit: batches with mas_workspace_bytes(B, T, S) > MAS_STATIC_SCRATCH_BYTES
 *     return MAS_ERR_SCRATCH and enqueue nothing (80 MiB holds, e.g.,
 *     B = 64, T = 1024, S = 4096).
 *   - The first call on a device enqueues the array's initialisation (a fill
 *     kernel, no memset) on `stream` ahead of the work; it must not be a call
 *     under graph capture.
 *   - Every call on one device shares that device's array, which keeps the
 *     last call's state: calls on one device must not overlap (issue them on
 *     one stream, or synchronise); overlapping calls race.
 */
#define MAS_STATIC_SCRATCH_BYTES ((size_t)80 << 20)
mas_status mas_forward_static(const float* value, const int32_t* t_x, const int32_t* t_y,
                              uint8_t* path_out, int32_t B, int32_t T, int32_t S,
                              float* score_out, int32_t* item_status_out, hipStream_t stream);

/* Human-readable name of a status code (static storage). */
const char* mas_status_string(mas_status status);

/* MAS_VERSION of the loaded library. */
int mas_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LIBMAS_MAS_H_ */
