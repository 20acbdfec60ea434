// Aligned text grid: every speech frame takes the features of the text token
// its alignment picks.  Sec. 5 (Conclusion) names this product of the MAS path
// with the text as the step that follows MAS in training; here it is a gather
// by row_start, so the [S, T] x [T, C] product with a 0/1 matrix is never
// formed and the dense path is not needed at all.
//
// One 256-thread workgroup per block of speech columns of one item:
//   1. every text row marks, in LDS, the columns of its segment
//      [row_start[i], row_start[i+1]) that fall in the block (row_start is
//      monotone, so each column is marked by at most one row);
//   2. each wave copies whole frames: lanes over the row's words, four
//      frames in flight per step, streaming (non-temporal) stores.
// The gather reads each used text row from HBM about once (neighbouring
// columns of a block share rows through L2) and writes every output byte
// once: an HBM-bound copy.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mas_internal.h"

namespace mas {
namespace {

constexpr int kTextThreads = 256;  // four waves
constexpr int kTextMaxCols = 256;  // speech columns per workgroup, at most
constexpr int kTextUnroll = 4;     // frames a wave moves per step

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <int W> struct Word;
template <> struct Word<16> { using type = u32x4; };
template <> struct Word<8> { using type = u32x2; };
template <> struct Word<4> { using type = uint32_t; };
template <> struct Word<2> { using type = uint16_t; };
template <> struct Word<1> { using type = uint8_t; };

// h [B][T][words], row_start [B][T+1], out [B][S][words]; words of W bytes.
template <int W>
__global__ void __launch_bounds__(kTextThreads)
    mas_text_kernel(const typename Word<W>::type* __restrict__ h, const int32_t* __restrict__ row_start,
                    typename Word<W>::type* __restrict__ out, int32_t T, int32_t S, int32_t words, int32_t cols,
                    int32_t col_blocks) {
  using V = typename Word<W>::type;
  __shared__ int32_t src[kTextMaxCols];
  const int b = blockIdx.x / col_blocks;
  const int j0 = (blockIdx.x - b * col_blocks) * cols;
  const int ncol = min(cols, S - j0);
  const int32_t* rs = row_start + (size_t)b * (T + 1);

  for (int k = threadIdx.x; k < cols; k += kTextThreads) src[k] = -1;
  __syncthreads();
  // Clamped to the block, so a malformed table cannot index outside it.
  for (int i = threadIdx.x; i < T; i += kTextThreads) {
    const int lo = max(rs[i], j0), hi = min(rs[i + 1], j0 + ncol);
    for (int j = lo; j < hi; ++j) src[j - j0] = i;
  }
  __syncthreads();

  const V* hb = h + (size_t)b * T * words;
  V* ob = out + ((size_t)b * S + j0) * words;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  constexpr int kWaves = kTextThreads / 64;
  for (int j = wave; j < ncol; j += kWaves * kTextUnroll) {
    int r[kTextUnroll];
#pragma unroll
    for (int u = 0; u < kTextUnroll; ++u) {
      const int jj = j + u * kWaves;
      r[u] = jj < ncol ? src[jj] : -2;  // -1: zero frame, -2: past the block
    }
    for (int c = lane; c < words; c += 64) {
      V v[kTextUnroll];
#pragma unroll
      for (int u = 0; u < kTextUnroll; ++u) v[u] = r[u] >= 0 ? hb[(size_t)r[u] * words + c] : V(0);
#pragma unroll
      for (int u = 0; u < kTextUnroll; ++u)
        if (r[u] != -2) __builtin_nontemporal_store(v[u], &ob[(size_t)(j + u * kWaves) * words + c]);
    }
  }
}

template <int W>
hipError_t launch_text_w(const void* h, const int32_t* row_start, int32_t B, int32_t T, int32_t S, size_t row_bytes,
                         void* out, int32_t cols, int32_t col_blocks, hipStream_t stream) {
  using V = typename Word<W>::type;
  hipLaunchKernelGGL(mas_text_kernel<W>, dim3((unsigned)B * (unsigned)col_blocks), dim3(kTextThreads), 0, stream,
                     static_cast<const V*>(h), row_start, static_cast<V*>(out), T, S, (int32_t)(row_bytes / W), cols,
                     col_blocks);
  return hipGetLastError();
}

}  // namespace

int32_t text_cols(int32_t B, int32_t S) {
  // Wide blocks when the batch fills the chip with them, narrow ones for
  // small batches (more workgroups, same work).
  const int64_t wide = (int64_t)B * ((S + kTextMaxCols - 1) / kTextMaxCols);
  return wide >= 1024 ? kTextMaxCols : 64;
}

hipError_t launch_text(const void* h, const int32_t* row_start, int32_t B, int32_t T, int32_t S, size_t row_bytes,
                       void* out, hipStream_t stream) {
  const int32_t cols = text_cols(B, S);
  const int32_t col_blocks = (S + cols - 1) / cols;
  const uintptr_t a = (uintptr_t)h | (uintptr_t)out | (uintptr_t)row_bytes;
  if (a % 16 == 0) return launch_text_w<16>(h, row_start, B, T, S, row_bytes, out, cols, col_blocks, stream);
  if (a % 8 == 0) return launch_text_w<8>(h, row_start, B, T, S, row_bytes, out, cols, col_blocks, stream);
  if (a % 4 == 0) return launch_text_w<4>(h, row_start, B, T, S, row_bytes, out, cols, col_blocks, stream);
  if (a % 2 == 0) return launch_text_w<2>(h, row_start, B, T, S, row_bytes, out, cols, col_blocks, stream);
  return launch_text_w<1>(h, row_start, B, T, S, row_bytes, out, cols, col_blocks, stream);
}

}  // namespace mas
