// Kernel parameter block and launchers shared by the libmas host code and
// kernel translation unit.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mas_layout.h"

namespace mas {

constexpr int32_t kDefaultWaitBound = 1 << 20;  // bound of a device-side wait, in polls without progress

struct KParams {
  const float* value;
  const int32_t* t_x;
  const int32_t* t_y;
  int32_t* row_start;   // [B][T+1]
  float* score;         // nullable [B]
  int32_t* status;      // nullable [B]
  int32_t* durations;   // nullable [B][T]
  uint8_t* path;        // nullable [B][T][S]; null: no path is written
  WsHeader* hdr;
  uint32_t* done;       // [B][NW] a wave's step masks published (tag)
  uint32_t* tmo;        // [B] a wave of the item gave up a wait in this call (tag)
  uint64_t* order;      // [B] items in the order their row_start tables were published: tag << 32 | item
  uint64_t* slots;      // [B][NB][NC*32] boundary words of each workgroup's last wave
  uint32_t* pm;         // [B][NC][EP] step masks (see mas_layout.h)
  uint8_t* pd;          // [B][NC][EP] descent bytes (see mas_layout.h)
  int32_t B, T, S, NW, NC, EP, NB;
  int32_t ntile;        // path tiles per item: ceil(T / kPathTileRows)
  int32_t path16;       // path 16-byte aligned and S % 16 == 0
  int32_t spin_limit;   // bound of a device-side wait, in polls without progress
  float neg;            // value of the cells no path reaches: -inf, or the finite sentinel of the legacy mode
  int32_t legacy;       // finite sentinel (mas_forward_sentinel): triangle cells hold neg exactly
};

// Timeline of one launch in the debug build (MAS_TRACE): indices of 64-bit
// 100 MHz wall-clock stamps.  wg: [grid][2] start and end of each workgroup;
// chunk: [B][NW][64] slot k: sweep wave g done with chunk 8k+7 (or its last
// chunk; chunks past 511 are not recorded); walk: [B][64] slot k: walker done
// with the chunks from 32k up (slot k = its start, for the first block);
// item: [B][8] step masks of every wave published (windows may start),
// walk start, walk end, row_start published, ticks the walker waited for
// windows, (unused) x3; tile: [B * ntile][2] start and
// end of path tile t; win: [B][4][2][64] window loader k's n-th window (its
// chunk C-1-k-4n, n < 8): issue, staged.
struct TraceLayout {
  size_t wg, chunk, walk, item, tile, win, total;
};
__host__ __device__ inline TraceLayout trace_layout(int B, int NW, int NC, int ntile, int grid) {
  TraceLayout t;
  t.wg = 0;
  t.chunk = t.wg + 2 * (size_t)grid;
  t.walk = t.chunk + (size_t)B * NW * 64;
  t.item = t.walk + (size_t)B * 64;
  t.tile = t.item + 8 * (size_t)B;
  t.win = t.tile + 2 * (size_t)B * ntile;
  t.total = t.win + (size_t)B * 4 * 2 * 64;
  return t;
}

// Forward sweep, backtrack and (when p.path) the dense path, in one launch:
// one 768-thread workgroup (four sweep waves, four loader waves, four
// finisher waves) per 252 text rows of every item, then (when p.path) the
// path-writer workgroups.
hipError_t launch_mas(const KParams& p, hipStream_t stream);
// Dense [B, T, S] u8 path from row_start [B, T+1].
hipError_t launch_path(const int32_t* row_start, int32_t B, int32_t T, int32_t S, uint8_t* path, hipStream_t stream);
// Aligned text grid out [B, S, row_bytes] from text [B, T, row_bytes] and
// row_start [B, T+1] (a gather; see mas_text.hip).
hipError_t launch_text(const void* h, const int32_t* row_start, int32_t B, int32_t T, int32_t S, size_t row_bytes,
                       void* out, hipStream_t stream);
// Gaussian log-likelihood of the band cells of value [B, T, S] from mu,
// log_sigma (nullable) [B, T, D] and z [B, S, D]; D <= kLoglikMaxD (see
// mas_loglik.hip).
constexpr int32_t kLoglikMaxD = 192;
constexpr int kLoglikMaxKs = (2 * kLoglikMaxD + 31) / 32;
hipError_t launch_loglik(const float* mu, const float* log_sigma, const float* z, const int32_t* t_x,
                         const int32_t* t_y, float* value, int32_t B, int32_t T, int32_t S, int32_t D,
                         hipStream_t stream);
// Workspace initialisation: zero-fill of `bytes` (a multiple of 16, at least
// the header) at a 256-byte aligned pointer, with the header's magic set.
hipError_t launch_ws_init(void* p, size_t bytes, hipStream_t stream);
// Zero-fill of `bytes` (a multiple of 16) at a 16-byte aligned pointer.
hipError_t launch_fill(void* p, size_t bytes, hipStream_t stream);

}  // namespace mas
