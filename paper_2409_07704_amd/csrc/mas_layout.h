// Workspace and bit layout shared by the libmas kernels and host code.
//
// Rows of an item are processed by 64-lane waves.  Lane 0 of wave g carries
// the row above the wave (row 63g-1, a copy handed down by the previous
// wave; for g = 0 the virtual -inf row above row 0) and lanes 1..63 own
// rows 63g .. 63g+62, one text row per lane.  Four such waves (252 rows)
// share a workgroup with the waves that feed them.  Speech columns are processed in chunks of 32, and every lane
// packs its row's 32 forward decisions of a chunk into one 32-bit word.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace mas {

constexpr int kWave = 64;                    // lanes per wavefront (CDNA)
constexpr int kRowsPerWave = kWave - 1;      // text rows a wave owns (lanes 1..63)
constexpr int kWavesPerBlock = 4;            // one wave per SIMD of a CU
constexpr int kThreadsPerBlock = kWave * kWavesPerBlock;
constexpr int kChunk = 32;                   // speech columns per decision word
constexpr size_t kAlign = 256;
constexpr int kMaxRows = 8192;               // largest T (the walker keeps row_start in LDS)

// Decision bit of text row i at speech column j (j >= 1): 1 when the forward
// max took the diagonal predecessor Q[i-1][j-1] (the backtrack then moves to
// row i-1), 0 when it kept Q[i][j-1].  A sweep wave packs a row's decisions
// of one chunk into one 32-bit word, the chunk's first column in bit 31.
// Those words never leave the CU: they are turned into step masks.
//
// Step mask of row i in chunk c: the set of positions p (column 32c + 31 - p)
// at which the backtrack, entering the chunk in row i at its last column,
// moves up one row while walking back to the chunk's first column; row i - k
// begins at the column of the k-th lowest position.  A wave stores, per chunk,
// kEntPerWave entries at pm[b][c][kEntPerWave * g + ...]:
//   entry r (r < 63):           the mask of its row 63g + r, for the path
//                               while it stays in the wave's rows; a path that
//                               climbs into the row above the wave ends there,
//                               with that step as its highest position p;
//   entry kMidOff + q (q < 32): the mask of the wave's last row entered at
//                               position q (column 32c + 31 - q), positions
//                               >= q, which completes such a path of the next
//                               wave at q = p + 1.
// A path climbs at most 32 rows per chunk, so it crosses at most one wave
// boundary in a chunk.
constexpr int kEntPerWave = 96;
constexpr int kMidOff = 64;
// Descent bytes, the walk's own copy of the step masks at a quarter of
// their size.  Per chunk, EP bytes: first one byte per mid entry of every
// wave (wave g's mid entry q at kChunk * g + q), then one byte per text row
// (row i at pd_row0(NW) + i), so that consecutive rows have consecutive
// bytes whatever waves they belong to:
//   row i (in wave g):  the number of rows the path climbs in the chunk while
//                       it stays in the wave's rows (the mask's popcount), or
//                       64 + p when it climbs into the row above the wave at
//                       position p (the highest position of the mask);
//   mid entry q:        the popcount of mid entry q's mask.
// (EP = 96 NW covers the 32 NW mid bytes and the 63 NW row bytes.)
constexpr uint32_t kEscape = 64;
__host__ __device__ constexpr int pd_row0(int NW) { return kChunk * NW; }

// Boundary hand-off between consecutive workgroups of an item: the last wave
// g of a workgroup publishes Q[63g+62][j] (its last row) for every column j it
// computes as one 64-bit word {low: fp32 bits, high: tag} (waves of one
// workgroup hand on through LDS).  The tag identifies the call (see
// WsHeader), so stale words from earlier calls are never mistaken for fresh
// ones.
// Dense path: written in tiles of kPathTileRows rows of one item, taken in
// the order the items' row_start tables are published, by at most
// kPathWorkgroups path-writer workgroups (three quarters of the MI355X's 256
// CUs: enough to keep up, while the stores of all 256 slow the sweeps still
// running more than they gain; timed on full batches of mixed lengths).
constexpr int kPathTileRows = 32;
constexpr int kPathWorkgroups = 192;

struct WsHeader {
  uint32_t gen;         // call generation; tag of a call = 2 * gen + 1
  uint32_t exit_count;  // workgroups that finished the current call
  uint32_t error;       // sticky: non-zero once a device-side wait timed out
  uint32_t walk_count;  // row_start tables published in the current call
  uint32_t tile_next;   // path tiles taken in the current call
  uint32_t magic;       // kWsMagic once the workspace has been initialised
  uint32_t path_fail;   // tag of the last call in which a path writer gave up a wait
  uint32_t pad[57];
};
constexpr uint32_t kWsMagic = 0x3153414du;  // "MAS1"
constexpr int kWsMagicPiece = 1;            // the header's 16-byte piece holding magic (bytes 16..31)
static_assert(sizeof(WsHeader) == kAlign, "header is one alignment unit");

__host__ __device__ inline size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct Layout {
  int32_t B, T, S;
  int32_t NW;      // waves per item = ceil(T / 63)
  int32_t NB;      // workgroups per item = ceil(NW / 4)
  int32_t NC;      // chunks per item = ceil(S / 32)
  int32_t EP;      // step-mask entries per chunk of an item = kEntPerWave * NW
  size_t off_done;   // uint32 [B][NW] sweep-finished flags (tag values)
  size_t off_tmo;    // uint32 [B] per-item timeout flags (tag values)
  size_t off_order;  // uint64 [B] items in the order their row_start tables were published: tag << 32 | item
  size_t off_slots;  // uint64 [B][NB][NC*32] boundary hand-off words of each workgroup's last wave
  size_t off_pm;     // uint32 [B][NC][EP] step masks
  size_t off_rs;     // int32  [B][T+1] row_start table (mas_forward_ex)
  size_t off_pd;     // uint8  [B][NC][EP] descent bytes
  size_t bytes;
};

// Returns false when the shape is invalid or its byte counts overflow.
__host__ inline bool make_layout(int32_t B, int32_t T, int32_t S, Layout* L) {
  if (B < 1 || T < 1 || S < 1 || T > kMaxRows) return false;
  L->B = B;
  L->T = T;
  L->S = S;
  L->NW = (T + kRowsPerWave - 1) / kRowsPerWave;
  L->NB = (L->NW + kWavesPerBlock - 1) / kWavesPerBlock;
  L->NC = (S + kChunk - 1) / kChunk;
  L->EP = kEntPerWave * L->NW;
  // Overflow guard: every product below stays far under 2^62 when these hold.
  if ((uint64_t)B * (uint64_t)L->NB + kPathWorkgroups > 0x7fffffffull) return false;  // grid size
  if ((uint64_t)B * (uint64_t)T * (uint64_t)S > (1ull << 46)) return false;
  // One item's value slab is addressed with signed 32-bit byte offsets.
  if ((uint64_t)T * (uint64_t)S * 4u >= (1ull << 31)) return false;
  size_t off = sizeof(WsHeader);
  L->off_done = off;
  off = round_up(off + (size_t)B * L->NW * sizeof(uint32_t), kAlign);
  L->off_tmo = off;
  off = round_up(off + (size_t)B * sizeof(uint32_t), kAlign);
  L->off_order = off;
  off = round_up(off + (size_t)B * sizeof(uint64_t), kAlign);
  L->off_slots = off;
  off = round_up(off + (size_t)B * L->NB * (size_t)L->NC * kChunk * sizeof(uint64_t), kAlign);
  L->off_pm = off;
  off = round_up(off + (size_t)B * L->NC * (size_t)L->EP * sizeof(uint32_t), kAlign);
  L->off_rs = off;
  off = round_up(off + (size_t)B * ((size_t)T + 1) * sizeof(int32_t), kAlign);
  L->off_pd = off;
  off = round_up(off + (size_t)B * L->NC * (size_t)L->EP, kAlign);
  L->bytes = off;
  return true;
}

// Per-item status codes (same values as MAS_ITEM_* in the public header).
enum ItemStatus : int32_t {
  kItemOk = 0,
  kItemEmpty = 1,
  kItemInfeasible = 2,
  kItemOutOfRange = 3,
  kItemSyncTimeout = 4,
  kItemBadWorkspace = 5
};

__host__ __device__ inline int32_t item_status(int32_t tx, int32_t ty, int32_t T, int32_t S) {
  if (tx < 0 || ty < 0 || tx > T || ty > S) return kItemOutOfRange;
  if (tx == 0 || ty == 0) return kItemEmpty;
  if (ty < tx) return kItemInfeasible;
  return kItemOk;
}

}  // namespace mas
