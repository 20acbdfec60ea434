// libmas kernels for gfx950 (MI355X): batched monotonic alignment search
// (Super-MAS Sec. 2, Algorithm 1; the column-parallel forward loop of
// Algorithm 2) and the dense path writer.
//
// One launch computes everything (mas_kernel).  A workgroup owns 252 text
// rows of one item and has twelve waves:
//   * four sweep waves (one per SIMD): wave w owns 63 rows, one text row per
//     lane in lanes 1..63, and lane 0 carries a copy of the row above the
//     wave.  A wave walks the speech axis in chunks of 32 columns.  The
//     diagonal predecessor Q[i-1][j-1] crosses lanes with one DPP wave_shr:1
//     per column, crosses waves of the workgroup through LDS ring slots, and
//     crosses workgroups through 64-bit {value, tag} words in global memory.
//     Wave g starts at chunk floor(63g / 32): every earlier cell of its rows
//     lies in the masked triangle i > j.
//   * four loader waves: loader w moves sweep wave w's value tiles (64 rows x
//     32 columns) from HBM into an LDS ring by buffer loads with the lds flag,
//     up to four chunks ahead, and publishes each tile once it has landed.
//     The sweep waves issue no loads of values; they read their tiles from LDS
//     while the next chunk's reads are already in flight.
//   * four finisher waves: finisher w turns each chunk's decision words of
//     sweep wave w into step masks (for every row the wave owns, the columns
//     at which the backtrack, entering the chunk in that row, moves up a row)
//     and stores them.
// The sweep wave holding row t_x-1 walks back from (t_x-1, t_y-1) once every
// wave of the item has published its masks, one lookup per chunk, while the
// four loaders of its workgroup stage the masks of upcoming chunks in LDS,
// and publishes the item's row_start table, appending the item to the call's
// completion order.  Path-writer workgroups, last in the grid, take
// tiles of 32 rows of one item from a shared counter in that order and write
// them from the table, every byte once (zeros and ones in one pass): an item
// that finishes late is written by many workgroups at once.
//
// Every wait is bounded, and a wave only waits on waves of its own workgroup
// or of workgroups with lower ids, which the hardware dispatches first:
// workgroup (band r, item b) has id r * B + b, and the path writers have the
// ids from B * NB on.
//
// Memory ordering across workgroups: data handed between workgroups (step
// masks, boundary words, row_start, flags) is written with device-scope
// (write-through) stores and read with device-scope loads, and a wave waits
// for its stores (vmcnt(0)) before raising a flag, so no cache write-back or
// invalidation is needed.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "mas_internal.h"

namespace mas {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

// Keeps the compiler from moving LDS accesses across this point; LDS
// operations of one wave execute in order, so no wait is needed.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Device-scope (write-through) stores and loads of data shared across
// workgroups.
__device__ __forceinline__ void st_dev(uint32_t* p, uint32_t v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ uint32_t ld_dev(const uint32_t* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }

__device__ __forceinline__ int lds_load(const int* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP); }
__device__ __forceinline__ void lds_store(int* p, int v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP); }
template <typename T>
__device__ __forceinline__ uint32_t lds_off(T* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) T*)p;
}
// Polled reads of mailbox words in waves that also move data into LDS with
// buffer loads: the compiler cannot tell a mailbox word from the tiles in
// flight and would wait for every load of the wave before each read, so these
// reads are issued directly, each with its own wait for LDS.
__device__ __forceinline__ int lds_poll(const int* p) {
  int v;
  asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(lds_off(p)) : "memory");
  return v;
}

__device__ __forceinline__ uint32_t call_tag(uint32_t gen) { return 2u * gen + 1u; }

// ---------------------------------------------------------------- timeline (debug build)
// With MAS_TRACE defined (the libmas_trace.so build), waves record 100 MHz
// wall-clock stamps of their milestones into the buffer set by mas_trace_set
// (layout: TraceLayout); otherwise every stamp compiles to nothing.  Stamps
// inside the sweep and walk loops are kept in one register (lane k: the k-th
// stamp, one per eight chunks) and stored once the loop is over, so that the
// traced loops issue no extra memory operations.
#ifdef MAS_TRACE
__device__ uint64_t* g_trace;
__device__ __forceinline__ void stamp(size_t idx) {
  uint64_t* const t = g_trace;
  if (t && __lane_id() == 0) t[idx] = __builtin_amdgcn_s_memrealtime();
}
// Time spent in some waits, summed (stored as one value).
struct Waited {
  uint64_t total = 0, since = 0;
  __device__ __forceinline__ void begin() { since = __builtin_amdgcn_s_memrealtime(); }
  __device__ __forceinline__ void end() {
    if (since) total += __builtin_amdgcn_s_memrealtime() - since;
    since = 0;
  }
  __device__ __forceinline__ void flush(size_t idx) {
    uint64_t* const t = g_trace;
    if (t && __lane_id() == 0) t[idx] = total;
  }
};
struct Stamps {
  uint64_t v = 0;
  __device__ __forceinline__ void at(int k) {
    const uint64_t now = __builtin_amdgcn_s_memrealtime();
    v = (int)__lane_id() == k ? now : v;
  }
  __device__ __forceinline__ void flush(size_t base) {
    uint64_t* const t = g_trace;
    if (t) t[base + __lane_id()] = v;
  }
};
#else
__device__ __forceinline__ void stamp(size_t) {}
struct Waited {
  __device__ __forceinline__ void begin() {}
  __device__ __forceinline__ void end() {}
  __device__ __forceinline__ void flush(size_t) {}
};
struct Stamps {
  __device__ __forceinline__ void at(int) {}
  __device__ __forceinline__ void flush(size_t) {}
};
#endif
__device__ __forceinline__ TraceLayout trace_of(const KParams& p) {
  return trace_layout(p.B, p.NW, p.NC, p.ntile, (int)gridDim.x);
}
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }


// State of the bounded waits of one wave: the bound (polls without progress;
// the host may lower it, see KParams::spin_limit) and whether a wait ran out.
// A wave whose wait runs out stops waiting from then on.  It first stores the
// call's tag into its flag (its item's timeout flag, or the call's path-writer
// flag) and waits for that store to land, so that the flag is visible before
// anything the wave does afterwards: the item's walker reads it after every
// wave whose work reaches the item's outputs has passed its last wait.
struct Bound {
  int limit;
  bool out;
  uint32_t* flag;
  uint32_t tag;
  __device__ __forceinline__ void expire();
};
constexpr int kLoaders = 4;          // loader waves per workgroup
constexpr int kFinishers = 4;        // finisher waves per workgroup (step masks to memory)
constexpr int kThreads = kThreadsPerBlock + (kLoaders + kFinishers) * kWave;
constexpr int kRing = 4;             // tile and boundary slots per sweep wave
constexpr int kPolicyDev = 16;       // cache policy sc1: device scope (write-through stores)
constexpr int kPolicyStream = 2;     // cache policy nt: streaming, data written once and not read back

// ---------------------------------------------------------------- LDS layout
// Sweep wave w owns kRing slots of kSlotStride bytes.  Slot k holds
//   * the value tile of one chunk: 64 tile rows (item rows 63g .. 63g+63; the
//     last one is loaded but unused) of 128 bytes.  Piece p (16 bytes,
//     columns 4p .. 4p+3) of tile row r sits at position p ^ swz(r) of the
//     row, swz(r) = (r >> 1) & 7: for any piece, 16 consecutive rows then
//     occupy 16 distinct four-bank groups of the 64-bank LDS, so the reads of
//     a wave (lane l reads row l-1) are conflict-free;
//   * at kBoundOff, the chunk's boundary row: Q of the row above the wave
//     for the chunk's 32 columns (lane 0's values);
//   * at kBitsOff, the chunk's decision words (lane l: word of row l-1, lane
//     0: a scratch word), left there by the sweep wave for its finisher.
// Chunk c uses slot (c - c_begin) % kRing of its wave.
constexpr int kTileBytes = kWave * kChunk * 4;  // 8192
constexpr int kBoundOff = kTileBytes;
constexpr int kBitsOff = kTileBytes + 256;
constexpr int kSlotStride = kTileBytes + 512;
constexpr int kWaveRegion = kRing * kSlotStride;
__host__ __device__ constexpr int swz(int r) { return (r >> 1) & 7; }

// The walk reuses the slot area (kWalkArea bytes): the row_start table under
// construction at its end (rs_bytes(T)), windows of descent bytes before it,
// one chunk per window, in nslot slots.  An item whose bytes for its rows
// < t_x fit kMinSlots windows gets windows of all of them (in as many slots
// as fit, at most kMaxSlots).  Otherwise windows are banded: the most slots
// S (at least kMinSlots) whose windows of band_bytes(S) bytes fit.  A window
// is staged for chunk c while the walker is at most S chunks above it, so
// the path can have climbed at most 32 * S rows by then; a banded window
// holds the rows from the lowest such row up to the walker's, and the mid
// entries of their waves and of the wave above them.
constexpr int kWalkArea = kWavesPerBlock * kWaveRegion;
constexpr int kMinSlots = 20;
constexpr int kMaxSlots = 48;   // (below 64 - 10: the window addresses are kept per chunk % 64)
constexpr int kWinLoaders = 4;  // loader waves staging windows: loader k takes chunks C-1-k, C-1-k-4, ...
constexpr int kMaxAhead = 8;    // windows in flight per loader, at most
__host__ __device__ constexpr int rs_bytes(int T) { return ((T + 1 + kWave) * 4 + 255) & ~255; }
__host__ __device__ constexpr int round_to(int x, int a) { return (x + a - 1) / a * a; }
// A banded window of an item with S slots: the rows the walk can still reach
// from the walker's row at issue time (32 per chunk over S chunks, and one
// more), then the mid entries of the waves those rows belong to and of the
// wave above them; 256-byte multiples.
__host__ __device__ constexpr int band_rows(int S) { return round_to(kChunk * S + 2, 256); }
__host__ __device__ constexpr int band_mids(int S) { return round_to(kChunk * ((kChunk * S + 1) / kRowsPerWave + 3), 256); }
__host__ __device__ constexpr int band_bytes(int S) { return band_rows(S) + band_mids(S); }
static_assert(kMinSlots * band_bytes(kMinSlots) <= kWalkArea - rs_bytes(kMaxRows), "banded windows fit");
// LDS-DMA loads of `bytes` (a multiple of 256): whole 1 KiB loads, then
// 256-byte ones (the LDS loads' rate goes by instructions more than by bytes).
__host__ __device__ constexpr int dma_loads(int bytes) { return bytes / 1024 + (bytes % 1024) / 256; }
// Window geometry of an item: bytes per window; slots; whether banded
// (otherwise a window is a chunk's descent bytes from the start: every mid
// entry and rows 0 .. t_x-1, rounded up to 1 KiB); windows in flight per
// loader; loads per window; and, when banded, the bytes of its row band and
// of its mid-entry band (which comes first in the window).
struct WinGeom {
  int ent, nslot, banded, ahead, loads, rows, mids;
};
__device__ __forceinline__ WinGeom win_geom(int tx, int NW, int T) {
  const int area = kWalkArea - rs_bytes(T);
  const int full = round_to(pd_row0(NW) + tx, 1024);
  WinGeom w;
  if (full * kMinSlots <= area) {
    w.ent = full;
    w.nslot = min(area / full, kMaxSlots);
    w.banded = 0;
    w.rows = 0;
    w.mids = 0;
    w.loads = dma_loads(full);
  } else {
    int S = kMinSlots;
    while (S < kMaxSlots && (S + 1) * band_bytes(S + 1) <= area) ++S;
    w.rows = band_rows(S);
    w.mids = band_mids(S);
    w.ent = w.rows + w.mids;
    w.nslot = S;
    w.banded = 1;
    w.loads = dma_loads(w.rows) + dma_loads(w.mids);
  }
  // (loads in flight stay below 64, the range of vmcnt)
  w.ahead = min(min(kMaxAhead, w.nslot / kWinLoaders), 63 / w.loads);
  return w;
}
// Walker position: (chunk << 16) | row (chunk < 2048, row < 8192), or -1
// once the walk is over.
__device__ __forceinline__ int walk_pos(int chunk, int row) { return (chunk << 16) | row; }
__device__ __forceinline__ int pos_chunk(int wp) { return wp >> 16; }
__device__ __forceinline__ int pos_row(int wp) { return wp & 0xFFFF; }

struct SweepLds {
  union {
    uint8_t ring[kWavesPerBlock][kWaveRegion];
    struct {
      uint8_t area[kWalkArea];  // windows from the start, row_start table at the end
    } walk;
  } u;
  // Mailbox of sweep wave w, read with one 16-byte load per chunk:
  //   .x ready: value tiles of chunks < ready are in w's slots (loader w);
  //   .y prod:  boundary rows of chunks < prod are in w's slots (wave w-1);
  //   .z cnext: progress of wave w+1: it has read every chunk < cnext, whose
  //             slots are free again (written by wave w+1);
  //   .w taken: the finisher has read the decision words of chunks < taken
  //             out of w's slots.
  // Wave 0's own progress goes to cons0.
  i32x4 box[kWavesPerBlock];
  int cons0;
  int wbase[kWave];             // walk window of chunk c (lane c % 64): LDS address of row 0's descent byte
  int wmid[kWave];              // ... and of wave 0's mid entry 0 (the addresses of bytes a banded window lacks are unused)
  i32x4 wready;                 // window loader k: its windows of chunks >= wready[k] are in LDS
  f32x4 sink[kWavesPerBlock][kChunk / 4 + 1];  // target of hand-offs nobody reads (a fixed LDS op count per step)
  int wpos;                     // walker position (walk_pos), or -1 once the walk is over
  int tile;                     // path writer: the tile taken next
  int pub;                      // path writer: the item of the tile taken (wave 0's poll), or -1
  uint64_t bpoll[4][kChunk];    // a workgroup's first loader: the boundary words of one poll (four chunks)
  uint32_t fdone[kWavesPerBlock];  // finisher w's step masks have all landed (the call's tag)
  // Row-start requests from the walker to its helper: records of up to 64
  // chunks (two buffers, request n in buffer n % 2), the chunk range they
  // cover, and the counts of requests posted and done.
  uint32_t req_d[2][kWave];
  int req_e[2][kWave];
  i32x4 req_arg[2];             // base chunk, lowest and highest chunk, last request (1) or not (0)
  int req_posted, req_done;
};
static_assert(sizeof(SweepLds) <= 160 * 1024, "LDS");
// The walk's row_start table (T + 1 entries, and up to 64 more that
// flush_records may touch) at the end of the walk area.
__device__ __forceinline__ int* walk_rs(SweepLds& L, int T) {
  return reinterpret_cast<int*>(L.u.walk.area + kWalkArea - rs_bytes(T));
}

// ---------------------------------------------------------------- vector memory
// Waits until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N <= 63, "vmcnt is a 6-bit counter");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// The same for a count known only at run time (n >= 0): waits until at most
// k operations are outstanding for the largest k <= n of a fixed set, which
// is at least as strict.  Compile-time branches only (a switch would become a
// jump table read through the scalar cache on every call).
__device__ __forceinline__ void vm_wait_le(int n) {
  if (n >= 16) {
    if (n >= 48) vm_wait<48>();
    else if (n >= 32) vm_wait<32>();
    else if (n >= 24) vm_wait<24>();
    else vm_wait<16>();
  } else if (n >= 4) {
    if (n >= 12) vm_wait<12>();
    else if (n >= 8) vm_wait<8>();
    else if (n >= 6) vm_wait<6>();
    else vm_wait<4>();
  } else {
    if (n >= 3) vm_wait<3>();
    else if (n >= 2) vm_wait<2>();
    else if (n >= 1) vm_wait<1>();
    else vm_wait<0>();
  }
}
// Waits until at most n operations are outstanding, n in [LO, HI] known only
// at run time (a tree of compile-time branches).
template <int LO, int HI>
__device__ __forceinline__ void vm_wait_exact(int n) {
  if constexpr (LO == HI) {
    vm_wait<LO>();
  } else {
    constexpr int MID = (LO + HI) / 2;
    if (n <= MID)
      vm_wait_exact<LO, MID>(n);
    else
      vm_wait_exact<MID + 1, HI>(n);
  }
}
// vm_wait_le with the call site's usual count first.
template <int USUAL>
__device__ __forceinline__ void vm_wait_usual(int n) {
  if (n == USUAL)
    vm_wait<USUAL>();
  else
    vm_wait_le(n);
}

__device__ __forceinline__ void Bound::expire() {
  if (out) return;
  out = true;
  if (flag) {
    st_dev(flag, tag);
    vm_wait<0>();
  }
}

// A buffer resource that moves forward through a region: base and number of
// bytes left.  Loads at per-lane offsets >= the count return 0 and such
// stores are dropped (the per-lane offset is range-checked, the scalar offset
// is not).  rsrc_s() reads every field back as wave-uniform, so the
// descriptor can feed scalar operands of inline assembly.
constexpr int kRsrcWord3 = 0x00020000;
struct Cursor {
  const char* base;
  int left;
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc() const {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), 0, left, kRsrcWord3);
  }
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_s() const {
    const uint64_t a = (uint64_t)(uintptr_t)base;
    const uint64_t lo = (uint32_t)uni((int)(uint32_t)a);
    const uint64_t hi = (uint32_t)uni((int)(uint32_t)(a >> 32));
    return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<char*>((uintptr_t)(lo | hi << 32)), 0, uni(left), kRsrcWord3);
  }
  __device__ __forceinline__ void advance(int step) {
    base += step;
    left = uni(max(left - step, 0));
  }
};
__device__ __forceinline__ Cursor make_cursor(const void* p, uint64_t bytes) {
  return Cursor{static_cast<const char*>(p), (int)(bytes < 0x7fffffffull ? bytes : 0x7fffffffull)};
}

// Loads into LDS: every lane's bytes at its voffset go to LDS at
// M0 + size * lane.  A scalar write of M0 needs one wait state before the
// load.  dma16 / dma4: read-only input (default cache policy); dma16_dev /
// dma4_dev: data written by other workgroups (device scope).
using lds_void = __attribute__((address_space(3))) void;
__device__ __forceinline__ lds_void* lds_at(uint32_t off) { return (lds_void*)(uintptr_t)uni((int)off); }
__device__ __forceinline__ void dma16(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds_at(lds), 16, voff, 0, 0, 0);
}
__device__ __forceinline__ void dma16_dev(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds_at(lds), 16, voff, 0, 0, kPolicyDev);
}
__device__ __forceinline__ void dma4_dev(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds_at(lds), 4, voff, 0, 0, kPolicyDev);
}
__device__ __forceinline__ void dma4(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds_at(lds), 4, voff, 0, 0, 0);
}

// ---------------------------------------------------------------- recurrence
// One text row per lane, lane 0 carrying the row above the wave.  Per column
// j (Algorithm 2's parallel step):
//   t       = max(Q[r-1][j-1], Q[r][j-1])   v_max_f32 with DPP wave_shr:1
//                                            (lane l reads lane l-1's Q);
//   Q[r][j] = t + value[r][j]                one fp32 add;
//   d       = sign(Q[r][j-1] - t)            1 iff the diagonal is strictly
//                                            greater (-0 below +0: the order
//                                            of v_max_f32);
//   bits    = bits << 1 | d                  v_alignbit (the chunk's first
//                                            column ends in bit 31).
// Lane 0 has no lane below it: DPP leaves its t untouched, and t is kept at
// -0 in lane 0 for the whole sweep, so lane 0's Q becomes -0 + value = value
// exactly: lane 0's "values" are the Q of the row above, handed down by the
// previous wave (or -inf above row 0).
// A VALU write followed by a DPP read of the same register needs two wait
// states: each column's add is followed by two other VALU instructions
// before the next column reads it, and each block starts with s_nop 1.
// (asm volatile: the compute must stay between the LDS reads issued before
// it and the wait after it.)
__device__ __forceinline__ void cols8(float& q, float& t, uint32_t& bits, float (&o)[8], const float* v) {
  float u;
  asm volatile("s_nop 1\n\t"
      "v_max_f32_dpp %[t], %[q], %[q] wave_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32 %[o0], %[t], %[v0]\n\t"
      "v_sub_f32 %[u], %[q], %[t]\n\t"
      "v_alignbit_b32 %[b], %[b], %[u], 31\n\t"
      "v_max_f32_dpp %[t], %[o0], %[o0] wave_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32 %[o1], %[t], %[v1]\n\t"
      "v_sub_f32 %[u], %[o0], %[t]\n\t"
      "v_alignbit_b32 %[b], %[b], %[u], 31\n\t"
      "v_max_f32_dpp %[t], %[o1], %[o1] wave_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32 %[o2], %[t], %[v2]\n\t"
      "v_sub_f32 %[u], %[o1], %[t]\n\t"
      "v_alignbit_b32 %[b], %[b], %[u], 31\n\t"
      "v_max_f32_dpp %[t], %[o2], %[o2] wave_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32 %[o3], %[t], %[v3]\n\t"
      "v_sub_f32 %[u], %[o2], %[t]\n\t"
      "v_alignbit_b32 %[b], %[b], %[u], 31\n\t"
      "v_max_f32_dpp %[t], %[o3], %[o3] wave_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32 %[o4], %[t], %[v4]\n\t"
      "v_sub_f32 %[u], %[o3], %[t]\n\t"
      "v_alignbit_b32 %[b], %[b], %[u], 31\n\t"
      "v_max_f32_dpp %[t], %[o4], %[o4] wave_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32 %[o5], %[t], %[v5]\n\t"
      "v_sub_f32 %[u], %[o4], %[t]\n\t"
      "v_alignbit_b32 %[b], %[b], %[u], 31\n\t"
      "v_max_f32_dpp %[t], %[o5], %[o5] wave_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32 %[o6], %[t], %[v6]\n\t"
      "v_sub_f32 %[u], %[o5], %[t]\n\t"
      "v_alignbit_b32 %[b], %[b], %[u], 31\n\t"
      "v_max_f32_dpp %[t], %[o6], %[o6] wave_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32 %[o7], %[t], %[v7]\n\t"
      "v_sub_f32 %[u], %[o6], %[t]\n\t"
      "v_alignbit_b32 %[b], %[b], %[u], 31"
      : [o0] "=&v"(o[0]), [o1] "=&v"(o[1]), [o2] "=&v"(o[2]), [o3] "=&v"(o[3]), [o4] "=&v"(o[4]), [o5] "=&v"(o[5]),
        [o6] "=&v"(o[6]), [o7] "=&v"(o[7]), [t] "+v"(t), [b] "+v"(bits), [u] "=&v"(u)
      : [q] "v"(q), [v0] "v"(v[0]), [v1] "v"(v[1]), [v2] "v"(v[2]), [v3] "v"(v[3]), [v4] "v"(v[4]), [v5] "v"(v[5]),
        [v6] "v"(v[6]), [v7] "v"(v[7]));
  q = o[7];
}

// One 32-column chunk for lanes 1..63 (rows row0 + lane - 1) and the carried
// row in lane 0.  v4: this lane's 32 values (lane 0: the row above's Q);
// qc: Q of every column (out); bits: decisions, first column in bit 31.
// Cells of the triangle i > j hold -inf in the tile (the loader writes it
// there): both predecessors of such a cell lie in the triangle too (lane 0's
// copies of the row above are -inf there already), so its Q comes out
// -inf + -inf = -inf, whatever the input held; decision bits of those cells
// are never read.  (The first cell Q[0][0] = value[0][0] comes from row 0's
// Q at column -1 being -0, see sweep_wave.)
__device__ __forceinline__ void sweep_chunk(float& q, float& t, const f32x4 (&v4)[8], float (&qc)[kChunk], uint32_t& bits) {
  float v[kChunk];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    v[4 * k + 0] = v4[k].x;
    v[4 * k + 1] = v4[k].y;
    v[4 * k + 2] = v4[k].z;
    v[4 * k + 3] = v4[k].w;
  }
  uint32_t w = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    float o[8];
    cols8(q, t, w, o, v + 8 * k);
#pragma unroll
    for (int m = 0; m < 8; ++m) qc[8 * k + m] = o[m];
  }
  bits = w;
}

// First n bytes of a u64 set to 0xFF (n in [0, 8]).
__device__ __forceinline__ uint64_t low_bytes(int n) { return n >= 8 ? ~0ull : ((1ull << (8 * n)) - 1ull); }

// 16 path bytes of one row starting at column j0: byte k = 1 iff lo <= j0+k < hi.
__device__ __forceinline__ uint4 path_piece(int lo, int hi, int j0) {
  const int a = min(max(lo - j0, 0), 16);
  const int e = min(max(hi - j0, 0), 16);
  const uint64_t ones = 0x0101010101010101ull;
  const uint64_t m0 = low_bytes(min(e, 8)) & ~low_bytes(min(a, 8)) & ones;
  const uint64_t m1 = low_bytes(max(e - 8, 0)) & ~low_bytes(max(a - 8, 0)) & ones;
  return make_uint4((uint32_t)m0, (uint32_t)(m0 >> 32), (uint32_t)m1, (uint32_t)(m1 >> 32));
}

// ---------------------------------------------------------------- per-wave context
struct WaveCtx {
  int lane, w, b, g, g_last, tx, ty, row, c_begin, c_end;
  int prev_end;    // chunks the previous wave computes (exclusive end)
  int mask_end;    // first chunk without a cell i > j of this wave
  int next_begin;  // the next wave's first chunk
};

// Chunks of wave g worth computing: from the first chunk holding a cell with
// i <= j of its rows, to the last chunk holding a cell of its rows that can
// still reach (t_x-1, t_y-1) (a path descends at most one row per column, so
// row r is useful up to column r + t_y - t_x).  Cells outside only feed
// cells outside (a reachable cell's two predecessors are reachable), so
// whatever they hold never reaches a decision the walk reads or the score.
__device__ __forceinline__ int chunk_begin(int g) { return (g * kRowsPerWave) / kChunk; }
__device__ __forceinline__ int chunk_end(int g, int tx, int ty) {
  const int by_len = (ty + kChunk - 1) / kChunk;
  const int by_reach = (g * kRowsPerWave + kRowsPerWave - 1 + ty - tx) / kChunk + 1;
  return by_len < by_reach ? by_len : by_reach;
}

__device__ __forceinline__ WaveCtx make_ctx(int b, int g, int w, int lane, int tx, int ty) {
  WaveCtx x;
  x.lane = lane;
  x.w = w;
  x.b = b;
  x.g = g;
  x.tx = tx;
  x.ty = ty;
  x.g_last = (tx - 1) / kRowsPerWave;
  x.row = g * kRowsPerWave + lane - 1;  // lane 0: the row above the wave
  x.c_begin = chunk_begin(g);
  x.c_end = chunk_end(g, tx, ty);
  x.prev_end = g > 0 ? chunk_end(g - 1, tx, ty) : 0;
  x.mask_end = (g * kRowsPerWave + kRowsPerWave - 2) / kChunk + 1;  // last masked column: 63g + 61
  x.next_begin = chunk_begin(g + 1);
  return x;
}

// Waits (bounded) until flag[k] == tag for every k in [0, n).  The bound
// counts polls since a flag last went up.
__device__ __forceinline__ void wait_flags(const uint32_t* flag, int n, uint32_t tag, int lane, Bound& bd) {
  for (int k0 = 0; k0 < n; k0 += kWave) {
    const int k = k0 + lane;
    int spins = 0;
    uint64_t missing = ~0ull;
    while (!bd.out) {
      const bool ready = k >= n || ld_dev(flag + k) == tag;
      const uint64_t m = __builtin_amdgcn_ballot_w64(!ready);
      if (m == 0) break;
      spins = m != missing ? 0 : spins + 1;
      missing = m;
      if (spins > bd.limit) bd.expire();
      __builtin_amdgcn_s_sleep(2);
    }
  }
}

// Waits (bounded) until the LDS words f[0 .. n) all hold tag.
__device__ __forceinline__ void wait_tags(const uint32_t* f, int n, uint32_t tag, Bound& bd) {
  for (int k = 0; k < n; ++k) {
    int spins = 0;
    while (!bd.out && (uint32_t)uni(lds_poll(reinterpret_cast<const int*>(f + k))) != tag) {
      if (++spins > bd.limit) bd.expire();
      __builtin_amdgcn_s_sleep(1);
    }
  }
}

// Spins (bounded) until the LDS word *p >= v; returns the last value read.
// The bound counts polls since the word last changed.
__device__ __forceinline__ int wait_at_least(const int* p, int v, Bound& bd) {
  int seen = uni(lds_poll(p));
  int spins = 0;
  while (seen < v && !bd.out) {
    __builtin_amdgcn_s_sleep(1);
    const int now = uni(lds_poll(p));
    spins = now != seen ? 0 : spins + 1;
    seen = now;
    if (spins > bd.limit) bd.expire();
  }
  return seen;
}

using lds_cchar = const __attribute__((address_space(3))) char;

// The LDS reads of the next chunk in slot K of a sweep wave: the wave's
// mailbox (ready, prod, cnext), then the lane's 8 pieces (byte offsets a[m]
// from the base of the shared block).  The empty asm statement with a memory
// clobber keeps the mailbox read ahead of the piece reads in issue order, and
// one wave's LDS reads execute in issue order, so pieces that the mailbox
// reports as delivered are read after their delivery.  These are ordinary
// loads for the compiler, which waits for each before its first use; callers
// pin them ahead of the compute with a scheduling barrier.
template <int K>
__device__ __forceinline__ void read_ahead(lds_cchar* Lb, uint32_t box_off, const uint32_t (&a)[8], f32x4 (&v)[8],
                                           i32x4& mb) {
  mb = *reinterpret_cast<const __attribute__((address_space(3))) i32x4*>(Lb + box_off);
  asm volatile("" ::: "memory");
#pragma unroll
  for (int m = 0; m < 8; ++m)
    v[m] = *reinterpret_cast<const __attribute__((address_space(3))) f32x4*>(Lb + a[m] + (uint32_t)(K * kSlotStride));
}
// s_waitcnt lgkmcnt(0) as a real instruction (vmcnt and expcnt at their
// maxima), which the compiler's own wait placement takes into account.
__device__ __forceinline__ void lgkm_wait0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// LDS stores without a branch: one lane (lane 0) writes v at addr; lanes
// 56..63 write f at their own addr (16 bytes each).  On this LDS every store
// instruction costs about the same whatever the number of active lanes, and
// a store from all lanes to one address serialises.
__device__ __forceinline__ void lds_put(uint32_t addr, int v) {
  uint64_t sv;
  asm volatile("s_mov_b64 %[sv], exec\n\ts_mov_b64 exec, 1\n\tds_write_b32 %[a], %[v]\n\ts_mov_b64 exec, %[sv]"
               : [sv] "=&s"(sv)
               : [a] "v"(addr), [v] "v"(v)
               : "memory");
}
__device__ __forceinline__ void lds_put_hi8(uint32_t addr, f32x4 f) {
  uint64_t sv;
  asm volatile("s_mov_b64 %[sv], exec\n\ts_mov_b64 exec, %[m]\n\tds_write_b128 %[a], %[f]\n\ts_mov_b64 exec, %[sv]"
               : [sv] "=&s"(sv)
               : [m] "s"(0xff00000000000000ull), [a] "v"(addr), [f] "v"(f)
               : "memory");
}
template <int N>
__device__ __forceinline__ float dpp_row_shl(float old, float src) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(src), 0x100 | N, 0xf, 0xf, false));
}
// Lanes 56..63 receive lane 63's q[4k .. 4k+3] (k = lane - 56), gathered by
// DPP row shifts inside the last 16-lane row: lane 56+k reads lane 63 with
// row_shl:(7-k); a lane whose source lies past the end of the row keeps its
// value, so the shifts run from the smallest up.
__device__ __forceinline__ f32x4 gather_last_row(const float (&q)[kChunk]) {
  f32x4 f = {q[28], q[29], q[30], q[31]};
#define MAS_GATHER(K)                                      \
  f.x = dpp_row_shl<7 - K>(f.x, q[4 * K + 0]);             \
  f.y = dpp_row_shl<7 - K>(f.y, q[4 * K + 1]);             \
  f.z = dpp_row_shl<7 - K>(f.z, q[4 * K + 2]);             \
  f.w = dpp_row_shl<7 - K>(f.w, q[4 * K + 3]);
  MAS_GATHER(6) MAS_GATHER(5) MAS_GATHER(4) MAS_GATHER(3) MAS_GATHER(2) MAS_GATHER(1) MAS_GATHER(0)
#undef MAS_GATHER
  return f;
}

// ---------------------------------------------------------------- sweep wave
// Sweeps the wave's rows over its chunks and returns the score candidate
// (Q at (row, t_y-1) of this lane; only meaningful for the wave holding row
// t_x-1).  IN: where the row above the wave comes from — 0 nowhere (the wave
// holds row 0: -inf), 1 the wave's slots and prod mailbox, filled by the
// previous wave of the workgroup or, for wave 0 of a later workgroup, by its
// loader from the previous workgroup's global boundary words.  OUT: 0 no
// consumer, 1 the next wave of the workgroup, 2 global boundary words for the
// next workgroup.
//
// Step c computes chunk c from registers while the LDS reads of chunk c+1
// (its tile, its boundary row and its mailbox) are in flight, hands the
// chunk's last row to the consumer, and then checks the mailbox: it only
// waits when the tile or the boundary row of chunk c+1 was not there yet.
template <int IN, int OUT>
__device__ __forceinline__ float sweep_wave(const KParams& p, SweepLds& L, const WaveCtx& x, uint32_t tag, Bound& bd) {
  constexpr bool IN1 = IN == 1;
  const int lane = x.lane, w = x.w;
  float t = -0.0f;  // lane 0 keeps -0 for the whole sweep (see cols8)
  char* const Lc = reinterpret_cast<char*>(&L);
  const uint32_t wbase = (uint32_t)w * kWaveRegion;
  auto bound_ptr = [&](int k) __attribute__((always_inline)) -> float* {
    return reinterpret_cast<float*>(Lc + wbase + (uint32_t)k * kSlotStride + kBoundOff);
  };
  // Per-lane LDS byte offsets of the 8 pieces of slot 0: lanes 1..63 read
  // tile row lane-1 (swizzled), lane 0 reads the boundary row.
  uint32_t ra[8];
  {
    const int r = lane > 0 ? lane - 1 : 0;
#pragma unroll
    for (int m = 0; m < 8; ++m)
      ra[m] = lane > 0 ? wbase + (uint32_t)(r * 128 + 16 * (m ^ swz(r))) : wbase + (uint32_t)(kBoundOff + 16 * m);
  }
  // Mailboxes: this wave's, the next wave's (OUT1: its prod), and where this
  // wave's progress goes (the previous wave's mailbox, or cons0).
  const uint32_t box_off = (uint32_t)((const char*)&L.box[w] - Lc);
  lds_cchar* const Lb = (lds_cchar*)Lc;
  const uint32_t next_prod = lds_off(&L.box[w < kWavesPerBlock - 1 ? w + 1 : w]) + 4u;
  const uint32_t my_cons = w > 0 ? lds_off(&L.box[w - 1]) + 8u : lds_off(&L.cons0);
  const int* const my_box = reinterpret_cast<const int*>(&L.box[w]);

  // Decision words: into the chunk's slot (the finisher wave turns them into
  // step masks); a lane's word of chunk c at bits_ptr(J)[lane].
  auto bits_ptr = [&](int k) __attribute__((always_inline)) -> uint32_t* {
    return reinterpret_cast<uint32_t*>(Lc + wbase + (uint32_t)k * kSlotStride + kBitsOff);
  };
  // Global boundary words of this wave (OUT2: the last wave of workgroup
  // g / 4): word 32c + j = {Q of the wave's last row at column 32c + j, tag}.
  const size_t slot_words = (size_t)p.NC * kChunk;
  const __amdgpu_buffer_rsrc_t sr =
      make_cursor(p.slots + ((size_t)x.b * p.NB + x.g / kWavesPerBlock) * slot_words, slot_words * 8u).rsrc();

  if (IN == 0) {
    // The row above row 0 is -inf in every slot.
    if (lane < kChunk) {
#pragma unroll
      for (int k = 0; k < kRing; ++k) bound_ptr(k)[lane] = neg_inf();
    }
  }

  // Lane 0's Q at the column before the first chunk: the previous wave's
  // last row there (its chunk c_begin-1, always computed), or -inf.  It
  // sits in slot kRing-1 (chunk c_begin-1).  Every other row's Q at the
  // column before its first chunk is -inf (the legacy mode's sentinel neg),
  // except row 0's at column -1: -0, so that the first cell comes out as
  // -0 + value[0][0] = value[0][0] exactly (its predecessors are -0 and the
  // row above row 0, -inf in both modes: row 0 is the running sum).
  float q = (IN == 0 && lane == 1) ? -0.0f : (IN == 0 && lane == 0) ? neg_inf() : p.neg;
  if (IN1) wait_at_least(my_box + 1, x.c_begin, bd);
  if (IN != 0) {
    wave_lds_sync();
    const float e = bound_ptr(kRing - 1)[kChunk - 1];
    q = lane == 0 ? e : q;
    wave_lds_sync();
    lds_put(my_cons, x.c_begin);
  }

  // The first chunk's tile and boundary row.  Values alternate between two
  // register sets by ring position: chunk c uses set (c - c_begin) % 2.
  f32x4 va[8], vb[8];
  wait_at_least(my_box + 0, x.c_begin + 1, bd);
  if (IN1 && x.c_begin < x.prev_end) wait_at_least(my_box + 1, x.c_begin + 1, bd);
  int cons_seen;  // the consumer's progress as last read (OUT1)
  {
    // (Through the same inline-assembly reads as the loop: values the
    // compiler loaded itself would make it wait for LDS inside the loop.)
    i32x4 mb;
    read_ahead<0>(Lb, box_off, ra, va, mb);
    cons_seen = uni(mb.z);
  }
  lds_put(my_cons, x.c_begin + 1);

  float qc[kChunk] = {};
  float score = neg_inf();
  const int row = x.g * kRowsPerWave + lane - 1;                 // this lane's text row (lanes 1..63)
  const int diag_last = (x.g * kRowsPerWave + kRowsPerWave - 1) / kChunk;  // the last chunk holding one of its diagonal cells
  Stamps stamps;  // (debug build) lane k: chunk 8k+7 (or the last chunk) done
  const int m_last = (x.ty - 1) % kChunk;

  // The last row of chunk cp (in lane 63's qc) for the next wave, right
  // after its compute: gathered into lanes 56..63 (four columns each).  OUT1:
  // one LDS write into the next wave's slot for chunk cp (once it has read
  // chunk cp-4 from that slot), then its mailbox's prod.  Chunks the next
  // wave does not read (cp < next_begin - 1) go to this wave's sink, so that
  // every step issues the same LDS operations and the compiler's waits stay
  // exact.  OUT2: two device-scope 16-byte stores per lane of {value, tag}
  // pairs; lanes outside 56..63 get offsets past the resource (dropped).
  const uint32_t sink = lds_off(&L.sink[w][0]);
  auto hand_off = [&](int cp) __attribute__((always_inline)) {
    const bool real = cp >= x.next_begin - 1;
    if (OUT == 1) {
      if (real && cons_seen < cp - (kRing - 1)) cons_seen = wait_at_least(my_box + 2, cp - (kRing - 1), bd);
      const int kn = (cp - x.next_begin) & (kRing - 1);
      const uint32_t ns = real ? wbase + kWaveRegion + (uint32_t)kn * kSlotStride + kBoundOff : sink;
      lds_put_hi8(ns + 16u * (uint32_t)(lane - (kWave - 8)), gather_last_row(qc));
      lds_put(real ? next_prod : sink + 128u, cp + 1);
    } else if (OUT == 2 && real) {
      const f32x4 f = gather_last_row(qc);
      const bool mine = lane >= kWave - 8;
      const int o = cp * (kChunk * 8) + 32 * (lane - (kWave - 8));
      const u32x4 lo = {__float_as_uint(f.x), tag, __float_as_uint(f.y), tag};
      const u32x4 hi = {__float_as_uint(f.z), tag, __float_as_uint(f.w), tag};
      __builtin_amdgcn_raw_buffer_store_b128(lo, sr, mine ? o : -1, 0, kPolicyDev);
      __builtin_amdgcn_raw_buffer_store_b128(hi, sr, mine ? o + 16 : -1, 0, kPolicyDev);
    }
  };

  // Chunk c at ring position J = (c - c_begin) % kRing, its values in vc,
  // the next chunk's read into vn.
  auto step = [&](auto pos_c, int c, f32x4 (&vc)[8], f32x4 (&vn)[8]) __attribute__((always_inline)) {
    constexpr int J = decltype(pos_c)::value;
    constexpr int J1 = (J + 1) & (kRing - 1);
    const bool has_next = c + 1 < x.c_end;
    const bool need_prod = IN1 && c + 1 < x.prev_end;
    // Reads of chunk c+1, in flight during the compute of chunk c: the
    // mailbox first, then the values (one LDS queue per wave: in order).
    // After the last chunk they read the next slot's stale contents, unused.
    i32x4 mb;
    read_ahead<J1>(Lb, box_off, ra, vn, mb);
    __builtin_amdgcn_sched_barrier(0);

    uint32_t bits = 0;
    sweep_chunk(q, t, vc, qc, bits);
    __builtin_amdgcn_sched_barrier(0);
    if (p.legacy && c <= diag_last) {
      // Legacy mode: the backtrack steps up at i == j whatever Q says (the
      // stay candidate is a masked cell); with a finite sentinel the
      // decision there can come out 0, so its bit is set.
      const int rel = row - c * kChunk;
      bits |= (lane > 0 && rel >= 0 && rel < kChunk) ? 1u << (kChunk - 1 - rel) : 0u;
    }
    hand_off(c);
    // The slot's decision words of chunk c-4 must have been taken (mailbox
    // .w, read with this step's mailbox; rarely not yet).
    if (uni(mb.w) < c - (kRing - 1)) {
      wait_at_least(my_box + 3, c - (kRing - 1), bd);
      lgkm_wait0();
    }
    bits_ptr(J)[lane] = bits;
    if (OUT == 0 && c == x.c_end - 1) {
#pragma unroll
      for (int m = 0; m < kChunk; ++m) score = (m == m_last) ? qc[m] : score;
    }

    if (has_next) {
      // The reads of chunk c+1 are usable if the tile and the boundary row
      // were there when they were issued; otherwise wait and read again.
      if (OUT == 1) cons_seen = max(cons_seen, uni(mb.z));
      if (uni(mb.x) < c + 2 || (need_prod && uni(mb.y) < c + 2)) {
        wait_at_least(my_box + 0, c + 2, bd);
        if (need_prod) wait_at_least(my_box + 1, c + 2, bd);
        read_ahead<J1>(Lb, box_off, ra, vn, mb);
        lgkm_wait0();
      }
      lds_put(my_cons, c + 2);
    }
    if ((c & 7) == 7 || c == x.c_end - 1) stamps.at(c >> 3);
  };
  for (int c = x.c_begin; c < x.c_end; c += kRing) {
    step(std::integral_constant<int, 0>(), c, va, vb);
    if (c + 1 < x.c_end) step(std::integral_constant<int, 1>(), c + 1, vb, va);
    if (c + 2 < x.c_end) step(std::integral_constant<int, 2>(), c + 2, va, vb);
    if (c + 3 < x.c_end) step(std::integral_constant<int, 3>(), c + 3, vb, va);
  }
  // Every chunk's decision words are in the slots (the finisher takes chunk
  // c once this progress passes c + 1).
  lds_put(my_cons, x.c_end + 1);
  stamps.flush(trace_of(p).chunk + ((size_t)x.b * p.NW + x.g) * kWave);
  vm_wait<0>();
  return score;
}

// ---------------------------------------------------------------- scheduling
// Critical-path-first start.  Every item runs as its own chain of waves, and
// the launch ends with the longest chain; HBM bandwidth, shared by every item
// sweeping at the same time, is the resource they compete for.  So each item
// waits, before loading more than its first tiles, for a share of the time by
// which its estimated run is shorter than the batch's longest: long items
// sweep first with little contention and short ones fill in behind them.
// Estimates are in wall-clock ticks (100 MHz): kTicksPerChunk per 32
// columns (about one chunk step of a sweep wave in a full batch) and
// kTicksPerGroup per 63 rows, chosen by timing full batches of mixed lengths
// (a per-wave term close to a wave's own start lag, about 270 ticks, delays
// items with few rows too long).  Batches larger than kDelayMaxBatch start
// at once (every workgroup would read every length), and no delay exceeds
// kDelayMaxTicks (1 ms, far below the bound of any device-side wait).
constexpr int kTicksPerChunk = 85;
constexpr int kTicksPerGroup = 100;
constexpr int kDelayPercent = 80;
constexpr int kDelayMaxBatch = 1024;
constexpr int kDelayMaxTicks = 100000;

__device__ __forceinline__ int est_ticks(int tx, int ty, int T, int S) {
  if (item_status(tx, ty, T, S) != kItemOk) return 0;
  return kTicksPerChunk * ((ty + kChunk - 1) / kChunk) + kTicksPerGroup * ((tx + kRowsPerWave - 1) / kRowsPerWave);
}

// Start delay of item b in ticks (wave-uniform).
__device__ __forceinline__ int start_delay(const KParams& p, int b, int lane) {
  if (p.B > kDelayMaxBatch) return 0;
  int m = 0;
  for (int i = lane; i < p.B; i += kWave) m = max(m, est_ticks(p.t_x[i], p.t_y[i], p.T, p.S));
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) m = max(m, __shfl_xor(m, off));
  const int mine = est_ticks(p.t_x[b], p.t_y[b], p.T, p.S);
  return uni(min((m - mine) / 100 * kDelayPercent, kDelayMaxTicks));
}

// ---------------------------------------------------------------- loader wave
// The value given to the tile cells of the triangle i > j.  Every cell there
// has only triangle cells as predecessors, so its Q is the max of theirs plus
// this value: -inf with -inf keeps them -inf (the method); in the legacy mode
// (a finite sentinel neg, as the paper's max_neg_val) +0 keeps them at neg
// exactly, the value Algorithm 1 initialises the cache to.  Row 0 starts from
// -0 at column -1 (so that Q[0][0] = value[0][0]), which cell (1, 0) also
// sees: in the legacy mode that cell gets neg as its value (-0 + neg = neg).
__device__ __forceinline__ float triangle_value(const KParams& p) { return p.legacy ? 0.0f : neg_inf(); }

// The cells of the triangle i > j in the landed tile of chunk c of wave g
// (slot at LDS byte address slot) become -inf: lane r rewrites tile row r
// (item row 63g + r), whose columns 32c .. 32c + nm - 1 lie in the triangle:
// whole pieces are overwritten, a piece cut by the diagonal is read and
// written back.  Only the first chunks of a wave cross the triangle.
__device__ __forceinline__ void mask_tile(const KParams& p, uint32_t slot, int g, int c, int lane) {
  const int nm = min(max(g * kRowsPerWave + lane - c * kChunk, 0), kChunk);
  using lds_f4 = __attribute__((address_space(3))) f32x4;
  const float tri = triangle_value(p);
  for (int pc = 0; 4 * pc < nm; ++pc) {
    lds_f4* const a = (lds_f4*)(uintptr_t)(slot + (uint32_t)lane * 128u + 16u * (uint32_t)(pc ^ swz(lane)));
    f32x4 v = {tri, tri, tri, tri};
    if (4 * pc + 4 > nm) {
      // (the piece has landed; other tiles may still be in flight)
      f32x4 old;
      asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(old) : "v"((uint32_t)(uintptr_t)a) : "memory");
      v.y = 4 * pc + 1 < nm ? tri : old.y;
      v.z = 4 * pc + 2 < nm ? tri : old.z;
      v.w = old.w;
    }
    // Legacy mode: cell (1, 0) follows row 0's -0 at column -1 (see
    // triangle_value), so its value is the sentinel itself.
    if (p.legacy && g == 0 && c == 0 && lane == 1 && pc == 0) v.x = p.neg;
    *a = v;
  }
}


// Value tiles of sweep wave w, chunks [c_begin, c_end), each into the slot
// its sweep wave has handed back; tiles that cross the triangle i > j get
// -inf there (mask_tile) before they are published.  ALIGNED (value 16-byte aligned, S % 4 ==
// 0): lane L of load k (k = 0..7) fetches tile row 8k + L/8, piece
// (L % 8) ^ swz(row), so each load covers eight 128-byte row segments and
// lands as eight contiguous swizzled LDS rows; up to kRing tiles in flight.
// Otherwise 4-byte loads of the same layout, one tile in flight.
//
// BOUND (the loader of wave 0 of every workgroup but an item's first): the
// sweep wave's boundary rows too.  The previous workgroup's last wave
// publishes Q of its last row as {value, tag} words in global memory; the
// loader polls four chunks per round trip (two chunks per device-scope
// load), and once a chunk's 32 words all carry this call's tag and its ring
// slot is free, moves the values into the slot's boundary row and raises the
// sweep wave's prod, as a wave of the same workgroup would.  So the sweep wave waits on LDS only: none of its
// steps waits for a global load (which would also wait for its own
// write-through stores).
template <bool ALIGNED, bool BOUND>
__device__ __forceinline__ void load_tiles(const KParams& p, SweepLds& L, const WaveCtx& x, uint32_t tag, Bound& bd) {
  const int lane = x.lane, w = x.w;
  const float* slab = p.value + (size_t)x.b * (size_t)p.T * (size_t)p.S;
  const uint64_t slab_bytes = (uint64_t)p.T * (uint64_t)p.S * 4u;
  Cursor vr = make_cursor(slab, slab_bytes);
  vr.advance((int)((uint64_t)x.g * kRowsPerWave * (uint64_t)p.S * 4u) + x.c_begin * (kChunk * 4));
  const uint32_t ring = lds_off(&L.u.ring[w][0]);
  constexpr int kOps = ALIGNED ? 8 : 32;  // loads per tile
  constexpr int kInflight = ALIGNED ? kRing : 1;
  // Per-lane byte offsets, relative to the chunk's first tile row; rows past
  // 2^31 bytes fall outside every resource.
  int voff[kOps];
#pragma unroll
  for (int k = 0; k < kOps; ++k) {
    const int r = ALIGNED ? 8 * k + (lane >> 3) : 2 * k + (lane >> 5);
    const int pos = ALIGNED ? (lane & 7) : ((lane & 31) >> 2);
    const uint32_t elem = ALIGNED ? 0u : 4u * (uint32_t)(lane & 3);
    const uint64_t o = (uint64_t)r * (uint64_t)p.S * 4u + 16u * (uint32_t)(pos ^ swz(r)) + elem;
    voff[k] = o < 0x80000000ull ? (int)o : (int)0x80000000u;
  }
  int issued = x.c_begin, readied = x.c_begin;
  bool held = x.g != 0;  // the item's first group waits for its start once its first tiles are in flight
  // The sweep wave's progress (its slots below it are free again).
  const int* const progress = w > 0 ? reinterpret_cast<const int*>(&L.box[w - 1]) + 2 : &L.cons0;
  const uint32_t ready_addr = lds_off(&L.box[w]);
  int cons = x.c_begin - 1;
  // BOUND: chunks bnext .. bend-1 still to deliver (from c_begin-1, which the
  // previous wave always computes).
  int bnext = x.c_begin - 1;
  const int bend = BOUND ? x.prev_end : bnext;
  // (the boundary words of the previous workgroup's last wave)
  const uint64_t* const bsrc = p.slots + ((size_t)x.b * p.NB + (x.g > 0 ? x.g / kWavesPerBlock - 1 : 0)) * ((size_t)p.NC * kChunk);
  const uint32_t prod_addr = lds_off(&L.box[w]) + 4u;
  const __amdgpu_buffer_rsrc_t brs = make_cursor(bsrc, (uint64_t)p.NC * kChunk * 8u).rsrc_s();
  const uint32_t bpoll_lds = lds_off(&L.bpoll[0][0]);
  int bspins = 0;
  // Issue while slots are free (the slot of chunk c held chunk c-4).
  auto issue_tiles = [&]() __attribute__((always_inline)) {
    while (issued < x.c_end && issued - readied < kInflight) {
      if (issued > cons + kRing - 1) {
        cons = uni(lds_poll(progress));
        if (issued > cons + kRing - 1) break;
      }
      const __amdgpu_buffer_rsrc_t r = vr.rsrc_s();
      const uint32_t dst = ring + (uint32_t)((issued - x.c_begin) & (kRing - 1)) * kSlotStride;
#pragma unroll
      for (int k = 0; k < kOps; ++k) {
        if (ALIGNED)
          dma16(dst + 1024u * k, r, voff[k]);
        else
          dma4(dst + 256u * k, r, voff[k]);
      }
      vr.advance(kChunk * 4);
      ++issued;
    }
  };
  while ((readied < x.c_end || bnext < bend) && !bd.out) {
    issue_tiles();
    if (!held) {
      held = true;
      const int delay = start_delay(p, x.b, lane);
      if (delay > 0) {
        const uint64_t until = wall_clock64() + (uint64_t)delay;
        while (wall_clock64() < until) __builtin_amdgcn_s_sleep(127);
      }
    }
    if (BOUND && bnext < bend) {
      if (bnext > cons + kRing - 1) cons = uni(lds_poll(progress));
      if (bnext <= cons + kRing - 1) {
        // The words of chunks c0 .. c0 + 3 (1 KiB, lane l: 16 bytes) into
        // LDS by one load past the caches, then the tiles for the slots that
        // are free now.  Loads complete in order, so waiting until only
        // those tiles are outstanding covers the poll and every tile before
        // it, and keeps the new tiles in flight: a poll does not drain the
        // loader's pipeline.  Words past the workgroup's region read as 0
        // (never a call's tag).
        const int c0 = bnext;
        dma16_dev(bpoll_lds, brs, c0 * (kChunk * 8) + 16 * lane);
        const int before = issued;
        issue_tiles();
        vm_wait_le(kOps * (issued - before));
        if (readied < before) {
          for (; readied < before; ++readied)
            if (readied < x.mask_end) mask_tile(p, ring + (uint32_t)((readied - x.c_begin) & (kRing - 1)) * kSlotStride, x.g, readied, lane);
          lds_put(ready_addr, readied);
        }
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const int c = c0 + h;
          const uint64_t wd = L.bpoll[h][lane & (kChunk - 1)];
          const uint64_t stale = __builtin_amdgcn_ballot_w64((uint32_t)(wd >> 32) != tag);
          if (bnext != c || c >= bend || c > cons + kRing - 1 || (uint32_t)stale != 0u) break;
          float* const brow = reinterpret_cast<float*>(reinterpret_cast<char*>(&L.u.ring[w][0]) +
                                                       ((c - x.c_begin) & (kRing - 1)) * kSlotStride + kBoundOff);
          if (lane < kChunk) brow[lane] = __uint_as_float((uint32_t)wd);
          lds_put(prod_addr, c + 1);
          ++bnext;
        }
        if (bnext == c0) {
          // Not published yet.
          if (++bspins > bd.limit) bd.expire();
          __builtin_amdgcn_s_sleep(1);
        } else {
          bspins = 0;
        }
        continue;
      }
    }
    if (issued == readied) {
      // Nothing in flight and no free slot: wait for the sweep wave.
      const int need = BOUND && bnext < bend ? min(issued, bnext) : issued;
      cons = wait_at_least(progress, need - (kRing - 1), bd);
      continue;
    }
    // The oldest tile in flight has landed once at most the younger ones
    // are outstanding.
    vm_wait_usual<kOps * (kInflight - 1)>(kOps * (issued - readied - 1));
    if (readied < x.mask_end) mask_tile(p, ring + (uint32_t)((readied - x.c_begin) & (kRing - 1)) * kSlotStride, x.g, readied, lane);
    ++readied;
    lds_put(ready_addr, readied);
  }
  vm_wait<0>();
}

// ---------------------------------------------------------------- step masks
// Eight columns of the step-mask recurrence (Algorithm 1's argmax loop read
// forward): the mask of (row r, column j) is d(r, j) ? mask(r-1, j-1) :
// mask(r, j-1), shifted left by one with d(r, j) as its new lowest bit, so
// that after the chunk's last column a step at column 32c + k sits at
// position 31 - k.  Everything is complemented:
//   v_lshrrev  b = wc >> 31        the lane's complemented decision;
//   v_add_co   wc += wc            the same bit into VCC, wc moves on one bit;
//   v_cndmask_dpp  xc = VCC ? pc : pc of the lane below (wave_shr:1);
//   v_lshl_or  pc = xc << 1 | b.
// Only the last two depend on the previous column (the first two fill the
// two wait states a DPP read needs after the VALU write of its source), and
// neither writes VCC, so consecutive columns do not wait on each other's
// carry.  Lane 0 (the row above the wave) has no lane below: DPP leaves its
// xc unwritten, all ones (mask 0), so a path that climbs into it contributes
// nothing more.
__device__ __forceinline__ void mask_cols8(uint32_t& wc, uint32_t& xc, uint32_t pc, uint32_t (&o)[8]) {
  uint32_t b0, b1;
#define MAS_MASK_COL(P, O, B)                                                         \
  "v_lshrrev_b32 %[" B "], 31, %[w]\n\t"                                              \
  "v_add_co_u32 %[w], vcc, %[w], %[w]\n\t"                                            \
  "v_cndmask_b32_dpp %[x], %[" P "], %[" P "], vcc wave_shr:1 row_mask:0xf bank_mask:0xf\n\t" \
  "v_lshl_or_b32 %[" O "], %[x], 1, %[" B "]\n\t"
  asm volatile(MAS_MASK_COL("p", "o0", "b0") MAS_MASK_COL("o0", "o1", "b1") MAS_MASK_COL("o1", "o2", "b0")
               MAS_MASK_COL("o2", "o3", "b1") MAS_MASK_COL("o3", "o4", "b0") MAS_MASK_COL("o4", "o5", "b1")
               MAS_MASK_COL("o5", "o6", "b0") MAS_MASK_COL("o6", "o7", "b1")
               : [o0] "=&v"(o[0]), [o1] "=&v"(o[1]), [o2] "=&v"(o[2]), [o3] "=&v"(o[3]), [o4] "=&v"(o[4]),
                 [o5] "=&v"(o[5]), [o6] "=&v"(o[6]), [o7] "=&v"(o[7]), [w] "+v"(wc), [x] "+v"(xc), [b0] "=&v"(b0),
                 [b1] "=&v"(b1)
               : [p] "v"(pc)
               : "vcc");
#undef MAS_MASK_COL
}

// A finisher wave: for every chunk of its sweep wave, once that wave's
// decision words of the chunk are in the ring slot (its progress passes c+1),
// reads them, frees the slot, computes the step masks of the wave's rows and
// of its last row entered at every position, and stores them to
// pm[b][c][kEntPerWave * g + ...] with device-scope write-through stores.
// Decisions at columns >= t_y (the last chunk's tail) count as "stay", so
// that the last row's mask describes the path from (t_x-1, t_y-1).  Once all
// of its stores have landed, the wave's done flag goes up.  The work is kept
// out of the sweep waves, whose column chain sets the pace, and out of the
// loaders, whose waits count their own loads only.
__device__ __forceinline__ void finisher_role(const KParams& p, SweepLds& L, const WaveCtx& x, uint32_t tag, Bound& bd) {
  const int lane = x.lane, w = x.w;
  if (x.g > x.g_last) return;
  const int C = (x.ty + kChunk - 1) / kChunk;
  const uint32_t top_keep = ~0u << (kChunk - 1 - (x.ty - 1) % kChunk);
  const __amdgpu_buffer_rsrc_t dr = make_cursor(p.pm + (size_t)x.b * p.NC * (size_t)p.EP, (uint64_t)p.NC * p.EP * 4u).rsrc();
  const __amdgpu_buffer_rsrc_t ddr = make_cursor(p.pd + (size_t)x.b * p.NC * (size_t)p.EP, (uint64_t)p.NC * p.EP).rsrc();
  const int base = kEntPerWave * x.g;
  const int row_off = lane > 0 ? 4 * (base + lane - 1) : -1;  // lane 0's mask (the row above) is not stored
  const int mid_off = lane >= kWave - 8 ? 4 * (base + kMidOff + 4 * (lane - (kWave - 8))) : -1;
  // Descent bytes: rows after every wave's mid entries (see mas_layout.h).
  const int row_doff = lane > 0 ? pd_row0(p.NW) + kRowsPerWave * x.g + lane - 1 : -1;
  const int mid_doff = lane >= kWave - 8 ? kChunk * x.g + 4 * (lane - (kWave - 8)) : -1;
  const int q0 = 4 * (lane - (kWave - 8));  // the first mid entry a lane in 56..63 stores
  const int* const progress = w > 0 ? reinterpret_cast<const int*>(&L.box[w - 1]) + 2 : &L.cons0;
  const uint32_t taken_addr = lds_off(&L.box[w]) + 12u;
  const uint32_t* const bits0 = reinterpret_cast<const uint32_t*>(&L.u.ring[w][kBitsOff]);
  for (int c = x.c_begin; c < x.c_end && !bd.out; ++c) {
    wait_at_least(progress, c + 2, bd);
    const uint32_t bits = bits0[((c - x.c_begin) & (kRing - 1)) * (kSlotStride / 4) + lane];
    lgkm_wait0();
    lds_put(taken_addr, c + 1);  // the slot is free again
    uint32_t wd = lane > 0 ? bits : 0u;
    if (c == C - 1) wd &= top_keep;
    uint32_t wc = ~wd, xc = ~0u;
    uint32_t h[kChunk];  // complemented masks after each column of the chunk
    {
      uint32_t o[8];
      mask_cols8(wc, xc, ~0u, o);
#pragma unroll
      for (int m = 0; m < 8; ++m) h[m] = o[m];
      mask_cols8(wc, xc, h[7], o);
#pragma unroll
      for (int m = 0; m < 8; ++m) h[8 + m] = o[m];
      mask_cols8(wc, xc, h[15], o);
#pragma unroll
      for (int m = 0; m < 8; ++m) h[16 + m] = o[m];
      mask_cols8(wc, xc, h[23], o);
#pragma unroll
      for (int m = 0; m < 8; ++m) h[24 + m] = o[m];
    }
    const int soff = c * p.EP * 4;
    const uint32_t pm_row = ~h[kChunk - 1];
    __builtin_amdgcn_raw_buffer_store_b32(pm_row, dr, row_off, soff, kPolicyDev);
    {
      // The row's descent byte (lane l: row l - 1 of the wave).
      const int s_row = __builtin_popcount(pm_row);
      const uint32_t d = s_row > lane - 1 ? kEscape + (31u - (uint32_t)__builtin_clz(pm_row | 1u)) : (uint32_t)s_row;
      __builtin_amdgcn_raw_buffer_store_b8((uint8_t)d, ddr, row_doff, c * p.EP, kPolicyDev);
    }
    // Mid entry q: the last row's mask after column 31 - q, its positions
    // raised by q; lane 63's values gathered into lanes 56..63, four each.
    float hq[kChunk];
#pragma unroll
    for (int q = 0; q < kChunk; ++q) hq[q] = __uint_as_float(h[kChunk - 1 - q]);
    const f32x4 f = gather_last_row(hq);
    const u32x4 mv = {~__float_as_uint(f.x) << q0, ~__float_as_uint(f.y) << (q0 + 1), ~__float_as_uint(f.z) << (q0 + 2),
                      ~__float_as_uint(f.w) << (q0 + 3)};
    __builtin_amdgcn_raw_buffer_store_b128(mv, dr, mid_off, soff, kPolicyDev);
    const uint32_t md = (uint32_t)__builtin_popcount(mv.x) | (uint32_t)__builtin_popcount(mv.y) << 8 |
                        (uint32_t)__builtin_popcount(mv.z) << 16 | (uint32_t)__builtin_popcount(mv.w) << 24;
    __builtin_amdgcn_raw_buffer_store_b32(md, ddr, mid_doff, c * p.EP, kPolicyDev);
  }
  vm_wait<0>();
  if (lane == 0) st_dev(p.done + (size_t)x.b * p.NW + x.g, tag);
  lds_put(lds_off(&L.fdone[w]), (int)tag);
}

// ---------------------------------------------------------------- backtrack
// Loader side of the walk: loader k (of kWinLoaders) stages the descent bytes
// of chunks C-1-k, C-1-k-4, ... down to 0, one window per chunk (WinGeom:
// its size, the slot count, up to `ahead` windows in flight), into slot
// ch % nslot once the walker has walked the chunk that slot held.  It
// publishes its progress in wready[k] as its lowest chunk staged so far
// minus 3 (its next chunk is 4 below): every chunk of its sequence at or
// above that value is staged, so that the windows of all chunks >= ch are
// in LDS once every loader's value is <= ch (-2^30 for a loader with no
// chunks).  A banded window holds the rows from the lowest one the walk can
// reach before it leaves the chunk (32 rows per chunk below the walker's row
// at issue time) up to the walker's row, after the mid entries of their waves
// and of the wave above them.  The LDS addresses that row 0's byte and wave
// 0's mid entry 0 would have in chunk ch's window go to wbase[ch % 64] and
// wmid[ch % 64] before the window is issued.
// Stops early once the walk is over.
__device__ __forceinline__ void load_windows(const KParams& p, SweepLds& L, int b, int tx, int ty, int k, int lane, Bound& bd) {
  const int C = (ty + kChunk - 1) / kChunk;
  const uint8_t* db = p.pd + (size_t)b * p.NC * (size_t)p.EP;
  const WinGeom wg = win_geom(tx, p.NW, p.T);
  const bool banded = wg.banded;
  const int nslot = wg.nslot;
  const int loads = wg.loads;
  const int row0 = pd_row0(p.NW);
  const uint32_t slot_bytes = (uint32_t)wg.ent;
  const uint32_t win0 = lds_off(&L.u.walk.area[0]);
  const uint32_t ready_addr = lds_off(&L.wready) + 4u * (uint32_t)k;
  const uint32_t base_addr = lds_off(&L.wbase[0]);
  const uint32_t mid_addr = lds_off(&L.wmid[0]);
  // `bytes` (a multiple of 256) of chunk ch's descent bytes from byte `off`
  // into LDS at dst; reads past the chunk's bytes are dropped.
  auto stage = [&](uint32_t dst, int ch, int off, int bytes) __attribute__((always_inline)) {
    const Cursor cr = make_cursor(db + (size_t)ch * p.EP + off, (uint64_t)(p.EP - off));
    const __amdgpu_buffer_rsrc_t r = cr.rsrc_s();
    const int n16 = bytes / 1024, n4 = (bytes % 1024) / 256;
    for (int q = 0; q < n16; ++q) dma16_dev(dst + 1024u * q, r, 16 * lane + 1024 * q);
    for (int q = 0; q < n4; ++q) dma4_dev(dst + 1024u * n16 + 256u * q, r, 4 * lane + 1024 * n16 + 256 * q);
  };
  constexpr int kStep = kWinLoaders;
  // Own chunks above `issued` are issued; own chunks >= `readied` are staged.
  int issued = C - 1 - k, readied = C - 1 - k + kStep;
  int slot = issued >= 0 ? issued % nslot : 0;  // slot of chunk `issued`
  if (issued < 0) lds_put(ready_addr, -(1 << 30));
  // Above the walker, which shares a SIMD with one of the loaders and issues
  // without pause: a loader's few instructions then go first.
  __builtin_amdgcn_s_setprio(3);
  // (debug build) lane n: the n-th window issued, staged; the first eight
  // only: a stamp costs the loader about as long as staging a window
  Stamps t_iss, t_rdy;
  int wpos = uni(lds_poll(&L.wpos));
  int spins = 0;
  while (readied - kStep >= 0 && wpos >= 0 && !bd.out) {
    while (issued >= 0 && readied - kStep - issued < kStep * wg.ahead) {
      // The slot holds chunk issued + nslot until the walker has walked it:
      // the published position is a chunk the walker has not walked yet.
      if (pos_chunk(wpos) >= issued + nslot) {
        wpos = uni(lds_poll(&L.wpos));
        if (wpos < 0 || pos_chunk(wpos) >= issued + nslot) break;
      }
      const uint32_t win = win0 + (uint32_t)slot * slot_bytes;
      const uint32_t at = 4u * (uint32_t)(issued & (kWave - 1));
      if (banded) {
        // Rows row_lo .. e (e: the walker's row at issue time) and the mid
        // entries of waves g_lo - 1 .. e / 63: the mid band first, then the
        // row band.
        const int e = uni(pos_row(wpos));
        const int row_lo = max(e - kChunk * nslot - 1, 0);
        const int g_mid = max(row_lo / kRowsPerWave - 1, 0);
        lds_put(base_addr + at, (int)(win + (uint32_t)wg.mids - (uint32_t)row_lo));
        lds_put(mid_addr + at, (int)(win - (uint32_t)(kChunk * g_mid)));
        stage(win, issued, kChunk * g_mid, wg.mids);
        stage(win + (uint32_t)wg.mids, issued, row0 + row_lo, wg.rows);
      } else {
        lds_put(base_addr + at, (int)(win + (uint32_t)row0));
        lds_put(mid_addr + at, (int)win);
        stage(win, issued, 0, wg.ent);
      }
      if ((C - 1 - k - issued) / kStep < 8) t_iss.at((C - 1 - k - issued) / kStep);
      issued -= kStep;
      slot -= kStep;
      if (slot < 0) slot += nslot;
      spins = 0;
    }
    const int inflight = (readied - kStep - issued) / kStep;
    if (inflight == 0) {
      // Nothing in flight: wait for the walker to free a slot.
      if (++spins > bd.limit) bd.expire();
      __builtin_amdgcn_s_sleep(1);
      wpos = uni(lds_poll(&L.wpos));
      continue;
    }
    vm_wait_exact<0, 63>(loads * (inflight - 1));
    readied -= kStep;
    lds_put(ready_addr, readied - (kStep - 1));
    if ((C - 1 - k - readied) / kStep < 8) t_rdy.at((C - 1 - k - readied) / kStep);
  }
  vm_wait<0>();
  t_iss.flush(trace_of(p).win + ((size_t)b * kWinLoaders + k) * 2 * kWave);
  t_rdy.flush(trace_of(p).win + ((size_t)b * kWinLoaders + k) * 2 * kWave + kWave);
}

// llvm.amdgcn.writelane (v_writelane_b32): lane l of `old` becomes v (v and l
// wave-uniform), the other lanes keep theirs.
extern "C" __device__ int mas_writelane(int v, int l, int old) __asm("llvm.amdgcn.writelane.i32");

// Row starts from the walk's records of up to 64 chunks: lane k holds the
// record of chunk base + k (valid when lo <= chunk <= hi): the step mask pm
// of its path and the row e the path entered it in.  The k-th lowest set bit
// p of pm is where row e - k begins: column 32 * chunk + 31 - p.  Steps from
// row 0 or below (possible only as the walk stops) are not rows.
__device__ __forceinline__ void flush_records(int* rsl, int base, int lo, int hi, uint32_t pm, int e, int lane) {
  const int c = base + lane;
  uint32_t m = (c >= lo && c <= hi) ? pm : 0u;
  int r = e;
  while (__builtin_amdgcn_ballot_w64(m != 0u) != 0) {
    if (m != 0u) {
      const int bit = __builtin_ctz(m);
      if (r >= 1) rsl[r] = c * kChunk + (kChunk - 1) - bit;
      --r;
      m &= m - 1u;
    }
  }
}

// The walker's helper, a finisher wave on another SIMD than the walker's:
// turns the walker's records into row starts as the walker hands them over,
// every 64 chunks, so that the walk does not stop for it.  A record is the
// row the path entered a chunk in and its descent byte there; the helper
// reads that row's step mask from memory (with the mid entry of the wave
// above that completes it when the path climbed out of its wave) and
// expands the masks (flush_records).  Ends after the request marked last.
__device__ __forceinline__ void walk_helper(const KParams& p, SweepLds& L, int b, int lane, Bound& bd) {
  const uint32_t* const pm_item = p.pm + (size_t)b * p.NC * (size_t)p.EP;
  for (int n = 0;; ++n) {
    // (polls spaced out: the wave may wait here through the sweep, beside
    // a sweep wave on its SIMD)
    int spins = 0;
    while (!bd.out && uni(lds_poll(&L.req_posted)) < n + 1) {
      if (++spins > bd.limit) bd.expire();
      __builtin_amdgcn_s_sleep(4);
    }
    if (bd.out) break;
    const int k = n & 1;
    const int base = uni(((volatile int*)&L.req_arg[k])[0]), lo = uni(((volatile int*)&L.req_arg[k])[1]);
    const int hi = uni(((volatile int*)&L.req_arg[k])[2]), last = uni(((volatile int*)&L.req_arg[k])[3]);
    const uint32_t d = *(volatile uint32_t*)&L.req_d[k][lane];
    const int e = *(volatile int*)&L.req_e[k][lane];
    const int c = base + lane;
    uint32_t pm = 0;
    if (c >= lo && c <= hi && e >= 0) {
      const int g = e / kRowsPerWave, rr = e - g * kRowsPerWave;
      const uint32_t* const chunk = pm_item + (size_t)c * p.EP;
      pm = ld_dev(chunk + kEntPerWave * g + rr);
      const uint32_t pos = d - kEscape;
      if (d >= kEscape && pos < kChunk - 1) pm |= ld_dev(chunk + kEntPerWave * (g - 1) + kMidOff + pos + 1);
    }
    flush_records(walk_rs(L, p.T), base, lo, hi, pm, e, lane);
    lgkm_wait0();
    lds_put(lds_off(&L.req_done), n + 1);
    if (last) break;
  }
}

// The walk of one item from (t_x-1, t_y-1) back to (0, 0) (Algorithm 1's
// argmax loop, read off the descent bytes): per chunk, from the top, the
// byte of the row the path enters the chunk in gives the row it leaves the
// chunk in: that many rows up, or, for a path that climbs into the row above
// its wave at position p, to the wave's row above and then as many rows as
// the mid entry p + 1 of the wave above says.  Each chunk's entry row and
// byte go into lane (chunk % 64) of two registers; every 64 chunks the
// helper turns them into row starts (walk_helper).  Builds row_start in
// walk_rs: the first column of every row, with rs[0] = 0 and
// rs[t_x .. T] = t_y.  Runs on the sweep wave that holds row t_x-1; the
// loaders of its workgroup stage the windows.
//
// A chunk's byte is one v_readlane of a register that holds the bytes of 64
// consecutive rows of the chunk, read from its window two chunks earlier,
// from the row the path enters the chunk above in (the path climbs at most
// 32 rows per chunk).  Only a climb into the row above a wave reads LDS on
// the chain (rare).  Chunks go in groups of four, 4q+3 down to 4q (the
// first group is partial): a group starts once the windows of its chunks and
// of the two below it are staged, checked against the staging progress read
// in the middle of the group before (read again, and waited for, only when
// that falls short); the window addresses come with the same read.  The
// walker publishes its position, by which the loaders free slots, once per
// group.  Once the path is in row 0 the rest of its group is walked
// all the same: row 0's bytes are zero.
__device__ __forceinline__ void walk(const KParams& p, SweepLds& L, int b, int tx, int ty, int lane, Bound& bd) {
  stamp(trace_of(p).item + 8 * (size_t)b + 1);
  int* rsl = walk_rs(L, p.T);
  Stamps wstamps;
  Waited waited;  // (debug build) ticks spent waiting for windows
  int e = tx - 1;                      // row of the path at the current chunk's last column
  int g = e / kRowsPerWave;            // its wave (changes only where the path climbs out of one)
  int cw = (ty - 1) / kChunk;          // chunk being walked
  const int c_top = cw;
  uint32_t rec_d = 0;   // lane k: descent byte of chunk (64-aligned base) + k
  int rec_e = 0;        // lane k: its entry row
  // Hands the records of chunks lo .. hi (lane k: chunk base + k) to the
  // helper, in request buffer posted % 2 once the request two back is done.
  int posted = 0;
  auto post = [&](int base, int lo, int hi, int last) __attribute__((always_inline)) {
    wait_at_least(&L.req_done, posted - 1, bd);
    const int k = posted & 1;
    *(volatile uint32_t*)&L.req_d[k][lane] = rec_d;
    *(volatile int*)&L.req_e[k][lane] = rec_e;
    if (lane < 4) ((volatile int*)&L.req_arg[k])[lane] = lane == 0 ? base : lane == 1 ? lo : lane == 2 ? hi : last;
    ++posted;
    lds_put(lds_off(&L.req_posted), posted);
  };
  if (e > 0) {
    // (debug build) lane k: chunks >= 32k walked; lane C/32+1: start.  A
    // stamp holds the walk for a scalar-memory round trip, so the walk takes
    // one every 32 chunks only.
    wstamps.at(min((cw >> 5) + 1, kWave - 1));
    using lds_u32 = __attribute__((address_space(3))) uint32_t;
    using lds_u8 = __attribute__((address_space(3))) uint8_t;
    using lds_i32x4 = __attribute__((address_space(3))) i32x4;
    const uint32_t wpos_addr = lds_off(&L.wpos);
    const lds_i32x4* const ready_p = (const lds_i32x4*)(uintptr_t)lds_off(&L.wready);
    const lds_u32* const base_p = (const lds_u32*)(uintptr_t)(lds_off(&L.wbase[0]) + 4u * (uint32_t)lane);
    const lds_u32* const mid_p = (const lds_u32*)(uintptr_t)(lds_off(&L.wmid[0]) + 4u * (uint32_t)lane);
    // Staging progress and window addresses as last read (the addresses
    // read after the progress: valid for every chunk it shows staged).
    // Chunks >= max_k ready[k] are staged; chunk ch's window addresses (of
    // row 0's byte and of wave 0's mid entry 0) are at lane ch % 64 of
    // `bases` and `mids`.
    auto staged_to = [&](const i32x4& r) __attribute__((always_inline)) -> int {
      return max(max(uni(r.x), uni(r.y)), max(uni(r.z), uni(r.w)));
    };
    i32x4 ready_v;
    uint32_t bases = 0, bases_n, mids = 0, mids_n;
    // Waits (bounded) until the windows of chunks >= ch are staged, reading
    // `bases` and `mids` along.
    auto ensure = [&](int ch) __attribute__((always_inline)) {
      waited.begin();
      int spins = 0;
      for (;;) {
        const i32x4 r = *(const volatile lds_i32x4*)ready_p;
        bases = *(const volatile lds_u32*)base_p;
        mids = *(const volatile lds_u32*)mid_p;
        if (staged_to(r) <= ch || bd.out) break;
        if (++spins > bd.limit) bd.expire();
        __builtin_amdgcn_s_sleep(1);
      }
      // (nothing left in flight: the group's waits count the prefetches alone)
      lgkm_wait0();
      waited.end();
    };
    // The bytes of chunk ch for rows e_b, e_b - 1, ..., e_b - 63 (lane k:
    // row e_b - k; rows are consecutive bytes), read from ch's window into
    // one register.  Lanes past row 0 or the window read whatever is there,
    // never used.
    const uint32_t lane_off = (uint32_t)(-lane);
    auto fetch = [&](int ch, int e_b) __attribute__((always_inline)) -> uint32_t {
      const uint32_t base = (uint32_t)__builtin_amdgcn_readlane((int)bases, ch & (kWave - 1));
      return *(const lds_u8*)(uintptr_t)(base + (uint32_t)e_b + lane_off);
    };
    // One chunk: its byte from lane bp - e of P (P holds the chunk's bytes
    // from row bp down), then P refilled with chunk cw - 2 from row e, the
    // row the path enters chunk cw - 1 in.
    auto body = [&](uint32_t& P, int& bp, bool publish) __attribute__((always_inline)) {
      const uint32_t d = (uint32_t)__builtin_amdgcn_readlane((int)P, bp - e);
      if (publish) lds_put(wpos_addr, walk_pos(cw, e));
      int s = (int)d;
      if (__builtin_expect(d >= kEscape, 0)) {
        // The path climbed into the row above the wave at position pos: up
        // to that row (the wave's last row above, e - 63 g + 1 rows), then
        // what the mid entry pos + 1 of the wave above adds; it goes on in
        // the wave above (a path climbs at most 32 rows per chunk).
        const uint32_t pos = d - kEscape;
        s = e - kRowsPerWave * g + 1;
        if (pos < kChunk - 1) {
          const uint32_t mb = (uint32_t)__builtin_amdgcn_readlane((int)mids, cw & (kWave - 1));
          s += uni((int)*(const lds_u8*)(uintptr_t)(mb + (uint32_t)(kChunk * (g - 1)) + pos + 1));
        }
        g -= 1;
      }
      rec_d = (uint32_t)mas_writelane((int)d, cw & (kWave - 1), (int)rec_d);
      rec_e = mas_writelane(e, cw & (kWave - 1), rec_e);
      e -= s;
      P = fetch(max(cw - 2, 0), e);  // (chunk 0 again near the end: never used)
      bp = e;
      cw -= 1;
      // The next chunk's v_readlane stays after this prefetch: hoisted above
      // it, it would wait for the prefetch it reads to be the last LDS load
      // in flight rather than the last but one.
      __builtin_amdgcn_sched_barrier(0);
    };
    // Records are complete for a 64-aligned group once its lowest chunk is
    // walked: the helper turns them into row starts.  (The wait after the
    // hand-off leaves nothing of its LDS stores outstanding, so that the
    // compiler can count the prefetches exactly.)
    auto flush_at = [&](int walked) __attribute__((always_inline)) {
      if ((walked & (kWave - 1)) == 0) {
        post(walked, walked, c_top, 0);
        lgkm_wait0();
      }
    };

    // The first group: windows down to two chunks below it, then the
    // first two registers.
    const int q_top = cw >> 2;
    ensure(max(4 * q_top - 2, 0));
    uint32_t Pa = fetch(cw, e), Pb = fetch(max(cw - 1, 0), e);
    int ba = e, bb = e;
    // Nothing may be outstanding on the LDS/scalar-memory counter when the
    // loops start: a scalar load still in flight (the compiler hoists
    // kernel-argument loads) would make every wait inside them a full one,
    // and the waits of the group loop count on the two prefetches alone.
    lgkm_wait0();
    while (cw >= 4 * q_top) {
      // Pa holds the chunk walked next: swap after each body.
      body(Pa, ba, true);
      flush_at(cw + 1);
      const uint32_t t = Pa;
      Pa = Pb;
      Pb = t;
      const int tb = ba;
      ba = bb;
      bb = tb;
    }
    // Whole groups of four: chunk 4q+3 uses Pa, 4q+2 Pb, and so on.  The
    // staging progress is read after the second chunk of a group, for the
    // check at the next group's start.
    bool have_read = false;
    while (cw >= 0 && e > 0) {
      const int need = max(cw - 5, 0);
      if (((cw + 1) & 31) == 0) wstamps.at((cw + 1) >> 5);
      if (have_read && staged_to(ready_v) <= need)
        bases = bases_n, mids = mids_n;
      else
        ensure(need);
      body(Pa, ba, true);
      body(Pb, bb, false);
      ready_v = *(const volatile lds_i32x4*)ready_p;
      bases_n = *(const volatile lds_u32*)base_p;
      mids_n = *(const volatile lds_u32*)mid_p;
      have_read = true;
      body(Pa, ba, false);
      body(Pb, bb, false);
      flush_at(cw + 1);
    }
    wstamps.at(max(cw + 1, 0) >> 5);
  }
  // The partial group of records the walk ended in (chunk cw + 1 was walked
  // last; none if that group was handed over already or nothing was
  // walked), marked last; then every request is done.
  if (tx > 1) {
    const int lo = cw + 1;
    post(lo & ~(kWave - 1), lo, (lo & (kWave - 1)) != 0 ? c_top : lo - 1, 1);
  } else {
    post(0, 0, -1, 1);
  }
  wait_at_least(&L.req_done, posted, bd);
  wstamps.flush(trace_of(p).walk + (size_t)b * kWave);
  waited.flush(trace_of(p).item + 8 * (size_t)b + 4);
  wave_lds_sync();
  lds_put(lds_off(&L.wpos), -1);
  if (lane == 0) rsl[0] = 0;
  for (int i = tx + lane; i <= p.T; i += kWave) rsl[i] = ty;
  wave_lds_sync();
}

// ---------------------------------------------------------------- path writer
// Rows [r0, r1) of the dense path of item b (Sec. 2: the alignment as a 0/1
// matrix of the input's size) from its published row_start table: row i
// holds ones at columns [rs[i], rs[i+1]) and zeros elsewhere (rows t_x .. T-1
// and invalid items: all zeros).  path16: per row, zero pieces by 16-byte
// stores (the pieces holding ones are skipped: offset past the resource),
// then the few pieces holding ones; otherwise bytes.  The stores are
// streaming (nt): the path is written once and never read here, and keeping
// it out of the caches leaves them to the sweeps still running (a launch on
// the bench batch took 206 us with cached stores, 179 us with these).  (Bounds are
// clamped to the row: the table is read back from memory, never trusted
// blindly.)
__device__ __forceinline__ void write_path_rows(const KParams& p, int b, int r0, int r1, int lane) {
  const uint32_t* const rs = reinterpret_cast<const uint32_t*>(p.row_start) + (size_t)b * ((size_t)p.T + 1);
  uint8_t* const item_path = p.path + (size_t)b * (size_t)p.T * (size_t)p.S;
  const __amdgpu_buffer_rsrc_t r = make_cursor(item_path, (uint64_t)p.T * p.S).rsrc();
  const u32x4 zero = {0u, 0u, 0u, 0u};
  for (int i0 = r0; i0 < r1; i0 += kWave) {
    const int n = min(kWave, r1 - i0);
    const int v = (int)ld_dev(rs + min(i0 + lane, p.T));
    const int vlast = (int)ld_dev(rs + min(i0 + kWave, p.T));
    for (int k2 = 0; k2 < n; ++k2) {
      const int a = __builtin_amdgcn_readlane(v, k2);
      const int e = k2 + 1 < kWave ? __builtin_amdgcn_readlane(v, k2 + 1) : vlast;
      const int lo = min(max(a, 0), p.S), hi = min(max(e, lo), p.S);
      const int row = i0 + k2;
      if (p.path16) {
        const int plo = lo >> 4, phi = hi > lo ? (hi + 15) >> 4 : plo;  // pieces holding ones
        for (int pc = lane; pc < p.S / 16; pc += kWave)
          __builtin_amdgcn_raw_buffer_store_b128(zero, r, (pc < plo || pc >= phi) ? row * p.S + 16 * pc : -1, 0, kPolicyStream);
        for (int pc = plo + lane; pc < phi; pc += kWave)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, path_piece(lo, hi, 16 * pc)), r, row * p.S + 16 * pc, 0,
                                                 kPolicyStream);
      } else {
        uint8_t* const rowp = item_path + (size_t)row * p.S;
        for (int j = lane; j < p.S; j += kWave) rowp[j] = (uint8_t)(j >= lo && j < hi);
      }
    }
  }
}

// The item published k-th in this call (its entry in the completion order
// carries the call's tag), or -1 once the bounded wait times out.  That wait
// spans whole sweeps and walks, so its bound grows with the longest item
// (limit polls per 256 chunks).
__device__ __forceinline__ int wait_published(const KParams& p, int k, uint32_t tag, int64_t limit, Bound& bd) {
  int64_t spins = 0;
  for (;;) {
    const uint64_t e = __hip_atomic_load(p.order + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((uint32_t)(e >> 32) == tag) {
      const int b = (int)(uint32_t)e;
      return b < p.B ? b : -1;
    }
    if (bd.out) return -1;
    if (++spins > limit) {
      // Raise the call's flag, then look once more: an item published after
      // this point reads the flag and reports itself as timed out.
      bd.expire();
      const uint64_t e2 = __hip_atomic_load(p.order + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int b = (int)(uint32_t)e2;
      return (uint32_t)(e2 >> 32) == tag && b < p.B ? b : -1;
    }
    __builtin_amdgcn_s_sleep(2);
  }
}

// A path-writer workgroup: takes tile t = (k, part) from the shared counter,
// rows [R part, R part + R) of the item published k-th (R = kPathTileRows),
// waits for that item, writes the tile (each wave an equal share of its rows)
// and goes on until the tiles run out.  The next tile is taken while the
// workgroup waits for this one's item.  Wave 0 alone polls the completion
// order (device-scope loads, which go past the caches) and hands the item to
// the other waves through LDS; they wait at the barrier meanwhile, so a
// waiting workgroup puts one poll rather than twelve on the memory system
// at a time, beside the sweeps still running.
__device__ __forceinline__ void path_writer(const KParams& p, SweepLds& L, uint32_t tag, int wv, int lane, Bound& bd) {
  constexpr int kWaves = kThreads / kWave;
  const int ntiles = p.B * p.ntile;
  int max_chunks = 0;
  for (int i = lane; i < p.B; i += kWave)
    if (item_status(p.t_x[i], p.t_y[i], p.T, p.S) == kItemOk) max_chunks = max(max_chunks, (p.t_y[i] + kChunk - 1) / kChunk);
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) max_chunks = max(max_chunks, __shfl_xor(max_chunks, off));
  const int64_t limit = (int64_t)bd.limit * (1 + uni(max_chunks) / 256);
  if (threadIdx.x == 0)
    L.tile = (int)__hip_atomic_fetch_add(&p.hdr->tile_next, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  int t = L.tile;
  while (t < ntiles) {
    const int k = t / p.ntile, part = t - k * p.ntile;
    if (wv == 0) {
      uint32_t next = 0;
      if (lane == 0) next = __hip_atomic_fetch_add(&p.hdr->tile_next, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int b0 = wait_published(p, k, tag, limit, bd);
      if (lane == 0) {
        L.pub = b0;
        L.tile = (int)next;
      }
    }
    __syncthreads();
    const int b = L.pub, tn = L.tile;
    const int q0 = part * kPathTileRows, q1 = min(q0 + kPathTileRows, p.T);
    const int per = (q1 - q0 + kWaves - 1) / kWaves;
    const int r0 = min(q0 + wv * per, q1), r1 = min(r0 + per, q1);
    if (wv == 0) stamp(trace_of(p).tile + 2 * (size_t)t + 0);
    if (r1 > r0 && b >= 0) write_path_rows(p, b, r0, r1, lane);
    if (wv == 0) stamp(trace_of(p).tile + 2 * (size_t)t + 1);
    __syncthreads();  // every wave has read L.pub and L.tile
    t = tn;
  }
}

// ---------------------------------------------------------------- roles
// Item b's row_start table is complete once this wave's stores have landed:
// append b to the call's completion order, which the path writers follow.
__device__ __forceinline__ void publish_item(const KParams& p, int b, uint32_t tag, int lane) {
  vm_wait<0>();
  if (lane == 0) {
    const uint32_t k = __hip_atomic_fetch_add(&p.hdr->walk_count, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (k < (uint32_t)p.B)
      __hip_atomic_store(p.order + k, ((uint64_t)tag << 32) | (uint32_t)b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// The workgroup of the wave holding row t_x-1 walks the item: that wave walks
// and publishes row_start, the workgroup's four loaders stage the decision
// windows.
__device__ __forceinline__ bool walker_workgroup(const WaveCtx& x) {
  return x.g / kWavesPerBlock == x.g_last / kWavesPerBlock;
}

__device__ __forceinline__ void sweep_role(const KParams& p, SweepLds& L, const WaveCtx& x, uint32_t tag, Bound& bd) {
  const int lane = x.lane, b = x.b, g = x.g, w = x.w, g_last = x.g_last;
  if (g > g_last) return;  // no rows of the alignment here
  float score;
  if (g == g_last) {
    score = g == 0 ? sweep_wave<0, 0>(p, L, x, tag, bd) : sweep_wave<1, 0>(p, L, x, tag, bd);
  } else if (w < kWavesPerBlock - 1) {
    score = g == 0 ? sweep_wave<0, 1>(p, L, x, tag, bd) : sweep_wave<1, 1>(p, L, x, tag, bd);
  } else {
    score = sweep_wave<1, 2>(p, L, x, tag, bd);
  }
  if (g != g_last) return;

  // The walker.
  if (lane == (x.tx - 1) - g_last * kRowsPerWave + 1 && p.score) p.score[b] = score;
  walk(p, L, b, x.tx, x.ty, lane, bd);
  stamp(trace_of(p).item + 8 * (size_t)b + 2);
  int32_t* rs_out = p.row_start + (size_t)b * ((size_t)p.T + 1);
  const int* const rsl = walk_rs(L, p.T);
  for (int i = lane; i <= p.T; i += kWave) st_dev(reinterpret_cast<uint32_t*>(rs_out + i), (uint32_t)rsl[i]);
  if (p.durations) {
    // Frames per text row (Sec. 2: what the duration predictor learns): the
    // row's span of columns; 0 for rows past t_x.
    int32_t* d = p.durations + (size_t)b * (size_t)p.T;
    for (int i = lane; i < p.T; i += kWave) d[i] = rsl[i + 1] - rsl[i];
  }
  publish_item(p, b, tag, lane);
  stamp(trace_of(p).item + 8 * (size_t)b + 3);
  // The item's status, once every wave whose work reaches its outputs has
  // passed its last wait: timed out if any of them (or this walker) gave up,
  // or if a path writer gave up before the publication became visible to it.
  vm_wait<0>();
  const bool tmo = bd.out || ld_dev(p.tmo + b) == tag || ld_dev(&p.hdr->path_fail) == tag;
  if (lane == 0 && p.status) p.status[b] = tmo ? kItemSyncTimeout : kItemOk;
}

template <bool ALIGNED>
__device__ __forceinline__ void loader_role(const KParams& p, SweepLds& L, const WaveCtx& x, uint32_t tag, Bound& bd) {
  const int lane = x.lane, b = x.b, g = x.g, g_last = x.g_last;
  if (g <= g_last) {
    if (g > 0 && x.w == 0)
      load_tiles<ALIGNED, true>(p, L, x, tag, bd);
    else
      load_tiles<ALIGNED, false>(p, L, x, tag, bd);
  }
  if (!walker_workgroup(x)) return;
  // Decision windows for the walk, once every wave of the item has published
  // its step masks: the waves of earlier workgroups through their done
  // flags in memory, this workgroup's through LDS (no memory round trip).
  const int g_own = (g_last / kWavesPerBlock) * kWavesPerBlock;
  wait_flags(p.done + (size_t)b * p.NW, g_own, tag, lane, bd);
  wait_tags(L.fdone, g_last - g_own + 1, tag, bd);
  if (x.w == 0) stamp(trace_of(p).item + 8 * (size_t)b + 0);
  load_windows(p, L, b, x.tx, x.ty, x.w, lane, bd);
}

// Items with invalid lengths: an all-zero slab, zero row_start, score -inf.
__device__ __forceinline__ void invalid_item(const KParams& p, int b, int g, bool is_loader, int lane, int st, uint32_t tag) {
  if (is_loader || g != 0) return;
  int32_t* rs_out = p.row_start + (size_t)b * ((size_t)p.T + 1);
  for (int i = lane; i <= p.T; i += kWave) st_dev(reinterpret_cast<uint32_t*>(rs_out + i), 0u);
  if (p.durations)
    for (int i = lane; i < p.T; i += kWave) p.durations[(size_t)b * (size_t)p.T + i] = 0;
  if (lane == 0) {
    if (p.score) p.score[b] = neg_inf();
    if (p.status) p.status[b] = st;
  }
  // The path writers write the all-zero slab from this table.
  publish_item(p, b, tag, lane);
}

// The last workgroup of the call to finish clears the call's counters and
// advances the generation (one counter update per workgroup: updates of one
// word serialise).
__device__ __forceinline__ void finish_call(const KParams& p, uint32_t gen) {
  vm_wait<0>();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t total = gridDim.x;
    const uint32_t prev = __hip_atomic_fetch_add(&p.hdr->exit_count, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == total - 1) {
      __hip_atomic_store(&p.hdr->walk_count, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&p.hdr->tile_next, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&p.hdr->exit_count, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&p.hdr->gen, gen + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Twelve waves per workgroup (four sweep waves, four loaders, four
// finishers), one workgroup per CU.
template <bool ALIGNED>
__global__ void __launch_bounds__(kThreads, 1) mas_kernel(KParams p) {
  __shared__ SweepLds L;
  if (threadIdx.x == 0) stamp(trace_of(p).wg + 2 * (size_t)blockIdx.x);
  if (__hip_atomic_load(&p.hdr->magic, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != kWsMagic) {
    // Not an initialised workspace: report it and touch nothing else.
    if (blockIdx.x == 0 && p.status)
      for (int i = threadIdx.x; i < p.B; i += blockDim.x) p.status[i] = kItemBadWorkspace;
    return;
  }
  const uint32_t gen = __hip_atomic_load(&p.hdr->gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t tag = call_tag(gen);
  const int sid = blockIdx.x;
  if (sid >= p.B * p.NB) {
    // A path writer.
    Bound bd{p.spin_limit, false, &p.hdr->path_fail, tag};
    path_writer(p, L, tag, uni(threadIdx.x / kWave), threadIdx.x & (kWave - 1), bd);
    if (bd.out) __hip_atomic_store(&p.hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x == 0) stamp(trace_of(p).wg + 2 * (size_t)blockIdx.x + 1);
    finish_call(p, gen);
    return;
  }
  const int b = sid % p.B;
  const int r = sid / p.B;
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = uni(threadIdx.x / kWave);
  const int w = wv & (kWavesPerBlock - 1);
  const bool is_finisher = wv >= 2 * kWavesPerBlock;
  const bool is_loader = wv >= kWavesPerBlock && !is_finisher;
  const int g = r * kWavesPerBlock + w;
  const int tx = p.t_x[b];
  const int ty = p.t_y[b];
  const int st = item_status(tx, ty, p.T, p.S);
  Bound bd{p.spin_limit, false, p.tmo + b, tag};

  // Workgroup set-up: the LDS holds whatever earlier workgroups left.
  if (threadIdx.x < kWavesPerBlock) {
    // Nothing loaded or delivered yet; every wave's progress is just below
    // its first chunk (it first reads the boundary row of chunk c_begin-1).
    const int gg = r * kWavesPerBlock + (int)threadIdx.x;
    L.box[threadIdx.x] = i32x4{chunk_begin(gg), chunk_begin(gg) - 1, chunk_begin(gg + 1) - 1, chunk_begin(gg)};
  }
  if (threadIdx.x == 0) {
    L.cons0 = chunk_begin(r * kWavesPerBlock) - 1;
    L.wready = i32x4{1 << 30, 1 << 30, 1 << 30, 1 << 30};
    // Walker not started: at chunk C (every window slot free), row t_x-1.
    lds_store(&L.wpos, walk_pos((ty + kChunk - 1) / kChunk, max(tx - 1, 0)));
  }
  if (threadIdx.x < kWave) L.wbase[threadIdx.x] = (int)lds_off(&L.u.walk.area[0]);
  if (threadIdx.x < kWavesPerBlock) L.fdone[threadIdx.x] = 0u;  // never a tag (tags are odd)
  if (threadIdx.x == 0) {
    L.req_posted = 0;
    L.req_done = 0;
  }
  __syncthreads();

  if (st != kItemOk) {
    invalid_item(p, b, g, is_loader || is_finisher, lane, st, tag);
  } else {
    const WaveCtx x = make_ctx(b, g, w, lane, tx, ty);
    if (is_finisher) {
      finisher_role(p, L, x, tag, bd);
      // (the finisher two SIMDs away from the walker helps it)
      if (walker_workgroup(x) && w == (((x.g_last & (kWavesPerBlock - 1)) + 2) & (kWavesPerBlock - 1)))
        walk_helper(p, L, x.b, lane, bd);
    }
    else if (is_loader)
      loader_role<ALIGNED>(p, L, x, tag, bd);
    else
      sweep_role(p, L, x, tag, bd);
  }
  if (bd.out) __hip_atomic_store(&p.hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  stamp(trace_of(p).wg + 2 * (size_t)blockIdx.x + 1);  // (one wave's stamp: the last to get here wins)
  finish_call(p, gen);
}

// ---------------------------------------------------------------- path writer
// Aligned variant: S % 16 == 0 and path 16-byte aligned.  One thread writes one
// 16-byte piece; consecutive threads write consecutive pieces of a row.
__global__ void __launch_bounds__(256) mas_path_kernel16(const int32_t* __restrict__ row_start, int32_t B, int32_t T, int32_t S,
                                                        uint4* __restrict__ path) {
  const int P = S / 16;
  const size_t n = (size_t)B * T * P;
  for (size_t k = (size_t)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) {
    const size_t bi = k / P;  // b * T + i
    const int pc = (int)(k - bi * P);
    const size_t b = bi / T;
    const int i = (int)(bi - b * T);
    const int32_t* rs = row_start + b * ((size_t)T + 1);
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4, path_piece(rs[i], rs[i + 1], pc * 16)),
                                reinterpret_cast<u32x4*>(path + k));
  }
}

// General variant: one thread per byte.
__global__ void __launch_bounds__(256) mas_path_kernel1(const int32_t* __restrict__ row_start, int32_t B, int32_t T, int32_t S,
                                                       uint8_t* __restrict__ path) {
  const size_t n = (size_t)B * T * S;
  for (size_t k = (size_t)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (size_t)gridDim.x * blockDim.x) {
    const size_t bi = k / S;
    const int j = (int)(k - bi * S);
    const size_t b = bi / T;
    const int i = (int)(bi - b * T);
    const int32_t* rs = row_start + b * ((size_t)T + 1);
    path[k] = (uint8_t)(rs[i] <= j && j < rs[i + 1]);
  }
}

// ---------------------------------------------------------------- workspace fill
// Zeros, except the header's magic word (its 16-byte piece is written by one
// thread, whole).
__global__ void __launch_bounds__(256) mas_ws_init_kernel(uint4* __restrict__ p, size_t n16) {
  for (size_t k = (size_t)blockIdx.x * blockDim.x + threadIdx.x; k < n16; k += (size_t)gridDim.x * blockDim.x)
    p[k] = k == (size_t)kWsMagicPiece ? make_uint4(0u, kWsMagic, 0u, 0u) : make_uint4(0u, 0u, 0u, 0u);
}

// ---------------------------------------------------------------- launchers
hipError_t launch_mas(const KParams& p, hipStream_t stream) {
  const int writers = p.path ? min(p.B * p.ntile, kPathWorkgroups) : 0;
  const dim3 grid((unsigned)(p.B * p.NB + writers)), block(kThreads);
  const bool aligned = (p.S % 4 == 0) && ((uintptr_t)p.value % 16 == 0);
  if (aligned)
    hipLaunchKernelGGL(mas_kernel<true>, grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL(mas_kernel<false>, grid, block, 0, stream, p);
  return hipGetLastError();
}

static unsigned stream_grid(size_t n, unsigned per_block) {
  const size_t want = (n + per_block - 1) / per_block;
  const size_t cap = 256 * 32;  // 32 workgroups per CU
  return (unsigned)(want < 1 ? 1 : (want > cap ? cap : want));
}

hipError_t launch_path(const int32_t* row_start, int32_t B, int32_t T, int32_t S, uint8_t* path, hipStream_t stream) {
  if (S % 16 == 0 && ((uintptr_t)path % 16) == 0) {
    const size_t n = (size_t)B * T * (S / 16);
    hipLaunchKernelGGL(mas_path_kernel16, dim3(stream_grid(n, 256)), dim3(256), 0, stream, row_start, B, T, S,
                       reinterpret_cast<uint4*>(path));
  } else {
    const size_t n = (size_t)B * T * S;
    hipLaunchKernelGGL(mas_path_kernel1, dim3(stream_grid(n, 256)), dim3(256), 0, stream, row_start, B, T, S, path);
  }
  return hipGetLastError();
}

__global__ void __launch_bounds__(256) mas_fill_kernel(uint4* __restrict__ p, size_t n16) {
  for (size_t k = (size_t)blockIdx.x * blockDim.x + threadIdx.x; k < n16; k += (size_t)gridDim.x * blockDim.x)
    p[k] = make_uint4(0u, 0u, 0u, 0u);
}

hipError_t launch_fill(void* p, size_t bytes, hipStream_t stream) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  hipLaunchKernelGGL(mas_fill_kernel, dim3(stream_grid(n16, 256)), dim3(256), 0, stream, reinterpret_cast<uint4*>(p), n16);
  return hipGetLastError();
}

hipError_t launch_ws_init(void* p, size_t bytes, hipStream_t stream) {
  static_assert(offsetof(WsHeader, magic) == 16 * kWsMagicPiece + 4, "magic is the second word of its piece");
  const size_t n16 = bytes / 16;
  hipLaunchKernelGGL(mas_ws_init_kernel, dim3(stream_grid(n16, 256)), dim3(256), 0, stream, reinterpret_cast<uint4*>(p), n16);
  return hipGetLastError();
}

}  // namespace mas

#ifdef MAS_TRACE
// Debug build only: where the kernels record their timeline (nullptr: off).
extern "C" int mas_trace_set(void* buffer) {
  return (int)hipMemcpyToSymbol(HIP_SYMBOL(mas::g_trace), &buffer, sizeof(buffer));
}
#endif
