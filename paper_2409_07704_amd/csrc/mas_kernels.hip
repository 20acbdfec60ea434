// libmas kernels for gfx950 (MI355X): batched monotonic alignment search
// (Super-MAS Sec. 2, Algorithm 1; column-parallel forward loop of
// Algorithm 2) and the dense path writer.
//
// One launch computes everything (mas_kernel).  A workgroup owns 256 text
// rows of one item: four waves, one text row per lane, 64 rows per wave.  A
// wave walks the speech axis in chunks of 32 columns.
//   * The recurrence's only cross-row dependency, the diagonal predecessor
//     Q[i-1][j-1], crosses lanes with one DPP wave_shr:1 per column, crosses
//     waves of a workgroup through an LDS ring, and crosses workgroups
//     through 64-bit {value, tag} words in global memory.  Wave g starts at
//     chunk floor(64g / 32): all earlier cells of its rows lie in the masked
//     triangle i > j, so waves are naturally skewed by 64 columns.
//   * Value tiles (64 rows x 32 columns) travel HBM -> LDS by buffer loads
//     with the lds flag, three chunks ahead, eight coalesced 16-byte pieces
//     per lane, into an XOR-swizzled layout from which each lane reads its
//     own row's 32 values.
//   * Q is never materialised: each lane keeps its row's previous column in
//     a register.  Each column's 64-row decision mask is the compare's SGPR
//     mask; every lane shifts its bit into a 32-bit word (v_addc with the
//     mask as carry-in), stored once per chunk.
//   * The dense path is cleared by the same waves: each wave zeroes its own
//     64 rows of the path, two 1 KiB stores per chunk step.
//   * The wave owning row t_x-1 then walks the decision words backwards from
//     (t_x-1, t_y-1), four chunks per block (words fetched two blocks ahead,
//     staged in LDS; one find-first-set per row change), builds row_start
//     in LDS and writes the item's ones into the cleared path.
//
// Vector-memory accounting: gfx9 retires a wave's vector-memory operations
// (loads and stores alike) in issue order, so "the operation issued N
// operations ago has completed" is s_waitcnt vmcnt(N).  Every vector-memory
// operation of the sweep loop is issued from inline assembly in a fixed
// sequence per step, and each step waits with a count derived from that
// sequence; the compiler neither sees these operations nor inserts waits
// for them.  Loads that feed the loop write LDS, never registers, so no
// register is written behind the compiler's back.
//
// Memory ordering across workgroups: data handed between workgroups
// (decision words, boundary words, flags, path bytes) is written with
// device-scope write-through stores and read with device-scope loads, and a
// wave waits for all its stores (vmcnt(0)) before raising a flag, so no cache
// write-back or invalidation is needed.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mas_internal.h"

namespace mas {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

// Keeps the compiler from moving LDS accesses across this point; LDS
// operations of one wave execute in order, so no wait is needed.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Device-scope (write-through) stores and loads of data shared across
// workgroups, outside the sweep loop.
__device__ __forceinline__ void st_dev(uint32_t* p, uint32_t v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ void st_dev(uint64_t* p, uint64_t v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ void st_dev(uint8_t* p, uint8_t v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ uint32_t ld_dev(const uint32_t* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }

__device__ __forceinline__ int lds_load(const int* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP); }
__device__ __forceinline__ void lds_store(int* p, int v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP); }

__device__ __forceinline__ uint32_t call_tag(uint32_t gen) { return 2u * gen + 1u; }

constexpr int kSpinLimit = 1 << 21;  // bound of every device-side wait (~seconds)
constexpr int kOnesPerLane = 128;    // path bytes a lane writes for its own row before the wave helps
constexpr int kDepth = 3;            // value tiles in flight ahead of the one computed
constexpr int kStages = 4;           // LDS tile slots per wave (kDepth + 1, a power of two)
constexpr int kPollSlots = 4;        // LDS slots of polled boundary words
static_assert(kStages == kDepth + 1 && (kStages & (kStages - 1)) == 0, "tile ring");

// ---------------------------------------------------------------- vector memory (inline asm)
// Byte offset of a __shared__ object inside the workgroup's LDS allocation.
template <typename T>
__device__ __forceinline__ uint32_t lds_off(T* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) T*)p;
}

// Waits until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N <= 63, "vmcnt is a 6-bit counter");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// A buffer resource that moves forward through a region: base and number of
// bytes left, turned into a descriptor (raw buffer, 32-bit data format) at
// each use.  Loads at offsets >= num_records return 0 and such stores are
// dropped (the per-lane offset is range-checked, the scalar offset is not).
constexpr int kRsrcWord3 = 0x00020000;
// The count update is written as scalar instructions: the compiler turns
// the saturating subtraction into a vector instruction otherwise, and the
// descriptor must live in scalar registers.  Byte counts are below 2^31.
struct Cursor {
  const char* base;
  int left;
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc() const {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), 0, left, kRsrcWord3);
  }
  __device__ __forceinline__ void advance(int step) {
    base += step;
    asm("s_sub_i32 %0, %0, %1\n\ts_max_i32 %0, %0, 0" : "+s"(left) : "s"(step) : "scc");
  }
};
__device__ __forceinline__ Cursor make_cursor(const void* p, int bytes) { return Cursor{static_cast<const char*>(p), bytes}; }

// Buffer resource over the bytes [off, total) of the region at p (empty
// when off >= total; total < 2^31).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t sub_rsrc(const void* p, uint64_t total, uint64_t off) {
  const uint64_t o = off < total ? off : total;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(static_cast<const char*>(p)) + o, 0, (int)(uint32_t)(total - o),
                                           kRsrcWord3);
}

// Loads into LDS (the lds flag): every lane's bytes at its voffset go to LDS
// at M0 + size * lane.  A scalar write of M0 needs one wait state before
// such a load.  OFF is added to the LDS base.
template <int OFF>
__device__ __forceinline__ void dma16(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  asm volatile("s_add_u32 m0, %[l], %[o]\n\ts_nop 0\n\tbuffer_load_dwordx4 %[v], %[r], 0 offen lds"
               :
               : [l] "s"(lds), [o] "n"(OFF), [r] "s"(r), [v] "v"(voff)
               : "memory", "m0", "scc");
}
template <int OFF>
__device__ __forceinline__ void dma4(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  asm volatile("s_add_u32 m0, %[l], %[o]\n\ts_nop 0\n\tbuffer_load_dword %[v], %[r], 0 offen lds"
               :
               : [l] "s"(lds), [o] "n"(OFF), [r] "s"(r), [v] "v"(voff)
               : "memory", "m0", "scc");
}
// Device-scope (sc1) variants for data written by other workgroups.
__device__ __forceinline__ void dma4_dev(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  asm volatile("s_mov_b32 m0, %[l]\n\ts_nop 0\n\tbuffer_load_dword %[v], %[r], 0 offen sc1 lds"
               :
               : [l] "s"(lds), [r] "s"(r), [v] "v"(voff)
               : "memory", "m0");
}
// One 16-byte load per lane, device-scope: the bytes at voff of the resource
// to LDS at lds + 16 lane.
__device__ __forceinline__ void dma_piece(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  asm volatile("s_mov_b32 m0, %[l]\n\ts_nop 0\n\tbuffer_load_dwordx4 %[v], %[r], 0 offen sc1 lds"
               :
               : [l] "s"(lds), [r] "s"(r), [v] "v"(voff)
               : "memory", "m0");
}

// Stores at voff + soff of a resource, device-scope (write-through).
__device__ __forceinline__ void buf_store32(uint32_t v, int voff, __amdgpu_buffer_rsrc_t r, uint32_t soff) {
  asm volatile("buffer_store_dword %[d], %[v], %[r], %[s] offen sc1" ::[d] "v"(v), [v] "v"(voff), [r] "s"(r), [s] "s"(soff)
               : "memory");
}
__device__ __forceinline__ void buf_store64(uint64_t v, int voff, __amdgpu_buffer_rsrc_t r, uint32_t soff) {
  asm volatile("buffer_store_dwordx2 %[d], %[v], %[r], %[s] offen sc1" ::[d] "v"(v), [v] "v"(voff), [r] "s"(r), [s] "s"(soff)
               : "memory");
}
// A 16-byte zero store (s_nop: a VALU write of store data needs one wait
// state).  Path bytes are only ever written by the wave that owns their row,
// so this needs no device-scope write-through.
__device__ __forceinline__ void vm_zero1(uint64_t a, u32x4 z) {
  asm volatile("global_store_dwordx4 %0, %1, off\n\ts_nop 0" ::"v"(a), "v"(z) : "memory");
}

// The recurrence, one text row per lane, lane 0 carrying the row above the
// wave.  Per column j (Algorithm 2's parallel step):
//   t      = max(Q[r-1][j-1], Q[r][j-1])    v_max_f32 with DPP wave_shr:1
//                                            (lane l reads lane l-1's Q);
//   Q[r][j] = t + value[r][j]               one fp32 add;
//   d      = sign(Q[r][j-1] - t)            1 iff the diagonal is strictly
//                                            greater (-0 below +0, the order
//                                            of v_max_f32 and of R2);
//   bits   = bits << 1 | d                  v_alignbit (first column ends in
//                                            bit 31 after 32 columns).
// Lane 0 has no lane below it: DPP leaves its t untouched, and t is kept at
// -0 in lane 0 for the whole sweep, so lane 0's Q becomes -0 + value = value
// exactly (x + -0 = x for every x): lane 0's "values" are the Q of the row
// above, handed down by the previous wave (or -inf above row 0).
// A VALU write followed by a DPP read of the same register needs two wait
// states: each column's add is followed by two other VALU instructions
// before the next column reads it, and each block starts with s_nop 1.
__device__ __forceinline__ void cols8(float& q, float& t, uint32_t& bits, float (&o)[8], const float* v) {
  float u;
  asm("s_nop 1\n\t"
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

// One column of the same step (for the chunks that cross the masked triangle).
__device__ __forceinline__ float col1(float q, float& t, uint32_t& bits, float v) {
  float o, u;
  asm("s_nop 1\n\t"
      "v_max_f32_dpp %[t], %[q], %[q] wave_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32 %[o], %[t], %[v]\n\t"
      "v_sub_f32 %[u], %[q], %[t]\n\t"
      "v_alignbit_b32 %[b], %[b], %[u], 31"
      : [o] "=&v"(o), [t] "+v"(t), [b] "+v"(bits), [u] "=&v"(u)
      : [q] "v"(q), [v] "v"(v));
  return o;
}

// One 32-column chunk for lanes 1..63 (rows row0 + lane - 1) and the carried
// row in lane 0.  v: this lane's 32 values (lane 0: the row above's Q);
// qc: Q of every column (out); bits: decisions, first column in bit 31.
// MASKED: the chunk crosses the triangle i > j, where Q is -inf (lane 0's
// copies already are), and holds the first cell Q[0][0] = value[0][0] when
// j0 == 0.
template <bool MASKED>
__device__ __forceinline__ void sweep_chunk(float& q, float& t, const f32x4 (&v4)[8], float (&qc)[kChunk], uint32_t& bits,
                                            int lane, int row, int j0) {
  float v[kChunk];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    v[4 * k + 0] = v4[k].x;
    v[4 * k + 1] = v4[k].y;
    v[4 * k + 2] = v4[k].z;
    v[4 * k + 3] = v4[k].w;
  }
  uint32_t w = bits;
  if (!MASKED) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float o[8];
      cols8(q, t, w, o, v + 8 * k);
#pragma unroll
      for (int m = 0; m < 8; ++m) qc[8 * k + m] = o[m];
    }
  } else {
    const bool own = lane > 0;
#pragma unroll
    for (int m = 0; m < kChunk; ++m) {
      const int j = j0 + m;
      float qn = col1(q, t, w, v[m]);
      qn = (own && row > j) ? neg_inf() : qn;
      if (j == 0) qn = (own && row == 0) ? v[m] : qn;
      qc[m] = qn;
      q = qn;
    }
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

// ---------------------------------------------------------------- LDS layout
// The walk fetches each chunk's decision words kWalkAhead chunks before it
// walks that chunk, as a window of kWalkWin rows below the walker's row e at
// fetch time.  One chunk before walking it, the walker reads the 64 rows
// below its current row from that window (a chunk holds at most 33 rows of
// the path, and the current row is at most 32 rows into the 64); the current
// row is then at least e - 32 (kWalkAhead - 1), as a chunk descends at most
// 32 rows.
constexpr int kWalkAhead = 14;
constexpr int kWalkLoads = 2;                      // 1 KiB loads per window
constexpr int kWalkWin = kWalkLoads * 4 * kWave;   // rows per window
constexpr int kWalkSlots = 16;                 // window ring (power of two > kWalkAhead)
static_assert(kWalkWin >= 32 * (kWalkAhead - 1) + kWave + 3, "walk window");

// Value tiles.  Each wave has kStages stages; the stage of chunk c is
// (c - c_begin) % kStages (c_begin: the wave's first chunk).  A stage holds
//   * 64 tile rows of 32 values: item rows 63g .. 63g+63 (row 63 unused), row
//     r at byte 144 r.  The 16 bytes of padding per row put piece k of 16
//     consecutive rows in distinct 4-bank groups of the 64-bank LDS
//     (36 r mod 64 differs for r mod 16), so the per-row reads of a wave are
//     conflict-free with one address per lane plus the piece offset;
//   * the boundary row at kBoundOff: the 32 Q values of the row above the
//     wave for the stage's chunk (word 2332 = 28 mod 64, a bank group that
//     rows 0 .. 14 do not use), then its tag (chunk + 1) at kTagOff.  The
//     previous wave of the workgroup writes it; a wave fed by another
//     workgroup copies its polled words there; the first wave of an item
//     fills it with -inf once.
constexpr int kRowBytes = 144;
constexpr int kBoundOff = 9328;
constexpr int kTagOff = kBoundOff + 4 * kChunk;
constexpr int kStageBytes = 9472;
static_assert(64 * kRowBytes <= kBoundOff && kBoundOff % 16 == 0 && (kBoundOff / 4) % 64 == 28, "boundary slot");
static_assert(kTagOff + 4 <= kStageBytes && kStageBytes % 256 == 0, "stage size");

struct SweepLds {
  union {
    uint8_t tile[kWavesPerBlock][kStages][kStageBytes];
    // The walker's staging, once every sweep of its item (and so of its
    // workgroup) has finished.
    struct {
      uint32_t win[kWalkSlots][kWalkWin];  // decision-word windows of upcoming chunks
      int rs[kMaxRows + 2 * kWave];        // row_start under construction
    } walk;
  } u;
  uint32_t poll[kPollSlots][kWave];        // polled boundary words {value, tag} x 32 (wave 0)
  f32x4 ostage[kChunk / 4];                // last row of wave 3 before its global hand-off
  uint32_t dummy[kWavesPerBlock][kWave];   // target of placeholder loads and idle lanes' writes
  int cons[kWavesPerBlock];                // next chunk wave w will consume
};
static_assert(sizeof(SweepLds) <= 160 * 1024, "LDS");

// ---------------------------------------------------------------- path clearing
// The bytes [p0, p1) of the path that one wave clears: its 63 rows of its
// item.  16-byte aligned pieces [a0, a1) go through the sweep schedule; the
// unaligned head and tail are cleared up front with byte stores.
struct ZeroPlan {
  uint64_t a0;    // address of the first aligned piece
  uint64_t last;  // address of the last aligned piece (a1 - 16)
  bool any;       // at least one aligned piece
};

__device__ __forceinline__ ZeroPlan zero_plan(const KParams& p, int b, int g, int lane) {
  const uint64_t base = (uint64_t)b * (uint64_t)p.T * (uint64_t)p.S;  // offsets from p.path
  const int r0 = min(g * kRowsPerWave, p.T), r1 = min(g * kRowsPerWave + kRowsPerWave, p.T);
  const uint64_t p0 = base + (uint64_t)r0 * (uint64_t)p.S, p1 = base + (uint64_t)r1 * (uint64_t)p.S;
  const uint64_t pa = (uint64_t)(uintptr_t)p.path;
  const uint64_t a0 = ((pa + p0 + 15) & ~15ull) - pa, a1 = ((pa + p1) & ~15ull) - pa;
  ZeroPlan z;
  z.any = a1 > a0 && a1 - a0 >= 16;
  z.a0 = pa + a0;
  z.last = pa + a1 - 16;
  // Unaligned head and tail bytes (at most 15 + 15; all bytes if no piece).
  const uint64_t h1 = z.any ? a0 : p1;
  for (uint64_t o = p0 + lane; o < h1; o += kWave) p.path[o] = 0;
  if (z.any)
    for (uint64_t o = a1 + lane; o < p1; o += kWave) p.path[o] = 0;
  return z;
}

// Clears the aligned pieces from address `from` to the last one with 1 KiB
// stores (outside the sweep schedule).
__device__ __forceinline__ void zero_rest(const ZeroPlan& z, uint64_t from, int lane) {
  const u32x4 zero = {0u, 0u, 0u, 0u};
  for (uint64_t a = from + 16u * (uint64_t)lane; a <= z.last; a += 16u * kWave) vm_zero1(a, zero);
}

// ---------------------------------------------------------------- sweep
// Per-wave constants of the sweep.
struct WaveCtx {
  int lane, wv, b, g, g_last, tx, ty, row, c_begin, c_end;
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
__device__ __forceinline__ int chunk_end(int g, int tx, int ty) {
  const int by_len = (ty + kChunk - 1) / kChunk;
  const int by_reach = (g * kRowsPerWave + kRowsPerWave - 1 + ty - tx) / kChunk + 1;
  return by_len < by_reach ? by_len : by_reach;
}

// Vector-memory operations of one sweep step, in issue order:
//   [poll of chunk c+2]        (IN == 2)
//   tile of chunk c+kDepth     (NL loads)
//   decision words of chunk c  (1 store)
//   [boundary words of c]      (OUT == 2: 1 store)
constexpr int step_ops(int nl, bool in2, bool out2) { return (in2 ? 1 : 0) + nl + 1 + (out2 ? 1 : 0); }
// Count for the wait at the start of step c: tile c was issued kDepth steps
// earlier (followed by that step's stores and kDepth-1 whole steps), the
// poll of chunk c two steps earlier (followed by that step's tile and stores
// and one whole step).  Counts above 63 are clamped: a wave has at most 63
// operations outstanding (issue stalls at the counter's limit), so anything
// issued earlier than that has completed.
constexpr int wait_count(int nl, bool in2, bool out2) {
  const int k = step_ops(nl, in2, out2);
  const int tail = 1 + (out2 ? 1 : 0);
  const int n_tile = tail + (kDepth - 1) * k;
  const int n_poll = nl + tail + k;
  const int n = in2 && n_poll < n_tile ? n_poll : n_tile;
  return n > 63 ? 63 : n;
}

// The 4-byte tile loads K .. N-1 (load k fills LDS bytes 256 k .. 256 k + 255).
template <int K, int N>
__device__ __forceinline__ void dma4_loads(uint32_t dst, __amdgpu_buffer_rsrc_t r, const int* vo) {
  if constexpr (K < N) {
    dma4<256 * K>(dst, r, vo[K]);
    dma4_loads<K + 1, N>(dst, r, vo);
  }
}
// The 16-byte tile loads K .. N-1 (load k fills LDS bytes 1024 k .. 1024 k + 1023).
template <int K, int N>
__device__ __forceinline__ void dma16_loads(uint32_t dst, __amdgpu_buffer_rsrc_t r, const int* vo) {
  if constexpr (K < N) {
    dma16<1024 * K>(dst, r, vo[K]);
    dma16_loads<K + 1, N>(dst, r, vo);
  }
}

// Byte offset of (tile row r, byte e of the row's 128) in the value slab
// relative to the tile's first row, or an offset no resource covers.
__device__ __forceinline__ int tile_voff(int r, int e, int S) {
  const uint64_t o = (uint64_t)r * (uint64_t)S * 4u + (uint64_t)e;
  return o < 0x80000000ull ? (int)o : -16;
}

// Sweeps this wave's rows over its chunks and returns the score candidate
// (Q at (row, t_y-1) of this lane; only meaningful for the wave holding row
// t_x-1).  IN: where the row above the wave comes from — 0 nowhere (the wave
// holds row 0), 1 the previous wave of the workgroup, 2 global boundary words
// of the previous workgroup.  OUT: 0 no consumer, 1 the next wave of the
// workgroup, 2 global boundary words for the next workgroup.
template <bool ALIGNED, int IN, int OUT>
__device__ __forceinline__ float sweep_rows(const KParams& p, SweepLds& L, const WaveCtx& x, uint32_t tag, bool& timed_out) {
  constexpr int NL = ALIGNED ? 9 : 36;  // tile loads per chunk (padding slots included)
  constexpr bool IN2 = IN == 2, OUT2 = OUT == 2;
  const int lane = x.lane, wv = x.wv;
  float t = -0.0f;  // lane 0 keeps -0 for the whole sweep (see cols8)

  // Value tiles: a resource from the wave's first tile row at the next chunk
  // to load; rows past the slab fall outside it and read 0.
  const float* slab = p.value + (size_t)x.b * (size_t)p.T * (size_t)p.S;
  const uint32_t slab_bytes = (uint32_t)((uint64_t)p.T * (uint64_t)p.S * 4u);
  const uint32_t first = (uint32_t)((uint64_t)x.g * kRowsPerWave * (uint64_t)p.S * 4u) + (uint32_t)x.c_begin * (kChunk * 4);
  Cursor vr = make_cursor(reinterpret_cast<const char*>(slab), (int)slab_bytes);
  vr.advance((int)first);
  // Per-lane load offsets: load k, lane L fills stage slot 64 k + L (16-byte
  // slots, nine per row: eight pieces and the padding) or word 64 k + L
  // (4-byte words, 36 per row).
  int voff[NL];
#pragma unroll
  for (int k = 0; k < NL; ++k) {
    if (ALIGNED) {
      const int sl = 64 * k + lane, r = sl / 9, pc = sl % 9;
      voff[k] = pc < 8 ? tile_voff(r, 16 * pc, p.S) : -16;
    } else {
      const int w = 64 * k + lane, r = w / 36, wi = w % 36;
      voff[k] = wi < 32 ? tile_voff(r, 4 * wi, p.S) : -16;
    }
  }
  // LDS: tile0 is this wave's stage 0 as an LDS address (for M0); the C++
  // accesses use byte offsets from the start of L (where the tiles begin).
  char* const Lc = reinterpret_cast<char*>(&L);
  const uint32_t tile_rel = (uint32_t)wv * (kStages * kStageBytes);
  const uint32_t tile0 = lds_off(&L.u.tile[wv][0][0]);
  // Lane l reads tile row l-1 of a stage; lane 0 reads the boundary row.
  const uint32_t rbase = tile_rel + (lane > 0 ? (uint32_t)(lane - 1) * kRowBytes : (uint32_t)kBoundOff);
  // Placeholder loads (steps with no store yet) read the slab's first 256 bytes.
  const uint32_t dummy = lds_off(&L.dummy[wv][0]);
  const __amdgpu_buffer_rsrc_t drsrc = make_cursor(slab, min((int)slab_bytes, 256)).rsrc();
  // Decision words: dec[b][c][row], lane 0 into the chunk's scratch word.
  const __amdgpu_buffer_rsrc_t dr = make_cursor(p.dec + (size_t)x.b * p.NC * (size_t)p.TP, p.NC * p.TP * 4).rsrc();
  const int dvo = 4 * (lane > 0 ? x.row : p.TP - 1);
  const uint32_t dstride = (uint32_t)p.TP * 4u;
  // Boundary words of this wave (OUT == 2) and of the previous one (IN == 2).
  const size_t slot_stride = (size_t)p.NC * kChunk;
  const int slot_bytes = (int)(slot_stride * 8u);
  const __amdgpu_buffer_rsrc_t sr = make_cursor(p.slots + ((size_t)x.b * p.NW + x.g) * slot_stride, slot_bytes).rsrc();
  const int svo = lane < kChunk ? 8 * lane : -16;
  const uint64_t* pslots = p.slots + ((size_t)x.b * p.NW + (x.g > 0 ? x.g - 1 : 0)) * slot_stride;
  Cursor pr = make_cursor(pslots, slot_bytes);
  if (IN2) pr.advance((x.c_begin - 1) * 256);  // first poll: chunk c_begin-1

  // Boundary words of chunk c are in poll slot c % 4 once all carry this
  // call's tag (re-polled until then); lane L's word is L % 32.
  auto polled_word = [&](int c) __attribute__((always_inline)) -> uint64_t {
    const uint64_t* pw = reinterpret_cast<const uint64_t*>(&L.poll[c & (kPollSlots - 1)][0]);
    uint64_t wd = pw[lane & (kChunk - 1)];
    int spins = 0;
    while (true) {
      // Lanes still seeing an old tag, as an opaque scalar: branching on the
      // ballot directly lets the compiler treat the loop as divergent.
      uint64_t stale = __builtin_amdgcn_ballot_w64((uint32_t)(wd >> 32) != tag);
      asm volatile("" : "+s"(stale));
      if (stale == 0) break;
      if (++spins > kSpinLimit) {
        timed_out = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      dma4_dev(lds_off(&L.poll[c & (kPollSlots - 1)][0]), make_cursor(pslots + (size_t)c * kChunk, kChunk * 8u).rsrc(), 4 * lane);
      vm_wait<0>();
      wd = pw[lane & (kChunk - 1)];
    }
    return wd;
  };
  // Waits for the boundary row of chunk c in the stage at byte offset so.
  auto bound_ready = [&](int c, uint32_t so) __attribute__((always_inline)) {
    const int* tg = reinterpret_cast<const int*>(Lc + tile_rel + so + kTagOff);
    int spins = 0;
    while (__builtin_amdgcn_readfirstlane(lds_load(tg)) != c + 1) {
      if (++spins > kSpinLimit) {
        timed_out = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  };

  if (IN == 0) {
    // The row above row 0 is -inf in every stage.
    if (lane < kChunk) {
#pragma unroll
      for (int st = 0; st < kStages; ++st)
        reinterpret_cast<float*>(&L.u.tile[wv][st][kBoundOff])[lane] = neg_inf();
    }
  }

  // Prologue: kDepth placeholder steps with the steady-state operation
  // sequence, so that the loop's wait counts hold from its first step.
#pragma unroll
  for (int k = 0; k < kDepth; ++k) {
    if (IN2) {
      dma4_dev(lds_off(&L.poll[(x.c_begin - 1 + k) & (kPollSlots - 1)][0]), pr.rsrc(), 4 * lane);
      pr.advance(256);
    }
    if (ALIGNED)
      dma16_loads<0, NL>(tile0 + k * kStageBytes, vr.rsrc(), voff);
    else
      dma4_loads<0, NL>(tile0 + k * kStageBytes, vr.rsrc(), voff);
    vr.advance(kChunk * 4);
    dma4<0>(dummy, drsrc, 4 * lane);
    if (OUT2) dma4<0>(dummy, drsrc, 4 * lane);
  }

  // Lane 0's Q at the column before the first chunk: the previous wave's
  // last row there (its chunk c_begin-1, always computed), or -inf.
  float q = neg_inf();
  if (IN == 1) {
    bound_ready(x.c_begin - 1, (kStages - 1) * kStageBytes);
    wave_lds_sync();
    const float e = reinterpret_cast<const float*>(&L.u.tile[wv][kStages - 1][kBoundOff])[kChunk - 1];
    q = lane == 0 ? e : q;
    wave_lds_sync();
    if (lane == 0) lds_store(&L.cons[wv], x.c_begin);
  } else if (IN == 2) {
    vm_wait<0>();
    const uint64_t wd = polled_word(x.c_begin - 1);
    const float e = __int_as_float(__builtin_amdgcn_readlane((int)(uint32_t)wd, kChunk - 1));
    q = lane == 0 ? e : q;
  }

  // Stage offsets: so of chunk c (the one computed), sd of chunk c+kDepth,
  // sn of chunk c in the next wave's stages.
  uint32_t so = 0, sd = (kStages - 1) * kStageBytes;
  uint32_t sn = (uint32_t)((x.c_begin - x.next_begin) & (kStages - 1)) * kStageBytes;
  const uint32_t tile_next = tile_rel + kStages * kStageBytes;
  // Lane 0 publishes the consumed-chunk counter; the other lanes write
  // their own dummy words (one store, no exec change).
  int* const cons_ptr = lane == 0 ? &L.cons[wv] : reinterpret_cast<int*>(&L.dummy[wv][lane]);
  // Lower bound of the consumer's counter: it starts at its own c_begin-1,
  // which is at least this wave's c_begin+1 (63 rows span >= 63 columns).
  int cons_seen = x.c_begin + 1;
  float qc[kChunk];
  uint32_t soff = (uint32_t)x.c_begin * dstride;
  for (int c = x.c_begin; c < x.c_end; ++c) {
    vm_wait<wait_count(NL, IN2, OUT2)>();
    if (IN2) {
      dma4_dev(lds_off(&L.poll[(c + 2) & (kPollSlots - 1)][0]), pr.rsrc(), 4 * lane);
      pr.advance(256);
    }
    if (ALIGNED)
      dma16_loads<0, NL>(tile0 + sd, vr.rsrc(), voff);
    else
      dma4_loads<0, NL>(tile0 + sd, vr.rsrc(), voff);
    vr.advance(kChunk * 4);

    // The row above: from the previous wave, or copied from the polled
    // words.  Beyond the previous wave's chunks the slot holds stale values:
    // they only reach cells that cannot reach (t_x-1, t_y-1).
    if (IN == 1 && c < x.prev_end) bound_ready(c, so);
    if (IN == 2 && c < x.prev_end) {
      const uint64_t wd = polled_word(c);
      reinterpret_cast<float*>(Lc + tile_rel + so + kBoundOff)[lane & (kChunk - 1)] = __uint_as_float((uint32_t)wd);
    }
    wave_lds_sync();
    f32x4 v[8];
    {
      const f32x4* base = reinterpret_cast<const f32x4*>(Lc + rbase + so);
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = base[k];
    }
    uint32_t bits = 0;
    if (c < x.mask_end)
      sweep_chunk<true>(q, t, v, qc, bits, lane, x.row, c * kChunk);
    else
      sweep_chunk<false>(q, t, v, qc, bits, lane, x.row, c * kChunk);
    buf_store32(bits, dvo, dr, soff);
    soff += dstride;
    if (IN == 1) {
      // The reads of this chunk's slot are done: the previous wave may
      // reuse it for chunk c + kStages.
      wave_lds_sync();
      lds_store(cons_ptr, c + 1);
    }
    if (OUT == 1) {
      // Wait until the consumer no longer needs the slot, then publish the
      // values, then the tag.
      int spins = 0;
      while (cons_seen < c - (kStages - 1)) {
        cons_seen = __builtin_amdgcn_readfirstlane(lds_load(&L.cons[wv + 1]));
        if (cons_seen >= c - (kStages - 1)) break;
        if (++spins > kSpinLimit) {
          timed_out = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      if (lane == kWave - 1) {
        f32x4* dst = reinterpret_cast<f32x4*>(Lc + tile_next + sn + kBoundOff);
#pragma unroll
        for (int k = 0; k < kChunk / 4; ++k) dst[k] = f32x4{qc[4 * k], qc[4 * k + 1], qc[4 * k + 2], qc[4 * k + 3]};
      }
      // Values before the tag (the LDS executes one wave's operations in
      // order; the fence keeps the compiler from reordering them).  Kept out
      // of the lane-63 branch: inside it, the compiler makes the whole chunk
      // loop divergent for the waves that feed no other wave of the group.
      wave_lds_sync();
      if (lane == kWave - 1) lds_store(reinterpret_cast<int*>(Lc + tile_next + sn + kTagOff), c + 1);
      sn = sn == (kStages - 1) * kStageBytes ? 0u : sn + kStageBytes;
    } else if (OUT == 2) {
      if (lane == kWave - 1) {
#pragma unroll
        for (int k = 0; k < kChunk / 4; ++k) L.ostage[k] = f32x4{qc[4 * k], qc[4 * k + 1], qc[4 * k + 2], qc[4 * k + 3]};
      }
      wave_lds_sync();
      const float val = reinterpret_cast<const float*>(L.ostage)[lane & (kChunk - 1)];
      buf_store64(((uint64_t)tag << 32) | (uint64_t)__float_as_uint(val), svo, sr, (uint32_t)c * 256u);
      wave_lds_sync();
    }
    so = so == (kStages - 1) * kStageBytes ? 0u : so + kStageBytes;
    sd = sd == (kStages - 1) * kStageBytes ? 0u : sd + kStageBytes;
  }
  vm_wait<0>();
  float score = neg_inf();
  if (OUT == 0) {
    const int m_last = (x.ty - 1) % kChunk;
#pragma unroll
    for (int m = 0; m < kChunk; ++m) score = (m == m_last) ? qc[m] : score;
  }
  return score;
}

// Waits (bounded) until flag[k] == tag for every k in [0, n).
__device__ __forceinline__ void wait_flags(const uint32_t* flag, int n, uint32_t tag, int lane, bool& timed_out) {
  for (int k0 = 0; k0 < n; k0 += kWave) {
    const int k = k0 + lane;
    int spins = 0;
    while (true) {
      const bool ready = k >= n || ld_dev(flag + k) == tag;
      if (__builtin_amdgcn_ballot_w64(!ready) == 0) break;
      if (++spins > kSpinLimit) {
        timed_out = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
}

// ---------------------------------------------------------------- backtrack
// One step of the walk inside a chunk, for row k >= 1 below the chunk's
// first row (its word, shifted right by one, in CUR), with the word of row
// k+1 read into NXT meanwhile.  q is the position of the previous row's
// step: the row's own step is the lowest set bit of its word above q, at
// q + 1 + ff1(word >> (q + 1)); none (shifted word zero, also for q = 31)
// ends the chunk.  s_lshr sets SCC to (result != 0), s_ff1 leaves it, so the
// s_addc adds the 1.
#define MAS_WALK_STEP(CUR, NXT)                  \
  "v_readlane_b32 %[" NXT "], %[wh], %[sl]\n\t" \
  "s_add_u32 %[sl], %[sl], 1\n\t"               \
  "s_lshr_b32 %[t], %[" CUR "], %[q]\n\t"       \
  "s_cbranch_scc0 .Lmas_walk_end%=\n\t"    \
  "s_ff1_i32_b32 %[t], %[t]\n\t"                \
  "s_addc_u32 %[q], %[q], %[t]\n\t"             \
  "s_bitset1_b32 %[pm], %[q]\n\t"
#define MAS_WALK_STEP2 MAS_WALK_STEP("y", "x") MAS_WALK_STEP("x", "y")
#define MAS_WALK_STEP8 MAS_WALK_STEP2 MAS_WALK_STEP2 MAS_WALK_STEP2 MAS_WALK_STEP2

// The steps of one chunk.  Row k of the chunk (k = 0 at the row the path
// enters the chunk in) is lane sl + k of w (and of wh = w >> 1).  The first
// row's step is its lowest set bit at or above position q0 (the column the
// path enters at); every later row's is its lowest set bit above the
// previous row's.  Returns the set of step positions: bit p set means one
// row starts at column 32c + 31 - p, the k-th lowest set bit for row k.  At
// most 32 rows step (one per column), so the 33rd row is never looked at.
__device__ __forceinline__ uint32_t walk_chunk(uint32_t w, uint32_t wh, int sl, int q0) {
  uint32_t pm, t, x, y;
  int q = q0;
  asm volatile(
      "s_mov_b32 %[pm], 0\n\t"
      "v_readlane_b32 %[x], %[w], %[sl]\n\t"
      "s_add_u32 %[sl], %[sl], 1\n\t"
      "v_readlane_b32 %[y], %[wh], %[sl]\n\t"
      "s_add_u32 %[sl], %[sl], 1\n\t"
      "s_lshr_b32 %[t], %[x], %[q]\n\t"
      "s_cbranch_scc0 .Lmas_walk_end%=\n\t"
      "s_ff1_i32_b32 %[t], %[t]\n\t"
      "s_add_u32 %[q], %[q], %[t]\n\t"
      "s_bitset1_b32 %[pm], %[q]\n\t"
      MAS_WALK_STEP8 MAS_WALK_STEP8 MAS_WALK_STEP8 MAS_WALK_STEP2 MAS_WALK_STEP2 MAS_WALK_STEP2
      MAS_WALK_STEP("y", "x")
      ".Lmas_walk_end%=:"
      : [pm] "=&s"(pm), [t] "=&s"(t), [x] "=&s"(x), [y] "=&s"(y), [q] "+s"(q), [sl] "+s"(sl)
      : [w] "v"(w), [wh] "v"(wh)
      : "scc");
  return pm;
}
#undef MAS_WALK_STEP8
#undef MAS_WALK_STEP2
#undef MAS_WALK_STEP

// The walk of one item from (t_x-1, t_y-1) back to (0, 0) (Algorithm 1's
// argmax loop, read off the decision words): in chunk c the path in row i
// stays there until the nearest column to the left whose decision bit is
// set, then continues one row up at the column before.  Builds row_start in
// L.u.walk.rs: the first column of every row, with rs[0] = 0 and
// rs[t_x .. T] = t_y.  Runs on the wave that holds row t_x-1, once every
// wave of the item has published its words.
__device__ __forceinline__ void walk(const KParams& p, SweepLds& L, int b, int tx, int ty, uint32_t tag, int lane,
                                     bool& timed_out) {
  const int g_last = (tx - 1) / kRowsPerWave;
  wait_flags(p.done + (size_t)b * p.NW, g_last, tag, lane, timed_out);
  // Every sweep of this workgroup has finished (lower waves: flags above;
  // higher waves hold no rows of the alignment), so the tile area is free.
  int* rsl = L.u.walk.rs;
  const uint32_t* db = p.dec + (size_t)b * p.NC * (size_t)p.TP;
  const uint64_t chunk_bytes = (uint64_t)p.TP * 4u;
  const int wvo = 16 * lane;
  int wlo = 0;  // lane s: first row of the window in ring slot s
  // Window of chunk ch: kWalkWin rows from a 16-byte aligned row lo in
  // [e - kWalkWin + 1, e - kWalkWin + 4] (or row 0) into slot ch % kWalkSlots;
  // an empty resource (reads 0) for chunks before the first.
  auto issue_win = [&](int ch, int e) __attribute__((always_inline)) {
    const int slot = ch & (kWalkSlots - 1);
    const int lo = max(e - kWalkWin + 4, 0) & ~3;
    wlo = lane == slot ? lo : wlo;
    const uint32_t dst = lds_off(&L.u.walk.win[slot][0]);
    const __amdgpu_buffer_rsrc_t rr = ch >= 0 ? sub_rsrc(db + (size_t)ch * p.TP, chunk_bytes, (uint64_t)lo * 4u)
                                              : sub_rsrc(db, chunk_bytes, chunk_bytes);
#pragma unroll
    for (int k = 0; k < kWalkLoads; ++k) dma_piece(dst + 1024 * k, rr, wvo + 1024 * k);
  };
  // Word of row e - lane of chunk ch (its window must be in LDS).
  auto read_row = [&](int ch, int e) __attribute__((always_inline)) -> uint32_t {
    const int slot = ch & (kWalkSlots - 1);
    const int r = e - lane - __builtin_amdgcn_readlane(wlo, slot);
    return L.u.walk.win[slot][r > 0 ? r : 0];
  };
  const uint32_t below = (1u << (lane & (kChunk - 1))) - 1u;  // positions below this lane's
  int idx = tx - 1;                  // row of the path at the chunk's last column
  int cw = (ty - 1) / kChunk;        // chunk being walked
  int q0 = 31 - (ty - 1) % kChunk;   // position of the path's column in chunk cw
  for (int k = 0; k < kWalkAhead; ++k) issue_win(cw - k, idx);
  vm_wait<kWalkLoads * (kWalkAhead - 1)>();  // window of chunk cw
  uint32_t W = read_row(cw, idx);    // rows e0 - lane of chunk cw
  int off = 0;                       // lane of row idx in W: idx = e0 - off
  bool walking = idx > 0;
  while (walking) {
    vm_wait<kWalkLoads * (kWalkAhead - 2)>();  // windows of chunks cw and cw-1
    issue_win(cw - kWalkAhead, idx);
    const uint32_t N = read_row(cw - 1, idx);  // the next chunk's rows below idx, read ahead
    const uint32_t pm = walk_chunk(W, W >> 1, off, q0);
    // Set bit p of pm belongs to the row (popcount of pm below p) under idx.
    if (lane < kChunk && ((pm >> lane) & 1u)) rsl[idx - (int)__builtin_popcount(pm & below)] = cw * kChunk + 31 - lane;
    const int kk = __builtin_popcount(pm);
    idx -= kk;
    q0 = 0;
    cw -= 1;
    W = N;
    off = kk;
    walking = idx > 0 && cw >= 0;
  }
  vm_wait<0>();  // no window load may land in LDS after this wave ends
  wave_lds_sync();
  if (lane == 0) rsl[0] = 0;
  for (int i = tx + lane; i <= p.T; i += kWave) rsl[i] = ty;
  wave_lds_sync();
}

template <bool ALIGNED>
__device__ __forceinline__ void sweep_block(const KParams& p, SweepLds& L, int sid, uint32_t tag, bool& timed_out) {
  const int lane = threadIdx.x & (kWave - 1);
  // The wave index is uniform across a wave; saying so keeps everything
  // derived from it (chunk indices, modes, loop bounds) in scalar registers.
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int b = sid % p.B;
  const int r = sid / p.B;
  const int g = r * kWavesPerBlock + wv;  // wave index inside the item
  const int tx = p.t_x[b];
  const int ty = p.t_y[b];
  const int st = item_status(tx, ty, p.T, p.S);
  const int c_begin = (g * kRowsPerWave) / kChunk;

  // Workgroup set-up: no boundary row is written yet (the LDS holds
  // whatever earlier workgroups left); each wave's first chunk to consume
  // (its carried row comes from chunk c_begin-1).
  if (threadIdx.x < kWavesPerBlock * kStages)
    lds_store(reinterpret_cast<int*>(&L.u.tile[threadIdx.x / kStages][threadIdx.x % kStages][kTagOff]), 0);
  if (lane == 0) lds_store(&L.cons[wv], c_begin - 1);
  __syncthreads();

  int32_t* rs_out = p.row_start + (size_t)b * ((size_t)p.T + 1);
  const bool has_rows = g * kRowsPerWave < p.T;
  ZeroPlan zp{};
  if (p.path && has_rows) zp = zero_plan(p, b, g, lane);
  const bool clear = p.path && has_rows && zp.any;
  if (st != kItemOk) {
    if (clear) zero_rest(zp, zp.a0, lane);
    if (g == 0) {
      for (int i = lane; i <= p.T; i += kWave) rs_out[i] = 0;
      if (lane == 0) {
        if (p.score) p.score[b] = neg_inf();
        if (p.status) p.status[b] = st;
      }
    }
    return;
  }
  const int g_last = (tx - 1) / kRowsPerWave;
  if (g > g_last) {
    // No rows of the alignment here: clear the path rows once the item's
    // sweep is over (the HBM is less busy then).
    if (clear) {
      if (lane == 0) {
        int spins = 0;
        while (ld_dev(p.done + (size_t)b * p.NW + g_last) != tag && ++spins <= kSpinLimit) __builtin_amdgcn_s_sleep(8);
      }
      zero_rest(zp, zp.a0, lane);
    }
    return;
  }
  if (g == 0 && lane == 0 && p.status) p.status[b] = kItemOk;
  // The walker's wave clears its rows first: it waits for the waves above
  // it anyway (for g_last > 0), and the walk then ends with only the ones
  // left to write.  The other waves clear theirs after their sweep.
  if (clear && g == g_last) zero_rest(zp, zp.a0, lane);

  WaveCtx x;
  x.lane = lane;
  x.wv = wv;
  x.b = b;
  x.g = g;
  x.g_last = g_last;
  x.tx = tx;
  x.ty = ty;
  x.row = g * kRowsPerWave + lane - 1;  // lane 0: the row above the wave
  x.c_begin = c_begin;
  x.c_end = chunk_end(g, tx, ty);
  x.prev_end = g > 0 ? chunk_end(g - 1, tx, ty) : 0;
  x.mask_end = (g * kRowsPerWave + kRowsPerWave - 2) / kChunk + 1;  // last masked column: 63g + 61
  x.next_begin = ((g + 1) * kRowsPerWave) / kChunk;
  float score;
  if (g == g_last) {
    score = g == 0 ? sweep_rows<ALIGNED, 0, 0>(p, L, x, tag, timed_out)
                   : (wv > 0 ? sweep_rows<ALIGNED, 1, 0>(p, L, x, tag, timed_out) : sweep_rows<ALIGNED, 2, 0>(p, L, x, tag, timed_out));
  } else if (wv < kWavesPerBlock - 1) {
    score = g == 0 ? sweep_rows<ALIGNED, 0, 1>(p, L, x, tag, timed_out)
                   : (wv > 0 ? sweep_rows<ALIGNED, 1, 1>(p, L, x, tag, timed_out) : sweep_rows<ALIGNED, 2, 1>(p, L, x, tag, timed_out));
  } else {
    score = sweep_rows<ALIGNED, 1, 2>(p, L, x, tag, timed_out);
  }

  // Publish this wave's decision words to the item's walker.
  if (lane == 0) st_dev(p.done + (size_t)b * p.NW + g, tag);
  int* rsl = L.u.walk.rs;
  if (g == g_last) {
    if (lane == (tx - 1) - g_last * kRowsPerWave + 1 && p.score) p.score[b] = score;
    walk(p, L, b, tx, ty, tag, lane, timed_out);
    for (int i = lane; i <= p.T; i += kWave) st_dev(reinterpret_cast<uint32_t*>(rs_out + i), (uint32_t)rsl[i]);
    if (!p.path) return;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if (lane == 0) st_dev(p.wdone + b, tag);
  } else {
    // Clear this wave's path rows while the walk runs, then wait for it.
    if (!p.path) return;
    if (clear) zero_rest(zp, zp.a0, lane);
    int spins = 0;
    while (ld_dev(p.wdone + b) != tag) {
      if (++spins > kSpinLimit) {
        timed_out = true;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  // Ones of this wave's rows: lane l's row 63g + l - 1 has columns [lo, hi),
  // from row_start entries 63g + l - 1 (lane l-1's) and 63g + l (its own).
  // Each lane writes the first kOnesPerLane bytes of its row's ones (one
  // 16-byte piece or one byte at a time); rows with more (a long stay in one
  // row) are finished by the whole wave, one such row at a time, 64 pieces
  // or bytes per store.
  const int ri = min(g * kRowsPerWave + lane, p.T);
  const int hi = g == g_last ? rsl[ri] : (int)ld_dev(reinterpret_cast<const uint32_t*>(rs_out + ri));
  const int lo = __builtin_amdgcn_update_dpp(0, hi, 0x138, 0xF, 0xF, false);  // lane l-1's entry
  const int row = g * kRowsPerWave + lane - 1;
  const bool mine = lane > 0 && row < tx;
  uint8_t* const item_path = p.path + (size_t)b * (size_t)p.T * (size_t)p.S;
  const int start = p.path16 ? (lo & ~15) : lo;
  const int split = mine ? min(hi, start + kOnesPerLane) : start;  // own part: [start, split)
  if (mine) {
    uint8_t* prow = item_path + (size_t)row * (size_t)p.S;
    if (p.path16) {
      for (int j0 = start; j0 < split; j0 += 16) *reinterpret_cast<uint4*>(prow + j0) = path_piece(lo, hi, j0);
    } else {
      for (int j = start; j < split; ++j) prow[j] = 1;
    }
  }
  uint64_t rest = __builtin_amdgcn_ballot_w64(mine && split < hi);
  while (rest) {
    const int l = __builtin_ctzll(rest);
    rest &= rest - 1;
    const int a = __builtin_amdgcn_readlane(split, l), e = __builtin_amdgcn_readlane(hi, l);
    uint8_t* prow = item_path + (size_t)(g * kRowsPerWave + l - 1) * (size_t)p.S;
    if (p.path16) {
      // a is a multiple of 16 and at least lo: every piece from a on holds
      // ones up to e.
      for (int j0 = a + 16 * lane; j0 < e; j0 += 16 * kWave) *reinterpret_cast<uint4*>(prow + j0) = path_piece(a, e, j0);
    } else {
      for (int j = a + lane; j < e; j += kWave) prow[j] = 1;
    }
  }
}

template <bool ALIGNED>
// One workgroup per CU: the value-tile ring takes most of the LDS.
__global__ void __launch_bounds__(kThreadsPerBlock, 1) mas_kernel(KParams p) {
  __shared__ SweepLds L;
  const uint32_t gen = __hip_atomic_load(&p.hdr->gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t tag = call_tag(gen);
  bool timed_out = false;
  const int item = (int)blockIdx.x % p.B;
  sweep_block<ALIGNED>(p, L, blockIdx.x, tag, timed_out);
  if (timed_out) {
    if (p.status) p.status[item] = kItemSyncTimeout;
    __hip_atomic_store(&p.hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // The last wave of the call to finish advances the generation.
  if ((threadIdx.x & (kWave - 1)) == 0) {
    const uint32_t total = gridDim.x * kWavesPerBlock;
    const uint32_t prev = __hip_atomic_fetch_add(&p.hdr->exit_count, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == total - 1) {
      __hip_atomic_store(&p.hdr->exit_count, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&p.hdr->gen, gen + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
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
    path[k] = path_piece(rs[i], rs[i + 1], pc * 16);
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
__global__ void __launch_bounds__(256) mas_zero_kernel(uint4* __restrict__ p, size_t n16) {
  for (size_t k = (size_t)blockIdx.x * blockDim.x + threadIdx.x; k < n16; k += (size_t)gridDim.x * blockDim.x)
    p[k] = make_uint4(0u, 0u, 0u, 0u);
}

// ---------------------------------------------------------------- launchers
hipError_t launch_mas(const KParams& p, bool aligned, hipStream_t stream) {
  const dim3 grid((unsigned)(p.B * p.NB)), block(kThreadsPerBlock);
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

hipError_t launch_zero(void* p, size_t bytes, hipStream_t stream) {
  const size_t n16 = bytes / 16;
  hipLaunchKernelGGL(mas_zero_kernel, dim3(stream_grid(n16, 256)), dim3(256), 0, stream, reinterpret_cast<uint4*>(p), n16);
  return hipGetLastError();
}

}  // namespace mas
