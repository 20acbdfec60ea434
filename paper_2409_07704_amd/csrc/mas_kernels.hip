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
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

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
constexpr int kGroup = 4;            // chunks per value load (512 contiguous bytes of each row)
constexpr int kSlots = 4;            // boundary-row slots per wave (a power of two, = kGroup)
constexpr int kPollSlots = 4;        // LDS slots of polled boundary words
static_assert((kSlots & (kSlots - 1)) == 0 && kSlots == kGroup, "slot ring");

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
// The compiler computes the saturating count update with a vector
// instruction; the descriptor must live in scalar registers, so the count
// is read back as a wave-uniform value.  Byte counts are below 2^31.
struct Cursor {
  const char* base;
  int left;
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc() const {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), 0, left, kRsrcWord3);
  }
  // The same, with every field read back as wave-uniform: for inline
  // assembly operands that must be scalar registers (under scalar-register
  // pressure the compiler may keep a uniform pointer in vector registers).
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_s() const {
    const uint64_t a = (uint64_t)(uintptr_t)base;
    const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
    return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<char*>((uintptr_t)(lo | hi << 32)), 0,
                                             __builtin_amdgcn_readfirstlane(left), kRsrcWord3);
  }
  __device__ __forceinline__ void advance(int step) {
    base += step;
    left = __builtin_amdgcn_readfirstlane(max(left - step, 0));
  }
};
__device__ __forceinline__ Cursor make_cursor(const void* p, int bytes) { return Cursor{static_cast<const char*>(p), bytes}; }

// Buffer resource over the bytes [off, total) of the region at p (empty
// when off >= total; total < 2^31).  Every field is read back as
// wave-uniform, so the descriptor can feed inline-assembly scalar operands.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t sub_rsrc(const void* p, uint64_t total, uint64_t off) {
  const uint64_t o = off < total ? off : total;
  return Cursor{static_cast<const char*>(p) + o, (int)(uint32_t)(total - o)}.rsrc_s();
}

// Loads into LDS (the lds flag): every lane's bytes at its voffset go to LDS
// at M0 + size * lane.  A scalar write of M0 needs one wait state before
// such a load.
// Device-scope (sc1) variants for data written by other workgroups.
__device__ __forceinline__ void dma4_dev(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  lds = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %[l]\n\ts_nop 0\n\tbuffer_load_dword %[v], %[r], 0 offen sc1 lds"
               :
               : [l] "s"(lds), [r] "s"(r), [v] "v"(voff)
               : "memory", "m0");
}
// One 16-byte load per lane, device-scope: the bytes at voff of the resource
// to LDS at lds + 16 lane.
__device__ __forceinline__ void dma_piece(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  lds = __builtin_amdgcn_readfirstlane(lds);
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

// Per-wave LDS region (kWaveLds bytes):
//   * kGroup value tiles, one per chunk of the current group of kGroup
//     chunks: 64 rows of 32 values, item rows 63g .. 63g+63 (row 63 unused),
//     row r at byte 144 r of its tile.  The 16 bytes of padding per row put
//     piece k of 16 consecutive rows in distinct 4-bank groups of the
//     64-bank LDS (36 r mod 64 differs for r mod 16), so the per-row reads of
//     a wave are conflict-free with one address per lane plus the piece
//     offset;
//   * kSlots boundary slots at kBoundOff + 256 k: the 32 Q values of the row
//     above the wave for chunk c in slot (c - c_begin) % kSlots (word
//     9244 + 64 k = 28 mod 64, a bank group rows 0 .. 14 do not use), then
//     its tag (chunk + 1).  The previous wave of the workgroup writes them; a
//     wave fed by another workgroup copies its polled words there; the first
//     wave of an item fills them with -inf once.
constexpr int kRowBytes = 144;
constexpr int kTileBytes = 64 * kRowBytes;
constexpr int kBoundOff = kGroup * kTileBytes + 112;
constexpr int kSlotBytes = 256;
constexpr int kTagOff = 4 * kChunk;  // inside a slot
constexpr int kWaveLds = 37888;
static_assert(kBoundOff % 16 == 0 && (kBoundOff / 4) % 64 == 28, "boundary slot");
static_assert(kBoundOff + (kSlots - 1) * kSlotBytes + kTagOff + 4 <= kWaveLds && kWaveLds % 256 == 0, "wave region");
static_assert(kBoundOff + (kSlots - 1) * kSlotBytes + kTagOff + 4 <= kWaveLds && kWaveLds % 256 == 0, "wave region");

struct SweepLds {
  union {
    uint8_t tile[kWavesPerBlock][kWaveLds];
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

// Byte offset of (tile row r, byte e of the row) in the value slab relative
// to the tile's first row, or INT_MIN: as an unsigned offset it stays at or
// above 2^31, outside every resource, after adding up to 2^31 - 1.
__device__ __forceinline__ int tile_voff(int r, int e, int S) {
  const uint64_t o = (uint64_t)r * (uint64_t)S * 4u + (uint64_t)e;
  return o < 0x80000000ull ? (int)o : (int)0x80000000u;
}

__device__ __forceinline__ f32x4 load16(__amdgpu_buffer_rsrc_t r, int voff) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0));
}

template <int V>
struct IntC {
  static constexpr int value = V;
};

// Cache policy of hand-off data between workgroups: sc1 (device scope).
constexpr int kPolicyDev = 16;

// Sweeps this wave's rows over its chunks and returns the score candidate
// (Q at (row, t_y-1) of this lane; only meaningful for the wave holding row
// t_x-1).  IN: where the row above the wave comes from — 0 nowhere (the wave
// holds row 0), 1 the previous wave of the workgroup, 2 global boundary words
// of the previous workgroup.  OUT: 0 no consumer, 1 the next wave of the
// workgroup, 2 global boundary words for the next workgroup.
//
// Value tiles travel HBM -> registers -> LDS in groups of kGroup chunks
// (512 contiguous bytes of each row: DRAM serves longer runs of a row
// faster than scattered 128-byte pieces).  While the kGroup tiles of one
// group sit in LDS and are swept, the next group is in flight in registers.
// Lane L loads piece L % 8 of chunk j of tile rows 8q + L/8 (q = 0..7):
// 16 bytes each, eight lanes per 128-byte row segment.  The compiler sees
// these loads and waits for them right before writing them to LDS.
template <int IN, int OUT>
__device__ __forceinline__ float sweep_rows(const KParams& p, SweepLds& L, const WaveCtx& x, uint32_t tag, bool& timed_out) {
  constexpr bool IN2 = IN == 2, OUT2 = OUT == 2;
  const int lane = x.lane, wv = x.wv;
  float t = -0.0f;  // lane 0 keeps -0 for the whole sweep (see cols8)

  // LDS: byte offsets from the start of L (where the wave regions begin).
  char* const Lc = reinterpret_cast<char*>(&L);
  const uint32_t wbase = (uint32_t)wv * kWaveLds;
  const uint32_t nbase = wbase + kWaveLds;  // the next wave's region
  auto slot_ptr = [&](uint32_t base, int k) __attribute__((always_inline)) -> char* {
    return Lc + base + kBoundOff + (uint32_t)(k & (kSlots - 1)) * kSlotBytes;
  };

  // Value tiles: a resource from the wave's first tile row at the next chunk
  // to load; rows past the slab fall outside it and read 0.
  const float* slab = p.value + (size_t)x.b * (size_t)p.T * (size_t)p.S;
  const int slab_bytes = (int)((uint64_t)p.T * (uint64_t)p.S * 4u);
  Cursor vr = make_cursor(slab, slab_bytes);
  vr.advance((int)((uint64_t)x.g * kRowsPerWave * (uint64_t)p.S * 4u) + x.c_begin * (kChunk * 4));
  int voff[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) voff[q] = tile_voff(8 * q + (lane >> 3), 16 * (lane & 7), p.S);
  // Where lane L's pieces go: row 8q + L/8, piece L % 8 (q * 1152 bytes apart).
  f32x4* const tile_w = reinterpret_cast<f32x4*>(Lc + wbase + (uint32_t)(lane >> 3) * kRowBytes + 16u * (uint32_t)(lane & 7));
  // Lane l >= 1 reads tile row l-1; lane 0 reads the chunk's boundary slot.
  const f32x4* const tile_r = reinterpret_cast<const f32x4*>(Lc + wbase + (uint32_t)(lane > 0 ? lane - 1 : 0) * kRowBytes);
  f32x4 buf[kGroup][8];
  auto load_group = [&]() __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t r = vr.rsrc();
#pragma unroll
    for (int q = 0; q < 8; ++q)
#pragma unroll
      for (int j = 0; j < kGroup; ++j) buf[j][q] = load16(r, voff[q] + j * (kChunk * 4));
    vr.advance(kGroup * kChunk * 4);
  };
  auto put_group = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < kGroup; ++j)
#pragma unroll
      for (int q = 0; q < 8; ++q) tile_w[j * (kTileBytes / 16) + q * (8 * kRowBytes / 16)] = buf[j][q];
  };

  // Decision words: dec[b][c][row], lane 0 into the chunk's scratch word.
  const __amdgpu_buffer_rsrc_t dr = make_cursor(p.dec + (size_t)x.b * p.NC * (size_t)p.TP, p.NC * p.TP * 4).rsrc();
  const int dvo = 4 * (lane > 0 ? x.row : p.TP - 1);
  const int dstride = p.TP * 4;
  // Boundary words of this wave (OUT == 2) and of the previous one (IN == 2).
  const size_t slot_stride = (size_t)p.NC * kChunk;
  const int slot_bytes = (int)(slot_stride * 8u);
  const __amdgpu_buffer_rsrc_t sr = make_cursor(p.slots + ((size_t)x.b * p.NW + x.g) * slot_stride, slot_bytes).rsrc();
  const int svo = lane < kChunk ? 8 * lane : -16;
  const uint64_t* pslots = p.slots + ((size_t)x.b * p.NW + (x.g > 0 ? x.g - 1 : 0)) * slot_stride;
  Cursor pr = make_cursor(pslots, slot_bytes);
  if (IN2) pr.advance((x.c_begin - 1) * 256);  // first poll: chunk c_begin-1

  // Boundary words of chunk c (256 bytes) into poll slot c % 4.  These
  // loads are the only vector-memory operations the compiler does not see:
  // the wait before reading a poll slot counts them by hand.
  auto issue_poll = [&](int c, __amdgpu_buffer_rsrc_t r) __attribute__((always_inline)) {
    dma4_dev(lds_off(&L.poll[c & (kPollSlots - 1)][0]), r, 4 * lane);
  };
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
      // (c is uniform; saying so keeps the descriptor in scalar registers.)
      const int cu = __builtin_amdgcn_readfirstlane(c);
      issue_poll(cu, make_cursor(pslots + (size_t)cu * kChunk, kChunk * 8).rsrc_s());
      vm_wait<0>();
      wd = pw[lane & (kChunk - 1)];
    }
    return wd;
  };
  // Waits for the boundary row of chunk c in this wave's slot k.
  auto bound_ready = [&](int c, int k) __attribute__((always_inline)) {
    const int* tg = reinterpret_cast<const int*>(slot_ptr(wbase, k) + kTagOff);
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
    // The row above row 0 is -inf in every slot.
    if (lane < kChunk) {
#pragma unroll
      for (int k = 0; k < kSlots; ++k) reinterpret_cast<float*>(slot_ptr(wbase, k))[lane] = neg_inf();
    }
  }
  if (IN2) {
    // Polls of chunks c_begin-1 .. c_begin+1 (the loop polls two ahead).
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      issue_poll(x.c_begin - 1 + k, pr.rsrc_s());
      pr.advance(256);
    }
  }
  // The first group in flight.
  load_group();

  // Lane 0's Q at the column before the first chunk: the previous wave's
  // last row there (its chunk c_begin-1, always computed), or -inf.
  float q = neg_inf();
  if (IN == 1) {
    bound_ready(x.c_begin - 1, -1);
    wave_lds_sync();
    const float e = reinterpret_cast<const float*>(slot_ptr(wbase, -1))[kChunk - 1];
    q = lane == 0 ? e : q;
    wave_lds_sync();
    if (lane == 0) lds_store(&L.cons[wv], x.c_begin);
  } else if (IN == 2) {
    vm_wait<0>();
    const uint64_t wd = polled_word(x.c_begin - 1);
    const float e = __int_as_float(__builtin_amdgcn_readlane((int)(uint32_t)wd, kChunk - 1));
    q = lane == 0 ? e : q;
  }

  // Lane 0 publishes the consumed-chunk counter; the other lanes write
  // their own dummy words (one store, no exec change).
  int* const cons_ptr = lane == 0 ? &L.cons[wv] : reinterpret_cast<int*>(&L.dummy[wv][lane]);
  // Lower bound of the consumer's counter: it starts at its own c_begin-1,
  // which is at least this wave's c_begin+1 (63 rows span >= 63 columns).
  int cons_seen = x.c_begin + 1;
  const int dk = x.c_begin - x.next_begin;  // the next wave's slot of chunk c: c - c_begin + dk
  float qc[kChunk];
  int soff = x.c_begin * dstride;
  // One chunk, at position J of its group: its tile and its boundary slot
  // are number J.
  auto step = [&](auto pos_c, int c) __attribute__((always_inline)) {
    constexpr int J = decltype(pos_c)::value;
    const int k = c - x.c_begin;  // k % kSlots == J
    if (IN2) {
      // Poll of chunk c: issued two steps ago, followed by the rest of that
      // step and the next one (the group's loads come first in position 0),
      // and nothing of this one yet.
      constexpr int tail = 1 + (OUT2 ? 1 : 0);
      constexpr int n = tail + (((J - 2) & (kGroup - 1)) == 0 ? 8 * kGroup : 0) + 1 + tail +
                        (((J - 1) & (kGroup - 1)) == 0 ? 8 * kGroup : 0);
      vm_wait<n>();
      issue_poll(c + 2, pr.rsrc_s());
      pr.advance(256);
    }
    if (J == 0) {
      // The group's tiles into LDS (the previous group's reads are done),
      // the next group into flight.
      wave_lds_sync();
      put_group();
      load_group();
    }
    // The row above: from the previous wave, or copied from the polled
    // words.  Beyond the previous wave's chunks the slot holds stale values:
    // they only reach cells that cannot reach (t_x-1, t_y-1).
    if (IN == 1 && c < x.prev_end) bound_ready(c, k);
    if (IN2 && c < x.prev_end) {
      const uint64_t wd = polled_word(c);
      reinterpret_cast<float*>(slot_ptr(wbase, k))[lane & (kChunk - 1)] = __uint_as_float((uint32_t)wd);
    }
    wave_lds_sync();
    f32x4 v[8];
    {
      const f32x4* src = lane > 0 ? tile_r + J * (kTileBytes / 16) : reinterpret_cast<const f32x4*>(slot_ptr(wbase, J));
#pragma unroll
      for (int m = 0; m < 8; ++m) v[m] = src[m];
    }
    uint32_t bits = 0;
    if (c < x.mask_end)
      sweep_chunk<true>(q, t, v, qc, bits, lane, x.row, c * kChunk);
    else
      sweep_chunk<false>(q, t, v, qc, bits, lane, x.row, c * kChunk);
    __builtin_amdgcn_raw_buffer_store_b32(bits, dr, dvo, soff, kPolicyDev);
    soff += dstride;
    if (IN == 1) {
      // The reads of this chunk's slot are done: the previous wave may
      // reuse it for chunk c + kSlots.
      lds_store(cons_ptr, c + 1);
    }
    if (OUT == 1) {
      // Wait until the consumer no longer needs the slot, then publish the
      // values, then the tag.
      int spins = 0;
      while (cons_seen < c - (kSlots - 1)) {
        cons_seen = __builtin_amdgcn_readfirstlane(lds_load(&L.cons[wv + 1]));
        if (cons_seen >= c - (kSlots - 1)) break;
        if (++spins > kSpinLimit) {
          timed_out = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      char* const ns = slot_ptr(nbase, k + dk);
      if (lane == kWave - 1) {
        f32x4* dst = reinterpret_cast<f32x4*>(ns);
#pragma unroll
        for (int m = 0; m < kChunk / 4; ++m) dst[m] = f32x4{qc[4 * m], qc[4 * m + 1], qc[4 * m + 2], qc[4 * m + 3]};
      }
      // Values before the tag (the LDS executes one wave's operations in
      // order; the fence keeps the compiler from reordering them).  Kept out
      // of the lane-63 branch: inside it, the compiler makes the whole chunk
      // loop divergent for the waves that feed no other wave of the group.
      wave_lds_sync();
      if (lane == kWave - 1) lds_store(reinterpret_cast<int*>(ns + kTagOff), c + 1);
    } else if (OUT2) {
      if (lane == kWave - 1) {
#pragma unroll
        for (int m = 0; m < kChunk / 4; ++m) L.ostage[m] = f32x4{qc[4 * m], qc[4 * m + 1], qc[4 * m + 2], qc[4 * m + 3]};
      }
      wave_lds_sync();
      const float val = reinterpret_cast<const float*>(L.ostage)[lane & (kChunk - 1)];
      const uint64_t word = ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(val);
      __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, word), sr, svo, c * 256, kPolicyDev);
      wave_lds_sync();
    }
  };
  for (int c = x.c_begin; c < x.c_end; c += kGroup) {
    step(IntC<0>(), c);
    if (c + 1 < x.c_end) step(IntC<1>(), c + 1);
    if (c + 2 < x.c_end) step(IntC<2>(), c + 2);
    if (c + 3 < x.c_end) step(IntC<3>(), c + 3);
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
  if (threadIdx.x < kWavesPerBlock * kSlots)
    lds_store(reinterpret_cast<int*>(&L.u.tile[threadIdx.x / kSlots][kBoundOff + (threadIdx.x % kSlots) * kSlotBytes + kTagOff]), 0);
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
    score = g == 0 ? sweep_rows<0, 0>(p, L, x, tag, timed_out)
                   : (wv > 0 ? sweep_rows<1, 0>(p, L, x, tag, timed_out) : sweep_rows<2, 0>(p, L, x, tag, timed_out));
  } else if (wv < kWavesPerBlock - 1) {
    score = g == 0 ? sweep_rows<0, 1>(p, L, x, tag, timed_out)
                   : (wv > 0 ? sweep_rows<1, 1>(p, L, x, tag, timed_out) : sweep_rows<2, 1>(p, L, x, tag, timed_out));
  } else {
    score = sweep_rows<1, 2>(p, L, x, tag, timed_out);
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

// One workgroup per CU.
__global__ void __launch_bounds__(kThreadsPerBlock, 1) mas_kernel(KParams p) {
  __shared__ SweepLds L;
  const uint32_t gen = __hip_atomic_load(&p.hdr->gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t tag = call_tag(gen);
  bool timed_out = false;
  const int item = (int)blockIdx.x % p.B;
  sweep_block(p, L, blockIdx.x, tag, timed_out);
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
hipError_t launch_mas(const KParams& p, hipStream_t stream) {
  const dim3 grid((unsigned)(p.B * p.NB)), block(kThreadsPerBlock);
  hipLaunchKernelGGL(mas_kernel, grid, block, 0, stream, p);
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
