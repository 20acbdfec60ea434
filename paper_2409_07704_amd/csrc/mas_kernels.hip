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
constexpr int kRing = 16;            // LDS hand-off ring depth (chunks)
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

// One value tile, 16-byte variant: load q (q = 0..7) brings every lane's
// 16-byte piece at byte offset voff[q] of the resource to LDS at
// lds + 1024 q + 16 lane.  Eight operations.  (Offsets are kept in the
// range-checked per-lane operand: the resource base moves per chunk.)
__device__ __forceinline__ void dma_tile16(uint32_t lds, __amdgpu_buffer_rsrc_t r, const int (&vo)[8]) {
  asm volatile(
      "s_mov_b32 m0, %[l]\n\ts_nop 0\n\t"
      "buffer_load_dwordx4 %[v0], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x400\n\ts_nop 0\n\t"
      "buffer_load_dwordx4 %[v1], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x800\n\ts_nop 0\n\t"
      "buffer_load_dwordx4 %[v2], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0xc00\n\ts_nop 0\n\t"
      "buffer_load_dwordx4 %[v3], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x1000\n\ts_nop 0\n\t"
      "buffer_load_dwordx4 %[v4], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x1400\n\ts_nop 0\n\t"
      "buffer_load_dwordx4 %[v5], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x1800\n\ts_nop 0\n\t"
      "buffer_load_dwordx4 %[v6], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x1c00\n\ts_nop 0\n\t"
      "buffer_load_dwordx4 %[v7], %[r], 0 offen lds"
      :
      : [l] "s"(lds), [r] "s"(r), [v0] "v"(vo[0]), [v1] "v"(vo[1]), [v2] "v"(vo[2]), [v3] "v"(vo[3]),
        [v4] "v"(vo[4]), [v5] "v"(vo[5]), [v6] "v"(vo[6]), [v7] "v"(vo[7])
      : "memory", "m0", "scc");
}

// Eight 4-byte loads: load k brings every lane's word at voff[k] of the
// resource to LDS at lds + 256 k + 4 lane.
__device__ __forceinline__ void dma_words8(uint32_t lds, __amdgpu_buffer_rsrc_t r, const int (&vo)[8]) {
  asm volatile(
      "s_mov_b32 m0, %[l]\n\ts_nop 0\n\t"
      "buffer_load_dword %[v0], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x100\n\ts_nop 0\n\t"
      "buffer_load_dword %[v1], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x200\n\ts_nop 0\n\t"
      "buffer_load_dword %[v2], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x300\n\ts_nop 0\n\t"
      "buffer_load_dword %[v3], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x400\n\ts_nop 0\n\t"
      "buffer_load_dword %[v4], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x500\n\ts_nop 0\n\t"
      "buffer_load_dword %[v5], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x600\n\ts_nop 0\n\t"
      "buffer_load_dword %[v6], %[r], 0 offen lds\n\t"
      "s_add_u32 m0, %[l], 0x700\n\ts_nop 0\n\t"
      "buffer_load_dword %[v7], %[r], 0 offen lds"
      :
      : [l] "s"(lds), [r] "s"(r), [v0] "v"(vo[0]), [v1] "v"(vo[1]), [v2] "v"(vo[2]), [v3] "v"(vo[3]),
        [v4] "v"(vo[4]), [v5] "v"(vo[5]), [v6] "v"(vo[6]), [v7] "v"(vo[7])
      : "memory", "m0", "scc");
}

// One 16-byte load per lane, device-scope: the bytes at voff of the resource
// to LDS at lds + 16 lane.
__device__ __forceinline__ void dma_piece(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  asm volatile("s_mov_b32 m0, %[l]\n\ts_nop 0\n\tbuffer_load_dwordx4 %[v], %[r], 0 offen sc1 lds"
               :
               : [l] "s"(lds), [r] "s"(r), [v] "v"(voff)
               : "memory", "m0");
}

// One 16-byte piece per lane, device-scope, to LDS at lds + 16 lane.
__device__ __forceinline__ void dma_poll(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  asm volatile("s_mov_b32 m0, %[l]\n\ts_nop 0\n\tbuffer_load_dwordx4 %[v], %[r], 0 offen sc1 lds"
               :
               : [l] "s"(lds), [r] "s"(r), [v] "v"(voff)
               : "memory", "m0");
}

// A placeholder operation that keeps a step's operation count when it has
// nothing to store: one 4-byte load per lane into a scratch LDS area.
__device__ __forceinline__ void dma_dummy(uint32_t lds, __amdgpu_buffer_rsrc_t r, int voff) {
  asm volatile("s_mov_b32 m0, %[l]\n\ts_nop 0\n\tbuffer_load_dword %[v], %[r], 0 offen lds"
               :
               : [l] "s"(lds), [r] "s"(r), [v] "v"(voff)
               : "memory", "m0");
}

__device__ __forceinline__ void vm_store32(uint64_t a, uint32_t v) {
  asm volatile("global_store_dword %0, %1, off sc1" ::"v"(a), "v"(v) : "memory");
}
__device__ __forceinline__ void vm_store64(uint64_t a, uint64_t v) {
  asm volatile("global_store_dwordx2 %0, %1, off sc1" ::"v"(a), "v"(v) : "memory");
}
// Two 16-byte zero stores (s_nop: a VALU write of store data needs one wait
// state).  Path bytes are only ever written by the wave that owns their row,
// so these need no device-scope write-through.
__device__ __forceinline__ void vm_zero2(uint64_t a0, uint64_t a1, u32x4 z) {
  asm volatile("global_store_dwordx4 %0, %2, off\n\tglobal_store_dwordx4 %1, %2, off\n\ts_nop 0" ::"v"(a0), "v"(a1), "v"(z)
               : "memory");
}
__device__ __forceinline__ void vm_zero1(uint64_t a, u32x4 z) {
  asm volatile("global_store_dwordx4 %0, %1, off\n\ts_nop 0" ::"v"(a), "v"(z) : "memory");
}

// Vector-memory operations of one sweep step, in issue order:
//   [poll of chunk c+2]  (waves fed by another workgroup)
//   tile of chunk c+kDepth (8 ops, or 32 for the 4-byte variant)
//   decision word of chunk c (1)
//   [boundary words of chunk c]  (waves that feed another workgroup)
//   [2 zero stores]      (when the path is written)
constexpr int step_ops(int nl, bool in2, bool h, bool z) { return (in2 ? 1 : 0) + nl + 1 + (h ? 1 : 0) + (z ? 2 : 0); }
// Count for the wait at the start of step c: tile c was issued kDepth steps
// earlier (followed by that step's stores and kDepth-1 whole steps), the
// poll of chunk c two steps earlier (followed by that step's tile and stores
// and one whole step).  Counts above 63 are clamped: at most 63 operations
// are ever outstanding, so the clamped wait still covers the operation.
constexpr int wait_count(int nl, bool in2, bool h, bool z) {
  const int k = step_ops(nl, in2, h, z);
  const int tail = 1 + (h ? 1 : 0) + (z ? 2 : 0);
  const int n_tile = tail + (kDepth - 1) * k;
  const int n_poll = nl + tail + k;
  const int n = in2 && n_poll < n_tile ? n_poll : n_tile;
  return n > 63 ? 63 : n;
}

template <int NL, bool IN2>
__device__ __forceinline__ void wait_step(bool h, bool z) {
  if (h) {
    if (z)
      vm_wait<wait_count(NL, IN2, true, true)>();
    else
      vm_wait<wait_count(NL, IN2, true, false)>();
  } else {
    if (z)
      vm_wait<wait_count(NL, IN2, false, true)>();
    else
      vm_wait<wait_count(NL, IN2, false, false)>();
  }
}

// Buffer resource over the bytes [off, total) of the region at p (empty
// when off >= total; total < 2^31).  Loads outside a resource return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t sub_rsrc(const void* p, uint64_t total, uint64_t off) {
  const uint64_t o = off < total ? off : total;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(static_cast<const char*>(p)) + o, 0, (int)(uint32_t)(total - o),
                                           0x00020000);
}

// XOR swizzle of 16-byte slots inside a tile row: slot (r, p) holds piece
// p ^ swz(r).  Distinct over 8 consecutive rows and over the 8 same-parity
// rows of any 16 consecutive rows, so 8- and 16-lane LDS phases are
// conflict-free for both the tile writes and the per-row reads.
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

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

// One hand-off slot between waves of a workgroup: the producer's last-row Q
// over one chunk, then a tag (chunk + 1) written after the values.
struct RingSlot {
  f32x4 q[kChunk / 4];
  int tag[4];
};

struct SweepLds {
  union {
    // Value tiles: [wave][slot] rows 63g .. 63g+63 x 32 columns, 16-byte unit
    // 8 r + s holds piece s ^ swz(r) of tile row r.
    f32x4 tile[kWavesPerBlock][kStages][8 * kWave];
    // The walker's staging, once every sweep of its item (and so of its
    // workgroup) has finished.
    struct {
      uint32_t win[kWalkSlots][kWalkWin];  // decision-word windows of upcoming chunks
      int rs[kMaxRows + 2 * kWave];        // row_start under construction
    } walk;
  } u;
  RingSlot ring[kWavesPerBlock - 1][kRing];       // wave w -> w+1 boundary rows
  uint64_t poll[kPollSlots][2 * kWave];           // polled boundary words (4 copies of 32)
  f32x4 stage[kWavesPerBlock][kChunk / 4];        // boundary row staging (global hand-off)
  f32x4 ninf[kChunk / 4];                         // a chunk of -inf (the row above row 0)
  uint32_t dummy[kWavesPerBlock][kWave];          // target of placeholder loads
  int cons[kWavesPerBlock];                       // next chunk wave w will consume
};

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
  int lane, wv, b, g, g_last, tx, ty, row, c_begin, c_end, out_mode;
  int prev_end;                     // chunks the previous wave computes (exclusive end)
  int mask_end;                     // first chunk without a cell i > j of this wave
  bool zero;                        // this wave clears its path rows during its steps
  const float* slab;                // the item's value slab [T][S]
  uint64_t slab_bytes;
  uint64_t row_off;                 // byte offset of the wave's first tile row in the slab
  const uint64_t* pslots;           // the previous wave's boundary words (IN == 2)
  uint64_t pslot_bytes;
  int voff[8];                      // per-lane byte offsets of the tile loads
  uint32_t tile0;                   // LDS offset of this wave's tile slot 0
  uint32_t dummy;                   // LDS offset of this wave's placeholder area
  uint64_t decp;                    // &dec[b][0][row] (lane 0: the scratch word)
  uint64_t slotp;                   // &slots[b][g][lane % 32] (boundary words out)
  ZeroPlan zp;
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

// Sweeps this wave's rows over its chunks and returns the score candidate
// (Q at (row, t_y-1) of this lane; only meaningful for the wave holding row
// t_x-1).  IN: where the row above the wave comes from — 0 nowhere (the wave
// holds row 0), 1 the LDS ring of the previous wave of the workgroup, 2
// global boundary words of the previous workgroup.  out_mode: 0 no
// consumer, 1 LDS ring, 2 global boundary words.
template <bool ALIGNED, int IN>
__device__ __forceinline__ float sweep_rows(const KParams& p, SweepLds& L, const WaveCtx& x, uint32_t tag, bool& timed_out) {
  constexpr int NL = ALIGNED ? 8 : 32;
  constexpr bool IN2 = IN == 2;
  const int lane = x.lane, wv = x.wv;
  const bool h = x.out_mode == 2, zero = x.zero;
  float score = neg_inf();
  float t = -0.0f;  // lane 0 keeps -0 for the whole sweep (see cols8)
  const u32x4 zv = {0u, 0u, 0u, 0u};
  const int dvo = 4 * lane;  // placeholder loads read the slab's first 256 bytes
  const __amdgpu_buffer_rsrc_t drsrc = sub_rsrc(x.slab, x.slab_bytes, 0);

  // Tile of chunk c into its slot.
  auto issue_tile = [&](int c) __attribute__((always_inline)) {
    const uint32_t dst = x.tile0 + (uint32_t)((c & (kStages - 1)) * 8 * kWave * 16);
    const uint64_t off = x.row_off + (uint64_t)c * (kChunk * 4);
    if (ALIGNED) {
      dma_tile16(dst, sub_rsrc(x.slab, x.slab_bytes, off), x.voff);
    } else {
      // Four groups of 8 loads; group hh covers tile rows 16hh .. 16hh+15.
#pragma unroll
      for (int hh = 0; hh < 4; ++hh)
        dma_words8(dst + hh * 2048, sub_rsrc(x.slab, x.slab_bytes, off + (uint64_t)hh * 16u * (uint64_t)p.S * 4u), x.voff);
    }
  };
  // Boundary words of chunk c (32 u64 = 256 bytes, 4 copies) into poll slot c % 4.
  const int pvo = 16 * (lane & 15);
  auto issue_poll = [&](int c) __attribute__((always_inline)) {
    dma_poll(lds_off(&L.poll[c & (kPollSlots - 1)][0]), sub_rsrc(x.pslots, x.pslot_bytes, (uint64_t)c * kChunk * 8u), pvo);
  };
  int zk = 0;  // zero steps issued
  auto issue_zero = [&]() __attribute__((always_inline)) {
    if (zero) {
      uint64_t a0 = x.zp.a0 + (uint64_t)zk * 2048u + 16u * (uint64_t)lane;
      uint64_t a1 = a0 + 1024u;
      a0 = a0 < x.zp.last ? a0 : x.zp.last;
      a1 = a1 < x.zp.last ? a1 : x.zp.last;
      vm_zero2(a0, a1, zv);
      ++zk;
    }
  };
  // Boundary words of chunk c in poll slot c % 4, word lane % 32, once every
  // one of them carries this call's tag (re-polled until then).
  auto polled_word = [&](int c) __attribute__((always_inline)) -> uint64_t {
    const int sl = c & (kPollSlots - 1);
    uint64_t wd = L.poll[sl][lane & (kChunk - 1)];
    int spins = 0;
    while (__builtin_amdgcn_ballot_w64((uint32_t)(wd >> 32) != tag) != 0) {
      if (++spins > kSpinLimit) {
        timed_out = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      issue_poll(c);
      vm_wait<0>();
      wd = L.poll[sl][lane & (kChunk - 1)];
    }
    return wd;
  };
  // Ring slot of chunk c from the previous wave, once its tag says it is
  // written (the tag is read before the values, and written after them).
  auto ring_ready = [&](int c) __attribute__((always_inline)) {
    const int* tg = &L.ring[wv - 1][c % kRing].tag[0];
    int spins = 0;
    while (lds_load(tg) != c + 1) {
      if (++spins > kSpinLimit) {
        timed_out = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  };

  // Pieces beyond what the steps will clear, up front.
  if (zero) zero_rest(x.zp, x.zp.a0 + (uint64_t)(kDepth + x.c_end - x.c_begin) * 2048u, lane);

  // Prologue: kDepth placeholder steps with the steady-state operation
  // sequence, so that the loop's wait counts hold from its first step.
  for (int c = x.c_begin - kDepth; c < x.c_begin; ++c) {
    if (IN2) issue_poll(c + 2);  // chunks c_begin-1 .. c_begin+1
    issue_tile(c + kDepth);
    dma_dummy(x.dummy, drsrc, dvo);
    if (h) dma_dummy(x.dummy, drsrc, dvo);
    issue_zero();
  }

  // Lane 0's Q at the column before the first chunk: the previous wave's
  // last row there (its chunk c_begin-1, always computed), or -inf.
  float q = neg_inf();
  if (IN == 1) {
    ring_ready(x.c_begin - 1);
    wave_lds_sync();
    const f32x4 e = L.ring[wv - 1][(x.c_begin - 1) % kRing].q[kChunk / 4 - 1];
    q = lane == 0 ? e.w : q;
  } else if (IN == 2) {
    vm_wait<0>();
    const uint64_t wd = polled_word(x.c_begin - 1);
    const float e = __int_as_float(__builtin_amdgcn_readlane((int)(uint32_t)wd, kChunk - 1));
    q = lane == 0 ? e : q;
  }
  if (lane == 0) lds_store(&L.cons[wv], x.c_begin);

  // This lane's 32 values come from its tile row (lanes 1..63: tile row
  // lane-1) or, for lane 0, from the row above's 32 Q values.
  const int tsw = lane > 0 ? swz(lane - 1) : 0;
  const int trow = lane > 0 ? lane - 1 : 0;
  // Lower bound of the consumer's counter: it starts at its own c_begin-1,
  // which is at least this wave's c_begin+1 (63 rows span >= 63 columns).
  int cons_seen = x.c_begin + 1;
  for (int c = x.c_begin; c < x.c_end; ++c) {
    wait_step<NL, IN2>(h, zero);
    if (IN2) issue_poll(c + 2);
    issue_tile(c + kDepth);

    // Source of lane 0's values for this chunk.
    const f32x4* gsrc = L.ninf;
    if (IN == 1 && c < x.prev_end) {
      ring_ready(c);
      gsrc = L.ring[wv - 1][c % kRing].q;
    } else if (IN == 2 && c < x.prev_end) {
      const uint64_t wd = polled_word(c);
      float* sf = reinterpret_cast<float*>(L.stage[wv]);
      if (lane < kChunk) sf[lane] = __uint_as_float((uint32_t)wd);
      gsrc = L.stage[wv];
    }
    wave_lds_sync();
    f32x4 v[8];
    {
      const f32x4* base = lane > 0 ? L.u.tile[wv][c & (kStages - 1)] + 8 * trow : gsrc;
      const int sw = lane > 0 ? tsw : 0;
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = base[k ^ sw];
    }
    wave_lds_sync();
    if (IN == 1 && lane == 0) lds_store(&L.cons[wv], c + 1);
    float qc[kChunk];
    uint32_t bits = 0;
    if (c < x.mask_end)
      sweep_chunk<true>(q, t, v, qc, bits, lane, x.row, c * kChunk);
    else
      sweep_chunk<false>(q, t, v, qc, bits, lane, x.row, c * kChunk);

    // Stores of the step: decision word, boundary row, path zeros.
    vm_store32(x.decp + (uint64_t)c * (uint64_t)p.TP * 4u, bits);
    if (x.out_mode == 1) {
      // Wait until the consumer no longer needs the ring slot, then publish
      // the values, then the tag.
      int spins = 0;
      while (cons_seen < c - (kRing - 2)) {
        cons_seen = lds_load(&L.cons[wv + 1]);
        if (cons_seen >= c - (kRing - 2)) break;
        if (++spins > kSpinLimit) {
          timed_out = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      RingSlot& rs = L.ring[wv][c % kRing];
      if (lane == kWave - 1) {
#pragma unroll
        for (int k = 0; k < kChunk / 4; ++k) rs.q[k] = f32x4{qc[4 * k], qc[4 * k + 1], qc[4 * k + 2], qc[4 * k + 3]};
      }
      wave_lds_sync();
      if (lane == kWave - 1) lds_store(&rs.tag[0], c + 1);
    } else if (h) {
      if (lane == kWave - 1) {
#pragma unroll
        for (int k = 0; k < kChunk / 4; ++k) L.stage[wv][k] = f32x4{qc[4 * k], qc[4 * k + 1], qc[4 * k + 2], qc[4 * k + 3]};
      }
      wave_lds_sync();
      const float val = reinterpret_cast<const float*>(L.stage[wv])[lane & (kChunk - 1)];
      const uint64_t word = ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(val);
      vm_store64(x.slotp + (uint64_t)c * kChunk * 8u, word);
      wave_lds_sync();
    }
    issue_zero();
    if (x.g == x.g_last && c == x.c_end - 1) {
      const int m_last = (x.ty - 1) % kChunk;
#pragma unroll
      for (int m = 0; m < kChunk; ++m) score = (m == m_last) ? qc[m] : score;
    }
  }
  vm_wait<0>();
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

  // Workgroup set-up: no ring slot is written yet; each wave's first chunk
  // to consume (its carried row starts at chunk c_begin-1); the -inf chunk.
  for (int i = threadIdx.x; i < (kWavesPerBlock - 1) * kRing; i += kThreadsPerBlock) lds_store(&L.ring[i / kRing][i % kRing].tag[0], 0);
  if (lane == 0) lds_store(&L.cons[wv], c_begin - 1);
  if (threadIdx.x < kChunk / 4) L.ninf[threadIdx.x] = f32x4{neg_inf(), neg_inf(), neg_inf(), neg_inf()};
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
  x.out_mode = g == g_last ? 0 : (wv < kWavesPerBlock - 1 ? 1 : 2);
  // The walker's wave clears its rows during its steps; the others after.
  x.zero = clear && g == g_last;
  x.zp = zp;
  x.slab = p.value + (size_t)b * (size_t)p.T * (size_t)p.S;
  x.slab_bytes = (uint64_t)p.T * (uint64_t)p.S * 4u;
  x.row_off = (uint64_t)g * kRowsPerWave * (uint64_t)p.S * 4u;
  const size_t slot_stride = (size_t)p.NC * kChunk;
  x.pslots = p.slots + ((size_t)b * p.NW + (g > 0 ? g - 1 : 0)) * slot_stride;
  x.pslot_bytes = slot_stride * 8u;
  // Tile rows 0..63 are item rows 63g .. 63g+63 (row 63 is not used); offsets
  // are relative to the first tile row at the chunk's first column, and rows
  // past the slab fall outside the resource and read 0.  Tile rows below 64
  // and S * 4 * 64 < 2^31 keep them in range of an int.
  if (ALIGNED) {
    // Load q: lane L reads tile row 8q + L/8, piece (L%8) ^ swz(row).
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int tr = 8 * q + (lane >> 3);
      const int pc = (lane & 7) ^ swz(tr);
      x.voff[q] = (tr * p.S + 4 * pc) * 4;
    }
  } else {
    // Load k of group hh: lane L writes LDS word 64k + L of the group, i.e.
    // tile row 16hh + 2k + L/32, slot (L%32)/4, word L%4 (swz has period 16).
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int tr = 2 * k + (lane >> 5);
      const int pc = ((lane & 31) >> 2) ^ swz(tr);
      x.voff[k] = (tr * p.S + 4 * pc + (lane & 3)) * 4;
    }
  }
  x.tile0 = lds_off(&L.u.tile[wv][0][0]);
  x.dummy = lds_off(&L.dummy[wv][0]);
  x.decp = (uint64_t)(uintptr_t)(p.dec + (size_t)b * p.NC * (size_t)p.TP + (lane > 0 ? (size_t)x.row : (size_t)p.TP - 1));
  x.slotp = (uint64_t)(uintptr_t)(p.slots + ((size_t)b * p.NW + g) * slot_stride + (lane & (kChunk - 1)));
  const float score = g == 0 ? sweep_rows<ALIGNED, 0>(p, L, x, tag, timed_out)
                             : (wv > 0 ? sweep_rows<ALIGNED, 1>(p, L, x, tag, timed_out)
                                       : sweep_rows<ALIGNED, 2>(p, L, x, tag, timed_out));

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
  // Ones of this wave's rows: lane l writes row 63g + l - 1, from row_start
  // entries 63g + l - 1 (lane l-1's) and 63g + l (its own).
  const int ri = min(g * kRowsPerWave + lane, p.T);
  const int hi = g == g_last ? rsl[ri] : (int)ld_dev(reinterpret_cast<const uint32_t*>(rs_out + ri));
  const int lo = __builtin_amdgcn_update_dpp(0, hi, 0x138, 0xF, 0xF, false);  // lane l-1's entry
  const int row = g * kRowsPerWave + lane - 1;
  if (lane > 0 && row < tx) {
    uint8_t* prow = p.path + ((size_t)b * (size_t)p.T + (size_t)row) * (size_t)p.S;
    if (p.path16) {
      for (int j0 = lo & ~15; j0 < hi; j0 += 16) *reinterpret_cast<uint4*>(prow + j0) = path_piece(lo, hi, j0);
    } else {
      for (int j = lo; j < hi; ++j) prow[j] = 1;
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
