// libmas kernels for gfx950 (MI355X): batched monotonic alignment search
// (Super-MAS Sec. 2, Algorithm 1; column-parallel forward loop of
// Algorithm 2) and the dense path writer.
//
// One launch computes everything (mas_kernel):
//   * Zero workgroups (the lowest block ids) stream zeros over the whole
//     [B, T, S] path while the sweep runs.
//   * Sweep workgroups own 256 text rows of one item: four waves, one text
//     row per lane, 64 rows per wave.  A wave walks the speech axis in
//     chunks of 32 columns.  The recurrence's only cross-row dependency, the
//     diagonal predecessor Q[i-1][j-1], crosses lanes with one DPP
//     wave_shr:1 per column, crosses waves of a workgroup through an LDS
//     ring, and crosses workgroups through 64-bit {value, tag} words in
//     global memory.  Wave g starts at chunk floor(64g / 32): all earlier
//     cells of its rows lie in the masked triangle i > j, so waves are
//     naturally skewed by 64 columns, which covers the hand-off latency.
//   * Each lane reads its own row's 32 values of a chunk (128 contiguous
//     bytes, eight 16-byte buffer loads with the chunk offset in a scalar
//     register) three chunks ahead, straight into the registers the
//     recurrence uses.
//   * Q is never materialised: each lane keeps its row's previous column in
//     a register.  Each column's 64-row decision mask is the compare's SGPR
//     mask; every lane shifts its bit into a 32-bit word (v_addc with the
//     mask as carry-in), stored once per chunk.
//   * The wave owning row t_x-1 then walks the decision words backwards
//     from (t_x-1, t_y-1), four chunks per block.  A block's words are
//     fetched two blocks ahead into registers (a block descends at most 128
//     rows, so a 448-row band bounds every word it can need) and staged in
//     LDS.  Within a chunk each row step is a find-first-set over one word
//     and sets one bit of a scalar path mask; the chunk's rows are then
//     scattered to row_start in LDS in one step.  Finally the wave writes
//     row_start and the item's ones into the zero-filled path.
//
// Memory ordering: data handed between workgroups (decision words, boundary
// words, progress flags, path bytes) is written with device-scope
// write-through stores and read with device-scope loads, and a wave waits
// for its own stores to complete (vmcnt(0)) before raising a flag, so no
// cache write-back or invalidation is needed.  On gfx9 the vector memory
// counter retires in issue order and counts stores too, so the loops keep a
// fixed sequence of loads per iteration (exact compiler waits) and keep
// loads that are waited on soon from queueing behind slow stores.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mas_internal.h"

namespace mas {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

// 64-bit lane mask of (a < b); NaN compares false as in C.
__device__ __forceinline__ uint64_t lt_mask(float a, float b) { return __builtin_amdgcn_ballot_w64(a < b); }

// mask ? t : f, per lane, from an SGPR lane mask.
__device__ __forceinline__ float select_mask(float f, float t, uint64_t m) {
  float r;
  asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(f), "v"(t), "s"(m));
  return r;
}

// bits * 2 + (this lane's bit of m): shifts a decision into a lane's word.
__device__ __forceinline__ uint32_t push_bit(uint32_t bits, uint64_t m) {
  uint32_t r;
  uint64_t carry;
  asm("v_addc_co_u32_e64 %0, %1, %2, %2, %3" : "=v"(r), "=s"(carry) : "v"(bits), "s"(m));
  return r;
}

// Lane l >= 1 receives src from lane l-1; lane 0 receives lane0 (DPP wave_shr:1).
__device__ __forceinline__ float shift_rows(float src, float lane0) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(lane0), __float_as_int(src), 0x138, 0xF, 0xF, false));
}

// acc[lane] = v for one (uniform) lane.
__device__ __forceinline__ void write_lane(int& acc, int v, int sel, int lane) { acc = lane == sel ? v : acc; }

// Keeps the compiler from moving LDS accesses across this point; LDS
// operations of one wave execute in order, so no wait is needed.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Device-scope (write-through) stores and loads of data shared across
// workgroups, and a wait for this wave's outstanding memory operations.
__device__ __forceinline__ void st_dev(uint32_t* p, uint32_t v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ void st_dev(uint64_t* p, uint64_t v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ uint32_t ld_dev(const uint32_t* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ uint64_t ld_dev(const uint64_t* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ __forceinline__ void wait_mem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ int lds_load(const int* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP); }
__device__ __forceinline__ void lds_store(int* p, int v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP); }

__device__ __forceinline__ uint32_t call_tag(uint32_t gen) { return 2u * gen + 1u; }

constexpr int kSpinLimit = 1 << 21;  // bound of every device-side wait (~seconds)
constexpr int kRing = 16;            // LDS hand-off ring depth (chunks)

// Buffer resource over one item's [T, S] value slab (T*S*4 < 2^31 bytes).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t slab_rsrc(const float* vb, int T, int S) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)vb, 0, T * S * 4, 0x00020000);
}
constexpr int kOob = 0x7fffff00;  // a byte offset past every slab: buffer loads return 0

// XOR swizzle of 16-byte slots inside a tile row: slot (r, p) holds piece
// p ^ swz(r).  Distinct over 8 consecutive rows and over the 8 same-parity
// rows of any 16 consecutive rows, so 8- and 16-lane LDS phases are
// conflict-free for both the transposing writes and the per-row reads.
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

template <bool ALIGNED>
struct TileLoader {
  // A chunk of the wave's 64 rows x 32 columns is fetched with 8 coalesced
  // 16-byte loads: lane L of load q reads tile row tr = 8q + L/8, piece
  // (L%8) ^ swz(tr), so 8 consecutive lanes cover one 128-byte row segment.
  // voff[q]: byte offset of the lane's piece in chunk 0 (or kOob for rows
  // past t_x).  Pieces at or past column t_y are not fetched (read as 0),
  // except inside the 16-byte piece holding column t_y-1.
  static __device__ __forceinline__ void load(f32x4 (&v)[8], __amdgpu_buffer_rsrc_t rsrc, const int (&voff)[8],
                                              const int (&col0)[8], int ty, int c) {
    const int soff = c * kChunk * 4;
    if ((c + 1) * kChunk <= ty) {  // whole chunk inside the extent
#pragma unroll
      for (int q = 0; q < 8; ++q) piece(v[q], rsrc, voff[q], soff);
      return;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) piece(v[q], rsrc, c * kChunk + col0[q] < ty ? voff[q] : kOob, soff);
  }
  static __device__ __forceinline__ void piece(f32x4& x, __amdgpu_buffer_rsrc_t rsrc, int vo, int so) {
    if (ALIGNED) {
      x = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, vo, so, 0));
    } else {
      x.x = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, vo, so + 0, 0));
      x.y = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, vo, so + 4, 0));
      x.z = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, vo, so + 8, 0));
      x.w = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, vo, so + 12, 0));
    }
  }
};

// One 32-column chunk of the recurrence for one row per lane.
//   q   : this lane's Q at the column before the chunk (updated)
//   v   : this lane's value[row][j0 .. j0+31]
//   bd  : Q[row0-1][j0-1 .. j0+30] (the row above the wave), read by lane 0
//   qc  : this lane's Q at every column of the chunk (out)
//   bits: decisions of the chunk, first column in bit 31 (out)
// MASKED handles the chunks that cross the triangle i > j (value not read
// there, Q = -inf) and the first cell Q[0][0] = value[0][0].
// FIRST: the wave holding row 0, whose row above is the virtual -inf row:
// `diag` keeps -inf in lane 0 (DPP leaves lane 0 untouched), so bd is unused.
template <bool MASKED, bool FIRST>
__device__ __forceinline__ void sweep_chunk(float& q, float& diag, const f32x4 (&v4)[8], const float (&bd)[kChunk],
                                            float (&qc)[kChunk], uint32_t& bits, int row, int j0) {
  uint32_t w = 0;
  float v[kChunk];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    v[4 * k + 0] = v4[k].x;
    v[4 * k + 1] = v4[k].y;
    v[4 * k + 2] = v4[k].z;
    v[4 * k + 3] = v4[k].w;
  }
#pragma unroll
  for (int m = 0; m < kChunk; ++m) {
    const float stay = q;
    diag = shift_rows(stay, FIRST ? diag : bd[m]);
    const uint64_t d = lt_mask(stay, diag);
    float qn = select_mask(stay, diag, d) + v[m];
    if (MASKED) {
      const int j = j0 + m;
      qn = (row > j) ? neg_inf() : qn;
      if (j == 0) qn = (row == 0) ? v[m] : neg_inf();
    }
    w = push_bit(w, d);
    qc[m] = qn;
    q = qn;
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
constexpr int kWalkChunks = 4;                 // chunks per walk block
constexpr int kWalkRows = 7 * kWave;           // rows staged per chunk of a block

struct SweepLds {
  f32x4 tile[kWavesPerBlock][8 * kWave];          // value tile of the chunk per wave (8 KiB)
  float ring[kWavesPerBlock - 1][kRing][kChunk];  // wave w -> w+1 boundary values
  f32x4 bout[kWavesPerBlock][kChunk / 4];         // boundary staging (global hand-off)
  int prod[kWavesPerBlock];                       // chunks wave w has published (exclusive end)
  int cons[kWavesPerBlock];                       // next chunk wave w will consume
  uint32_t blk[kWalkChunks][kWalkRows];           // decision words of the walk block
};

// Dynamic LDS: the walker's row_start table (T + 128 ints).
extern __shared__ int mas_rs_lds[];

// ---------------------------------------------------------------- zero fill
// Zero workgroup z writes its share of the whole path with device-scope
// stores, then publishes the call's tag in zprog[z].
__device__ __forceinline__ void zero_block(const KParams& p, int z, uint32_t tag) {
  const size_t total = (size_t)p.B * (size_t)p.T * (size_t)p.S;
  const size_t nthr = (size_t)p.NZ * blockDim.x;
  const size_t t0 = (size_t)z * blockDim.x + threadIdx.x;
  if (p.path16) {
    uint64_t* q = reinterpret_cast<uint64_t*>(p.path);
    const size_t n = total / 8;
    for (size_t k = t0; k < n; k += nthr) st_dev(q + k, 0ull);
  } else {
    for (size_t k = t0; k < total; k += nthr) __hip_atomic_store(p.path + k, (uint8_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  wait_mem();
  __syncthreads();
  if (threadIdx.x == 0) st_dev(p.zprog + z, (uint64_t)tag);
}

// ---------------------------------------------------------------- sweep
// Per-wave constants of the sweep.
struct WaveCtx {
  int lane, wv, b, g, g_last, tx, ty, row, c_begin, c_end, out_mode;
  __amdgpu_buffer_rsrc_t rsrc;
  int voff[8];  // byte offset of this lane's piece of load q in chunk 0
  int col0[8];  // its first column in chunk 0
  uint32_t* decp;
  const uint64_t* poll_base;
  uint64_t* slots_out;
};

// Sweeps this wave's 64 rows over all chunks of its item and returns the
// score candidate (Q at (row, t_y-1) of this lane; only meaningful for the
// wave holding row t_x-1).  IN: where the row above the wave comes from —
// 0 nowhere (the wave holds row 0), 1 the LDS ring of the previous wave of
// the workgroup, 2 global hand-off words of the previous workgroup.
// out_mode: 0 no consumer, 1 LDS ring, 2 global hand-off words.
template <bool ALIGNED, int IN>
__device__ __forceinline__ float sweep_rows(const KParams& p, SweepLds& L, const WaveCtx& x, uint32_t tag, bool& timed_out) {
  const int lane = x.lane, wv = x.wv;
  float q = neg_inf();
  float diag = neg_inf();  // lane 0 keeps -inf when IN == 0
  float score = neg_inf();

  // Global boundary words (IN == 2), polled two chunks ahead into a ring of
  // three registers that follows the three value buffers; waiting for a poll
  // then only waits for stores issued three chunks earlier.  Every lane loads
  // (lanes 32..63 repeat lanes 0..31) so the loads stay outside divergent
  // control flow.
  uint64_t bwa = 0, bwb = 0, bwc = 0;
  auto poll_issue = [&](uint64_t& bw, int c) __attribute__((always_inline)) {
    const int cc = c < x.c_end ? c : x.c_end - 1;  // past the end: re-read valid words
    bw = ld_dev(x.poll_base + (size_t)cc * kChunk);
  };
  auto poll_wait = [&](uint64_t& bw, int c) __attribute__((always_inline)) {
    if (__builtin_amdgcn_ballot_w64((uint32_t)(bw >> 32) != tag) == 0) return;
    int spins = 0;
    do {
      if (++spins > kSpinLimit) {
        timed_out = true;
        return;
      }
      __builtin_amdgcn_s_sleep(1);
      poll_issue(bw, c);
    } while (__builtin_amdgcn_ballot_w64((uint32_t)(bw >> 32) != tag) != 0);
  };
  if (IN == 2) {
    poll_issue(bwa, x.c_begin);
    poll_issue(bwb, x.c_begin + 1);
  }

  // bw: this chunk's polled words; bw2: the register chunk c+2 will check.
  const int rsw = swz(lane);
  int prod_seen = 0;                    // last value read of the producer's counter
  int cons_seen = x.c_begin + 2;        // last value read of the consumer's counter
  uint32_t bits_prev = 0;               // decision word of the previous chunk (stored one step late)
  auto step = [&](int c, const f32x4 (&stg)[8], uint64_t& bw, uint64_t& bw2) __attribute__((always_inline)) {
    // Transpose the chunk's tile through LDS: this lane's row, 32 values.
#pragma unroll
    for (int k = 0; k < 8; ++k) L.tile[wv][64 * k + lane] = stg[k];
    wave_lds_sync();
    f32x4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = L.tile[wv][8 * lane + (k ^ rsw)];
    // Boundary column values bd[m] = Q[row0-1][j0-1+m].
    float bd[kChunk];
    if (IN == 1) {
      int spins = 0;
      while (prod_seen <= c) {
        prod_seen = lds_load(&L.prod[wv - 1]);
        if (prod_seen > c) break;
        if (++spins > kSpinLimit) {
          timed_out = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      wave_lds_sync();
      const float* cur = L.ring[wv - 1][c % kRing];
      bd[0] = L.ring[wv - 1][(c + kRing - 1) % kRing][kChunk - 1];
#pragma unroll
      for (int m = 1; m < kChunk; ++m) bd[m] = cur[m - 1];
      wave_lds_sync();
      if (lane == 0) lds_store(&L.cons[wv], c + 1);
    } else if (IN == 2) {
      poll_wait(bw, c);
      reinterpret_cast<float*>(L.bout[wv])[lane & (kChunk - 1)] = __uint_as_float((uint32_t)bw);
      wave_lds_sync();
#pragma unroll
      for (int k = 0; k < kChunk / 4; ++k) {
        const f32x4 t = L.bout[wv][k];
        bd[4 * k + 0] = t.x;
        bd[4 * k + 1] = t.y;
        bd[4 * k + 2] = t.z;
        bd[4 * k + 3] = t.w;
      }
      poll_issue(bw2, c + 2);
    }
    wave_lds_sync();
    float qc[kChunk];
    uint32_t bits;
    if (c < x.c_begin + 2)
      sweep_chunk<true, IN == 0>(q, diag, v, bd, qc, bits, x.row, c * kChunk);
    else
      sweep_chunk<false, IN == 0>(q, diag, v, bd, qc, bits, x.row, c * kChunk);
    if (c > x.c_begin) st_dev(x.decp + (size_t)(c - 1) * p.TP, bits_prev);
    bits_prev = bits;
    if (x.out_mode == 1) {
      // Wait until the consumer no longer needs the ring slot, then publish.
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
      if (lane == kWave - 1) {
        f32x4* dst = reinterpret_cast<f32x4*>(L.ring[wv][c % kRing]);
#pragma unroll
        for (int k = 0; k < kChunk / 4; ++k) dst[k] = f32x4{qc[4 * k], qc[4 * k + 1], qc[4 * k + 2], qc[4 * k + 3]};
      }
      wave_lds_sync();
      if (lane == 0) lds_store(&L.prod[wv], c + 1);
    } else if (x.out_mode == 2) {
      if (lane == kWave - 1) {
#pragma unroll
        for (int k = 0; k < kChunk / 4; ++k) L.bout[wv][k] = f32x4{qc[4 * k], qc[4 * k + 1], qc[4 * k + 2], qc[4 * k + 3]};
      }
      wave_lds_sync();
      const float val = reinterpret_cast<const float*>(L.bout[wv])[lane & (kChunk - 1)];
      const uint64_t word = ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(val);
      st_dev(x.slots_out + (size_t)c * kChunk + (lane & (kChunk - 1)), word);
      wave_lds_sync();
    }
    if (x.g == x.g_last && c == x.c_end - 1) {
      const int m_last = (x.ty - 1) % kChunk;
#pragma unroll
      for (int m = 0; m < kChunk; ++m) score = (m == m_last) ? qc[m] : score;
    }
  };

  // Three chunks of values in flight; loads past the last chunk read
  // nothing (out of range).  Full triples first: every iteration issues the
  // same memory operations, so wait counts stay exact.
  f32x4 va[8], vbk[8], vc[8];
  TileLoader<ALIGNED>::load(va, x.rsrc, x.voff, x.col0, x.ty, x.c_begin);
  TileLoader<ALIGNED>::load(vbk, x.rsrc, x.voff, x.col0, x.ty, x.c_begin + 1);
  TileLoader<ALIGNED>::load(vc, x.rsrc, x.voff, x.col0, x.ty, x.c_begin + 2);
  int c = x.c_begin;
  for (; c + 2 < x.c_end; c += 3) {
    step(c, va, bwa, bwc);
    TileLoader<ALIGNED>::load(va, x.rsrc, x.voff, x.col0, x.ty, c + 3);
    step(c + 1, vbk, bwb, bwa);
    TileLoader<ALIGNED>::load(vbk, x.rsrc, x.voff, x.col0, x.ty, c + 4);
    step(c + 2, vc, bwc, bwb);
    TileLoader<ALIGNED>::load(vc, x.rsrc, x.voff, x.col0, x.ty, c + 5);
  }
  if (c < x.c_end) step(c, va, bwa, bwc);
  if (c + 1 < x.c_end) step(c + 1, vbk, bwb, bwa);
  st_dev(x.decp + (size_t)(x.c_end - 1) * p.TP, bits_prev);
  return score;
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
  const int c_begin = (g * kWave) / kChunk;

  if (lane == 0) {
    lds_store(&L.prod[wv], 0);
    lds_store(&L.cons[wv], c_begin);
  }
  __syncthreads();

  int32_t* rs_out = p.row_start + (size_t)b * ((size_t)p.T + 1);
  if (st != kItemOk) {
    if (g == 0) {
      for (int i = lane; i <= p.T; i += kWave) rs_out[i] = 0;
      if (lane == 0) {
        if (p.score) p.score[b] = neg_inf();
        if (p.status) p.status[b] = st;
      }
    }
    return;
  }
  if (g * kWave >= tx) return;  // no rows of this item here
  if (g == 0 && lane == 0 && p.status) p.status[b] = kItemOk;

  WaveCtx x;
  x.lane = lane;
  x.wv = wv;
  x.b = b;
  x.g = g;
  x.g_last = (tx - 1) / kWave;
  x.tx = tx;
  x.ty = ty;
  x.row = g * kWave + lane;
  x.c_begin = c_begin;
  x.c_end = (ty + kChunk - 1) / kChunk;
  x.out_mode = g == x.g_last ? 0 : (wv < kWavesPerBlock - 1 ? 1 : 2);
  x.rsrc = slab_rsrc(p.value + (size_t)b * (size_t)p.T * (size_t)p.S, p.T, p.S);
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int tr = 8 * q + (lane >> 3);
    const int pc = (lane & 7) ^ swz(tr);
    const int trow = g * kWave + tr;
    x.col0[q] = 4 * pc;
    x.voff[q] = trow < tx ? (trow * p.S + 4 * pc) * 4 : kOob;
  }
  x.decp = p.dec + (size_t)b * p.NC * (size_t)p.TP + x.row;
  const size_t slot_stride = (size_t)p.NC * kChunk;
  x.poll_base = p.slots + ((size_t)b * p.NW + (g > 0 ? g - 1 : 0)) * slot_stride + (lane & (kChunk - 1)) - 1;
  x.slots_out = p.slots + ((size_t)b * p.NW + g) * slot_stride;
  const int g_last = x.g_last;
  const float score = g == 0 ? sweep_rows<ALIGNED, 0>(p, L, x, tag, timed_out)
                             : (wv > 0 ? sweep_rows<ALIGNED, 1>(p, L, x, tag, timed_out)
                                       : sweep_rows<ALIGNED, 2>(p, L, x, tag, timed_out));

  // Publish this wave's decision words to the item's walker.
  wait_mem();
  if (lane == 0) st_dev(p.done + (size_t)b * p.NW + g, tag);
  if (g != g_last) return;

  // ------------------------------------------------------------ backtrack
  if (lane == ((tx - 1) & (kWave - 1)) && p.score) p.score[b] = score;
  for (int k0 = 0; k0 < g_last; k0 += kWave) {
    const int k = k0 + lane;
    int spins = 0;
    while (true) {
      const bool ready = k >= g_last || ld_dev(p.done + (size_t)b * p.NW + k) == tag;
      if (__builtin_amdgcn_ballot_w64(!ready) == 0) break;
      if (++spins > kSpinLimit) {
        timed_out = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }

  // Walk blocks of kWalkChunks chunks from the right.  Within a block the
  // path descends at most 32 * kWalkChunks rows, and a chunk reads rows down
  // to 32 below its entry row, so every row block n+2 reads lies within
  // 3 * 32 * kWalkChunks + 1 (<= kWalkRows) rows below the entry row of
  // block n: block n+2's words (rows [e - kWalkRows + 1, e] of each of its
  // chunks, e = entry row of block n) are fetched while block n is walked.
  const uint32_t* db = p.dec + (size_t)b * p.NC * (size_t)p.TP;
  auto fetch = [&](uint32_t (&w)[kWalkChunks][kWalkRows / kWave], int cb, int e) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kWalkChunks; ++k) {
      const int ch = cb - k;
      const size_t base = (size_t)(ch > 0 ? ch : 0) * p.TP;
#pragma unroll
      for (int i = 0; i < kWalkRows / kWave; ++i) {
        const int r = e - (kWalkRows - 1) + i * kWave + lane;  // rows ascending
        w[k][i] = ld_dev(db + base + (r > 0 ? r : 0));
      }
    }
  };
  auto stage = [&](const uint32_t (&w)[kWalkChunks][kWalkRows / kWave]) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kWalkChunks; ++k)
#pragma unroll
      for (int i = 0; i < kWalkRows / kWave; ++i) L.blk[k][i * kWave + lane] = w[k][i];
  };
  int idx = tx - 1;                  // entry row of the chunk being walked
  int cw = (ty - 1) / kChunk;        // chunk being walked
  int sh0 = 31 - (ty - 1) % kChunk;  // bits >= sh0 are columns not yet passed in chunk cw
  bool walking = idx > 0;
  // Walks the kWalkChunks chunks staged in L.blk (rows [eb - kWalkRows + 1,
  // eb] of chunks cb, cb-1, ...); clears `walking` when the walk is over.
  auto walk_block = [&](int eb) __attribute__((always_inline)) {
    for (int k = 0; k < kWalkChunks && walking; ++k) {
      // Window of this chunk: lane l holds the word of row idx - l.
      const int wr = idx - lane - (eb - (kWalkRows - 1));
      const uint32_t W = L.blk[k][wr > 0 ? wr : 0];
      int kk = 0, sh = sh0;
      uint32_t pm = 0;  // bit p set: the kk-th recorded row starts at column 32cw + 31 - p
      while (true) {
        const uint32_t w = __builtin_amdgcn_readlane(W, kk);
        const uint64_t t = (uint64_t)w & (~0ull << sh);
        if (t == 0) break;  // the row continues left of this chunk (row 0 never steps)
        const int pos = __builtin_ctzll(t);
        pm |= 1u << pos;
        sh = pos + 1;
        kk += 1;
      }
      // Scatter: set bit p of pm belongs to the row (popcount of pm below p) under idx.
      if (lane < kChunk && ((pm >> lane) & 1u))
        mas_rs_lds[idx - (int)__builtin_popcount(pm & ((1u << lane) - 1u))] = cw * kChunk + 31 - lane;
      idx -= kk;
      sh0 = 0;
      cw -= 1;
      walking = idx > 0 && cw >= 0;
    }
  };
  {
    uint32_t wa[kWalkChunks][kWalkRows / kWave], wb[kWalkChunks][kWalkRows / kWave];
    fetch(wa, cw, idx);
    fetch(wb, cw - kWalkChunks, idx);
    int ea = idx, eb_ = idx;  // band tops of the blocks held in wa / wb
    while (walking) {
      wave_lds_sync();
      stage(wa);
      wave_lds_sync();
      const int e0 = idx;
      fetch(wa, cw - 2 * kWalkChunks, e0);
      walk_block(ea);
      ea = e0;
      if (!walking) break;
      wave_lds_sync();
      stage(wb);
      wave_lds_sync();
      const int e1 = idx;
      fetch(wb, cw - 2 * kWalkChunks, e1);
      walk_block(eb_);
      eb_ = e1;
    }
  }
  wave_lds_sync();
  if (lane == 0) mas_rs_lds[0] = 0;
  for (int i = tx + lane; i <= p.T; i += kWave) mas_rs_lds[i] = ty;
  wave_lds_sync();
  for (int i = lane; i <= p.T; i += kWave) rs_out[i] = mas_rs_lds[i];

  if (!p.path) return;
  // Ones of the item's path, once the zero fill has finished.
  for (int z0 = 0; z0 < p.NZ; z0 += kWave) {
    const int z = z0 + lane;
    int spins = 0;
    while (true) {
      const bool ready = z >= p.NZ || (uint32_t)ld_dev(p.zprog + z) == tag;
      if (__builtin_amdgcn_ballot_w64(!ready) == 0) break;
      if (++spins > kSpinLimit) {
        timed_out = true;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  uint8_t* pb = p.path + (size_t)b * (size_t)p.T * (size_t)p.S;
  for (int i = lane; i < tx; i += kWave) {
    const int lo = mas_rs_lds[i], hi = mas_rs_lds[i + 1];
    uint8_t* prow = pb + (size_t)i * (size_t)p.S;
    if (p.path16) {
      for (int j0 = lo & ~15; j0 < hi; j0 += 16) {
        const uint4 x = path_piece(lo, hi, j0);
        uint64_t* d = reinterpret_cast<uint64_t*>(prow + j0);
        st_dev(d, ((uint64_t)x.y << 32) | x.x);
        st_dev(d + 1, ((uint64_t)x.w << 32) | x.z);
      }
    } else {
      for (int j = lo; j < hi; ++j) __hip_atomic_store(prow + j, (uint8_t)1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

template <bool ALIGNED>
// Two waves per SIMD: a sweep workgroup and a zero-fill workgroup share a CU.
__global__ void __launch_bounds__(kRowsPerBlock, 2) mas_kernel(KParams p) {
  __shared__ SweepLds L;
  const uint32_t gen = __hip_atomic_load(&p.hdr->gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t tag = call_tag(gen);
  bool timed_out = false;
  int item = -1;
  if ((int)blockIdx.x < p.NZ) {
    zero_block(p, blockIdx.x, tag);
  } else {
    const int sid = blockIdx.x - p.NZ;
    item = sid % p.B;
    sweep_block<ALIGNED>(p, L, sid, tag, timed_out);
  }
  if (timed_out) {
    if (p.status && item >= 0) p.status[item] = kItemSyncTimeout;
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
  const dim3 grid((unsigned)(p.NZ + p.B * p.NB)), block(kRowsPerBlock);
  const size_t lds = ((size_t)p.T + 2 * kWave) * sizeof(int);
  if (aligned)
    hipLaunchKernelGGL(mas_kernel<true>, grid, block, lds, stream, p);
  else
    hipLaunchKernelGGL(mas_kernel<false>, grid, block, lds, stream, p);
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
