// libmas kernels for gfx950 (MI355X): forward max-plus sweep with decision
// bits and backtrack (Super-MAS Sec. 2, Algorithms 1-2), and the dense path
// writer.
//
// Forward sweep design:
//   * One text row per lane, 64 rows per wave, waves of an item chained
//     along the text axis.  A wave walks the speech axis in chunks of 32
//     columns; the only cross-row dependency of the recurrence is the
//     diagonal predecessor Q[i-1][j-1], which crosses lanes with one DPP
//     wave_shr:1 per column and crosses waves through 64-bit {value, tag}
//     words in global memory (one per column, published a chunk at a time).
//   * Wave g starts at chunk floor(64g / 32): every earlier cell of its rows
//     lies in the masked triangle i > j, so its previous column starts at
//     -inf.  The waves of an item are therefore naturally skewed by 64
//     columns, which covers the hand-off latency.
//   * The value tile of a chunk (64 rows x 32 columns = 8 KiB) is read with
//     coalesced 16-byte loads (8 lanes per 128-byte row segment), staged in
//     LDS with an XOR swizzle that keeps both the writes and the per-row
//     reads free of bank conflicts, and read back one row per lane.
//   * Q is never materialised: each lane keeps its row's previous column in
//     a register.  The per-column decision mask of the wave comes out of the
//     compare as a 64-bit SGPR mask; each lane shifts its own bit into a
//     32-bit word (v_addc with the mask as carry-in), stored once per chunk.
//   * After its last chunk the wave owning row t_x-1 waits for the other
//     waves of the item, then walks the decision words backwards from
//     (t_x-1, t_y-1) and writes row_start[].  Within a 32-column chunk the
//     path visits at most 32 rows, so a 64-row window of words, fetched one
//     chunk ahead, holds every word the walk can need; each row step is a
//     find-first-set over one word.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mas_internal.h"

namespace mas {

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

// Orders this wave's LDS traffic between lanes (same wave, so no s_barrier).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// XOR swizzle of 16-byte slots inside a tile row: slot (r, p) holds piece
// p ^ swz(r).  Distinct for 8 consecutive rows and for the 8 same-parity rows
// of any 16 consecutive rows, so 8- and 16-lane LDS phases are conflict-free.
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

template <bool ALIGNED>
struct TileLoader {
  // Lane L of load q (q = 0..7) fetches tile row 8q + L/8, piece (L%8) ^ swz(row),
  // and later stores it to LDS slot 64q + L; a row's 8 pieces come from 8
  // consecutive lanes, so every 128-byte segment is read by one coalesced group.
  static __device__ __forceinline__ void load(float4 (&stg)[8], const float* __restrict__ vb, int S, int row0, int tx,
                                              int ty, int c, int lane) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int tr = 8 * q + (lane >> 3);
      const int p = (lane & 7) ^ swz(tr);
      const int row = row0 + tr;
      const int col = c * kChunk + 4 * p;
      float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
      if (row < tx && col < ty) {
        const float* src = vb + (size_t)row * (size_t)S + col;
        if (ALIGNED) {
          x = *reinterpret_cast<const float4*>(src);
        } else {
          x.x = src[0];
          if (col + 1 < ty) x.y = src[1];
          if (col + 2 < ty) x.z = src[2];
          if (col + 3 < ty) x.w = src[3];
        }
      }
      stg[q] = x;
    }
  }
};

// One 32-column chunk of the recurrence for one row per lane.
//   q      : this lane's Q at the column before the chunk (updated)
//   v      : this lane's value[row][j0 .. j0+31]
//   bd     : Q[row0-1][j0-1 .. j0+30] (the row above the wave), any lane
//   qc     : this lane's Q at every column of the chunk (out)
//   bits   : decisions of the chunk, first column in bit 31 (out)
// MASKED handles the chunks that cross the triangle i > j (value not read
// there, Q = -inf) and the first cell Q[0][0] = value[0][0].
template <bool MASKED>
__device__ __forceinline__ void sweep_chunk(float& q, const float (&v)[kChunk], const float (&bd)[kChunk],
                                            float (&qc)[kChunk], uint32_t& bits, int row, int j0) {
  uint32_t w = 0;
#pragma unroll
  for (int m = 0; m < kChunk; ++m) {
    const float stay = q;
    const float diag = shift_rows(stay, bd[m]);
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

__device__ __forceinline__ uint32_t call_tag(uint32_t gen) { return 2u * gen + 1u; }

constexpr int kSpinLimit = 1 << 21;

template <bool ALIGNED>
__global__ void __launch_bounds__(kRowsPerBlock) mas_search_kernel(SearchParams p) {
  __shared__ float4 tile[kWavesPerBlock][8 * kWave];       // 8 KiB per wave
  __shared__ float4 bnd_lds[kWavesPerBlock][kChunk / 4];   // boundary values in
  __shared__ float4 bout_lds[kWavesPerBlock][kChunk / 4];  // boundary values out

  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int b = blockIdx.x % p.B;
  const int g = (blockIdx.x / p.B) * kWavesPerBlock + wv;  // wave index inside the item
  const uint32_t gen = __hip_atomic_load(&p.hdr->gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t tag = call_tag(gen);
  bool timed_out = false;

  const int tx = p.t_x[b];
  const int ty = p.t_y[b];
  const int st = item_status(tx, ty, p.T, p.S);
  int32_t* rs = p.row_start + (size_t)b * ((size_t)p.T + 1);

  if (st != kItemOk) {
    if (g == 0) {
      for (int i = lane; i <= p.T; i += kWave) rs[i] = 0;
      if (lane == 0) {
        if (p.score) p.score[b] = neg_inf();
        if (p.status) p.status[b] = st;
      }
    }
  } else if (g * kWave < tx) {
    if (g == 0 && lane == 0 && p.status) p.status[b] = kItemOk;
    const int row0 = g * kWave;
    const int row = row0 + lane;
    const int g_last = (tx - 1) / kWave;
    const int c_begin = row0 / kChunk;
    const int c_end = (ty + kChunk - 1) / kChunk;
    const float* vb = p.value + (size_t)b * (size_t)p.T * (size_t)p.S;
    uint32_t* decp = p.dec + (size_t)b * p.NC * (size_t)p.TP + row;
    const size_t slot_stride = (size_t)p.NC * kChunk;
    const uint64_t* slots_in = p.slots + ((size_t)b * p.NW + (g > 0 ? g - 1 : 0)) * slot_stride;
    uint64_t* slots_out = p.slots + ((size_t)b * p.NW + g) * slot_stride;
    const bool publish = g < g_last;
    const int rsw = swz(lane);

    float q = neg_inf();
    float score = neg_inf();
    float4 stg0[8], stg1[8];
    TileLoader<ALIGNED>::load(stg0, vb, p.S, row0, tx, ty, c_begin, lane);
    if (c_begin + 1 < c_end) TileLoader<ALIGNED>::load(stg1, vb, p.S, row0, tx, ty, c_begin + 1, lane);

    // Boundary words of the chunk being processed; polled one chunk ahead.
    uint64_t bw = 0;
    auto poll_issue = [&](int c) {
      if (g > 0 && lane < kChunk) bw = __hip_atomic_load(slots_in + (size_t)c * kChunk - 1 + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    auto poll_wait = [&](int c) {
      if (g == 0) return;
      int spins = 0;
      while (true) {
        const bool ready = lane >= kChunk || (uint32_t)(bw >> 32) == tag;
        if (__builtin_amdgcn_ballot_w64(!ready) == 0) break;
        if (++spins > kSpinLimit) {
          timed_out = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
        poll_issue(c);
      }
    };
    poll_issue(c_begin);

    auto step = [&](int c, float4 (&stg)[8]) {
      // Stage the value tile and read this lane's row back.
#pragma unroll
      for (int k = 0; k < 8; ++k) tile[wv][64 * k + lane] = stg[k];
      wave_lds_sync();
      float v[kChunk];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float4 x = tile[wv][8 * lane + (k ^ rsw)];
        v[4 * k + 0] = x.x;
        v[4 * k + 1] = x.y;
        v[4 * k + 2] = x.z;
        v[4 * k + 3] = x.w;
      }
      // Boundary column values Q[row0-1][j0-1 .. j0+30].
      float bd[kChunk];
      if (g == 0) {
#pragma unroll
        for (int m = 0; m < kChunk; ++m) bd[m] = neg_inf();
      } else {
        poll_wait(c);
        if (lane < kChunk) reinterpret_cast<float*>(bnd_lds[wv])[lane] = __uint_as_float((uint32_t)bw);
        wave_lds_sync();
#pragma unroll
        for (int k = 0; k < kChunk / 4; ++k) {
          const float4 x = bnd_lds[wv][k];
          bd[4 * k + 0] = x.x;
          bd[4 * k + 1] = x.y;
          bd[4 * k + 2] = x.z;
          bd[4 * k + 3] = x.w;
        }
        if (c + 1 < c_end) poll_issue(c + 1);
      }
      wave_lds_sync();
      float qc[kChunk];
      uint32_t bits;
      if (c < c_begin + 2)
        sweep_chunk<true>(q, v, bd, qc, bits, row, c * kChunk);
      else
        sweep_chunk<false>(q, v, bd, qc, bits, row, c * kChunk);
      decp[(size_t)c * p.TP] = bits;
      if (publish) {
        if (lane == kWave - 1) {
#pragma unroll
          for (int k = 0; k < kChunk / 4; ++k) bout_lds[wv][k] = make_float4(qc[4 * k], qc[4 * k + 1], qc[4 * k + 2], qc[4 * k + 3]);
        }
        wave_lds_sync();
        if (lane < kChunk) {
          const float val = reinterpret_cast<const float*>(bout_lds[wv])[lane];
          const uint64_t word = ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(val);
          __hip_atomic_store(slots_out + (size_t)c * kChunk + lane, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      if (g == g_last && c == c_end - 1) {
        const int m_last = (ty - 1) % kChunk;
#pragma unroll
        for (int m = 0; m < kChunk; ++m) score = (m == m_last) ? qc[m] : score;
      }
    };

    for (int c = c_begin; c < c_end; c += 2) {
      step(c, stg0);
      if (c + 2 < c_end) TileLoader<ALIGNED>::load(stg0, vb, p.S, row0, tx, ty, c + 2, lane);
      if (c + 1 < c_end) {
        step(c + 1, stg1);
        if (c + 3 < c_end) TileLoader<ALIGNED>::load(stg1, vb, p.S, row0, tx, ty, c + 3, lane);
      }
    }

    // Publish completion of this wave's decision words to the item's walker.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    if (lane == 0) __hip_atomic_store(p.done + (size_t)b * p.NW + g, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

    if (g == g_last) {
      if (lane == ((tx - 1) & (kWave - 1)) && p.score) p.score[b] = score;
      // Wait until every other wave of the item has stored its words.
      for (int k0 = 0; k0 < g_last; k0 += kWave) {
        const int k = k0 + lane;
        int spins = 0;
        while (true) {
          const bool ready = k >= g_last ||
                             __hip_atomic_load(p.done + (size_t)b * p.NW + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == tag;
          if (__builtin_amdgcn_ballot_w64(!ready) == 0) break;
          if (++spins > kSpinLimit) {
            timed_out = true;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");

      for (int i = tx + lane; i <= p.T; i += kWave) rs[i] = ty;

      // Backtrack over the decision words.
      const uint32_t* db = p.dec + (size_t)b * p.NC * (size_t)p.TP;
      auto window = [&](int c, int base) -> uint32_t {
        const int r = base - lane;
        return r >= 0 ? db[(size_t)c * p.TP + r] : 0u;
      };
      int idx = tx - 1;
      int j = ty - 1;
      int c = j / kChunk;
      int wb = idx;                 // window base of chunk c
      uint32_t W = window(c, wb);
      int wnb = idx;                // window base of chunk c-1
      uint32_t Wn = c > 0 ? window(c - 1, wnb) : 0u;
      int32_t acc = 0;              // row_start values of rows [idx & ~63, +64)
      // With valid decision words the walk stays inside each window and
      // reaches row 0 at a chunk c >= 0; the guards only keep a corrupted
      // workspace (after a timed-out wait) from reading out of bounds.
      while (idx > 0 && c >= 0) {
        const uint32_t w = __builtin_amdgcn_readlane(W, (wb - idx) & (kWave - 1));
        const int m = j - c * kChunk;
        const uint32_t masked = w & (0xFFFFFFFFu << (31 - m));
        bool next_chunk;
        if (masked) {
          const int jj = c * kChunk + 31 - __builtin_ctz(masked);
          acc = lane == (idx & (kWave - 1)) ? jj : acc;
          if ((idx & (kWave - 1)) == 0 && idx + lane < tx) rs[idx + lane] = acc;
          idx -= 1;
          j = jj - 1;
          next_chunk = j < c * kChunk;
        } else {
          j = c * kChunk - 1;
          next_chunk = true;
        }
        if (next_chunk && idx > 0) {
          c -= 1;
          W = Wn;
          wb = wnb;
          wnb = idx;
          if (c > 0) Wn = window(c - 1, wnb);
        }
      }
      // Row 0 starts at column 0; flush the partial group of rows [0, 64).
      acc = lane == 0 ? 0 : acc;
      if (lane < tx) rs[lane] = acc;
    }
  }

  if (timed_out) {
    if (p.status) p.status[b] = kItemSyncTimeout;
    __hip_atomic_store(&p.hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // The last wave of the call to finish advances the generation.
  if (lane == 0) {
    const uint32_t total = gridDim.x * kWavesPerBlock;
    const uint32_t prev = __hip_atomic_fetch_add(&p.hdr->exit_count, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == total - 1) {
      __hip_atomic_store(&p.hdr->exit_count, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&p.hdr->gen, gen + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// ---------------------------------------------------------------- path writer
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
hipError_t launch_search(const SearchParams& p, bool aligned, hipStream_t stream) {
  const int nb = (p.T + kRowsPerBlock - 1) / kRowsPerBlock;
  const dim3 grid((unsigned)(p.B * nb)), block(kRowsPerBlock);
  if (aligned)
    hipLaunchKernelGGL(mas_search_kernel<true>, grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL(mas_search_kernel<false>, grid, block, 0, stream, p);
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
