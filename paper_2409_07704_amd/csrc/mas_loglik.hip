// Gaussian log-likelihood producer: the MAS input q[b][i][j] = log N(z_j;
// mu_i, sigma_i) (Sec. 2; diagonal covariance over D channels), computed for
// the cells MAS reads and nothing else.  Sec. 5 (Conclusion) names this
// calculation as the step to fuse with MAS.
//
// Arithmetic.  With r = exp(-2 log_sigma), every cell is a dot product plus
// a per-row constant:
//   q[i][j] = a_i + sum_k F[i][k] G[j][k],
//   a_i     = sum_d ( -ln(2 pi)/2 - log_sigma[i][d] - mu[i][d]^2 r[i][d] / 2 ),
//   F[i]    = [ mu[i][d] r[i][d] (d < D),  -r[i][d] / 2 (d < D) ],
//   G[j]    = [ z[j][d],                   z[j][d]^2          ],
// so the cells form a [T, 2D] x [2D, S] product: MFMA work.  Without
// log_sigma (sigma = 1) the z^2 part is a per-frame constant c_j =
// -sum_d z[j][d]^2 / 2 and the product shrinks to [T, D] x [D, S] with
// F[i] = mu[i], G[j] = z[j].  To keep fp32
// accuracy on fp16 matrix cores, every operand row is scaled by a power of 2
// to magnitudes in [2^13, 2^14) and split into fp16 hi + lo (x = hi + lo up to
// 2^-22 relative); the product takes hi*hi + hi*lo + lo*hi (three MFMAs per
// step, fp32 accumulation) and the scales come off exactly with ldexp.
//
// Work split.  Work units of 128 text rows of an item by up to 1024 speech
// columns, cut to the item's band, go to one persistent workgroup per CU by
// a static cost-balanced schedule that every workgroup computes from the
// lengths (no atomics in memory, no host round trip).  In a workgroup, eight
// MFMA waves of 16 text rows keep their rows' F as A-fragments in registers
// while four or eight builder waves stream the unit's speech frames in tiles
// of 32 columns, two tiles ahead, and build the B-fragments into LDS
// (double-buffered, one barrier per tile), each lane taking 8 channels of
// one frame straight from its own loads.  Only cells of the feasible band
// (i <= j, j - i <= t_y - t_x, inside the item's lengths) are written;
// waves whose 16 x 32 block holds none skip the MFMAs.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mas_internal.h"

namespace mas {
namespace {

constexpr int kLlWaves = 8;                       // MFMA waves: 16 text rows each
constexpr int kLlRows = kLlWaves * 16;            // text rows per work unit
constexpr int kLlCols = 32;                       // speech columns per tile
constexpr int kScaleExp = 14;                     // scaled operands lie in [2^13, 2^14)
constexpr int kMinExp = -113;                     // scale exponents stay in range of a normal float
constexpr int kXcds = 8;                          // MI355X: workgroups go to its 8 XCDs round-robin
constexpr int kUnitStartCost = 3;                 // a unit's start-up, in tiles, for the schedule
constexpr int kMaxWaves = 16;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int KS>
struct LlLds {
  // B-fragments of two tiles: [tile % 2][k-step][n-block][hi, lo][slot],
  // slot = gb_slot(lane, k-step) for the lane that reads it.
  half8 gb[2][KS][2][2][64];
  int col_e[2][kLlCols];  // exponent of the columns' scale, per tile buffer
  float col_c[2][kLlCols];  // unit variance: -|z_j|^2 / 2 of the columns, per tile buffer
  int64_t wsum[kMaxWaves];        // schedule: per-wave sums of a block reduction or scan
  long long first, last;          // schedule: this workgroup's first and last tile, unit << 32 | tile
};

// Where the fragment that lane `slot` of k-step ks reads is stored: the low
// three bits of the 16-byte slot are XORed with the lane's k-group and the
// k-step's parity, so that both the readers (eight consecutive lanes) and
// the writers (eight consecutive k-groups of one frame) touch eight
// different bank groups.
__device__ __forceinline__ int gb_slot(int slot, int ks) { return slot ^ (((slot >> 4) & 3) | ((ks & 1) << 2)); }

// Workgroup barrier that orders LDS only.  __syncthreads() also orders
// global memory, which would make every wave drain its outstanding global
// stores and loads at each barrier; the barriers here guard LDS buffers only.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ float wave_xor_max(float v, int mask) {
  return fmaxf(v, __shfl_xor(v, mask, 64));
}

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}

// Maximum over groups of N (2, 4, 8 or 16) consecutive lanes, every lane of a
// group getting it, with DPP moves inside 16-lane rows (no LDS round trips):
// swaps within pairs and quads, then rotations of the row by 4 and 8.
template <int N>
__device__ __forceinline__ float group_max(float v) {
  static_assert(N == 2 || N == 4 || N == 8 || N == 16, "group size");
  v = fmaxf(v, dpp_mov<0xB1>(v));                 // quad_perm [1, 0, 3, 2]
  if (N >= 4) v = fmaxf(v, dpp_mov<0x4E>(v));     // quad_perm [2, 3, 0, 1]
  if (N == 8) v = fmaxf(v, __shfl_xor(v, 4, 64));
  if (N == 16) {
    v = fmaxf(v, dpp_mov<0x124>(v));              // row_ror 4
    v = fmaxf(v, dpp_mov<0x128>(v));              // row_ror 8
  }
  return v;
}

// Sum over groups of N consecutive lanes (as group_max).
template <int N>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(N == 2 || N == 4 || N == 8 || N == 16, "group size");
  v += dpp_mov<0xB1>(v);
  if (N >= 4) v += dpp_mov<0x4E>(v);
  if (N == 8) v += __shfl_xor(v, 4, 64);
  if (N == 16) {
    v += dpp_mov<0x124>(v);
    v += dpp_mov<0x128>(v);
  }
  return v;
}

// hi + lo split of x * 2^(kScaleExp - e): hi is the scaled value rounded to
// fp16, lo the (exact) remainder rounded to fp16.  Pairs go through the
// packed conversion.
__device__ __forceinline__ void split8(const float (&x)[8], int e, half8& hi, half8& lo) {
  const float sc = __builtin_bit_cast(float, (127 + kScaleExp - e) << 23);  // 2^(kScaleExp - e), a normal float
#pragma unroll
  for (int k = 0; k < 8; k += 2) {
    const float s0 = x[k] * sc, s1 = x[k + 1] * sc;
    const _Float16 h0 = (_Float16)s0, h1 = (_Float16)s1;
    hi[k] = h0;
    hi[k + 1] = h1;
    lo[k] = (_Float16)(s0 - (float)h0);
    lo[k + 1] = (_Float16)(s1 - (float)h1);
  }
}

// 8 consecutive floats from p (16-byte aligned when VEC, and in bounds);
// without VEC only the first `valid` are read (the others repeat p[0]).
// The caller masks the elements past `valid` where it uses them, so that a
// prefetch is not waited for at the load.
template <bool VEC>
__device__ __forceinline__ void load8(const float* p, int valid, float (&x)[8]) {
  if (VEC) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    const float4 w = *reinterpret_cast<const float4*>(p + 4);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
    x[4] = w.x; x[5] = w.y; x[6] = w.z; x[7] = w.w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = p[e < valid ? e : 0];
  }
}

__device__ __forceinline__ void mask8(int valid, float (&x)[8]) {
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = e < valid ? x[e] : 0.f;
}

// F for 8 channels of one row, k = k0 .. k0 + 7 (the mu r part below Dp,
// the -r / 2 part from Dp), and that row's share of a_i.  r = exp(-2 ls) is
// formed as 2^(ls * (-2 / ln 2)) with the hardware exp2 (about 1 ulp, plus
// the rounding of the product, relative |ls| 2^-23).
template <bool VEC, bool UNIT>
__device__ __forceinline__ void f_group(const float* mu_row, const float* ls_row, int k0, int D, int Dp, bool row_ok,
                                        float (&f)[8], float& asum) {
  const bool zpart = k0 < Dp;
  const int d0 = zpart ? k0 : k0 - Dp;
  const int valid = row_ok && (UNIT ? zpart : k0 < 2 * Dp) && d0 < D ? min(8, D - d0) : 0;
  float mv[8], lv[8];
  load8<VEC>(mu_row + (valid ? d0 : 0), zpart ? valid : 0, mv);
  mask8(zpart ? valid : 0, mv);
  if (ls_row) {
    load8<VEC>(ls_row + (valid ? d0 : 0), valid, lv);
    mask8(valid, lv);
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) lv[e] = 0.f;
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float r = ls_row ? __builtin_amdgcn_exp2f(lv[e] * -2.88539008177792681f) : 1.f;
    f[e] = 0.f;
    if (e < valid) {
      if (zpart) {
        f[e] = mv[e] * r;
        asum += -0.918938533204672742f - lv[e] - 0.5f * (mv[e] * mv[e]) * r;
      } else {
        f[e] = -0.5f * r;
      }
    }
  }
}

// One work unit: rows [i0, i0 + 128) of item b, over the speech columns of
// their feasible band from jlo (a multiple of 32) in tiles of 32.
// ntiles = 0: nothing to do.
struct LlUnit {
  int i0, ilast, slack, ty, jlo, ntiles;
};

__device__ __forceinline__ LlUnit ll_unit(int rb, int tx, int ty, int T, int S) {
  LlUnit u;
  u.i0 = rb * kLlRows;
  u.ty = ty;
  u.ntiles = 0;
  if (!(tx >= 1 && tx <= ty && tx <= T && ty <= S) || u.i0 >= tx) return u;
  u.ilast = min(u.i0 + kLlRows, tx) - 1;
  u.slack = ty - tx;
  u.jlo = u.i0 & ~(kLlCols - 1);
  const int jhi = min(ty, u.ilast + u.slack + 1);
  u.ntiles = (jhi - u.jlo + kLlCols - 1) / kLlCols;
  return u;
}

// Schedule cost of a unit (its tiles plus a start-up charge) and of an item.
__device__ __forceinline__ int64_t ll_cost(const LlUnit& u) { return u.ntiles ? u.ntiles + kUnitStartCost : 0; }
__device__ __forceinline__ int64_t ll_item_cost(int tx, int ty, int T, int S, int nrb) {
  int64_t c = 0;
  for (int rb = 0; rb < nrb; ++rb) {
    const LlUnit u = ll_unit(rb, tx, ty, T, S);
    if (!u.ntiles) break;
    c += ll_cost(u);
  }
  return c;
}

// Block-wide inclusive scan of one int64 per thread (all threads call it).
template <int kWaves, class Lds>
__device__ __forceinline__ int64_t block_scan(int64_t x, Lds& L, int64_t* total) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) L.wsum[wave] = x;
  __syncthreads();
  int64_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int64_t t = L.wsum[w];
    before += w < wave ? t : 0;
    all += t;
  }
  __syncthreads();
  *total = all;
  return before + x;
}

// KS = k-steps of 32 (the padded 2 * Dp channels); VEC: D % 8 == 0 and mu,
// log_sigma and z 16-byte aligned (16-byte loads of 8 channels); NB =
// builder waves (8 while the MFMA waves fit in 128 VGPRs, else 4).
//
// Persistent workgroups with a static schedule: every workgroup reads the
// lengths, prices each work unit (item, row block, column piece) by its tile
// count plus a start-up charge, and takes the units whose running cost
// starts in its share [v C / G, (v + 1) C / G) of the total C.  The shares
// of XCD x are its eighth of the batch in order, so each XCD's L2 holds few
// items' frames.  Waves 0-7 hold A-fragments, run the MFMAs and store;
// waves 8.. load the frames and build the B-fragments.  Each kind of wave
// issues only one kind of global memory operation (stores, or loads), so
// no wave ever waits on the other kind.
template <int KS, bool VEC, int NB, bool UNIT>
__global__ void __launch_bounds__((kLlWaves + NB) * 64)
    mas_loglik_kernel(const float* __restrict__ mu, const float* __restrict__ log_sigma, const float* __restrict__ z,
                      const int32_t* __restrict__ t_x, const int32_t* __restrict__ t_y, float* __restrict__ value,
                      int32_t B, int32_t T, int32_t S, int32_t D, int32_t Dp, int32_t nrb) {
  __shared__ LlLds<KS> L;
  constexpr int kThreads = (kLlWaves + NB) * 64;
  constexpr int FPW = kLlCols / NB;              // frames per builder wave
  constexpr int LPF = 64 / FPW;                  // lanes per frame
  constexpr int P = ((UNIT ? 4 : 2) * KS + LPF - 1) / LPF;  // z channel groups per lane: Dp / 8 <= LPF P
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

  // ---- Schedule (identical in every workgroup).  Units (item, row block)
  // in order; a unit's cost positions are its start-up charge, then one per
  // tile.  This workgroup takes the tiles whose positions fall in its share
  // [v C / G, (v + 1) C / G) of the total cost C.
  const int G = gridDim.x;
  const int v = (blockIdx.x % kXcds) * (G / kXcds) + blockIdx.x / kXcds;  // XCD x: shares [x G/8, (x+1) G/8)
  if (threadIdx.x == 0) {
    L.first = 0x7fffffffffffffffLL;
    L.last = -1;
  }
  // Zero every B-fragment once: the padding channels stay zero.
  {
    uint4* g = reinterpret_cast<uint4*>(&L.gb[0][0][0][0][0]);
    constexpr int n16 = (int)(sizeof(L.gb) / 16);
    for (int k = threadIdx.x; k < n16; k += kThreads) g[k] = make_uint4(0u, 0u, 0u, 0u);
  }
  // Items in chunks of one per thread: an inclusive scan of their costs
  // gives each item's first position.  With more items than threads, a
  // first pass finds the total.
  int64_t total = 0;
  if (B > kThreads) {
    int64_t mine = 0;
    for (int b = threadIdx.x; b < B; b += kThreads) mine += ll_item_cost(t_x[b], t_y[b], T, S, nrb);
    block_scan<kLlWaves + NB>(mine, L, &total);
  }
  int64_t run = 0;  // cost before the current chunk of items
  for (int c0 = 0; c0 < B; c0 += kThreads) {
    const int b = c0 + threadIdx.x;
    const int tx = b < B ? t_x[b] : 0, ty = b < B ? t_y[b] : 0;
    const int64_t mine = b < B ? ll_item_cost(tx, ty, T, S, nrb) : 0;
    int64_t chunk = 0;
    int64_t at = run + block_scan<kLlWaves + NB>(mine, L, &chunk) - mine;  // this item's first position
    if (B <= kThreads) total = chunk;
    const int64_t lo = total * v / G, hi = total * (v + 1) / G;
    if (mine > 0 && at < hi && at + mine > lo) {
      for (int rb = 0; rb < nrb; ++rb) {
        const LlUnit u = ll_unit(rb, tx, ty, T, S);
        if (!u.ntiles) break;
        const int64_t t0 = at + kUnitStartCost;  // position of tile 0
        const int64_t ta = max(lo - t0, (int64_t)0), tb = min(hi - t0, (int64_t)u.ntiles);
        if (ta < tb) {
          const long long key = (long long)(b * nrb + rb) << 32;
          atomicMin(&L.first, key | ta);
          atomicMax(&L.last, key | (tb - 1));
        }
        at += ll_cost(u);
      }
    }
    run += chunk;
  }
  __syncthreads();
  const long long s_first = L.first, s_last = L.last;
  const int u_first = (int)(s_first >> 32), u_last = (int)(s_last >> 32);
  const int t_first = (int)(s_first & 0xffffffff), t_last = (int)(s_last & 0xffffffff);

  if (wave >= kLlWaves) {
    // ---------------------------------------------------------- builders
    // Lane (n, g0): frame n of a tile, channel groups g = g0 + LPF p.
    const int n = (wave - kLlWaves) * FPW + lane / LPF, g0 = lane % LPF;
    for (int u = u_first; u <= u_last; ++u) {
      const int b = u / nrb, rb = u % nrb;
      const LlUnit U = ll_unit(rb, t_x[b], t_y[b], T, S);
      // Tiles ta .. ta + ntiles - 1 of the unit are this workgroup's.
      const int ta = u == u_first ? t_first : 0;
      const int ntiles = (u == u_last ? t_last + 1 : U.ntiles) - ta;
      if (ntiles <= 0) continue;
      // Frame loads.  Frames past the unit's tiles or the tensor re-read
      // the item's first frame, and channels past D (only without VEC)
      // repeat the group's first one: such values only ever meet zero rows
      // of F or land in columns that are never stored, so they need no
      // masking (inputs are finite).
      const float* zitem = z + (size_t)b * S * D;
      const int jfirst = U.jlo + ta * kLlCols + n;
      auto load_tile = [&](int t, float (&zr)[P][8]) {
        const int j = jfirst + t * kLlCols;
        const float* src = zitem + (size_t)(t < ntiles && j < S ? j : 0) * D;
#pragma unroll
        for (int p = 0; p < P; ++p) {
          const int d0 = 8 * (g0 + LPF * p);
          const int valid = d0 < D ? min(8, D - d0) : 0;
          load8<VEC>(src + (valid ? d0 : 0), valid, zr[p]);
        }
      };
      // Channel group g of frame n is k-group g of the z part and Dp / 8 + g
      // of the z^2 part; the frame's scale comes from max |z| (max z^2 is
      // its square).
      auto build_tile = [&](int buf, const float (&zr)[P][8]) {
        float m = 0.f, ss = 0.f;
#pragma unroll
        for (int p = 0; p < P; ++p)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            m = fmaxf(m, fabsf(zr[p][e]));
            if (UNIT && 8 * (g0 + LPF * p) + e < D) ss += zr[p][e] * zr[p][e];
          }
        m = group_max<LPF>(m);
        const int ec = max(__builtin_amdgcn_frexp_expf(UNIT ? m : fmaxf(m, m * m)), kMinExp);
        const int nb = n >> 4;
#pragma unroll
        for (int p = 0; p < P; ++p) {
          const int g = g0 + LPF * p;
          if (8 * g < Dp) {
            half8 hi, lo;
            split8(zr[p], ec, hi, lo);
            int kg = g;
            int slot = gb_slot((n & 15) + 16 * (kg & 3), kg >> 2);
            L.gb[buf][kg >> 2][nb][0][slot] = hi;
            L.gb[buf][kg >> 2][nb][1][slot] = lo;
            if (!UNIT) {
              float sq[8];
#pragma unroll
              for (int e = 0; e < 8; ++e) sq[e] = zr[p][e] * zr[p][e];
              split8(sq, ec, hi, lo);
              kg = Dp / 8 + g;
              slot = gb_slot((n & 15) + 16 * (kg & 3), kg >> 2);
              L.gb[buf][kg >> 2][nb][0][slot] = hi;
              L.gb[buf][kg >> 2][nb][1][slot] = lo;
            }
          }
        }
        if (UNIT) ss = group_sum<LPF>(ss);
        if (g0 == 0) {
          L.col_e[buf][n] = ec;
          if (UNIT) L.col_c[buf][n] = -0.5f * ss;
        }
      };
      // Frames of the next kDepth tiles in registers: at MFMA step m the
      // builders turn tile m + 1 (register set (m + 1) % kDepth) into
      // B-fragments and refill that set with tile m + 1 + kDepth.  Full
      // rounds of kDepth steps issue their loads on every path (past the
      // last tile they re-read the item's first frame), so the compiler's
      // wait before each build counts exactly the newer loads; the last
      // partial round issues none.
      constexpr int kDepth = 4;
      float zr[kDepth][P][8];
#pragma unroll
      for (int k = 0; k < kDepth; ++k) load_tile(k, zr[k]);
      build_tile(0, zr[0]);
      load_tile(kDepth, zr[0]);
      lds_barrier();
      int m0 = 0;
      for (; m0 + kDepth <= ntiles; m0 += kDepth) {
#pragma unroll
        for (int j = 0; j < kDepth; ++j) {
          const int m = m0 + j;
          if (m + 1 < ntiles) build_tile((m + 1) & 1, zr[(j + 1) % kDepth]);
          load_tile(m + 1 + kDepth, zr[(j + 1) % kDepth]);
          lds_barrier();
        }
      }
#pragma unroll
      for (int j = 0; j < kDepth; ++j) {
        const int m = m0 + j;
        if (m < ntiles) {
          if (m + 1 < ntiles) build_tile((m + 1) & 1, zr[(j + 1) % kDepth]);
          lds_barrier();
        }
      }
    }
    return;
  }

  // ------------------------------------------------------------ MFMA waves
  const int m = lane & 15, q = lane >> 4;
  for (int u = u_first; u <= u_last; ++u) {
    const int b = u / nrb, rb = u % nrb;
    const LlUnit U = ll_unit(rb, t_x[b], t_y[b], T, S);
    const int ta = u == u_first ? t_first : 0;
    const int ntiles = (u == u_last ? t_last + 1 : U.ntiles) - ta;
    if (ntiles <= 0) continue;
    const int r0 = U.i0 + wave * 16;
    const int ilast = U.ilast, slack = U.slack, ty = U.ty;
    half8 ahi[KS], alo[KS];
    float ra[4];
    int re[4];
    {
      // A-fragments of this wave's 16 rows: lane (m, q) holds row m and
      // channels k = 32 ks + 8 q + e of F.  Small contractions keep F in
      // registers between the row maximum and the split; large ones read mu
      // and log_sigma a second time (from cache) instead.
      const int i = r0 + m;
      const bool row_ok = i <= ilast;
      const size_t roff = ((size_t)b * T + (row_ok ? i : 0)) * D;
      const float* mu_row = mu + roff;
      const float* ls_row = log_sigma ? log_sigma + roff : nullptr;
      constexpr bool kKeep = KS <= 8;
      float fv[kKeep ? KS : 1][8];
      float amax = 0.f, asum = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        float f[8];
        f_group<VEC, UNIT>(mu_row, ls_row, 32 * ks + 8 * q, D, Dp, row_ok, f, asum);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          amax = fmaxf(amax, fabsf(f[e]));
          if constexpr (kKeep) fv[ks][e] = f[e];
        }
      }
      amax = wave_xor_max(wave_xor_max(amax, 16), 32);
      asum += __shfl_xor(asum, 16, 64);
      asum += __shfl_xor(asum, 32, 64);
      const int er = max(__builtin_amdgcn_frexp_expf(amax), kMinExp);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if constexpr (kKeep) {
          split8(fv[ks], er, ahi[ks], alo[ks]);
        } else {
          float f[8], unused = 0.f;
          f_group<VEC, UNIT>(mu_row, ls_row, 32 * ks + 8 * q, D, Dp, row_ok, f, unused);
          split8(f, er, ahi[ks], alo[ks]);
        }
      }
      // Row constants of the four rows this lane's results fall in (rows
      // 4 q + r, held by lane 4 q + r).
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        ra[r] = __shfl(asum, 4 * q + r, 64);
        re[r] = __shfl(er, 4 * q + r, 64);
      }
    }
    // The item's slab of value as a buffer: lanes with nothing to write
    // store to offset -1, which the buffer bounds check drops.
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(value + (size_t)b * T * S, 0,
                                                                        (int)((size_t)T * S * 4), 0x00020000);
    const int ilo_w = r0, ihi_w = min(r0 + 15, ilast);
    // Per result row: its index (rows past the item's last get one no
    // column can be within `slack` of) and its byte offset in the slab.
    int rr[4], roffb[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ii = r0 + 4 * q + r;
      rr[r] = ii <= ilast ? ii : (1 << 30);
      roffb[r] = ii <= ilast ? ii * S * 4 : 0;
    }
    lds_barrier();  // tile 0 is built
    for (int t = 0; t < ntiles; ++t) {
      const int buf = t & 1;
      const int c = U.jlo + (ta + t) * kLlCols;
      // Does this wave's 16 x 32 block hold a band cell?
      if (ilo_w <= ihi_w && c + kLlCols - 1 >= ilo_w && c <= ihi_w + slack && c < ty) {
        f32x4 h0 = {0.f, 0.f, 0.f, 0.f}, h1 = h0, x0 = h0, x1 = h0;
        // B-fragments read ahead of their MFMAs (two k-steps with eight
        // builder waves' register budget to spare, else one); the
        // scheduling barriers keep the compiler from sinking each read onto
        // its use.
        constexpr int kAhead = NB == 8 ? 1 : 2;
        half8 bf[kAhead + 1][4];
        auto read_b = [&](int ks, half8 (&o)[4]) {
          const int sl = gb_slot(lane, ks);
          o[0] = L.gb[buf][ks][0][0][sl];
          o[1] = L.gb[buf][ks][1][0][sl];
          o[2] = L.gb[buf][ks][0][1][sl];
          o[3] = L.gb[buf][ks][1][1][sl];
        };
#pragma unroll
        for (int a = 0; a < kAhead; ++a)
          if (a < KS) read_b(a, bf[a]);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          if (ks + kAhead < KS) read_b(ks + kAhead, bf[(ks + kAhead) % (kAhead + 1)]);
          __builtin_amdgcn_sched_barrier(0);
          const half8(&cb)[4] = bf[ks % (kAhead + 1)];
          x0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(alo[ks], cb[0], x0, 0, 0, 0);
          x1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(alo[ks], cb[1], x1, 0, 0, 0);
          h0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ahi[ks], cb[0], h0, 0, 0, 0);
          h1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ahi[ks], cb[1], h1, 0, 0, 0);
          x0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ahi[ks], cb[2], x0, 0, 0, 0);
          x1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ahi[ks], cb[3], x1, 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        }
        // Lane l holds column l % 16 of each n-block, rows 4 (l / 16) + r.
        // A cell is in the band when 0 <= j - i <= slack and j < t_y; a
        // block wholly inside the band stores without per-cell checks.
        const int j0 = c + (lane & 15), j1 = j0 + 16;
        const int ce0 = L.col_e[buf][lane & 15] - 2 * kScaleExp, ce1 = L.col_e[buf][16 + (lane & 15)] - 2 * kScaleExp;
        const float cc0 = UNIT ? L.col_c[buf][lane & 15] : 0.f, cc1 = UNIT ? L.col_c[buf][16 + (lane & 15)] : 0.f;
        const bool inside = r0 + 15 <= ilast && c >= r0 + 15 && c + kLlCols - 1 - r0 <= slack && c + kLlCols <= ty;
        if (inside) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v0 = (ra[r] + cc0) + ldexpf(h0[r] + x0[r], re[r] + ce0);
            const float v1 = (ra[r] + cc1) + ldexpf(h1[r] + x1[r], re[r] + ce1);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v0), vr, roffb[r] + j0 * 4, 0, 0);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v1), vr, roffb[r] + j1 * 4, 0, 0);
          }
        } else {
          const bool c0 = j0 < ty, c1 = j1 < ty;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v0 = (ra[r] + cc0) + ldexpf(h0[r] + x0[r], re[r] + ce0);
            const float v1 = (ra[r] + cc1) + ldexpf(h1[r] + x1[r], re[r] + ce1);
            const bool in0 = c0 && (unsigned)(j0 - rr[r]) <= (unsigned)slack;
            const bool in1 = c1 && (unsigned)(j1 - rr[r]) <= (unsigned)slack;
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v0), vr, in0 ? roffb[r] + j0 * 4 : -1, 0, 0);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v1), vr, in1 ? roffb[r] + j1 * 4 : -1, 0, 0);
          }
        }
      }
      lds_barrier();  // tile t + 1 is built; buffer t % 2 may be rebuilt
    }
  }
}

template <int KS, bool UNIT>
hipError_t launch_ll_ks(const float* mu, const float* log_sigma, const float* z, const int32_t* t_x,
                        const int32_t* t_y, float* value, int32_t B, int32_t T, int32_t S, int32_t D, int32_t Dp,
                        bool vec, int grid, hipStream_t stream) {
  const int32_t nrb = (T + kLlRows - 1) / kLlRows;
  constexpr int NB = KS <= 5 ? 8 : 4;
  constexpr int kThreads = (kLlWaves + NB) * 64;
  if (vec)
    hipLaunchKernelGGL((mas_loglik_kernel<KS, true, NB, UNIT>), dim3(grid), dim3(kThreads), 0, stream, mu, log_sigma, z,
                       t_x, t_y, value, B, T, S, D, Dp, nrb);
  else
    hipLaunchKernelGGL((mas_loglik_kernel<KS, false, NB, UNIT>), dim3(grid), dim3(kThreads), 0, stream, mu, log_sigma, z,
                       t_x, t_y, value, B, T, S, D, Dp, nrb);
  return hipGetLastError();
}

template <int KS>
hipError_t dispatch_ll(int ks, const float* mu, const float* log_sigma, const float* z, const int32_t* t_x,
                       const int32_t* t_y, float* value, int32_t B, int32_t T, int32_t S, int32_t D, int32_t Dp,
                       bool vec, int grid, hipStream_t stream) {
  if (ks == KS)
    return log_sigma ? launch_ll_ks<KS, false>(mu, log_sigma, z, t_x, t_y, value, B, T, S, D, Dp, vec, grid, stream)
                     : launch_ll_ks<KS, true>(mu, log_sigma, z, t_x, t_y, value, B, T, S, D, Dp, vec, grid, stream);
  if constexpr (KS > 1)
    return dispatch_ll<KS - 1>(ks, mu, log_sigma, z, t_x, t_y, value, B, T, S, D, Dp, vec, grid, stream);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_loglik(const float* mu, const float* log_sigma, const float* z, const int32_t* t_x,
                         const int32_t* t_y, float* value, int32_t B, int32_t T, int32_t S, int32_t D,
                         hipStream_t stream) {
  const int32_t Dp = (D + 7) & ~7;
  const int ks = ((log_sigma ? 2 : 1) * Dp + 31) / 32;
  const bool vec = D % 8 == 0 && ((uintptr_t)z | (uintptr_t)mu | (uintptr_t)log_sigma) % 16 == 0;
  // One persistent workgroup per CU, in whole rounds of the eight XCDs.
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int grid = max(kXcds, (cus + kXcds - 1) / kXcds * kXcds);
  return dispatch_ll<kLoglikMaxKs>(ks, mu, log_sigma, z, t_x, t_y, value, B, T, S, D, Dp, vec, grid, stream);
}

}  // namespace mas
