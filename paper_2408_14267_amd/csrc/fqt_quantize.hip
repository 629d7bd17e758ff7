// AGP + SCQ quantization of the output gradient dY on gfx950.
//
//   k_stats         one pass over dY in 64 (channel) x 64 (unfolded row r = n*P + pixel)
//                   tiles: per-tile min/max of every channel row and every r column,
//                   written as partials (no atomics: same-address atomics from the
//                   eight XCDs serialise at the memory side)
//   k_select_fused  (N, D <= 1024) one workgroup per group set: min/max of each group's
//                   partials (Section 3.2 range and zero point; Section 5.2 / 5.3
//                   groups), then AGP keep probabilities, Bernoulli masks, kept-id
//                   compaction, scale/offset (Section 5.2, AGP)
//   k_stats_reduce  (larger sets) one workgroup per group: min/max of its partials,
//   k_select        then one workgroup per group set for the AGP steps
//   k_qpack         second pass over dY: stochastic rounding of every element of a
//                   kept sample / kept channel, bit-plane split and packing, and the
//                   byte codes the MFMA products read
//                   (Section 3.2 SR; Section 5.2 decomposition; Appendix C encoders)
//
// A tile holds whole 64-bit words of both packings: a PSQ word runs along the 64
// channels of one row r, a PCQ word along the 64 rows of one channel.
#include <climits>
#include <type_traits>

#include "fqt_internal.hpp"
#include "fqt_signs.hpp"

namespace fqt {
namespace {

constexpr int TILE = 64;
constexpr int THREADS = 512;                 // tile kernels: 8 elements (2 quads) per thread
constexpr int WAVES = THREADS / 64;
constexpr int QUADS = TILE * TILE / (4 * THREADS);
static_assert(TILE / WAVES == 8, "qpack: a wave stores 8 lines, 8 lanes per line");
constexpr int PITCH = TILE + 4;   // bytes per LDS code row; 68 keeps transposed reads conflict-free

// How a thread walks its 8 tile elements (2 quads of 4).
//  PIX    (P % 4 == 0): a quad is 4 consecutive rows r of one channel (one 16-byte load)
//  CHAN   (P == 1, D % 4 == 0): a quad is 4 consecutive channels of one row
//  SCALAR otherwise: single elements
enum TileMode { TILE_PIX = 0, TILE_CHAN = 1, TILE_SCALAR = 2 };

struct TileGeom {
  uint32_t D, P, R;
  FastDiv divP;
};

template <int MODE>
__device__ __forceinline__ void quad_coord(int t, int q, int k, int &dd, int &rr) {
  if (MODE == TILE_PIX) {
    dd = (t >> 4) + (THREADS / 16) * q;
    rr = 4 * (t & 15) + k;
  } else if (MODE == TILE_CHAN) {
    dd = 4 * (t & 15) + k;
    rr = (t >> 4) + (THREADS / 16) * q;
  } else {
    const int idx = t + THREADS * (4 * q + k);
    dd = idx >> 6;
    rr = idx & 63;
  }
}

// NCHW index of (channel d, unfolded row r); every index is below 2^31.
__device__ __forceinline__ uint32_t elem_index(const TileGeom &g, uint32_t d, uint32_t r) {
  const uint32_t n = fdiv(r, g.divP);
  return (n * g.D + d) * g.P + (r - n * g.P);
}

__device__ __forceinline__ int wave_min(int v) { return wave_min_all(v); }
__device__ __forceinline__ int wave_max(int v) { return wave_max_all(v); }

// ----------------------------------------------------------------------------- stats

// Partial layouts.  Channel partials: part_c[rb][d] for row blocks rb of rs * 64 rows
// (rs = stats_rows_per_block: enough blocks to cover the chip, few partials).  Sample partials: part_s[(dt * nrt + rt) * SL + k] for the 64-row tile rt and
// 64-channel tile dt, slot k holding sample n_first(rt) + k, n_first(rt) = rt * 64 / P, and
// SL = min(64, ceil(63 / P) + 1) slots (a 64-row tile meets at most that many samples).
// With P = 1 (a sample per row) they are part_s[r * ndt + dt] instead, so that the partials
// of one sample are contiguous for the reduction.
struct StatsGeom {
  TileGeom g;
  uint32_t nrt, SL, rs;
  uint32_t chan_fast;   // grid x walks the channel tiles, y the row blocks
  uint32_t ndt;         // channel tiles
};

// Load the quads of tile rows [r0, r0 + 64) x channels [d0, d0 + 64) into x (element 0 of
// dY outside the layer, so the loads issue back to back).
template <int MODE, int DT>
__device__ __forceinline__ void stats_load(const void *dy, const TileGeom &g, uint32_t r0,
                                           uint32_t d0, int t, float (&x)[QUADS][4],
                                           bool (&ok)[QUADS]) {
  for (int q = 0; q < QUADS; ++q) {
    int dd, rr;
    quad_coord<MODE>(t, q, 0, dd, rr);
    ok[q] = d0 + dd < g.D && r0 + rr < g.R;      // quads are all-valid or all-invalid
    load_quad<DT>(dy, ok[q] ? elem_index(g, d0 + dd, r0 + rr) : 0, x[q]);
  }
}

// Merged key encoding: max key as its unsigned order (k ^ 2^31), min key as the complement
// of that, so that both combine with an unsigned atomic max and 0 is the identity of both.
__device__ __forceinline__ void merge_key(uint2 *mk, int lo, int hi) {
  uint32_t *p = reinterpret_cast<uint32_t *>(mk);
  __hip_atomic_fetch_max(p, ~(uint32_t(lo) ^ 0x80000000u), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_fetch_max(p + 1, uint32_t(hi) ^ 0x80000000u, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int2 merged_key(uint2 u) {
  return make_int2(int(~u.x ^ 0x80000000u), int(u.y ^ 0x80000000u));
}

// One block per (rs row tiles, 64 channels).  Each 64 x 64 tile goes through LDS as
// order-preserving integer keys; channel rows are reduced over the rows (kept across the
// block's row tiles), row columns over the channels and then over the rows of each sample
// in the tile.
// With mks / mkc set (merged keys), the sample and channel keys are combined into them
// with atomics instead of being stored as partials: channel keys into replica
// (row block) % MKEY_REP, sample keys into replica (channel tile) % MKEY_REP.
template <int MODE, int DT>
__global__ __launch_bounds__(THREADS) void k_stats(const void *__restrict__ dy, StatsGeom sg,
                                                   int2 *__restrict__ part_c,
                                                   int2 *__restrict__ part_s,
                                                   uint2 *__restrict__ mks,
                                                   uint2 *__restrict__ mkc) {
  __shared__ int32_t key[TILE][TILE + 1];
  __shared__ int32_t pmin[WAVES][TILE], pmax[WAVES][TILE];
  const TileGeom &g = sg.g;
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const uint32_t bxr = sg.chan_fast ? blockIdx.y : blockIdx.x;   // row block
  const uint32_t byc = sg.chan_fast ? blockIdx.x : blockIdx.y;   // channel tile
  const uint32_t d0 = byc * TILE;
  const uint32_t rt0 = bxr * sg.rs;
  int clo = INT_MAX, chi = INT_MIN;             // channel d0 + lane over this wave's rows
  // Two register sets of row tiles: two tiles' loads are in flight behind each reduction.
  float xa[QUADS][4], xb[QUADS][4];
  bool oka[QUADS], okb[QUADS];
  if (MODE != TILE_SCALAR) {
    stats_load<MODE, DT>(dy, g, rt0 * TILE, d0, t, xa, oka);
    if (sg.rs > 1 && rt0 + 1 < sg.nrt) stats_load<MODE, DT>(dy, g, (rt0 + 1) * TILE, d0, t, xb, okb);
  }
  auto tile = [&](uint32_t s, float (&x)[QUADS][4], bool (&ok)[QUADS]) -> bool {
    const uint32_t rt = rt0 + s;
    if (rt >= sg.nrt) return false;
    const uint32_t r0 = rt * TILE;
    if (MODE != TILE_SCALAR) {
      for (int q = 0; q < QUADS; ++q) {
        if (!ok[q]) continue;
        for (int k = 0; k < 4; ++k) {
          int dk, rk;
          quad_coord<MODE>(t, q, k, dk, rk);
          key[dk][rk] = f2key(x[q][k] + 0.0f);
        }
      }
      // The row tile two ahead loads into these registers while this one is reduced.
      if (s + 2 < sg.rs && rt + 2 < sg.nrt)
        stats_load<MODE, DT>(dy, g, r0 + 2 * TILE, d0, t, x, ok);
    } else {
      for (int q = 0; q < 4 * QUADS; ++q) {
        int dd, rr;
        quad_coord<MODE>(t, q >> 2, q & 3, dd, rr);
        if (d0 + dd < g.D && r0 + rr < g.R)
          key[dd][rr] = f2key(load_elem<DT>(dy, elem_index(g, d0 + dd, r0 + rr)) + 0.0f);
      }
    }
    __syncthreads();

    const bool row_ok = r0 + lane < g.R;
    // Channels of the tile: lane d0 + lane reduces the wave's rows (read across the key
    // rows; the odd pitch keeps them on distinct banks), no cross-lane step.
#pragma unroll
    for (int i = 0; i < TILE / WAVES; ++i) {
      const int rr = (TILE / WAVES) * wave + i;
      if (r0 + rr >= g.R) break;
      const int k = key[lane][rr];
      clo = min(clo, k);
      chi = max(chi, k);
    }
    // Columns r of the tile: reduce over the tile's channels.
    int lo = INT_MAX, hi = INT_MIN;
    for (int i = 0; i < TILE / WAVES; ++i) {
      const int dd = (TILE / WAVES) * wave + i;
      if (d0 + dd >= g.D) break;
      const int k = key[dd][lane];
      lo = min(lo, k);
      hi = max(hi, k);
    }
    pmin[wave][lane] = lo;
    pmax[wave][lane] = hi;
    __syncthreads();
    if (wave == 0) {
      for (int v = 1; v < WAVES; ++v) {
        lo = min(lo, pmin[v][lane]);
        hi = max(hi, pmax[v][lane]);
      }
      // Rows of one sample are adjacent lanes: slot k of this tile reduces the rows of
      // sample n_first + k.
      const uint32_t n_first = fdiv(r0, g.divP);
      const uint32_t slot = row_ok ? fdiv(r0 + lane, g.divP) - n_first : 0xFFFFFFFFu;
      int2 *ps = part_s + (size_t(byc) * sg.nrt + rt) * sg.SL;
      if (g.P == 1) {
        // One sample per row: its partials are stored sample-major, [R][ndt].
        if (mks) {
          if (row_ok) merge_key(mks + (byc % MKEY_REP) * MKEY_GROUPS + r0 + lane, lo, hi);
        } else if (row_ok) {
          part_s[size_t(r0 + lane) * sg.ndt + byc] = make_int2(lo, hi);
        }
      } else if (mks && (TILE % g.P) == 0) {
        // P divides 64: every sample of the tile is an aligned group of P lanes.  A
        // butterfly within the groups leaves each group's key in all of its lanes, and the
        // first lane of each group merges it (one atomic instruction for all the samples).
        if (!row_ok) {
          lo = INT_MAX;
          hi = INT_MIN;
        }
        auto fold = [&](auto m) {
          constexpr int M = decltype(m)::value;
          lo = min(lo, int(lane_xor<M>(uint32_t(lo))));
          hi = max(hi, int(lane_xor<M>(uint32_t(hi))));
        };
        if (g.P > 1) fold(std::integral_constant<int, 1>());
        if (g.P > 2) fold(std::integral_constant<int, 2>());
        if (g.P > 4) fold(std::integral_constant<int, 4>());
        if (g.P > 8) fold(std::integral_constant<int, 8>());
        if (g.P > 16) fold(std::integral_constant<int, 16>());
        if (g.P > 32) fold(std::integral_constant<int, 32>());
        if (row_ok && (uint32_t(lane) & (g.P - 1)) == 0)
          merge_key(mks + (byc % MKEY_REP) * MKEY_GROUPS + n_first + uint32_t(lane) / g.P, lo,
                    hi);
      } else {
        for (uint32_t k = 0; k < sg.SL; ++k) {
          const int l = wave_min(slot == k ? lo : INT_MAX);
          const int h = wave_max(slot == k ? hi : INT_MIN);
          if (mks) {
            // A slot holds data only for a sample that the tile meets (then n < N).
            if (lane == 0 && l <= h)
              merge_key(mks + (byc % MKEY_REP) * MKEY_GROUPS + n_first + k, l, h);
          } else if (lane == 0) {
            ps[k] = make_int2(l, h);
          }
        }
      }
    }
    // (The next tile's key stores wait for every read of this one.)
    __syncthreads();
      return true;
  };
  for (uint32_t s = 0; s < sg.rs; s += 2) {
    if (!tile(s, xa, oka) || s + 1 >= sg.rs || !tile(s + 1, xb, okb)) break;
  }
  // Channel partials of this row block, [row block][D]: the waves' partials combined,
  // then one coalesced store.
  pmin[wave][lane] = clo;
  pmax[wave][lane] = chi;
  __syncthreads();
  if (wave == 1 && d0 + lane < g.D) {
    int lo = pmin[0][lane], hi = pmax[0][lane];
#pragma unroll
    for (int v = 1; v < WAVES; ++v) {
      lo = min(lo, pmin[v][lane]);
      hi = max(hi, pmax[v][lane]);
    }
    if (mkc) merge_key(mkc + (bxr % MKEY_REP) * MKEY_GROUPS + d0 + lane, lo, hi);
    else part_c[size_t(bxr) * g.D + d0 + lane] = make_int2(lo, hi);
  }
}

// Large maps (Ho*Wo >= 1024): the (min, max) key of every (sample, channel) plane of dY,
// each a contiguous run of P elements, streamed by one wave with 8 quads per lane in
// flight; ppl[n * D + d].  A sample's key is the reduction of its D planes, a channel's of
// its N planes.
constexpr int PLANE_U = 8;
template <int DT>
__global__ __launch_bounds__(256) void k_stats_planes(const void *__restrict__ dy,
                                                      uint32_t planes, uint32_t P4,
                                                      int2 *__restrict__ ppl) {
  const int lane = threadIdx.x & 63;
  const uint32_t nwaves = gridDim.x * 4;
  for (uint32_t pl = blockIdx.x * 4 + (threadIdx.x >> 6); pl < planes; pl += nwaves) {
    int lo = INT_MAX, hi = INT_MIN;
    const int64_t base = int64_t(pl) * P4 * 4;
    // Whole batches (no per-lane test: every load issues before the first use), then the
    // tail with out-of-plane quads reading element 0 and masked.
    uint32_t qb = 0;
    for (; qb + 64 * PLANE_U <= P4; qb += 64 * PLANE_U) {
      float v[PLANE_U][4];
#pragma unroll
      for (int u = 0; u < PLANE_U; ++u)
        load_quad<DT>(dy, base + 4 * int64_t(qb + 64 * u + lane), v[u]);
#pragma unroll
      for (int u = 0; u < PLANE_U; ++u)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int key = f2key(v[u][k] + 0.0f);
          lo = min(lo, key);
          hi = max(hi, key);
        }
    }
    if (qb < P4) {
      float v[PLANE_U][4];
#pragma unroll
      for (int u = 0; u < PLANE_U; ++u) {
        const uint32_t q = qb + 64 * u + lane;
        load_quad<DT>(dy, q < P4 ? base + 4 * int64_t(q) : 0, v[u]);
      }
#pragma unroll
      for (int u = 0; u < PLANE_U; ++u) {
        const bool in = qb + 64 * u + lane < P4;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int key = f2key(v[u][k] + 0.0f);
          lo = min(lo, in ? key : INT_MAX);
          hi = max(hi, in ? key : INT_MIN);
        }
      }
    }
    lo = wave_min(lo);
    hi = wave_max(hi);
    if (lane == 0) ppl[pl] = make_int2(lo, hi);
  }
}

// Large group sets: block b < N reduces sample b over its slots, block N + d channel d
// over its row-block partials.
constexpr int RED_THREADS = 256;
__global__ __launch_bounds__(RED_THREADS) void k_stats_reduce(const int2 *__restrict__ part_c,
                                                          const int2 *__restrict__ part_s,
                                                          StatsGeom sg, uint32_t nrb,
                                                          uint32_t ndt,
                                                          int2 *__restrict__ skey,
                                                          int2 *__restrict__ ckey) {
  __shared__ int32_t smn[RED_THREADS / 64], smx[RED_THREADS / 64];
  const TileGeom &g = sg.g;
  const uint32_t b = blockIdx.x;
  const uint32_t N = g.R / g.P;
  int lo = INT_MAX, hi = INT_MIN;
  if (b < N && g.P == 1) {
#pragma unroll 8
    for (uint32_t i = threadIdx.x; i < ndt; i += RED_THREADS) {
      const int2 v = part_s[size_t(b) * ndt + i];
      lo = min(lo, v.x);
      hi = max(hi, v.y);
    }
  } else if (b < N) {
    const uint32_t rt_lo = (b * g.P) / TILE, rt_hi = min(sg.nrt - 1, (b * g.P + g.P - 1) / TILE);
    const uint32_t cnt = rt_hi - rt_lo + 1;
#pragma unroll 8
    for (uint32_t i = threadIdx.x; i < ndt * cnt; i += RED_THREADS) {
      const uint32_t dt = i / cnt, rt = rt_lo + i % cnt;
      const uint32_t k = b - fdiv(rt * TILE, g.divP);
      const int2 v = part_s[(size_t(dt) * sg.nrt + rt) * sg.SL + k];
      lo = min(lo, v.x);
      hi = max(hi, v.y);
    }
  } else {
    const uint32_t d = b - N;
#pragma unroll 8
    for (uint32_t i = threadIdx.x; i < nrb; i += RED_THREADS) {
      const int2 v = part_c[size_t(i) * g.D + d];
      lo = min(lo, v.x);
      hi = max(hi, v.y);
    }
  }
  lo = wave_min(lo);
  hi = wave_max(hi);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    smn[wave] = lo;
    smx[wave] = hi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < RED_THREADS / 64; ++w) {
      lo = min(lo, smn[w]);
      hi = max(hi, smx[w]);
    }
    if (b < N) skey[b] = make_int2(lo, hi);
    else ckey[b - N] = make_int2(lo, hi);
  }
}

// ----------------------------------------------------------------------------- select

struct SetArgs {
  const int2 *key;     // [G] (min, max) keys (k_select)
  const int2 *part;    // partials (k_select_fused)
  uint32_t slots;      // 0: group g reduces part[u * ld + g], u < U (channels)
                       // 1: sample slots of part_s (P, nrt, SL, ndt)
                       // 2: key[g] already holds the group's key (k_stats_reduce ran)
                       // 3: group g reduces part[g * ld + u], u < U (per-plane partials)
                       // 4: key[r * MKEY_GROUPS + g], r < MKEY_REP, are the group's merged
                       //    key replicas (cleared once read)
  uint32_t U, ld;
  uint32_t P, nrt, SL, ndt;
  FastDiv divP;
  int32_t G;
  uint32_t stream;
  int32_t *kept;
  int32_t *count;
  float *scale, *offset, *prob;
  GroupParam *gp;
  float2 *slot;        // [G] (scale, offset) of the kept group in each slot
};

struct SelectArgs {
  SetArgs set[2];      // [0] samples, [1] channels
  int bits, mode;
  uint64_t seed;
  uint32_t step, layer;
};

constexpr int ID_BITS = 14;                   // group ids < 2^14 = FQT_MAX_AGP_GROUPS

__device__ __forceinline__ float group_range(int2 k) {
  return (key2f(k.y) - key2f(k.x)) + 0.0f;
}

// w_i = floor(2^40 * R_i / R_max): one correctly rounded float64 division, exact scaling.
__device__ __forceinline__ uint64_t agp_weight(float R, float Rmax) {
  if (!(Rmax > 0.0f) || !(R > 0.0f)) return 0;
  return static_cast<uint64_t>(floor(ldexp(static_cast<double>(R) / static_cast<double>(Rmax), 40)));
}

__device__ __forceinline__ uint64_t sort_key(uint64_t w, int i) {
  return (w << ID_BITS) | static_cast<uint64_t>((FQT_MAX_AGP_GROUPS - 1) - i);
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

template <int NT, typename T>
__device__ T block_sum(T v, T *scratch) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  T r = 0;
  for (int i = 0; i < NT / 64; ++i) r += scratch[i];
  __syncthreads();
  return r;
}

template <int NT>
__device__ float block_max_f(float v, float *scratch) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  float r = scratch[0];
  for (int i = 1; i < NT / 64; ++i) r = fmaxf(r, scratch[i]);
  __syncthreads();
  return r;
}

template <int NT>
__device__ uint64_t block_max_u64(uint64_t v, uint64_t *scratch) {
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t y = __shfl_xor(v, o);
    v = v > y ? v : y;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  uint64_t r = scratch[0];
  for (int i = 1; i < NT / 64; ++i) r = r > scratch[i] ? r : scratch[i];
  __syncthreads();
  return r;
}

// Exclusive prefix of `v` over thread order; `total` receives the block total.
template <int NT, typename T>
__device__ T block_exscan(T v, T *scratch, T &total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  T x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const T y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) scratch[wave] = x;
  __syncthreads();
  T off = 0, tot = 0;
  for (int i = 0; i < NT / 64; ++i) {
    if (i < wave) off += scratch[i];
    tot += scratch[i];
  }
  __syncthreads();
  total = tot;
  return off + x - v;
}

// a * b for a < 2^32, b < 2^64, as a 128-bit (hi, lo) pair.
__device__ __forceinline__ void mul_32x64(uint32_t a, uint64_t b, uint64_t &hi, uint64_t &lo) {
  const uint64_t p_lo = uint64_t(a) * (b & 0xFFFFFFFFull);
  const uint64_t p_hi = uint64_t(a) * (b >> 32);
  lo = p_lo + (p_hi << 32);
  hi = (p_hi >> 32) + (lo < p_lo ? 1 : 0);
}

// One workgroup of NT threads per group set (blockIdx.x = 0 samples, 1 channels).
// GP is the power-of-two capacity of the LDS sort (>= G).
template <int GP, int NT>
__global__ __launch_bounds__(NT) void k_select(SelectArgs a) {
  extern __shared__ uint64_t skey[];
  __shared__ uint64_t scr_u[NT / 64];
  __shared__ int32_t scr_i[NT / 64];
  __shared__ float scr_f[NT / 64];
  const SetArgs S = blockIdx.x ? a.set[1] : a.set[0];
  const int G = S.G;
  const int t = threadIdx.x;
  const int b = a.bits;
  const int B = (1 << b) - 1;

  // Thread t owns the groups [i0, i1) (at most CH of them): their keys are read once, all
  // loads issued together, and kept in registers (every loop below walks the same chunk,
  // unrolled, so the indices into the key registers are compile-time constants).
  constexpr int CH = (GP + NT - 1) / NT;
  const int chunk = (G + NT - 1) / NT;       // <= CH
  const int i0 = t * chunk;
  const int i1 = min(i0 + chunk, G);
  int2 keys[CH];
#pragma unroll
  for (int m = 0; m < CH; ++m)
    keys[m] = (m < chunk && i0 + m < G) ? S.key[i0 + m] : make_int2(0, 0);
  float rmax = 0.0f;
#pragma unroll
  for (int m = 0; m < CH; ++m)
    if (i0 + m < i1) rmax = fmaxf(rmax, group_range(keys[m]));
  rmax = block_max_f<NT>(rmax, scr_f);
  // The groups' AGP weights, once each while they fit in registers (up to 8 groups per
  // thread; 16 would spill, and are recomputed at each use instead).
  constexpr bool WCACHE = CH <= 8;
  uint64_t wts[WCACHE ? CH : 1];
  if constexpr (WCACHE) {
#pragma unroll
    for (int m = 0; m < CH; ++m)
      wts[m] = (a.mode != FQT_AGP_OFF && i0 + m < i1) ? agp_weight(group_range(keys[m]), rmax)
                                                       : 0ull;
  }
  auto wt = [&](int m) -> uint64_t {
    if constexpr (WCACHE) return wts[m];
    else return agp_weight(group_range(keys[m]), rmax);
  };

  int64_t s_sat = 0;           // number of saturated groups (p capped at 1)
  uint64_t w_thr = 0;          // weight of the last saturated group
  uint64_t w_rem = 0;          // weight of the unsaturated groups
  uint64_t key_thr = 0;        // TOPK: smallest kept sort key
  bool need_sort = a.mode == FQT_AGP_TOPK;
  if (a.mode == FQT_AGP_BERNOULLI) {
    // Saturation by rounds, as in the one-key-per-thread selection: with s groups
    // saturated and W the weight of the others, every unsaturated group with
    // (G - b s) w >= b W saturates; the rounds end (at s_sat) when none does, else the
    // sort below decides.  Equal weights pass or fail together, so the saturated groups
    // are exactly those with w >= w_thr, the smallest saturated weight.
    constexpr int SAT_ROUNDS = 8;
    const int c0 = i0, c1 = i1;
    uint64_t wsum = 0;
#pragma unroll
    for (int m = 0; m < CH; ++m) {
      if (c0 + m >= c1) break;
      const uint64_t w = wt(m);
      skey[c0 + m] = w;                   // this thread's weights, kept in LDS
      wsum += w;
    }
    uint64_t W = block_sum<NT, uint64_t>(wsum, scr_u);
    uint32_t satbits = 0;                 // groups c0 + m saturated
    int64_t sc = 0;
    bool done = false;
    for (int round = 0; round < SAT_ROUNDS; ++round) {
      const int64_t A = int64_t(G) - int64_t(b) * sc;
      uint64_t rs = 0;
      int32_t rc = 0;
      for (int i = c0; i < c1; ++i) {
        const uint64_t w = skey[i];
        const bool pass = !((satbits >> (i - c0)) & 1u) && w > 0 &&
                          A * int64_t(w) >= int64_t(b) * int64_t(W);
        if (pass) {
          satbits |= 1u << (i - c0);
          rs += w;
          ++rc;
        }
      }
      const int32_t cnt = block_sum<NT, int32_t>(rc, scr_i);
      const uint64_t sum = block_sum<NT, uint64_t>(rs, scr_u);
      if (cnt == 0) {
        done = true;
        break;
      }
      sc += cnt;
      W -= sum;
    }
    if (done) {
      s_sat = sc;
      w_rem = sc < G ? W : 0;
      uint64_t wmin = ~0ull;
      for (int i = c0; i < c1; ++i)
        if ((satbits >> (i - c0)) & 1u) wmin = min(wmin, skey[i]);
      // Smallest saturated weight: a block minimum as the negated maximum.
      const uint64_t neg = block_max_u64<NT>(~wmin, scr_u);
      w_thr = sc > 0 ? ~neg : 0;
    } else {
      need_sort = true;
    }
    __syncthreads();                      // the weights in skey are read; the sort reuses it
  }
  if (need_sort) {
#pragma unroll
    for (int m = 0; m < CH; ++m)
      if (i0 + m < i1) skey[i0 + m] = sort_key(wt(m), i0 + m);
    for (int i = G + t; i < GP; i += NT) skey[i] = 0ull;
    __syncthreads();
    // Bitonic sort, descending.
    for (int k = 2; k <= GP; k <<= 1) {
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int i = t; i < GP; i += NT) {
          const int ixj = i ^ j;
          if (ixj > i) {
            const uint64_t x = skey[i], y = skey[ixj];
            if (((i & k) == 0) ? (x < y) : (x > y)) {
              skey[i] = y;
              skey[ixj] = x;
            }
          }
        }
        __syncthreads();
      }
    }
    if (a.mode == FQT_AGP_TOPK) {
      key_thr = skey[max(1, G / b) - 1];
    } else {
      // Position s saturates iff (G - b s) w_(s) >= b * (weight at positions >= s); the
      // test holds on a prefix of the positions, so its pass count is s_sat.
      constexpr int CHUNK = (GP + NT - 1) / NT;
      const int p0 = t * CHUNK;
      uint64_t local = 0;
      for (int p = p0; p < min(p0 + CHUNK, G); ++p) local += skey[p] >> ID_BITS;
      uint64_t wtot;
      uint64_t excl = block_exscan<NT, uint64_t>(local, scr_u, wtot);
      int32_t pass = 0;
      for (int p = p0; p < min(p0 + CHUNK, G); ++p) {
        const uint64_t w = skey[p] >> ID_BITS;
        const int64_t lhs = (int64_t(G) - int64_t(b) * p) * int64_t(w);
        const int64_t rhs = int64_t(b) * int64_t(wtot - excl);
        pass += (w > 0 && lhs >= rhs) ? 1 : 0;
        excl += w;
      }
      s_sat = block_sum<NT, int32_t>(pass, scr_i);
      uint64_t rem = 0;
      for (int p = max(p0, int(s_sat)); p < min(p0 + CHUNK, G); ++p) rem += skey[p] >> ID_BITS;
      w_rem = block_sum<NT, uint64_t>(rem, scr_u);
      w_thr = s_sat > 0 ? (skey[s_sat - 1] >> ID_BITS) : 0;
    }
  }

  // Masks in id order, then the stable partition kept-ascending | pruned-ascending.
  const int64_t A = int64_t(G) - int64_t(b) * s_sat;
  uint32_t keepbits = 0;
  int32_t nkeep = 0;
#pragma unroll
  for (int m = 0; m < CH; ++m) {
    const int i = i0 + m;
    if (i >= i1) break;
    bool keep;
    if (a.mode == FQT_AGP_OFF) {
      keep = true;
    } else {
      const uint64_t w = wt(m);
      if (a.mode == FQT_AGP_TOPK) {
        keep = sort_key(w, i) >= key_thr;
      } else if (s_sat > 0 && w > 0 && w >= w_thr) {
        keep = true;
      } else if (A > 0 && w_rem > 0 && w > 0) {
        const Ctr4 u = philox_block(uint64_t(i) >> 2, S.stream, a.seed, a.step, a.layer);
        const uint32_t u32 = ctr_word(u, uint32_t(i) & 3u);
        uint64_t lh, ll;
        mul_32x64(u32, uint64_t(b) * w_rem, lh, ll);
        const uint64_t aw = uint64_t(A) * w;     // < 2^55
        const uint64_t rh = aw >> 32, rl = aw << 32;
        keep = lh < rh || (lh == rh && ll < rl);
      } else {
        keep = false;
      }
    }
    keepbits |= (keep ? 1u : 0u) << m;
    nkeep += keep ? 1 : 0;
  }
  int32_t count;
  int32_t rank = block_exscan<NT, int32_t>(nkeep, scr_i, count);
  if (t == 0) *S.count = count;
#pragma unroll
  for (int m = 0; m < CH; ++m) {
    const int i = i0 + m;
    if (i >= i1) break;
    const bool keep = (keepbits >> m) & 1u;
    const int2 k = keys[m];
    const float R = group_range(k);
    const float Z = key2f(k.x);
    float Sc = 0.0f, Zp = 0.0f, p = 0.0f;
    bool unit_p = a.mode != FQT_AGP_BERNOULLI;
    uint64_t w = 0;
    if (a.mode == FQT_AGP_BERNOULLI) {
      w = wt(m);
      unit_p = s_sat > 0 && w > 0 && w >= w_thr;
    }
    if (a.mode == FQT_AGP_OFF) {
      p = 1.0f;
    } else if (a.mode == FQT_AGP_TOPK) {
      p = keep ? 1.0f : 0.0f;
    } else if (unit_p) {
      p = 1.0f;
    } else if (w_rem > 0 && A > 0) {
      p = static_cast<float>(static_cast<double>(uint64_t(A) * w) /
                             static_cast<double>(uint64_t(b) * w_rem));
    }
    if (keep) {
      if (unit_p) {
        Sc = static_cast<float>(static_cast<double>(R) / static_cast<double>(B));
        Zp = Z;
      } else {
        const double bw = static_cast<double>(uint64_t(b) * w_rem);
        const double aw = static_cast<double>(uint64_t(A) * w);
        Sc = static_cast<float>((static_cast<double>(R) * bw) / (static_cast<double>(B) * aw));
        Zp = static_cast<float>((static_cast<double>(Z) * bw) / aw);
      }
    }
    S.prob[i] = p;
    S.scale[i] = Sc;
    S.offset[i] = Zp + 0.0f;
    if (keep) S.slot[rank] = make_float2(Sc, Zp + 0.0f);
    GroupParam gp;
    gp.z = Z;
    gp.inv = R > 0.0f ? __fdiv_rn(float(B), R) : 0.0f;
    gp.rank = keep ? rank : -1;
    gp.pad = 0;
    S.gp[i] = gp;
    if (keep) {
      S.kept[rank] = i;
      ++rank;
    } else {
      S.kept[count + (i - rank)] = i;
    }
  }
}

// AGP off (Section 5.2: every group kept, p = 1) over large group sets: one thread per
// group writes what the one-workgroup selection writes for it (rank = group id), so the
// whole chip takes the per-group work.  Grid: ceil(max G / 256) x 2 sets.
__global__ __launch_bounds__(256) void k_select_off(SelectArgs a) {
  const SetArgs &S = blockIdx.y ? a.set[1] : a.set[0];
  const int i = int(blockIdx.x) * 256 + int(threadIdx.x);
  if (i == 0) *S.count = S.G;
  if (i >= S.G) return;
  const int B = (1 << a.bits) - 1;
  const int2 k = S.key[i];
  const float R = group_range(k);
  const float Z = key2f(k.x);
  const float Sc = static_cast<float>(static_cast<double>(R) / static_cast<double>(B));
  S.prob[i] = 1.0f;
  S.scale[i] = Sc;
  S.offset[i] = Z + 0.0f;
  S.slot[i] = make_float2(Sc, Z + 0.0f);
  GroupParam gp;
  gp.z = Z;
  gp.inv = R > 0.0f ? __fdiv_rn(float(B), R) : 0.0f;
  gp.rank = i;
  gp.pad = 0;
  S.gp[i] = gp;
  S.kept[i] = i;
}

// Select for group sets of at most GP <= 1024 groups, one 1024-thread workgroup per set,
// with the partial reduction folded in.  One sort key per thread: the bitonic stages
// whose partner lies in the same wave exchange through shuffles, the others through a
// double-buffered LDS array (one barrier per stage); the water-filling scan, the
// saturation count and the kept-id ranks are wave scans plus one LDS combine each.
constexpr int SEL_NT = 1024;
constexpr int SEL_NW = SEL_NT / 64;

// v of lane (lane ^ j) for a wave-internal bitonic partner distance j < 64.
__device__ __forceinline__ uint64_t xor_partner(uint64_t v, int j) {
  switch (j) {
    case 32: return lane_xor64<32>(v);
    case 16: return lane_xor64<16>(v);
    case 8: return lane_xor64<8>(v);
    case 4: return lane_xor64<4>(v);
    case 2: return lane_xor64<2>(v);
    default: return lane_xor64<1>(v);
  }
}

// Inclusive prefix sum of v over the block's thread order, and the block total, when only
// the first NWR waves hold non-zero values (the others get their offsets wrong).
template <int NWR, typename T>
__device__ T block_incl_scan(T v, T *scr, T &total, int lane, int wave) {
  if constexpr (sizeof(T) == 8) v = wave_scan_add_u64(v);
  else v = wave_scan_i32(v, 0, [](int a, int b) { return a + b; });
  if (lane == 63) scr[wave] = v;
  __syncthreads();
  T off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NWR; ++w) {
    const T x = scr[w];
    off += w < wave ? x : T(0);
    tot += x;
  }
  __syncthreads();
  total = tot;
  return off + v;
}

template <int GP>
__device__ __forceinline__ void select_fused_body(const SelectArgs &a, int set) {
  static_assert(GP <= SEL_NT && GP % 64 == 0, "one sort key per thread");
  __shared__ int2 gk[GP];
  __shared__ int2 tmpk[SEL_NT];
  __shared__ uint64_t sbuf[2][GP];
  __shared__ uint64_t scr_u[SEL_NW];
  __shared__ int32_t scr_i[SEL_NW];
  __shared__ float scr_f[SEL_NW];
  __shared__ uint64_t sat_w[2];          // W(s_sat), w at s_sat - 1
  const SetArgs S = set ? a.set[1] : a.set[0];
  const int G = S.G;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int b = a.bits;
  const int B = (1 << b) - 1;

  // Group keys: min over the minima, max over the maxima of the group's partials.  Loads
  // are issued in batches of 16 per thread so that a group set costs a few memory
  // latencies.
  // SEL_NT / GP threads per group: thread t takes group t % GP and every (SEL_NT / GP)-th
  // of its partials from t / GP; the shares meet in LDS.
  {
    constexpr int SPLIT = SEL_NT / GP;
    const int g = t % GP, r0 = t / GP;
    int lo = INT_MAX, hi = INT_MIN;
    if (S.slots == 2) {                 // keys reduced beforehand
      if (g < G && r0 == 0) {
        const int2 k = S.key[g];
        lo = k.x;
        hi = k.y;
      }
    } else if (S.slots == 4) {          // merged keys, left zero for the next call
      if (g < G) {
        uint2 *mk = reinterpret_cast<uint2 *>(const_cast<int2 *>(S.key));
        uint2 u[(MKEY_REP + SPLIT - 1) / SPLIT];
#pragma unroll
        for (int i = 0; i < (MKEY_REP + SPLIT - 1) / SPLIT; ++i) {
          const int r = r0 + i * SPLIT;
          u[i] = r < MKEY_REP ? mk[r * MKEY_GROUPS + g] : make_uint2(0u, 0u);
        }
#pragma unroll
        for (int i = 0; i < (MKEY_REP + SPLIT - 1) / SPLIT; ++i) {
          const int r = r0 + i * SPLIT;
          const int2 k = merged_key(u[i]);
          lo = min(lo, k.x);
          hi = max(hi, k.y);
          if (r < MKEY_REP) mk[r * MKEY_GROUPS + g] = make_uint2(0u, 0u);
        }
      }
    } else if (g < G && !S.slots) {     // channels: row-block partials, adjacent per row
      // One per-lane offset (the group) and a wave-uniform one per row block (r0 is
      // uniform across each wave).
      const __amdgpu_buffer_rsrc_t prs = buffer_of(S.part, S.U * S.ld * 8);
      const uint32_t voff = uint32_t(g) * 8;
      for (uint32_t u0 = r0; u0 < S.U; u0 += 16 * SPLIT) {
        uint64_t v[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const uint32_t u = u0 + k * SPLIT;
          v[k] = load8(prs, u < S.U ? voff : BUF_NONE, u < S.U ? u * S.ld * 8 : 0);
        }
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          if (u0 + k * SPLIT >= S.U) break;
          lo = min(lo, int(uint32_t(v[k])));
          hi = max(hi, int(uint32_t(v[k] >> 32)));
        }
      }
    } else if (g < G && S.slots == 3) { // group g reduces part[g * ld + u], u < U
      const __amdgpu_buffer_rsrc_t prs = buffer_of(S.part, uint32_t(S.G) * S.ld * 8);
      for (uint32_t u0 = r0; u0 < S.U; u0 += 16 * SPLIT) {
        uint64_t v[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const uint32_t u = u0 + k * SPLIT;
          v[k] = load8(prs, u < S.U ? (uint32_t(g) * S.ld + u) * 8 : BUF_NONE, 0);
        }
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          if (u0 + k * SPLIT >= S.U) break;
          lo = min(lo, int(uint32_t(v[k])));
          hi = max(hi, int(uint32_t(v[k] >> 32)));
        }
      }
    } else if (g < G) {                 // samples: the slots of the 64-row tiles they meet
      const uint32_t first = uint32_t(g) * S.P;
      const uint32_t rt_lo = first / TILE, rt_hi = min(S.nrt - 1, (first + S.P - 1) / TILE);
      for (uint32_t dt = r0; dt < S.ndt; dt += SPLIT) {
#pragma unroll 4
        for (uint32_t rt = rt_lo; rt <= rt_hi; ++rt) {
          const uint32_t k = uint32_t(g) - fdiv(rt * TILE, S.divP);
          const int2 v = S.part[(size_t(dt) * S.nrt + rt) * S.SL + k];
          lo = min(lo, v.x);
          hi = max(hi, v.y);
        }
      }
    }
    tmpk[t] = make_int2(lo, hi);
    __syncthreads();
    if (t < G) {
      int2 k = tmpk[t];
#pragma unroll
      for (int s2 = 1; s2 < SPLIT; ++s2) {
        const int2 o = tmpk[t + s2 * GP];
        k.x = min(k.x, o.x);
        k.y = max(k.y, o.y);
      }
      gk[t] = k;
    }
  }
  __syncthreads();

  // Largest range: ranges are non-negative, so their float bits order like ints.
  float rmax = 0.0f;
  for (int i = t; i < G; i += SEL_NT) rmax = fmaxf(rmax, group_range(gk[i]));
  {
    const int m = wave_max_all(__float_as_int(rmax));
    if (lane == 0) scr_f[wave] = __int_as_float(m);
    __syncthreads();
    rmax = 0.0f;
#pragma unroll
    for (int w = 0; w < GP / 64; ++w) rmax = fmaxf(rmax, scr_f[w]);   // groups: t < G <= GP
  }
  const int2 own = t < G ? gk[t] : make_int2(0, 0);
  const float own_R = group_range(own);
  const uint64_t own_w = t < G ? agp_weight(own_R, rmax) : 0;

  int64_t s_sat = 0;           // number of saturated groups (p capped at 1)
  uint64_t w_rem = 0;          // weight of the unsaturated groups
  uint64_t key_thr = 0;        // TOPK: smallest kept sort key
  bool own_sat = false;        // group t is saturated
  bool need_sort = a.mode == FQT_AGP_TOPK;
  if (a.mode == FQT_AGP_BERNOULLI) {
    // Saturation by rounds.  With s groups saturated and W the weight of the others, every
    // unsaturated group with (G - b s) w >= b W saturates; the rounds end when none does.
    // A group that passes a round passes the sorted-order test at its own position (the
    // weights ranked between it and the saturated ones are at least its own), and a round
    // that adds none fails that test at position s, so the rounds end at s_sat.  They
    // usually take a few rounds (ranges that decay geometrically over the groups take the
    // most); past SAT_ROUNDS the sort below decides instead.
    constexpr int SAT_ROUNDS = 8;
    if constexpr (GP <= 256) {
      // Each wave that holds groups runs the rounds itself over all G weights (lane l holds
      // groups l + 64 m): wave scans and ballots, no barrier per round; all of them reach the
      // same result, and one barrier hands the outcome to the other waves.  The weights
      // pass through sbuf[0], which the sort below reuses only after that barrier.
      constexpr int M = GP / 64;
      const int nw = (G + 63) / 64;
      __shared__ uint64_t sat_out[2];        // s_sat (or ~0 when the rounds did not settle), W
      if (t < GP) sbuf[0][t] = t < G ? own_w : 0ull;
      __syncthreads();
      if (wave < nw) {
        uint64_t wl[M];
        uint64_t tot = 0;
#pragma unroll
        for (int m = 0; m < M; ++m) {
          wl[m] = m < nw ? sbuf[0][lane + 64 * m] : 0ull;
          tot += wl[m];
        }
        uint64_t W = wave_total_u64(tot);
        int64_t s = 0;
        bool done = false;
        uint32_t satm = 0;                   // bit m: group lane + 64 m saturated
        for (int round = 0; round < SAT_ROUNDS; ++round) {
          const int64_t A = int64_t(G) - int64_t(b) * s;
          uint64_t ps = 0;
          uint32_t pm = 0;
          int32_t cnt = 0;
#pragma unroll
          for (int m = 0; m < M; ++m) {
            if (m >= nw) break;
            // Groups past G hold weight 0 and never pass.
            const bool pass = !((satm >> m) & 1u) && wl[m] > 0 &&
                              A * int64_t(wl[m]) >= int64_t(b) * int64_t(W);
            ps += pass ? wl[m] : 0ull;
            pm |= pass ? (1u << m) : 0u;
            cnt += __builtin_popcountll(__ballot(pass));
          }
          if (cnt == 0) {
            done = true;
            break;
          }
          const uint64_t sum = wave_total_u64(ps);
          satm |= pm;
          s += cnt;
          W -= sum;
        }
        own_sat = t < G && ((satm >> wave) & 1u);
        if (t == 0) {
          sat_out[0] = done ? uint64_t(s) : ~0ull;
          sat_out[1] = W;
        }
      }
      __syncthreads();
      if (sat_out[0] != ~0ull) {
        s_sat = int64_t(sat_out[0]);
        w_rem = s_sat < G ? sat_out[1] : 0;
      } else {
        own_sat = false;
        need_sort = true;
      }
    } else {
      // Up to 1024 groups: one group per thread, the round sums combined through LDS.
      __shared__ uint64_t rsum[2][SEL_NW];
      __shared__ int32_t rcnt[2][SEL_NW];
      uint64_t W = 0;
      {
        const uint64_t ws = wave_scan_add_u64(own_w);
        if (lane == 63) rsum[1][wave] = ws;
        __syncthreads();
#pragma unroll
        for (int w = 0; w < GP / 64; ++w) W += rsum[1][w];
      }
      int64_t s = 0;
      bool done = false;
      for (int round = 0; round < SAT_ROUNDS; ++round) {
        const int64_t A = int64_t(G) - int64_t(b) * s;
        const bool pass = t < G && !own_sat && own_w > 0 &&
                          A * int64_t(own_w) >= int64_t(b) * int64_t(W);
        const uint64_t ws = wave_scan_add_u64(pass ? own_w : 0ull);
        const int32_t wc = __builtin_popcountll(__ballot(pass));
        const int buf = round & 1;
        if (lane == 63) {
          rsum[buf][wave] = ws;
          rcnt[buf][wave] = wc;
        }
        __syncthreads();
        uint64_t sum = 0;
        int32_t cnt = 0;
#pragma unroll
        for (int w = 0; w < GP / 64; ++w) {
          sum += rsum[buf][w];
          cnt += rcnt[buf][w];
        }
        if (cnt == 0) {
          done = true;
          break;
        }
        own_sat = own_sat || pass;
        s += cnt;
        W -= sum;
      }
      if (done) {
        s_sat = s;
        w_rem = s < G ? W : 0;
      } else {
        own_sat = false;
        need_sort = true;
      }
    }
  }
  if (need_sort) {
    // Bitonic sort of one key per thread, descending.
    uint64_t x = t < G ? sort_key(own_w, t) : 0ull;
    int buf = 0;
    // Only the GP / 64 waves holding keys work; the others just meet the LDS stages'
    // barriers (they would otherwise take VALU issue slots from the sorting waves).
    const bool sorter = wave < GP / 64;
    // Fully unrolled (GP is a compile-time constant): every stage is straight-line code
    // with its exchange pattern fixed.
#pragma unroll
    for (int k = 2; k <= GP; k <<= 1) {
#pragma unroll
      for (int j = k >> 1; j > 0; j >>= 1) {
        uint64_t y = 0;
        if (j >= 64) {
          if (sorter) sbuf[buf][t] = x;
          __syncthreads();
          if (sorter) y = sbuf[buf][t ^ j];
          buf ^= 1;
        } else if (sorter) {
          y = xor_partner(x, j);
        }
        if (sorter) {
          const bool lower = (t & j) == 0, desc = (t & k) == 0;
          x = (lower == desc) ? (x > y ? x : y) : (x < y ? x : y);
        }
      }
    }
    if (a.mode == FQT_AGP_TOPK) {
      if (t < GP) sbuf[buf][t] = x;
      __syncthreads();
      key_thr = sbuf[buf][max(1, G / b) - 1];
    } else {
      // Position p = t of the descending order saturates iff (G - b p) w_(p) >= b W(p),
      // W(p) = weight at positions >= p; the test holds on a prefix, so its pass count
      // is s_sat.
      const uint64_t w = t < G ? (x >> ID_BITS) : 0ull;
      uint64_t total;
      const uint64_t incl = block_incl_scan<GP / 64, uint64_t>(w, scr_u, total, lane, wave);
      const uint64_t Wp = total - incl + w;
      const bool pass = t < G && w > 0 &&
                        (int64_t(G) - int64_t(b) * t) * int64_t(w) >= int64_t(b) * int64_t(Wp);
      int32_t cnt_total;
      block_incl_scan<GP / 64, int32_t>(pass ? 1 : 0, scr_i, cnt_total, lane, wave);
      s_sat = cnt_total;
      if (t == s_sat) sat_w[0] = Wp;
      if (t == s_sat - 1) sat_w[1] = w;
      __syncthreads();
      w_rem = s_sat < G ? sat_w[0] : 0;
      const uint64_t w_thr = s_sat > 0 ? sat_w[1] : 0;   // weight of the last saturated
      own_sat = s_sat > 0 && own_w > 0 && own_w >= w_thr;
    }
  }

  // Mask of group i = t, then the stable partition kept-ascending | pruned-ascending.
  const int64_t A = int64_t(G) - int64_t(b) * s_sat;
  bool keep = false;
  if (t < G) {
    if (a.mode == FQT_AGP_OFF) {
      keep = true;
    } else if (a.mode == FQT_AGP_TOPK) {
      keep = sort_key(own_w, t) >= key_thr;
    } else if (own_sat) {
      keep = true;
    } else if (A > 0 && w_rem > 0 && own_w > 0) {
      const Ctr4 u = philox_block(uint64_t(t) >> 2, S.stream, a.seed, a.step, a.layer);
      const uint32_t u32 = ctr_word(u, uint32_t(t) & 3u);
      uint64_t lh, ll;
      mul_32x64(u32, uint64_t(b) * w_rem, lh, ll);
      const uint64_t aw = uint64_t(A) * own_w;     // < 2^55
      const uint64_t rh = aw >> 32, rl = aw << 32;
      keep = lh < rh || (lh == rh && ll < rl);
    }
  }
  // Rank among the kept groups: kept lanes below this one in the wave (mbcnt of the
  // ballot) plus the kept counts of the waves before it.
  const uint64_t kb = __ballot(keep);
  const int32_t below = int32_t(__builtin_amdgcn_mbcnt_hi(
      uint32_t(kb >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(kb), 0u)));
  if (lane == 0) scr_i[wave] = int32_t(__builtin_popcountll(kb));
  __syncthreads();
  int32_t count = 0, rank = below;
#pragma unroll
  for (int w = 0; w < GP / 64; ++w) {
    const int32_t c = scr_i[w];
    rank += w < wave ? c : 0;
    count += c;
  }
  if (t == 0) *S.count = count;
  if (t >= G) return;
  const float R = own_R;
  const float Z = key2f(own.x);
  float Sc = 0.0f, Zp = 0.0f, p = 0.0f;
  const bool unit_p = a.mode != FQT_AGP_BERNOULLI || own_sat;
  if (a.mode == FQT_AGP_OFF) {
    p = 1.0f;
  } else if (a.mode == FQT_AGP_TOPK) {
    p = keep ? 1.0f : 0.0f;
  } else if (unit_p) {
    p = 1.0f;
  } else if (w_rem > 0 && A > 0) {
    p = static_cast<float>(static_cast<double>(uint64_t(A) * own_w) /
                           static_cast<double>(uint64_t(b) * w_rem));
  }
  if (keep) {
    if (unit_p) {
      Sc = static_cast<float>(static_cast<double>(R) / static_cast<double>(B));
      Zp = Z;
    } else {
      const double bw = static_cast<double>(uint64_t(b) * w_rem);
      const double aw = static_cast<double>(uint64_t(A) * own_w);
      Sc = static_cast<float>((static_cast<double>(R) * bw) / (static_cast<double>(B) * aw));
      Zp = static_cast<float>((static_cast<double>(Z) * bw) / aw);
    }
  }
  S.prob[t] = p;
  S.scale[t] = Sc;
  S.offset[t] = Zp + 0.0f;
  if (keep) S.slot[rank] = make_float2(Sc, Zp + 0.0f);
  GroupParam gp;
  gp.z = Z;
  gp.inv = R > 0.0f ? __fdiv_rn(float(B), R) : 0.0f;
  gp.rank = keep ? rank : -1;
  gp.pad = 0;
  S.gp[t] = gp;
  S.kept[keep ? rank : count + (t - rank)] = t;
}

// One workgroup per group set.
template <int GP>
__global__ __launch_bounds__(SEL_NT) void k_select_fused(SelectArgs a) {
  select_fused_body<GP>(a, int(blockIdx.x));
}

// The same two selection workgroups, then spare workgroups that pack the products' sign
// operands (they do not depend on dY): blocks [2, 2 + npw) the weight bytes, the rest the
// im2col of X, in one of three forms: bit-level (block order of bit_im2col_body), through
// the band (word group fastest, then 64-channel groups), or a wave per 64 positions of
// IM2COL_CPW channels (any convolution; work items in wave order); for a linear layer the
// sign words of X down its rows (a wave per work item of rows_wave_body).
enum SignForm { SIGN_BITS = 0, SIGN_BAND = 1, SIGN_WAVE = 2, SIGN_ROWS = 3 };
constexpr uint32_t SIGN_IPB = 4;     // work items per workgroup of the wave and rows forms
struct SignArgs {
  const void *x;
  BandGeom bg;
  BitGeom bt;
  Im2colGeom ig;
  uint64_t *xsign;
  uint32_t nwb;          // word-group blocks of the band (samples x word groups)
  FastDiv divNwb;
  const void *w;
  PackWGeom pg;
  int8_t *wsb;
  int32_t *wlsum;
  uint32_t npw;
  uint32_t ipb;          // work items per workgroup of the wave and rows forms (waves past it idle)
};
// DT: dtype of X; WDT: dtype of W; KH, KW: the kernel size of the band and wave forms
// (0: read from the geometry).
template <int GP, int DT, int FORM, int KH, int KW, int WDT = DT>
__global__ __launch_bounds__(SEL_NT) __attribute__((amdgpu_waves_per_eu(8))) void k_select_signs(
    SelectArgs a, SignArgs sg) {
  extern __shared__ uint32_t band[];
  __shared__ PackWLds pws;
  const uint32_t b = blockIdx.x;
  if (b < 2) {
    select_fused_body<GP>(a, int(b));
  } else if (b - 2 < sg.npw) {
    pack_w_body<WDT>(sg.w, sg.pg, sg.wsb, sg.wlsum, b - 2, pws);
  } else if constexpr (FORM == SIGN_BITS) {
    bit_im2col_body<DT, SEL_NT>(sg.x, sg.bt, sg.xsign, b - 2 - sg.npw,
                                reinterpret_cast<uint64_t *>(band));
  } else if constexpr (FORM == SIGN_BAND) {
    const uint32_t f = b - 2 - sg.npw;
    const uint32_t cb = fdiv(f, sg.divNwb);
    band_im2col_body<DT, KH, KW, SEL_NT>(sg.x, sg.bg, sg.xsign, f - cb * sg.nwb, cb, band);
  } else {
    // Work items spread over workgroups: a CU's address unit, not the memory latency, bounds
    // these gathers when one workgroup takes sixteen waves of them.
    const uint32_t wave = threadIdx.x >> 6;
    if (wave >= sg.ipb) return;
    const uint32_t item = (b - 2 - sg.npw) * sg.ipb + wave;
    if constexpr (FORM == SIGN_WAVE) wave_im2col_body<DT, KH, KW, true>(sg.x, sg.ig, sg.xsign, item);
    else rows_wave_body<DT>(sg.x, sg.ig.R, sg.ig.C, sg.xsign, item);
  }
}
// Static LDS of k_select_signs<GP>: the selection's arrays and the weight-byte tile.
constexpr size_t select_signs_static_lds(int GP) {
  return size_t(24) * GP + 8 * SEL_NT + 16 * SEL_NW + 16 + sizeof(PackWLds);
}

// ----------------------------------------------------------------------------- quantize + pack

// The 24-bit uniform of a Philox word as the float u24 * 2^-24 (exact).
__device__ __forceinline__ float unit24(uint32_t u) {
  return __fmul_rn(static_cast<float>(u >> 8), 5.9604644775390625e-8f);
}

// b-bit stochastic rounding code of x (Section 3.2): v = clamp((x - Z) * inv, 0, B),
// q = floor(v) + [u < v - floor(v)] for the uniform u = u24 * 2^-24 (the same test as
// u24 < frac(v) * 2^24: both sides scale by a power of two).  inv = 0 (R = 0) gives q = 0.
// For 0 <= v <= 255 the truncating conversion is floor(v) and v_fract_f32 gives
// v - floor(v) exactly.  The clamp is one v_med3_f32; a NaN product (inf * 0) makes it
// return the minimum of its three inputs, 0, as max-then-min would.
__device__ __forceinline__ uint32_t sr_code(float x, float z, float inv, float Bf, float u) {
  float v = __fmul_rn(__fsub_rn(x, z), inv);
  v = __builtin_amdgcn_fmed3f(v, 0.0f, Bf);
  return static_cast<uint32_t>(v) + (u < __builtin_amdgcn_fractf(v) ? 1u : 0u);
}
// b = 1: v is clamped to [0, 1], so q = [u < v]; as u < 1, the test on the unclamped
// product gives the same bit (true for v >= 1, false for v <= 0 and for NaN).
__device__ __forceinline__ uint32_t sr_bit(float x, float z, float inv, float u) {
  return u < __fmul_rn(__fsub_rn(x, z), inv) ? 1u : 0u;
}
// The code of x in group p, whose parameters in LDS have inv = 0 when the group is pruned:
// then v = (x - z) * 0 is 0 or NaN and both rounding forms give 0 (also for R = 0).
template <bool ONE>
__device__ __forceinline__ uint32_t sr_any(float x, const GroupParam &p, float Bf, float u) {
  return ONE ? sr_bit(x, p.z, p.inv, u) : sr_code(x, p.z, p.inv, Bf, u);
}

struct QPackArgs {
  const void *dy;
  TileGeom g;
  const GroupParam *sp;
  const GroupParam *cp;
  uint64_t *psq;        // [bits][R][Wd]
  uint64_t *pcq;        // [bits][D][Wr]
  uint8_t *psq_codes;   // [2*Wd][R][32]  chunk-major: byte d of row r at ((d/32)*R + r)*32 + d%32
  uint8_t *pcq_codes;   // [2*Wr][D][32]  byte r of kept channel j at ((r/32)*D + j)*32 + r%32
  uint32_t Wd, Wr;
  int bits;
  uint64_t seed;
  uint32_t step, layer;
  uint32_t eager;       // read every quad of the layer before the parameters
  uint32_t chan_fast;   // grid x walks the channel tiles (rows of dY read as long runs)
  uint32_t planes;      // 1: also write the bit planes (0: the byte codes only)
};

// Codes of a thread's quads into the LDS tiles.  The four codes of a quad share one
// Philox block (element e takes word e % 4; both encodings use the element's word); the
// encoding whose lines run along the quad gets them as one 32-bit store.
template <int MODE, bool ONE>
__device__ __forceinline__ void qpack_quads(const QPackArgs &a, const TileGeom &g, uint32_t d0,
                                            uint32_t r0, int t, const float (&x)[QUADS][4],
                                            const bool (&need)[QUADS], float Bf,
                                            const GroupParam *spar, const GroupParam *cpar,
                                            uint8_t (*cs)[PITCH], uint8_t (*cc)[PITCH]) {
#pragma unroll
  for (int q = 0; q < QUADS; ++q) {
    int dd, rr;
    quad_coord<MODE>(t, q, 0, dd, rr);
    uint32_t qs[4] = {0, 0, 0, 0}, qc[4] = {0, 0, 0, 0};
    if (need[q]) {
      const uint32_t e = elem_index(g, d0 + dd, r0 + rr);
      const Ctr4 u = philox_block(e >> 2, STREAM_ELEM, a.seed, a.step, a.layer);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int dk = MODE == TILE_CHAN ? dd + k : dd;
        const int rk = MODE == TILE_PIX ? rr + k : rr;
        const float uf = unit24(u.v[k]);
        qs[k] = sr_any<ONE>(x[q][k], spar[rk], Bf, uf);
        qc[k] = sr_any<ONE>(x[q][k], cpar[dk], Bf, uf);
      }
    }
    const uint32_t ws = qs[0] | (qs[1] << 8) | (qs[2] << 16) | (qs[3] << 24);
    const uint32_t wc = qc[0] | (qc[1] << 8) | (qc[2] << 16) | (qc[3] << 24);
    if (MODE == TILE_CHAN) {            // row rr, channels dd .. dd + 3
      *reinterpret_cast<uint32_t *>(&cs[rr][dd]) = ws;
#pragma unroll
      for (int k = 0; k < 4; ++k) cc[dd + k][rr] = uint8_t(qc[k]);
    } else {                            // channel dd, rows rr .. rr + 3
#pragma unroll
      for (int k = 0; k < 4; ++k) cs[rr + k][dd] = uint8_t(qs[k]);
      *reinterpret_cast<uint32_t *>(&cc[dd][rr]) = wc;
    }
  }
}

template <int MODE, int DT>
__global__ __launch_bounds__(THREADS) void k_qpack(QPackArgs a) {
  __shared__ __align__(16) uint8_t cs[TILE][PITCH];   // PSQ codes, [rr][dd]
  __shared__ __align__(16) uint8_t cc[TILE][PITCH];   // PCQ codes, [dd][rr]
  __shared__ __align__(8) uint8_t pbuf[WAVES][8][8][8];  // per wave: [line][plane][8-code chunk]
  __shared__ GroupParam spar[TILE];     // sample params of each column rr
  __shared__ GroupParam cpar[TILE];     // channel params of each row dd
  __shared__ int32_t prow[TILE];        // PSQ row of column rr, -1 if pruned/outside
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const TileGeom &g = a.g;
  const uint32_t r0 = (a.chan_fast ? blockIdx.y : blockIdx.x) * TILE;
  const uint32_t d0 = (a.chan_fast ? blockIdx.x : blockIdx.y) * TILE;
  const float Bf = float((1 << a.bits) - 1);

  // Eager form (most elements kept): the dY loads issue before the group parameters
  // arrive, so the two memory round trips overlap; otherwise only quads with a kept
  // sample or channel are read, after the parameters.
  float x[QUADS][4];
  if (MODE != TILE_SCALAR && a.eager) {
    for (int q = 0; q < QUADS; ++q) {
      int dd, rr;
      quad_coord<MODE>(t, q, 0, dd, rr);
      const bool in = d0 + dd < g.D && r0 + rr < g.R;
      load_quad<DT>(a.dy, in ? elem_index(g, d0 + dd, r0 + rr) : 0, x[q]);
    }
  }

  if (t < TILE) {
    const uint32_t r = r0 + t;
    GroupParam p;
    p.z = 0.0f; p.inv = 0.0f; p.rank = -1; p.pad = 0;
    int32_t row = -1;
    if (r < g.R) {
      const uint32_t n = fdiv(r, g.divP);
      p = a.sp[n];
      if (p.rank >= 0) row = int32_t(uint32_t(p.rank) * g.P + (r - n * g.P));
      else p.inv = 0.0f;                        // pruned: every code 0
    }
    spar[t] = p;
    prow[t] = row;
  } else if (t < 2 * TILE) {
    const uint32_t d = d0 + (t - TILE);
    GroupParam p;
    p.z = 0.0f; p.inv = 0.0f; p.rank = -1; p.pad = 0;
    if (d < g.D) p = a.cp[d];
    if (p.rank < 0) p.inv = 0.0f;               // pruned: every code 0
    cpar[t - TILE] = p;
  }
  __syncthreads();

  if (MODE != TILE_SCALAR) {
    bool need[QUADS];
    for (int q = 0; q < QUADS; ++q) {
      int dd, rr;
      quad_coord<MODE>(t, q, 0, dd, rr);
      // Quads are all inside or all outside the layer; inside, draw only if some
      // element belongs to a kept sample or a kept channel.
      bool nd = false;
      if (d0 + dd < g.D && r0 + rr < g.R) {
        for (int k = 0; k < 4; ++k) {
          const int dk = MODE == TILE_CHAN ? dd + k : dd;
          const int rk = MODE == TILE_PIX ? rr + k : rr;
          nd |= (spar[rk].rank >= 0) | (cpar[dk].rank >= 0);
        }
      }
      need[q] = nd;
      if (!a.eager) load_quad<DT>(a.dy, nd ? elem_index(g, d0 + dd, r0 + rr) : 0, x[q]);
    }
    if (a.bits == 1) qpack_quads<MODE, true>(a, g, d0, r0, t, x, need, Bf, spar, cpar, cs, cc);
    else qpack_quads<MODE, false>(a, g, d0, r0, t, x, need, Bf, spar, cpar, cs, cc);
  } else {
    for (int m = 0; m < 4 * QUADS; ++m) {
      int dd, rr;
      quad_coord<MODE>(t, m >> 2, m & 3, dd, rr);
      const uint32_t d = d0 + dd, r = r0 + rr;
      uint32_t qs = 0, qc = 0;
      const GroupParam ps = spar[rr], pc = cpar[dd];
      if (d < g.D && r < g.R && (ps.rank >= 0 || pc.rank >= 0)) {
        const uint32_t e = elem_index(g, d, r);
        const float xv = load_elem<DT>(a.dy, e) + 0.0f;
        const Ctr4 u = philox_block(e >> 2, STREAM_ELEM, a.seed, a.step, a.layer);
        const float uf = unit24(ctr_word(u, e & 3u));
        qs = sr_any<false>(xv, ps, Bf, uf);
        qc = sr_any<false>(xv, pc, Bf, uf);
      }
      cs[rr][dd] = uint8_t(qs);
      cc[dd][rr] = uint8_t(qc);
    }
  }
  __syncthreads();

  // Each wave stores its 8 lines of each encoding (line i = wave + WAVES * i).  Lane
  // 8 i + k holds code bytes 8 k .. 8 k + 7 of line i: it stores them, transposes them as
  // an 8 x 8 bit matrix (byte p = plane p of those 8 codes) and leaves the plane bytes in
  // LDS, from where lane 8 i + p reads the whole 64-bit word of plane p.
  const int li = lane >> 3, lk = lane & 7;
  // PCQ: channel rows dd, lanes along r (column encoder).
  {
    const int dd = wave + WAVES * li;
    const int rank = cpar[dd].rank;             // -1 for pruned channels and past D
    const uint32_t *src = reinterpret_cast<const uint32_t *>(&cc[dd][8 * lk]);
    const uint32_t lo = src[0], hi = src[1];
    if (rank >= 0)
      *reinterpret_cast<uint2 *>(a.pcq_codes + ((size_t(r0 >> 5) + (lk >> 2)) * g.D + rank) * 32 +
                                 8 * (lk & 3)) = make_uint2(lo, hi);
    if (a.planes) {
      const uint64_t y = bit_transpose8((uint64_t(hi) << 32) | lo);
#pragma unroll
      for (int p = 0; p < 8; ++p)
        if (p < a.bits) pbuf[wave][li][p][lk] = uint8_t(y >> (8 * p));
      __builtin_amdgcn_wave_barrier();          // LDS operations of a wave run in order
      const uint64_t pw = *reinterpret_cast<const uint64_t *>(&pbuf[wave][li][lk][0]);
      if (rank >= 0 && lk < a.bits) a.pcq[(size_t(lk) * g.D + rank) * a.Wr + (r0 >> 6)] = pw;
    }
  }
  __builtin_amdgcn_wave_barrier();
  // PSQ: sample rows rr, lanes along d (row encoder).
  {
    const int rr = wave + WAVES * li;
    const int row = prow[rr];                   // -1 for pruned samples and past R
    const uint32_t *src = reinterpret_cast<const uint32_t *>(&cs[rr][8 * lk]);
    const uint32_t lo = src[0], hi = src[1];
    if (row >= 0)
      *reinterpret_cast<uint2 *>(a.psq_codes + ((size_t(d0 >> 5) + (lk >> 2)) * g.R + row) * 32 +
                                 8 * (lk & 3)) = make_uint2(lo, hi);
    if (a.planes) {
      const uint64_t y = bit_transpose8((uint64_t(hi) << 32) | lo);
#pragma unroll
      for (int p = 0; p < 8; ++p)
        if (p < a.bits) pbuf[wave][li][p][lk] = uint8_t(y >> (8 * p));
      __builtin_amdgcn_wave_barrier();
      const uint64_t pw = *reinterpret_cast<const uint64_t *>(&pbuf[wave][li][lk][0]);
      if (row >= 0 && lk < a.bits) a.psq[(size_t(lk) * g.R + row) * a.Wd + (d0 >> 6)] = pw;
    }
  }
}

// Zero-fill of a quantize / layer workspace's state bytes (the merged group keys): one
// 16-byte store per thread.  A kernel, not hipMemsetAsync, so that a captured graph replays
// it like any other node.
__global__ __launch_bounds__(256) void k_state_clear(uint4 *state, uint32_t n16) {
  const uint32_t e = blockIdx.x * 256 + threadIdx.x;
  if (e < n16) state[e] = make_uint4(0u, 0u, 0u, 0u);
}

template <int GP, int NT>
int launch_select(const SelectArgs &sa, hipStream_t s) {
  const size_t lds = size_t(GP) * sizeof(uint64_t);
  int dev = 0, max_lds = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return FQT_E_HIP;
  if (lds + 1024 > size_t(max_lds)) return FQT_E_SHAPE;   // the group set does not fit in LDS
  if (lds > 65536) {
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(&k_select<GP, NT>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
      return FQT_E_HIP;
  }
  hipLaunchKernelGGL((k_select<GP, NT>), dim3(2), dim3(NT), lds, s, sa);
  return last_launch_status();
}

}  // namespace

uint32_t stats_slots(const Layer &L) {
  const int64_t per = (63 + L.P - 1) / L.P + 1;
  return uint32_t(per < 64 ? per : 64);
}
// Row tiles per stats block: one while that still gives 256 blocks, else up to 8 (each
// row block adds a partial per channel that the selection reads from one workgroup).
uint32_t stats_rows_per_block(const Layer &L) {
  int64_t rs = 1;
  while (rs < 8 && L.Wr * L.Wd / (rs * 2) >= 256) rs *= 2;
  return uint32_t(rs);
}
int64_t stats_row_blocks(const Layer &L) {
  const int64_t rs = stats_rows_per_block(L);
  return (L.Wr + rs - 1) / rs;
}

int launch_state_clear(void *state, hipStream_t s) {
  constexpr uint32_t n16 = FQT_WS_STATE_BYTES / 16;
  hipLaunchKernelGGL(k_state_clear, dim3((n16 + 255) / 256), dim3(256), 0, s,
                     static_cast<uint4 *>(state), n16);
  return last_launch_status();
}

int launch_quantize(const Layer &L, const fqt_quant_cfg &cfg, const void *dY, const fqt_qgrad &q,
                    const QuantWs &w, hipStream_t s, SignJob *signs, bool write_planes) {
  TileGeom g{uint32_t(L.D), uint32_t(L.P), uint32_t(L.R), make_fastdiv(uint32_t(L.P))};
  const uint32_t nrt = uint32_t(L.Wr), ndt = uint32_t(L.Wd);
  const uint32_t nrb = uint32_t(stats_row_blocks(L));
  const int mode = (L.P % 4 == 0) ? TILE_PIX : (L.P == 1 && L.D % 4 == 0) ? TILE_CHAN : TILE_SCALAR;
  // With channels contiguous in dY (P = 1) the channel tiles go fastest, so the blocks in
  // flight read whole rows of dY in order.
  const uint32_t chan_fast = (mode == TILE_CHAN && nrb <= 65535) ? 1u : 0u;
  const StatsGeom sg{g, nrt, stats_slots(L), stats_rows_per_block(L), chan_fast, ndt};
  const dim3 grid = chan_fast ? dim3(ndt, nrb) : dim3(nrb, ndt);
  const int64_t gmax = L.N > L.D ? L.N : L.D;
  // Large maps with both group sets in one-workgroup selections: per-plane statistics
  // (part_c holds the N * D plane keys: it has D * stats_row_blocks >= D * N entries).
  const bool planes = L.P >= 1024 && L.P % 4 == 0 && gmax <= 1024;
  // The one-workgroup selection reduces the partials itself; with many partials per group
  // (large N*Ho*Wo) a workgroup per group reduces them first.  With few partials per group
  // the statistics merge the keys with atomics instead (the selection then reads one key
  // per group).
  const bool many_partials =
      !planes && (nrb > 256 || int64_t(ndt) * ((L.P + TILE - 1) / TILE + 1) > 256);
  const bool merged = !planes && !many_partials && gmax <= 1024;
  uint2 *mks = merged ? w.mkeys : nullptr;
  uint2 *mkc = merged ? w.mkeys + L.N : nullptr;
  if (planes) {
    const uint32_t np = uint32_t(L.N * L.D);
    const uint32_t blocks = std::min<uint32_t>((np + 3) / 4, 4096);
    dispatch_dtype(L.dy_t, [&]<int DT>() {
      hipLaunchKernelGGL(k_stats_planes<DT>, dim3(blocks), dim3(256), 0, s, dY, np,
                         uint32_t(L.P / 4), w.part_c);
    });
  } else dispatch_dtype(L.dy_t, [&]<int DT>() {
    if (mode == TILE_PIX)
      hipLaunchKernelGGL((k_stats<TILE_PIX, DT>), grid, dim3(THREADS), 0, s, dY, sg, w.part_c,
                         w.part_s, mks, mkc);
    else if (mode == TILE_CHAN)
      hipLaunchKernelGGL((k_stats<TILE_CHAN, DT>), grid, dim3(THREADS), 0, s, dY, sg, w.part_c,
                         w.part_s, mks, mkc);
    else
      hipLaunchKernelGGL((k_stats<TILE_SCALAR, DT>), grid, dim3(THREADS), 0, s, dY, sg,
                         w.part_c, w.part_s, mks, mkc);
  });
  if (last_launch_status() != FQT_OK) return FQT_E_HIP;

  SelectArgs sa;
  sa.set[0] = SetArgs{w.skey, w.part_s, 1u, 0u, 0u, uint32_t(L.P), nrt, sg.SL, ndt,
                      make_fastdiv(uint32_t(L.P)), int32_t(L.N), STREAM_SAMPLE, q.psq_kept,
                      q.psq_count, q.psq_scale, q.psq_offset, q.psq_prob, w.sp, w.sslot};
  sa.set[1] = SetArgs{w.ckey, w.part_c, 0u, nrb, uint32_t(L.D), 0u, 0u, 0u, 0u,
                      make_fastdiv(1u), int32_t(L.D), STREAM_CHANNEL, q.pcq_kept, q.pcq_count,
                      q.pcq_scale, q.pcq_offset, q.pcq_prob, w.cp, w.cslot};
  sa.bits = cfg.bits; sa.mode = cfg.agp_mode; sa.seed = cfg.seed; sa.step = cfg.step;
  sa.layer = cfg.layer_id;
  if (planes) {
    sa.set[0].slots = 3; sa.set[0].part = w.part_c; sa.set[0].U = uint32_t(L.D);
    sa.set[0].ld = uint32_t(L.D);
    sa.set[1].slots = 0; sa.set[1].U = uint32_t(L.N); sa.set[1].ld = uint32_t(L.D);
  }
  if (merged) {
    sa.set[0].slots = 4; sa.set[0].key = reinterpret_cast<const int2 *>(mks);
    sa.set[1].slots = 4; sa.set[1].key = reinterpret_cast<const int2 *>(mkc);
  }
  int st;
  if (gmax <= 1024 && many_partials) {
    hipLaunchKernelGGL(k_stats_reduce, dim3(unsigned(L.N + L.D)), dim3(RED_THREADS), 0, s,
                       w.part_c, w.part_s, sg, nrb, ndt, w.skey, w.ckey);
    if (last_launch_status() != FQT_OK) return FQT_E_HIP;
    sa.set[0].slots = 2;          // the selection reads the reduced keys
    sa.set[1].slots = 2;
  }
  // Sign operands in the selection launch.  Convolutions: bit-level for stride-1
  // same-padded convolutions whose staging fits the LDS left beside the selection (64 KB per
  // workgroup in all; at most about 448 im2col workgroups: with two 1024-thread workgroups
  // per CU the launch fits the chip in one round), else through the band where X and W share
  // a dtype and its staging fits, else a wave per 64 positions.  Linear layers: the rows
  // form.
  BitGeom bt;
  BandGeom bg;
  size_t sign_lds = 0;
  const int gp = gmax <= 256 ? 256 : 1024;
  const size_t lds_left = 65536 - 512 - select_signs_static_lds(gp);
  const bool sign_ok = signs && gmax <= 1024;
  const bool with_bits = sign_ok && bit_geom(L, SEL_NT, 448, lds_left, &bt, &sign_lds);
  const bool with_band = sign_ok && !with_bits && L.x_t == L.w_t &&
                         band_geom(L, signs->X, L.x_t, SEL_NT, lds_left, &bg, &sign_lds);
  const bool with_wave = sign_ok && !with_bits && !with_band && L.kind == FQT_CONV2D;
  const bool with_rows = sign_ok && L.kind == FQT_LINEAR;
  if (with_bits || with_band || with_wave || with_rows) {
    SignArgs sg{};
    sg.x = signs->X; sg.xsign = signs->xsign;
    sg.w = signs->W; sg.pg = pack_w_geom(L); sg.wsb = signs->wsb; sg.wlsum = signs->wlsum;
    sg.npw = pack_w_blocks(L);
    uint32_t xblocks;
    if (with_bits) {
      bit_geom_vec(&bt, signs->X);
      sg.bt = bt;
      xblocks = bit_blocks(bt);
    } else if (with_wave) {
      sg.ig = im2col_geom(L);
      sg.ipb = SIGN_IPB;
      xblocks = uint32_t((int64_t(sg.ig.cgroups) * sg.ig.nw + SIGN_IPB - 1) / SIGN_IPB);
    } else if (with_rows) {
      sg.ig = Im2colGeom{};
      sg.ig.R = uint32_t(L.N);       // rows of X
      sg.ig.C = uint32_t(L.C);       // columns of X
      sg.ipb = SIGN_IPB;
      const int64_t items = ((L.N + 63) / 64) * ((L.C + 15) / 16);
      xblocks = uint32_t((items + SIGN_IPB - 1) / SIGN_IPB);
    } else {
      sg.bg = bg;
      sg.nwb = band_word_blocks(L, bg); sg.divNwb = make_fastdiv(sg.nwb);
      xblocks = sg.nwb * uint32_t((L.C + BAND_CPW * SEL_NW - 1) / (BAND_CPW * SEL_NW));
    }
    const dim3 grid(2 + sg.npw + xblocks);
    dispatch_dtype(L.x_t, [&]<int DT>() {
      auto go = [&]<int GPT>() {
        // The band form needs X and W of one dtype; the others take W's dtype apart.
        auto launch = [&]<int FORM, int KH, int KW>() {
          if constexpr (FORM != SIGN_BAND) {
            if (L.w_t != DT) {
              dispatch_dtype(L.w_t, [&]<int WDT>() {
                hipLaunchKernelGGL((k_select_signs<GPT, DT, FORM, KH, KW, WDT>), grid,
                                   dim3(SEL_NT), sign_lds, s, sa, sg);
              });
              return;
            }
          }
          hipLaunchKernelGGL((k_select_signs<GPT, DT, FORM, KH, KW>), grid, dim3(SEL_NT),
                             sign_lds, s, sa, sg);
        };
        if (with_rows) launch.template operator()<SIGN_ROWS, 0, 0>();
        else if (with_bits) launch.template operator()<SIGN_BITS, 0, 0>();
        else if (with_band && L.kh == 3 && L.kw == 3) launch.template operator()<SIGN_BAND, 3, 3>();
        else if (with_band && L.kh == 1 && L.kw == 1) launch.template operator()<SIGN_BAND, 1, 1>();
        else if (with_band) launch.template operator()<SIGN_BAND, 0, 0>();
        else if (L.kh == 3 && L.kw == 3) launch.template operator()<SIGN_WAVE, 3, 3>();
        else if (L.kh == 1 && L.kw == 1) launch.template operator()<SIGN_WAVE, 1, 1>();
        else launch.template operator()<SIGN_WAVE, 0, 0>();
      };
      if (gp == 256) go.template operator()<256>();
      else go.template operator()<1024>();
    });
    st = last_launch_status();
    signs->done = st == FQT_OK;
  } else if (gmax <= 1024) {
    if (gmax <= 256) hipLaunchKernelGGL(k_select_fused<256>, dim3(2), dim3(SEL_NT), 0, s, sa);
    else hipLaunchKernelGGL(k_select_fused<1024>, dim3(2), dim3(SEL_NT), 0, s, sa);
    st = last_launch_status();
  } else {
    hipLaunchKernelGGL(k_stats_reduce, dim3(unsigned(L.N + L.D)), dim3(RED_THREADS), 0, s,
                       w.part_c, w.part_s, sg, nrb, ndt, w.skey, w.ckey);
    if (last_launch_status() != FQT_OK) return FQT_E_HIP;
    if (cfg.agp_mode == FQT_AGP_OFF) {
      hipLaunchKernelGGL(k_select_off, dim3(unsigned((gmax + 255) / 256), 2), dim3(256), 0, s, sa);
      st = last_launch_status();
    } else if (gmax <= 4096) st = launch_select<4096, 1024>(sa, s);
    else st = launch_select<16384, 1024>(sa, s);
  }
  if (st != FQT_OK) {
    // The statistics merged their keys but no selection will read and clear them: clear
    // them here, so that the workspace stays fit for the next call.
    if (merged) launch_state_clear(w.mkeys, s);
    return st;
  }

  // One block per 64 x 64 tile.  With channels contiguous in dY (P = 1), the channel
  // tiles go fastest, so the blocks in flight read whole rows of dY in order.
  QPackArgs qa;
  qa.chan_fast = (mode == TILE_CHAN && nrt <= 65535) ? 1u : 0u;
  const dim3 qgrid = qa.chan_fast ? dim3(ndt, nrt) : dim3(nrt, ndt);
  qa.dy = dY; qa.g = g; qa.sp = w.sp; qa.cp = w.cp;
  qa.psq = q.psq_planes; qa.pcq = q.pcq_planes;
  qa.psq_codes = q.psq_codes; qa.pcq_codes = q.pcq_codes;
  qa.Wd = uint32_t(L.Wd); qa.Wr = uint32_t(L.Wr);
  qa.bits = cfg.bits; qa.seed = cfg.seed; qa.step = cfg.step; qa.layer = cfg.layer_id;
  // Kept fraction of the elements: 1 without AGP; with AGP about 1 - (1 - 1/b)^2 (G/b
  // groups of each encoding kept), above 3/4 for b <= 2.
  qa.eager = (cfg.agp_mode == FQT_AGP_OFF || cfg.bits <= 2) ? 1u : 0u;
  qa.planes = write_planes ? 1u : 0u;
  dispatch_dtype(L.dy_t, [&]<int DT>() {
    if (mode == TILE_PIX)
      hipLaunchKernelGGL((k_qpack<TILE_PIX, DT>), qgrid, dim3(THREADS), 0, s, qa);
    else if (mode == TILE_CHAN)
      hipLaunchKernelGGL((k_qpack<TILE_CHAN, DT>), qgrid, dim3(THREADS), 0, s, qa);
    else
      hipLaunchKernelGGL((k_qpack<TILE_SCALAR, DT>), qgrid, dim3(THREADS), 0, s, qa);
  });
  return last_launch_status();
}

}  // namespace fqt
