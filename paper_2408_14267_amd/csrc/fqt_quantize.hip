// AGP + SCQ quantization of the output gradient dY on gfx950.
//
//   k_stats         one pass over dY in 64 (channel) x 64 (unfolded row r = n*P + pixel)
//                   tiles: per-tile min/max of every channel row and every r column,
//                   written as partials (no atomics: same-address atomics from the
//                   eight XCDs serialise at the memory side)
//   k_stats_reduce  one workgroup per group: min/max of its partials
//                   (Section 3.2 range and zero point; Section 5.2 / 5.3 groups)
//   k_select        one workgroup per group set: AGP keep probabilities, Bernoulli
//                   masks, kept-id compaction, scale/offset (Section 5.2, AGP)
//   k_qpack         second pass over dY: stochastic rounding of every element of a
//                   kept sample / kept channel, bit-plane split and packing, and the
//                   byte codes the MFMA products read
//                   (Section 3.2 SR; Section 5.2 decomposition; Appendix C encoders)
//
// A tile holds whole 64-bit words of both packings: a PSQ word runs along the 64
// channels of one row r, a PCQ word along the 64 rows of one channel.
#include <climits>

#include "fqt_internal.hpp"

namespace fqt {
namespace {

constexpr int TILE = 64;
constexpr int THREADS = 512;                 // tile kernels: 8 elements (2 quads) per thread
constexpr int WAVES = THREADS / 64;
constexpr int QUADS = TILE * TILE / (4 * THREADS);
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

__device__ __forceinline__ int wave_min(int v) {
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ int wave_max(int v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
  return v;
}

// ----------------------------------------------------------------------------- stats

template <int MODE, int DT>
__global__ __launch_bounds__(THREADS) void k_stats(const void *__restrict__ dy,
                                                   TileGeom g, uint32_t nrt,
                                                   int2 *__restrict__ part_c,
                                                   int2 *__restrict__ part_s) {
  __shared__ int32_t key[TILE][TILE + 1];
  __shared__ int32_t pmin[WAVES][TILE], pmax[WAVES][TILE];
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const uint32_t r0 = blockIdx.x * TILE, d0 = blockIdx.y * TILE;

  if (MODE != TILE_SCALAR) {
    float x[QUADS][4];
    bool ok[QUADS];
    for (int q = 0; q < QUADS; ++q) {
      int dd, rr;
      quad_coord<MODE>(t, q, 0, dd, rr);
      ok[q] = d0 + dd < g.D && r0 + rr < g.R;      // quads are all-valid or all-invalid
      // Unconditional (element 0 outside the layer) so the loads issue back to back.
      load_quad<DT>(dy, ok[q] ? elem_index(g, d0 + dd, r0 + rr) : 0, x[q]);
    }
    for (int q = 0; q < QUADS; ++q) {
      if (!ok[q]) continue;
      for (int k = 0; k < 4; ++k) {
        int dk, rk;
        quad_coord<MODE>(t, q, k, dk, rk);
        key[dk][rk] = f2key(x[q][k] + 0.0f);
      }
    }
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
  // Channel rows of the tile: reduce over the tile's 64 rows r.
  for (int i = 0; i < TILE / WAVES; ++i) {
    const int dd = wave + WAVES * i;
    const uint32_t d = d0 + dd;
    if (d >= g.D) break;
    const int k = key[dd][lane];
    const int lo = wave_min(row_ok ? k : INT_MAX);
    const int hi = wave_max(row_ok ? k : INT_MIN);
    if (lane == 0) part_c[size_t(d) * nrt + blockIdx.x] = make_int2(lo, hi);
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
  if (wave == 0 && row_ok) {
    for (int v = 1; v < WAVES; ++v) {
      lo = min(lo, pmin[v][lane]);
      hi = max(hi, pmax[v][lane]);
    }
    part_s[size_t(blockIdx.y) * g.R + r0 + lane] = make_int2(lo, hi);
  }
}

// Block b < N reduces sample b over part_s[*][b*P .. b*P+P); block N + d reduces
// channel d over part_c[d][*].
constexpr int RED_THREADS = 256;
__global__ __launch_bounds__(RED_THREADS) void k_stats_reduce(const int2 *__restrict__ part_c,
                                                          const int2 *__restrict__ part_s,
                                                          uint32_t N, uint32_t P, uint32_t R,
                                                          uint32_t nrt, uint32_t ndt,
                                                          int2 *__restrict__ skey,
                                                          int2 *__restrict__ ckey) {
  __shared__ int32_t smn[RED_THREADS / 64], smx[RED_THREADS / 64];
  const uint32_t b = blockIdx.x;
  int lo = INT_MAX, hi = INT_MIN;
  if (b < N) {
    for (uint32_t dt = 0; dt < ndt; ++dt)
      for (uint32_t p = threadIdx.x; p < P; p += RED_THREADS) {
        const int2 v = part_s[size_t(dt) * R + b * P + p];
        lo = min(lo, v.x);
        hi = max(hi, v.y);
      }
  } else {
    const uint32_t d = b - N;
    for (uint32_t i = threadIdx.x; i < nrt; i += RED_THREADS) {
      const int2 v = part_c[size_t(d) * nrt + i];
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
  const int2 *key;     // [G] (min, max) keys
  int32_t G;
  uint32_t stream;
  int32_t *kept;
  int32_t *count;
  float *scale, *offset, *prob;
  GroupParam *gp;
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

  // The first group of each thread is read once and kept in registers (G <= NT: all).
  const int2 own = t < G ? S.key[t] : make_int2(0, 0);
#define GROUP_KEY(i) ((i) == t ? own : S.key[(i)])
  float rmax = 0.0f;
  for (int i = t; i < G; i += NT) rmax = fmaxf(rmax, group_range(GROUP_KEY(i)));
  rmax = block_max_f<NT>(rmax, scr_f);

  int64_t s_sat = 0;           // number of saturated groups (p capped at 1)
  uint64_t w_thr = 0;          // weight of the last saturated group
  uint64_t w_rem = 0;          // weight of the unsaturated groups
  uint64_t key_thr = 0;        // TOPK: smallest kept sort key
  if (a.mode != FQT_AGP_OFF) {
    for (int i = t; i < GP; i += NT)
      skey[i] = i < G ? sort_key(agp_weight(group_range(GROUP_KEY(i)), rmax), i) : 0ull;
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
  const int chunk = (G + NT - 1) / NT;       // <= 16 for G <= 16384 and NT >= 1024
  const int i0 = t * chunk;
  const int i1 = min(i0 + chunk, G);
  uint32_t keepbits = 0;
  int32_t nkeep = 0;
  for (int i = i0; i < i1; ++i) {
    bool keep;
    if (a.mode == FQT_AGP_OFF) {
      keep = true;
    } else {
      const uint64_t w = agp_weight(group_range(GROUP_KEY(i)), rmax);
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
    keepbits |= (keep ? 1u : 0u) << (i - i0);
    nkeep += keep ? 1 : 0;
  }
  int32_t count;
  int32_t rank = block_exscan<NT, int32_t>(nkeep, scr_i, count);
  if (t == 0) *S.count = count;
  for (int i = i0; i < i1; ++i) {
    const bool keep = (keepbits >> (i - i0)) & 1u;
    const int2 k = GROUP_KEY(i);
    const float R = group_range(k);
    const float Z = key2f(k.x);
    float Sc = 0.0f, Zp = 0.0f, p = 0.0f;
    bool unit_p = a.mode != FQT_AGP_BERNOULLI;
    uint64_t w = 0;
    if (a.mode == FQT_AGP_BERNOULLI) {
      w = agp_weight(R, rmax);
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
#undef GROUP_KEY
}

// ----------------------------------------------------------------------------- quantize + pack

// b-bit stochastic rounding code of x (Section 3.2): v = clamp((x - Z) * inv, 0, B),
// q = floor(v) + [u24 < frac(v) * 2^24].  inv = 0 (R = 0) gives q = 0.
__device__ __forceinline__ uint32_t sr_code(float x, float z, float inv, float Bf, uint32_t u) {
  float v = __fmul_rn(__fsub_rn(x, z), inv);
  v = fminf(fmaxf(v, 0.0f), Bf);
  const float fl = floorf(v);
  const float fr = v - fl;
  return static_cast<uint32_t>(fl) + (static_cast<float>(u >> 8) < fr * 16777216.0f ? 1u : 0u);
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
};

template <int MODE, int DT>
__global__ __launch_bounds__(THREADS) void k_qpack(QPackArgs a) {
  __shared__ uint8_t cs[TILE][PITCH];   // PSQ codes, [rr][dd]
  __shared__ uint8_t cc[TILE][PITCH];   // PCQ codes, [dd][rr]
  __shared__ GroupParam spar[TILE];     // sample params of each column rr
  __shared__ GroupParam cpar[TILE];     // channel params of each row dd
  __shared__ int32_t prow[TILE];        // PSQ row of column rr, -1 if pruned/outside
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const TileGeom &g = a.g;
  const uint32_t r0 = blockIdx.x * TILE, d0 = blockIdx.y * TILE;
  const float Bf = float((1 << a.bits) - 1);

  if (t < TILE) {
    const uint32_t r = r0 + t;
    GroupParam p;
    p.z = 0.0f; p.inv = 0.0f; p.rank = -1; p.pad = 0;
    int32_t row = -1;
    if (r < g.R) {
      const uint32_t n = fdiv(r, g.divP);
      p = a.sp[n];
      if (p.rank >= 0) row = int32_t(uint32_t(p.rank) * g.P + (r - n * g.P));
    }
    spar[t] = p;
    prow[t] = row;
  } else if (t < 2 * TILE) {
    const uint32_t d = d0 + (t - TILE);
    GroupParam p;
    p.z = 0.0f; p.inv = 0.0f; p.rank = -1; p.pad = 0;
    if (d < g.D) p = a.cp[d];
    cpar[t - TILE] = p;
  }
  __syncthreads();

  if (MODE != TILE_SCALAR) {
    float x[QUADS][4];
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
      load_quad<DT>(a.dy, nd ? elem_index(g, d0 + dd, r0 + rr) : 0, x[q]);
    }
    for (int q = 0; q < QUADS; ++q) {
      int dd, rr;
      quad_coord<MODE>(t, q, 0, dd, rr);
      uint32_t qs[4] = {0, 0, 0, 0}, qc[4] = {0, 0, 0, 0};
      if (need[q]) {
        const uint32_t e = elem_index(g, d0 + dd, r0 + rr);
        const Ctr4 u = philox_block(e >> 2, STREAM_ELEM, a.seed, a.step, a.layer);
        for (int k = 0; k < 4; ++k) {
          const int dk = MODE == TILE_CHAN ? dd + k : dd;
          const int rk = MODE == TILE_PIX ? rr + k : rr;
          const float xv = x[q][k] + 0.0f;
          const GroupParam ps = spar[rk], pc = cpar[dk];
          if (ps.rank >= 0) qs[k] = sr_code(xv, ps.z, ps.inv, Bf, u.v[k]);
          if (pc.rank >= 0) qc[k] = sr_code(xv, pc.z, pc.inv, Bf, u.v[k]);
        }
      }
      for (int k = 0; k < 4; ++k) {
        int dk, rk;
        quad_coord<MODE>(t, q, k, dk, rk);
        cs[rk][dk] = uint8_t(qs[k]);
        cc[dk][rk] = uint8_t(qc[k]);
      }
    }
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
        const uint32_t uw = ctr_word(u, e & 3u);
        if (ps.rank >= 0) qs = sr_code(xv, ps.z, ps.inv, Bf, uw);
        if (pc.rank >= 0) qc = sr_code(xv, pc.z, pc.inv, Bf, uw);
      }
      cs[rr][dd] = uint8_t(qs);
      cc[dd][rr] = uint8_t(qc);
    }
  }
  __syncthreads();

  // PCQ: channel row dd of the tile, lanes along r (column encoder) and its 64 code bytes.
  for (int i = 0; i < TILE / WAVES; ++i) {
    const int dd = wave + WAVES * i;
    if (d0 + dd >= g.D) break;
    const int rank = cpar[dd].rank;
    if (rank < 0) continue;
    const uint32_t code = cc[dd][lane];
    for (int p = 0; p < a.bits; ++p) {
      const uint64_t m = __ballot((code >> p) & 1u);
      if (lane == p) a.pcq[(size_t(p) * g.D + rank) * a.Wr + (r0 >> 6)] = m;
    }
    if (lane < 16)        // lanes 0-7 fill 32-byte chunk r0/32, lanes 8-15 the next one
      *reinterpret_cast<uint32_t *>(
          a.pcq_codes + ((size_t(r0 >> 5) + (lane >> 3)) * g.D + rank) * 32 + 4 * (lane & 7)) =
          reinterpret_cast<const uint32_t *>(&cc[dd][0])[lane];
  }
  // PSQ: row rr of the tile, lanes along d (row encoder) and its 64 code bytes.
  for (int i = 0; i < TILE / WAVES; ++i) {
    const int rr = wave + WAVES * i;
    const int row = prow[rr];
    if (row < 0) continue;
    const uint32_t code = cs[rr][lane];
    for (int p = 0; p < a.bits; ++p) {
      const uint64_t m = __ballot((code >> p) & 1u);
      if (lane == p) a.psq[(size_t(p) * g.R + row) * a.Wd + (d0 >> 6)] = m;
    }
    if (lane < 16)
      *reinterpret_cast<uint32_t *>(
          a.psq_codes + ((size_t(d0 >> 5) + (lane >> 3)) * g.R + row) * 32 + 4 * (lane & 7)) =
          reinterpret_cast<const uint32_t *>(&cs[rr][0])[lane];
  }
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

int launch_quantize(const Layer &L, const fqt_quant_cfg &cfg, const void *dY, const fqt_qgrad &q,
                    const QuantWs &w, hipStream_t s) {
  TileGeom g{uint32_t(L.D), uint32_t(L.P), uint32_t(L.R), make_fastdiv(uint32_t(L.P))};
  const uint32_t nrt = uint32_t(L.Wr), ndt = uint32_t(L.Wd);
  const dim3 grid(nrt, ndt);
  const int mode = (L.P % 4 == 0) ? TILE_PIX : (L.P == 1 && L.D % 4 == 0) ? TILE_CHAN : TILE_SCALAR;
  dispatch_dtype(L.dy_t, [&]<int DT>() {
    if (mode == TILE_PIX)
      hipLaunchKernelGGL((k_stats<TILE_PIX, DT>), grid, dim3(THREADS), 0, s, dY, g, nrt, w.part_c,
                         w.part_s);
    else if (mode == TILE_CHAN)
      hipLaunchKernelGGL((k_stats<TILE_CHAN, DT>), grid, dim3(THREADS), 0, s, dY, g, nrt,
                         w.part_c, w.part_s);
    else
      hipLaunchKernelGGL((k_stats<TILE_SCALAR, DT>), grid, dim3(THREADS), 0, s, dY, g, nrt,
                         w.part_c, w.part_s);
  });
  if (last_launch_status() != FQT_OK) return FQT_E_HIP;
  hipLaunchKernelGGL(k_stats_reduce, dim3(unsigned(L.N + L.D)), dim3(RED_THREADS), 0, s, w.part_c,
                     w.part_s, uint32_t(L.N), uint32_t(L.P), uint32_t(L.R), nrt, ndt, w.skey,
                     w.ckey);
  if (last_launch_status() != FQT_OK) return FQT_E_HIP;

  SelectArgs sa;
  sa.set[0] = SetArgs{w.skey, int32_t(L.N), STREAM_SAMPLE, q.psq_kept, q.psq_count, q.psq_scale,
                      q.psq_offset, q.psq_prob, w.sp};
  sa.set[1] = SetArgs{w.ckey, int32_t(L.D), STREAM_CHANNEL, q.pcq_kept, q.pcq_count, q.pcq_scale,
                      q.pcq_offset, q.pcq_prob, w.cp};
  sa.bits = cfg.bits; sa.mode = cfg.agp_mode; sa.seed = cfg.seed; sa.step = cfg.step;
  sa.layer = cfg.layer_id;
  const int64_t gmax = L.N > L.D ? L.N : L.D;
  int st;
  if (gmax <= 256) st = launch_select<256, 256>(sa, s);
  else if (gmax <= 1024) st = launch_select<1024, 1024>(sa, s);
  else if (gmax <= 4096) st = launch_select<4096, 1024>(sa, s);
  else st = launch_select<16384, 1024>(sa, s);
  if (st != FQT_OK) return st;

  QPackArgs qa;
  qa.dy = dY; qa.g = g; qa.sp = w.sp; qa.cp = w.cp;
  qa.psq = q.psq_planes; qa.pcq = q.pcq_planes;
  qa.psq_codes = q.psq_codes; qa.pcq_codes = q.pcq_codes;
  qa.Wd = uint32_t(L.Wd); qa.Wr = uint32_t(L.Wr);
  qa.bits = cfg.bits; qa.seed = cfg.seed; qa.step = cfg.step; qa.layer = cfg.layer_id;
  dispatch_dtype(L.dy_t, [&]<int DT>() {
    if (mode == TILE_PIX)
      hipLaunchKernelGGL((k_qpack<TILE_PIX, DT>), grid, dim3(THREADS), 0, s, qa);
    else if (mode == TILE_CHAN)
      hipLaunchKernelGGL((k_qpack<TILE_CHAN, DT>), grid, dim3(THREADS), 0, s, qa);
    else
      hipLaunchKernelGGL((k_qpack<TILE_SCALAR, DT>), grid, dim3(THREADS), 0, s, qa);
  });
  return last_launch_status();
}

}  // namespace fqt
