// AGP + SCQ quantization of the output gradient dY on gfx950.
//
//   k_init_stats  min/max keys of both group sets to their identities
//   k_stats       one pass over dY: per-sample and per-channel min/max
//                 (Section 3.2 range and zero point; Section 5.2 / 5.3 groups)
//   k_select      one workgroup per group set: AGP keep probabilities, Bernoulli
//                 masks, kept-id compaction, scale/offset (Section 5.2, AGP)
//   k_qpack       second pass over dY: stochastic rounding of every element of a
//                 kept sample / kept channel, bit-plane split and packing
//                 (Section 3.2 SR; Section 5.2 decomposition; Appendix C encoders)
//
// dY is read as 64 (channel) x 64 (unfolded row r = n*P + pixel) tiles.  A tile
// holds whole 64-bit words of both packings: a PSQ word runs along the 64
// channels of one row, a PCQ word along the 64 rows of one channel.
#include <climits>

#include "fqt_internal.hpp"

namespace fqt {
namespace {

constexpr int TILE = 64;
constexpr int THREADS = 256;
constexpr int LDS_PITCH = TILE + 4;   // bytes per code row; 68 keeps column reads conflict-free

// How a thread walks its 16 tile elements.
//  PIX    (P % 4 == 0): 4 consecutive rows r of one channel per quad, a 16-byte load
//  CHAN   (P == 1, D % 4 == 0): 4 consecutive channels of one row per quad
//  SCALAR otherwise: single elements
enum TileMode { TILE_PIX = 0, TILE_CHAN = 1, TILE_SCALAR = 2 };

struct TileGeom {
  int64_t D, P, R;
};

// Tile coordinates (dd, rr) of element k of quad q of thread t.
template <int MODE>
__device__ __forceinline__ void quad_coord(int t, int q, int k, int &dd, int &rr) {
  if (MODE == TILE_PIX) {
    dd = (t >> 4) + 16 * q;
    rr = 4 * (t & 15) + k;
  } else if (MODE == TILE_CHAN) {
    dd = 4 * (t & 15) + k;
    rr = (t >> 4) + 16 * q;
  } else {
    const int idx = t + THREADS * (4 * q + k);
    dd = idx >> 6;
    rr = idx & 63;
  }
}

__device__ __forceinline__ int64_t elem_index(const TileGeom &g, int64_t d, int64_t r) {
  const int64_t n = r / g.P;
  const int64_t pix = r - n * g.P;
  return (n * g.D + d) * g.P + pix;
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

__global__ void k_init_stats(int32_t *smin, int32_t *smax, int64_t N, int32_t *cmin,
                             int32_t *cmax, int64_t D) {
  const int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  if (i < N) {
    smin[i] = INT_MAX;
    smax[i] = INT_MIN;
  }
  if (i < D) {
    cmin[i] = INT_MAX;
    cmax[i] = INT_MIN;
  }
}

template <int MODE>
__global__ __launch_bounds__(THREADS) void k_stats(const void *__restrict__ dy, int dtype,
                                                   TileGeom g, int32_t *smin, int32_t *smax,
                                                   int32_t *cmin, int32_t *cmax) {
  __shared__ int32_t key[TILE][TILE + 1];
  __shared__ int32_t pmin[4][TILE], pmax[4][TILE];
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int64_t r0 = int64_t(blockIdx.x) * TILE, d0 = int64_t(blockIdx.y) * TILE;

  for (int q = 0; q < 4; ++q) {
    if (MODE != TILE_SCALAR) {
      int dd, rr;
      quad_coord<MODE>(t, q, 0, dd, rr);
      const int64_t d = d0 + dd, r = r0 + rr;
      if (d < g.D && r < g.R) {           // quads are all-valid or all-invalid
        float x[4];
        load_quad(dy, dtype, elem_index(g, d, r), x);
        for (int k = 0; k < 4; ++k) {
          int dk, rk;
          quad_coord<MODE>(t, q, k, dk, rk);
          key[dk][rk] = f2key(x[k] + 0.0f);
        }
      }
    } else {
      for (int k = 0; k < 4; ++k) {
        int dd, rr;
        quad_coord<MODE>(t, q, k, dd, rr);
        const int64_t d = d0 + dd, r = r0 + rr;
        if (d < g.D && r < g.R) key[dd][rr] = f2key(load_elem(dy, dtype, elem_index(g, d, r)) + 0.0f);
      }
    }
  }
  __syncthreads();

  const bool row_ok = r0 + lane < g.R;
  // Channel groups: wave-reduce each tile row over its 64 rows r.
  for (int i = 0; i < 16; ++i) {
    const int dd = wave + 4 * i;
    const int64_t d = d0 + dd;
    if (d >= g.D) break;
    const int k = key[dd][lane];
    const int lo = wave_min(row_ok ? k : INT_MAX);
    const int hi = wave_max(row_ok ? k : INT_MIN);
    if (lane == 0) {
      atomicMin(&cmin[d], lo);
      atomicMax(&cmax[d], hi);
    }
  }
  // Sample groups: column reduce over channels, then a segmented reduce over the
  // lanes of each sample (a tile may span several samples when P < 64).
  int lo = INT_MAX, hi = INT_MIN;
  for (int i = 0; i < 16; ++i) {
    const int dd = 16 * wave + i;
    if (d0 + dd >= g.D) break;
    const int k = key[dd][lane];
    lo = min(lo, k);
    hi = max(hi, k);
  }
  pmin[wave][lane] = lo;
  pmax[wave][lane] = hi;
  __syncthreads();
  if (wave == 0) {
    lo = min(min(pmin[0][lane], pmin[1][lane]), min(pmin[2][lane], pmin[3][lane]));
    hi = max(max(pmax[0][lane], pmax[1][lane]), max(pmax[2][lane], pmax[3][lane]));
    const int64_t n = row_ok ? (r0 + lane) / g.P : -1;
    for (int o = 1; o < 64; o <<= 1) {
      const int lo2 = __shfl_down(lo, o);
      const int hi2 = __shfl_down(hi, o);
      const int64_t n2 = __shfl_down(n, o);
      if (lane + o < 64 && n2 == n) {
        lo = min(lo, lo2);
        hi = max(hi, hi2);
      }
    }
    const int64_t nprev = __shfl_up(n, 1);
    if (row_ok && (lane == 0 || nprev != n)) {
      atomicMin(&smin[n], lo);
      atomicMax(&smax[n], hi);
    }
  }
}

// ----------------------------------------------------------------------------- select

struct SelectArgs {
  const int32_t *kmin[2];
  const int32_t *kmax[2];
  int32_t G[2];
  int32_t *kept[2];
  int32_t *count[2];
  float *scale[2];
  float *offset[2];
  float *prob[2];
  GroupParam *gp[2];
  int bits, mode;
  uint64_t seed;
  uint32_t step, layer;
};

constexpr int SEL_THREADS = 1024;
constexpr int SEL_WAVES = SEL_THREADS / 64;
constexpr int ID_BITS = 14;                   // group ids < 2^14 = FQT_MAX_AGP_GROUPS

__device__ __forceinline__ float group_range(const int32_t *kmin, const int32_t *kmax, int i) {
  return (key2f(kmax[i]) - key2f(kmin[i])) + 0.0f;
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

template <typename T>
__device__ T block_sum(T v, T *scratch) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  T r = 0;
  for (int i = 0; i < SEL_WAVES; ++i) r += scratch[i];
  __syncthreads();
  return r;
}

__device__ float block_max_f(float v, float *scratch) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  float r = scratch[0];
  for (int i = 1; i < SEL_WAVES; ++i) r = fmaxf(r, scratch[i]);
  __syncthreads();
  return r;
}

// Exclusive prefix of `v` over thread order; `total` receives the block total.
template <typename T>
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
  for (int i = 0; i < SEL_WAVES; ++i) {
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

// One workgroup per group set (blockIdx.x = 0 samples, 1 channels).  GP is the
// power-of-two capacity of the LDS sort (>= G).
template <int GP>
__global__ __launch_bounds__(SEL_THREADS) void k_select(SelectArgs a) {
  extern __shared__ uint64_t skey[];
  __shared__ uint64_t scr_u[SEL_WAVES];
  __shared__ int32_t scr_i[SEL_WAVES];
  __shared__ float scr_f[SEL_WAVES];
  const int set = blockIdx.x;
  const int G = a.G[set];
  const int32_t *kmin = a.kmin[set], *kmax = a.kmax[set];
  const int t = threadIdx.x;
  const int b = a.bits;
  const int B = (1 << b) - 1;

  float rmax = 0.0f;
  for (int i = t; i < G; i += SEL_THREADS) rmax = fmaxf(rmax, group_range(kmin, kmax, i));
  rmax = block_max_f(rmax, scr_f);

  // Water-filling result (BERNOULLI) or top-k threshold (TOPK).
  int64_t s_sat = 0;           // number of saturated groups
  uint64_t w_thr = 0;          // weight of the last saturated group
  uint64_t w_rem = 0;          // weight of the unsaturated groups
  uint64_t key_thr = 0;        // TOPK: smallest kept sort key
  if (a.mode != FQT_AGP_OFF) {
    for (int i = t; i < GP; i += SEL_THREADS)
      skey[i] = i < G ? sort_key(agp_weight(group_range(kmin, kmax, i), rmax), i) : 0ull;
    __syncthreads();
    // Bitonic sort, descending.
    for (int k = 2; k <= GP; k <<= 1) {
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int i = t; i < GP; i += SEL_THREADS) {
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
      const int kk = max(1, G / b);
      key_thr = skey[kk - 1];
    } else {
      // Saturation test at sorted position s: (G - b s) w_(s) >= b * (sum of w at positions >= s).
      // It holds on a prefix of positions, so the number of positions passing is s_sat.
      const int chunk = (GP + SEL_THREADS - 1) / SEL_THREADS;
      const int p0 = t * chunk;
      uint64_t local = 0;
      for (int p = p0; p < min(p0 + chunk, G); ++p) local += skey[p] >> ID_BITS;
      uint64_t wtot;
      uint64_t excl = block_exscan<uint64_t>(local, scr_u, wtot);
      int32_t pass = 0;
      for (int p = p0; p < min(p0 + chunk, G); ++p) {
        const uint64_t w = skey[p] >> ID_BITS;
        const int64_t lhs = (int64_t(G) - int64_t(b) * p) * int64_t(w);
        const int64_t rhs = int64_t(b) * int64_t(wtot - excl);
        pass += (w > 0 && lhs >= rhs) ? 1 : 0;
        excl += w;
      }
      s_sat = block_sum<int32_t>(pass, scr_i);
      uint64_t rem = 0;
      for (int p = max(p0, int(s_sat)); p < min(p0 + chunk, G); ++p) rem += skey[p] >> ID_BITS;
      w_rem = block_sum<uint64_t>(rem, scr_u);
      w_thr = s_sat > 0 ? (skey[s_sat - 1] >> ID_BITS) : 0;
    }
  }

  // Masks in id order, then the stable partition kept-ascending | pruned-ascending.
  const int64_t A = int64_t(G) - int64_t(b) * s_sat;
  const int chunk = (G + SEL_THREADS - 1) / SEL_THREADS;
  const int i0 = t * chunk;
  const int i1 = min(i0 + chunk, G);
  uint32_t keepbits = 0;   // chunk <= 16 for G <= 16384
  int32_t nkeep = 0;
  for (int i = i0; i < i1; ++i) {
    bool keep;
    if (a.mode == FQT_AGP_OFF) {
      keep = true;
    } else {
      const uint64_t w = agp_weight(group_range(kmin, kmax, i), rmax);
      if (a.mode == FQT_AGP_TOPK) {
        keep = sort_key(w, i) >= key_thr;
      } else if (s_sat > 0 && w > 0 && w >= w_thr) {
        keep = true;
      } else if (A > 0 && w_rem > 0 && w > 0) {
        const Ctr4 u = philox_block(uint64_t(i) >> 2, set ? STREAM_CHANNEL : STREAM_SAMPLE,
                                    a.seed, a.step, a.layer);
        const uint32_t u32 = u.v[i & 3];
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
  int32_t rank = block_exscan<int32_t>(nkeep, scr_i, count);
  if (t == 0) *a.count[set] = count;
  for (int i = i0; i < i1; ++i) {
    const bool keep = (keepbits >> (i - i0)) & 1u;
    const float R = group_range(kmin, kmax, i);
    const float Z = key2f(kmin[i]);
    float S = 0.0f, Zp = 0.0f, p = 0.0f;
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
        S = static_cast<float>(static_cast<double>(R) / static_cast<double>(B));
        Zp = Z;
      } else {
        const double bw = static_cast<double>(uint64_t(b) * w_rem);
        const double aw = static_cast<double>(uint64_t(A) * w);
        S = static_cast<float>((static_cast<double>(R) * bw) / (static_cast<double>(B) * aw));
        Zp = static_cast<float>((static_cast<double>(Z) * bw) / aw);
      }
    }
    a.prob[set][i] = p;
    a.scale[set][i] = S;
    a.offset[set][i] = Zp + 0.0f;
    GroupParam gp;
    gp.z = Z;
    gp.inv = R > 0.0f ? __fdiv_rn(float(B), R) : 0.0f;
    gp.rank = keep ? rank : -1;
    gp.pad = 0;
    a.gp[set][i] = gp;
    if (keep) {
      a.kept[set][rank] = i;
      ++rank;
    } else {
      a.kept[set][count + (i - rank)] = i;
    }
  }
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
  int dtype;
  TileGeom g;
  const GroupParam *sp;
  const GroupParam *cp;
  uint64_t *psq;   // [bits][R][Wd]
  uint64_t *pcq;   // [bits][D][Wr]
  int64_t Wd, Wr;
  int bits;
  uint64_t seed;
  uint32_t step, layer;
};

template <int MODE>
__global__ __launch_bounds__(THREADS) void k_qpack(QPackArgs a) {
  __shared__ uint8_t cs[TILE][LDS_PITCH];   // PSQ codes [dd][rr]
  __shared__ uint8_t cc[TILE][LDS_PITCH];   // PCQ codes [dd][rr]
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const TileGeom &g = a.g;
  const int64_t r0 = int64_t(blockIdx.x) * TILE, d0 = int64_t(blockIdx.y) * TILE;
  const float Bf = float((1 << a.bits) - 1);

  for (int q = 0; q < 4; ++q) {
    if (MODE != TILE_SCALAR) {
      int dd, rr;
      quad_coord<MODE>(t, q, 0, dd, rr);
      const int64_t d = d0 + dd, r = r0 + rr;
      uint8_t qs[4] = {0, 0, 0, 0}, qc[4] = {0, 0, 0, 0};
      if (d < g.D && r < g.R) {
        const int64_t e = elem_index(g, d, r);
        GroupParam ps[4], pc[4];
        bool need = false;
        for (int k = 0; k < 4; ++k) {
          const int64_t dk = MODE == TILE_CHAN ? d + k : d;
          const int64_t rk = MODE == TILE_PIX ? r + k : r;
          ps[k] = a.sp[rk / g.P];
          pc[k] = a.cp[dk];
          need |= (ps[k].rank >= 0) | (pc[k].rank >= 0);
        }
        if (need) {
          float x[4];
          load_quad(a.dy, a.dtype, e, x);
          const Ctr4 u = philox_block(uint64_t(e) >> 2, STREAM_ELEM, a.seed, a.step, a.layer);
          for (int k = 0; k < 4; ++k) {
            const float xv = x[k] + 0.0f;
            if (ps[k].rank >= 0) qs[k] = uint8_t(sr_code(xv, ps[k].z, ps[k].inv, Bf, u.v[k]));
            if (pc[k].rank >= 0) qc[k] = uint8_t(sr_code(xv, pc[k].z, pc[k].inv, Bf, u.v[k]));
          }
        }
      }
      for (int k = 0; k < 4; ++k) {
        int dk, rk;
        quad_coord<MODE>(t, q, k, dk, rk);
        cs[dk][rk] = qs[k];
        cc[dk][rk] = qc[k];
      }
    } else {
      for (int k = 0; k < 4; ++k) {
        int dd, rr;
        quad_coord<MODE>(t, q, k, dd, rr);
        const int64_t d = d0 + dd, r = r0 + rr;
        uint8_t qs = 0, qc = 0;
        if (d < g.D && r < g.R) {
          const GroupParam ps = a.sp[r / g.P];
          const GroupParam pc = a.cp[d];
          if (ps.rank >= 0 || pc.rank >= 0) {
            const int64_t e = elem_index(g, d, r);
            const float xv = load_elem(a.dy, a.dtype, e) + 0.0f;
            const Ctr4 u = philox_block(uint64_t(e) >> 2, STREAM_ELEM, a.seed, a.step, a.layer);
            const uint32_t uw = u.v[e & 3];
            if (ps.rank >= 0) qs = uint8_t(sr_code(xv, ps.z, ps.inv, Bf, uw));
            if (pc.rank >= 0) qc = uint8_t(sr_code(xv, pc.z, pc.inv, Bf, uw));
          }
        }
        cs[dd][rr] = qs;
        cc[dd][rr] = qc;
      }
    }
  }
  __syncthreads();

  // PCQ words: channel row dd, lanes along r (column encoder).
  for (int i = 0; i < 16; ++i) {
    const int dd = wave + 4 * i;
    const int64_t d = d0 + dd;
    if (d >= g.D) break;
    const int rank = a.cp[d].rank;
    if (rank < 0) continue;
    const uint32_t code = cc[dd][lane];
    for (int p = 0; p < a.bits; ++p) {
      const uint64_t m = __ballot((code >> p) & 1u);
      if (lane == p) a.pcq[(int64_t(p) * g.D + rank) * a.Wr + (r0 >> 6)] = m;
    }
  }
  // PSQ words: row rr, lanes along d (row encoder).
  for (int i = 0; i < 16; ++i) {
    const int rr = wave + 4 * i;
    const int64_t r = r0 + rr;
    if (r >= g.R) break;
    const int64_t n = r / g.P;
    const int rank = a.sp[n].rank;
    if (rank < 0) continue;
    const uint32_t code = cs[lane][rr];
    const int64_t row = int64_t(rank) * g.P + (r - n * g.P);
    for (int p = 0; p < a.bits; ++p) {
      const uint64_t m = __ballot((code >> p) & 1u);
      if (lane == p) a.psq[(int64_t(p) * g.R + row) * a.Wd + (d0 >> 6)] = m;
    }
  }
}

template <int GP>
int launch_select(const SelectArgs &sa, hipStream_t s) {
  const size_t lds = size_t(GP) * sizeof(uint64_t);
  int dev = 0, max_lds = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return FQT_E_HIP;
  if (lds + 1024 > size_t(max_lds)) return FQT_E_SHAPE;   // the group set does not fit in LDS
  if (lds > 65536) {
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(&k_select<GP>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
      return FQT_E_HIP;
  }
  hipLaunchKernelGGL(k_select<GP>, dim3(2), dim3(SEL_THREADS), lds, s, sa);
  return last_launch_status();
}

}  // namespace

int launch_quantize(const Layer &L, const fqt_quant_cfg &cfg, const void *dY, const fqt_qgrad &q,
                    const QuantWs &w, hipStream_t s) {
  const int64_t gmax = L.N > L.D ? L.N : L.D;
  hipLaunchKernelGGL(k_init_stats, dim3(unsigned((gmax + 255) / 256)), dim3(256), 0, s, w.smin,
                     w.smax, L.N, w.cmin, w.cmax, L.D);
  if (last_launch_status() != FQT_OK) return FQT_E_HIP;

  TileGeom g{L.D, L.P, L.R};
  const dim3 grid(unsigned((L.R + TILE - 1) / TILE), unsigned((L.D + TILE - 1) / TILE));
  const int mode = (L.P % 4 == 0) ? TILE_PIX : (L.P == 1 && L.D % 4 == 0) ? TILE_CHAN : TILE_SCALAR;
  if (mode == TILE_PIX)
    hipLaunchKernelGGL(k_stats<TILE_PIX>, grid, dim3(THREADS), 0, s, dY, L.dy_t, g, w.smin, w.smax,
                       w.cmin, w.cmax);
  else if (mode == TILE_CHAN)
    hipLaunchKernelGGL(k_stats<TILE_CHAN>, grid, dim3(THREADS), 0, s, dY, L.dy_t, g, w.smin,
                       w.smax, w.cmin, w.cmax);
  else
    hipLaunchKernelGGL(k_stats<TILE_SCALAR>, grid, dim3(THREADS), 0, s, dY, L.dy_t, g, w.smin,
                       w.smax, w.cmin, w.cmax);
  if (last_launch_status() != FQT_OK) return FQT_E_HIP;

  SelectArgs sa;
  sa.kmin[0] = w.smin; sa.kmax[0] = w.smax; sa.G[0] = int32_t(L.N);
  sa.kmin[1] = w.cmin; sa.kmax[1] = w.cmax; sa.G[1] = int32_t(L.D);
  sa.kept[0] = q.psq_kept; sa.count[0] = q.psq_count; sa.scale[0] = q.psq_scale;
  sa.offset[0] = q.psq_offset; sa.prob[0] = q.psq_prob; sa.gp[0] = w.sp;
  sa.kept[1] = q.pcq_kept; sa.count[1] = q.pcq_count; sa.scale[1] = q.pcq_scale;
  sa.offset[1] = q.pcq_offset; sa.prob[1] = q.pcq_prob; sa.gp[1] = w.cp;
  sa.bits = cfg.bits; sa.mode = cfg.agp_mode; sa.seed = cfg.seed; sa.step = cfg.step;
  sa.layer = cfg.layer_id;
  int st;
  if (gmax <= 1024) st = launch_select<1024>(sa, s);
  else if (gmax <= 4096) st = launch_select<4096>(sa, s);
  else st = launch_select<16384>(sa, s);
  if (st != FQT_OK) return st;

  QPackArgs qa;
  qa.dy = dY; qa.dtype = L.dy_t; qa.g = g; qa.sp = w.sp; qa.cp = w.cp;
  qa.psq = q.psq_planes; qa.pcq = q.pcq_planes; qa.Wd = L.Wd; qa.Wr = L.Wr;
  qa.bits = cfg.bits; qa.seed = cfg.seed; qa.step = cfg.step; qa.layer = cfg.layer_id;
  if (mode == TILE_PIX) hipLaunchKernelGGL(k_qpack<TILE_PIX>, grid, dim3(THREADS), 0, s, qa);
  else if (mode == TILE_CHAN) hipLaunchKernelGGL(k_qpack<TILE_CHAN>, grid, dim3(THREADS), 0, s, qa);
  else hipLaunchKernelGGL(k_qpack<TILE_SCALAR>, grid, dim3(THREADS), 0, s, qa);
  return last_launch_status();
}

}  // namespace fqt
