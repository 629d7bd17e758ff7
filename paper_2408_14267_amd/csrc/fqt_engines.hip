// Two further engines for the weight-gradient product, both reading the paper's packed
// operands: the PCQ code planes (Section 5.2's lossless decomposition q = sum_p 2^p q_p,
// packed along N*Ho*Wo by the column encoder) and sign(unfold(X)) packed along the same
// contraction (Appendix C, Alg. 2 and the Unfolder), with its line sums.
//
//   I[j][k] = sum_r q_j(r) s_k(r) = sum_p 2^p (2 popc(a_p & t) - popc(a_p))      (App. C)
//   dW[kept_j][k] = S_j I + Z'_j c_k,  c_k = sum_r s_k(r) = 2 popc(t) - R
//
// FQT_ENGINE_POPCOUNT (the paper's own engine, on the VALU): AND + v_bcnt over 64-bit words,
//   tiled through LDS, 4 x 4 outputs per thread.
// FQT_ENGINE_FP4 (gfx950 matrix cores): both operands expanded once to e2m1 nibbles, a code
//   bit as 1.0 (0x2) or 0.0 and a sign bit t as 1.0 or 0.0, so that one
//   v_mfma_scale_f32_32x32x64_f8f6f4 per plane (its A scale 2^p carries the plane weight)
//   gives sum_p 2^p sum_r a_p t exactly in float32 (integers below 2^24), and
//   I = 2 sum q t - sum q.  The expansion writes a chunk-major layout ([64-position step]
//   [row][32 bytes]) so that a wave's operand load reads 1 KB of contiguous memory.
#include "fqt_internal.hpp"

namespace fqt {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int acc_row(int v, int g) { return 8 * (v >> 2) + 4 * g + (v & 3); }
__device__ __forceinline__ float rescale(float S, int I, float Zp, float c) {
  return __fadd_rn(__fmul_rn(S, float(I)), __fmul_rn(Zp, c));
}

struct PlaneArgs {
  const uint64_t *planes;        // [b][D][Wr] PCQ code planes, kept channels compacted
  const int32_t *kept, *count;   // [D], [1]
  const float *scale, *offset;   // [D] by channel id
  const uint64_t *xbits;         // [K][Wr] sign(unfold(X)) along N*Ho*Wo
  const int32_t *xsum;           // [K] 2 popc - N*Ho*Wo
  int32_t *qsum;                 // [D] sum of the codes of kept slot j
  float *dW;                     // [D][K]
  int32_t *I_out;
  uint32_t D, K, Wr, bits;
};

// Sum of the codes of every kept slot (slots >= count get 0): sum_p 2^p popc over the row.
__global__ __launch_bounds__(256) void k_code_sums(PlaneArgs a) {
  const uint32_t j = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (j >= a.D) return;
  const int count = *a.count;
  uint32_t s = 0;
  if (int(j) < count)
    for (uint32_t p = 0; p < a.bits; ++p)
      for (uint32_t w = lane; w < a.Wr; w += 64)
        s += uint32_t(__popcll(a.planes[(size_t(p) * a.D + j) * a.Wr + w])) << p;
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m);
  if (lane == 0) a.qsum[j] = int32_t(s);
}

// The epilogue of both engines for one output: I from sum q t, the rescale, the stores.
__device__ __forceinline__ void plane_store(const PlaneArgs &a, uint32_t j, uint32_t k, int count,
                                            int qt) {
  if (j >= a.D || k >= a.K) return;
  const size_t d = size_t(a.kept[j]);
  int I = 0;
  float out = 0.0f;
  if (int(j) < count) {
    I = 2 * qt - a.qsum[j];
    out = rescale(a.scale[d], I, a.offset[d], float(a.xsum[k]));
  }
  a.dW[d * a.K + k] = out;
  if (a.I_out) a.I_out[d * a.K + k] = I;
}

// ----------------------------------------------------------------------------- popcount

constexpr int PC_T = 64;            // output tile: 64 slots x 64 columns, 256 threads
constexpr int PC_KW = 8;            // words of the contraction per LDS stage
template <int BITS>
__global__ __launch_bounds__(256) void k_popc_dw(PlaneArgs a) {
  __shared__ uint64_t As[BITS][PC_T][PC_KW + 1];
  __shared__ uint64_t Bs[PC_T][PC_KW + 1];
  const int t = threadIdx.x, tr = t >> 4, tc = t & 15;
  const uint32_t j0 = blockIdx.y * PC_T, k0 = blockIdx.x * PC_T;
  const int count = *a.count;
  uint32_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[i][c] = 0u;
  if (int(j0) < count) {
    for (uint32_t w0 = 0; w0 < a.Wr; w0 += PC_KW) {
      // Stage the plane words of the block's 64 slots and the sign words of its 64 columns.
      for (int idx = t; idx < BITS * PC_T * PC_KW; idx += 256) {
        const int p = idx / (PC_T * PC_KW), rr = (idx / PC_KW) % PC_T, ww = idx % PC_KW;
        const uint32_t j = j0 + rr, w = w0 + ww;
        As[p][rr][ww] = (int(j) < count && w < a.Wr) ? a.planes[(size_t(p) * a.D + j) * a.Wr + w] : 0ull;
      }
      for (int idx = t; idx < PC_T * PC_KW; idx += 256) {
        const int cc = idx / PC_KW, ww = idx % PC_KW;
        const uint32_t k = k0 + cc, w = w0 + ww;
        Bs[cc][ww] = (k < a.K && w < a.Wr) ? a.xbits[size_t(k) * a.Wr + w] : 0ull;
      }
      __syncthreads();
#pragma unroll
      for (int ww = 0; ww < PC_KW; ++ww) {
        uint64_t bv[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) bv[c] = Bs[tc + 16 * c][ww];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
          for (int p = 0; p < BITS; ++p) {
            const uint64_t av = As[p][4 * tr + i][ww];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              const uint64_t m = av & bv[c];
              if (p == 0) acc[i][c] += __popc(uint32_t(m)) + __popc(uint32_t(m >> 32));
              else acc[i][c] += uint32_t(__popc(uint32_t(m)) + __popc(uint32_t(m >> 32))) << p;
            }
          }
        }
      }
      __syncthreads();
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) plane_store(a, j0 + 4 * tr + i, k0 + tc + 16 * c, count, int(acc[i][c]));
}

// ----------------------------------------------------------------------------- fp4

// Bits -> e2m1 nibbles (bit 1 -> 0x2 = 1.0, bit 0 -> 0x0), chunk-major: word w of line l
// (64 positions) becomes the 32 bytes at (w * Lp + l) * 32, byte m holding positions 2m
// (low nibble) and 2m + 1.  Lines l < L come from src [L][Wr]; lines L <= l < Lp are zero.
// One thread per (word, line); the lines of a word are consecutive threads, so both the
// reads (stride Wr words) and the 32-byte writes of a wave cover contiguous memory on the
// written side.
__global__ __launch_bounds__(256) void k_bits_to_fp4(const uint64_t *__restrict__ src,
                                                     uint32_t L, uint32_t Lp, uint32_t Wr,
                                                     uint8_t *__restrict__ dst) {
  const uint64_t e = uint64_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= uint64_t(Wr) * Lp) return;
  const uint32_t w = uint32_t(e / Lp), l = uint32_t(e - uint64_t(w) * Lp);
  const uint64_t x = l < L ? src[size_t(l) * Wr + w] : 0ull;
  uint32_t out[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    // Byte m of dword q: positions 8q + 2m and 8q + 2m + 1.  A nibble pair from two bits:
    // bit0 * 0x02 | bit1 * 0x20.
    const uint32_t b8 = uint32_t(x >> (8 * q)) & 0xFFu;
    uint32_t v = 0;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const uint32_t two = (b8 >> (2 * m)) & 3u;
      v |= ((two & 1u) * 0x02u | (two >> 1) * 0x20u) << (8 * m);
    }
    out[q] = v;
  }
  uint4 *o = reinterpret_cast<uint4 *>(dst + (size_t(w) * Lp + l) * 32);
  o[0] = make_uint4(out[0], out[1], out[2], out[3]);
  o[1] = make_uint4(out[4], out[5], out[6], out[7]);
}

struct Fp4Args {
  PlaneArgs p;
  const uint8_t *A;              // [b][Wr][Dp][32] nibbles of the code planes
  const uint8_t *B;              // [Wr][Kp][32] nibbles of the sign bits (t = 1 for +1)
  uint32_t Dp, Kp, a_bytes, b_bytes, kgroups;
};

// The e2m1 operand of the scaled MFMA: four dwords (32 nibbles) per lane; the instruction
// reads no more for fp4.
__device__ __forceinline__ v8i as_v8(v4i v) { return v8i{v.x, v.y, v.z, v.w, 0, 0, 0, 0}; }

// Wave tile 64 x 64 (2 x 2 MFMA tiles); a block's four waves take four adjacent column
// tiles of the same 64 slots.  Grid: ceil(Dp / 64) slot blocks (slowest) x ceil(Kp / 256).
template <int BITS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_fp4_dw(Fp4Args f) {
  const PlaneArgs &a = f.p;
  const int lane = threadIdx.x & 63, i = lane & 31, g = lane >> 5;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t rb = blockIdx.x / f.kgroups;
  const uint32_t j0 = rb * 64;
  const uint32_t k0 = ((blockIdx.x - rb * f.kgroups) * 4 + wave) * 64;
  const int count = *a.count;
  if (k0 >= a.K) return;
  v16f acc[2][2];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int c = 0; c < 2; ++c) acc[r][c] = v16f{0};
  if (int(j0) < count) {
    const __amdgpu_buffer_rsrc_t ars = buffer_of(f.A, f.a_bytes);
    const __amdgpu_buffer_rsrc_t brs = buffer_of(f.B, f.b_bytes);
    uint32_t aoff[2], boff[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const uint32_t j = j0 + 32 * r + i;
      aoff[r] = int(j) < count ? j * 32 + 16 * g : BUF_NONE;
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const uint32_t k = k0 + 32 * c + i;
      boff[c] = k < a.K ? k * 32 + 16 * g : BUF_NONE;
    }
    constexpr int ST = BITS <= 2 ? 2 : 1;     // 64-position steps per batch, double-buffered
    v4i Ab[2][ST][BITS][2], Bb[2][ST][2];
    auto issue = [&](int buf, uint32_t s0) {
#pragma unroll
      for (int u = 0; u < ST; ++u) {
        const uint32_t s = min(s0 + u, a.Wr - 1);
        const uint32_t bs = __builtin_amdgcn_readfirstlane(s * f.Kp * 32);
#pragma unroll
        for (int c = 0; c < 2; ++c) Bb[buf][u][c] = load16(brs, boff[c], bs);
#pragma unroll
        for (int p = 0; p < BITS; ++p) {
          const uint32_t as = __builtin_amdgcn_readfirstlane((uint32_t(p) * a.Wr + s) * f.Dp * 32);
#pragma unroll
          for (int r = 0; r < 2; ++r) Ab[buf][u][p][r] = load16(ars, aoff[r], as);
        }
      }
    };
    auto consume = [&](int buf, uint32_t s0) {
#pragma unroll
      for (int u = 0; u < ST; ++u) {
        if (s0 + u >= a.Wr) break;
#pragma unroll
        for (int p = 0; p < BITS; ++p)
#pragma unroll
          for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int c = 0; c < 2; ++c)
              acc[r][c] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                  as_v8(Ab[buf][u][p][r]), as_v8(Bb[buf][u][c]), acc[r][c], 4, 4, 0, 127 + p, 0,
                  127);
      }
    };
    issue(0, 0);
    for (uint32_t s0 = 0; s0 < a.Wr; s0 += 2 * ST) {
      if (s0 + ST < a.Wr) issue(1, s0 + ST);
      __builtin_amdgcn_sched_barrier(0);
      consume(0, s0);
      if (s0 + 2 * ST < a.Wr) issue(0, s0 + 2 * ST);
      __builtin_amdgcn_sched_barrier(0);
      if (s0 + ST < a.Wr) consume(1, s0 + ST);
    }
  }
  // Every partial sum is an integer below 2^24 (checked on the host), so the float32
  // accumulators hold sum q t exactly.
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        plane_store(a, j0 + 32 * r + uint32_t(acc_row(v, g)), k0 + 32 * c + i, count,
                    int(acc[r][c][v]));
}

}  // namespace

size_t engine_ws_bytes(const Layer &L, const fqt_quant_cfg &cfg, int engine) {
  const size_t Dp = size_t((L.D + 63) / 64) * 64, Kp = size_t((L.K + 255) / 256) * 256;
  size_t n = align256(size_t(L.D) * 4);                           // code sums
  if (engine == FQT_ENGINE_FP4)
    n += align256(size_t(cfg.bits) * L.Wr * Dp * 32) + align256(size_t(L.Wr) * Kp * 32);
  return n;
}

int launch_gemm_dw_planes(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                          const uint64_t *xbits, const int32_t *xsum, float *dW, int32_t *I_out,
                          int engine, void *ws, hipStream_t s) {
  PlaneArgs a;
  a.planes = q.pcq_planes; a.kept = q.pcq_kept; a.count = q.pcq_count;
  a.scale = q.pcq_scale; a.offset = q.pcq_offset; a.xbits = xbits; a.xsum = xsum;
  a.qsum = static_cast<int32_t *>(ws);
  a.dW = dW; a.I_out = I_out;
  a.D = uint32_t(L.D); a.K = uint32_t(L.K); a.Wr = uint32_t(L.Wr); a.bits = uint32_t(cfg.bits);
  hipLaunchKernelGGL(k_code_sums, dim3(unsigned((L.D + 3) / 4)), dim3(256), 0, s, a);
  if (last_launch_status() != FQT_OK) return FQT_E_HIP;
  const int b = cfg.bits;
  if (engine == FQT_ENGINE_POPCOUNT) {
    const dim3 grid(unsigned((L.K + PC_T - 1) / PC_T), unsigned((L.D + PC_T - 1) / PC_T));
    switch (b) {
      case 1: hipLaunchKernelGGL(k_popc_dw<1>, grid, dim3(256), 0, s, a); break;
      case 2: hipLaunchKernelGGL(k_popc_dw<2>, grid, dim3(256), 0, s, a); break;
      case 3: hipLaunchKernelGGL(k_popc_dw<3>, grid, dim3(256), 0, s, a); break;
      case 4: hipLaunchKernelGGL(k_popc_dw<4>, grid, dim3(256), 0, s, a); break;
      case 5: hipLaunchKernelGGL(k_popc_dw<5>, grid, dim3(256), 0, s, a); break;
      case 6: hipLaunchKernelGGL(k_popc_dw<6>, grid, dim3(256), 0, s, a); break;
      case 7: hipLaunchKernelGGL(k_popc_dw<7>, grid, dim3(256), 0, s, a); break;
      case 8: hipLaunchKernelGGL(k_popc_dw<8>, grid, dim3(256), 0, s, a); break;
      default: return FQT_E_INVAL;
    }
    return last_launch_status();
  }
  // FP4: expand both operands to nibbles, then the scaled-MFMA product.
  Fp4Args f;
  f.p = a;
  f.Dp = uint32_t((L.D + 63) / 64 * 64);
  f.Kp = uint32_t((L.K + 255) / 256 * 256);
  uint8_t *A = static_cast<uint8_t *>(ws) + align256(size_t(L.D) * 4);
  uint8_t *Bn = A + align256(size_t(b) * L.Wr * f.Dp * 32);
  f.A = A; f.B = Bn;
  f.a_bytes = uint32_t(size_t(b) * L.Wr * f.Dp * 32);
  f.b_bytes = uint32_t(size_t(L.Wr) * f.Kp * 32);
  f.kgroups = f.Kp / 256;
  for (int p = 0; p < b; ++p) {
    const uint64_t n = uint64_t(L.Wr) * f.Dp;
    hipLaunchKernelGGL(k_bits_to_fp4, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s,
                       q.pcq_planes + size_t(p) * L.D * L.Wr, uint32_t(L.D), f.Dp, uint32_t(L.Wr),
                       A + size_t(p) * L.Wr * f.Dp * 32);
  }
  {
    const uint64_t n = uint64_t(L.Wr) * f.Kp;
    hipLaunchKernelGGL(k_bits_to_fp4, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s, xbits,
                       uint32_t(L.K), f.Kp, uint32_t(L.Wr), Bn);
  }
  if (last_launch_status() != FQT_OK) return FQT_E_HIP;
  const dim3 grid(unsigned((f.Dp / 64) * f.kgroups));
  switch (b) {
    case 1: hipLaunchKernelGGL(k_fp4_dw<1>, grid, dim3(256), 0, s, f); break;
    case 2: hipLaunchKernelGGL(k_fp4_dw<2>, grid, dim3(256), 0, s, f); break;
    case 3: hipLaunchKernelGGL(k_fp4_dw<3>, grid, dim3(256), 0, s, f); break;
    case 4: hipLaunchKernelGGL(k_fp4_dw<4>, grid, dim3(256), 0, s, f); break;
    default: return FQT_E_INVAL;
  }
  return last_launch_status();
}

int check_engine(const Layer &L, const fqt_quant_cfg &cfg, int engine) {
  if (engine != FQT_ENGINE_POPCOUNT && engine != FQT_ENGINE_FP4) return FQT_E_INVAL;
  if (engine == FQT_ENGINE_FP4) {
    if (cfg.bits > 4) return FQT_E_INVAL;
    // float32 partials exact: every sum below 2^24; operand buffers below 2^31 bytes.
    if (int64_t((1 << cfg.bits) - 1) * L.R >= (int64_t(1) << 24)) return FQT_E_SHAPE;
    const int64_t Dp = (L.D + 63) / 64 * 64, Kp = (L.K + 255) / 256 * 256;
    if (int64_t(cfg.bits) * L.Wr * Dp * 32 >= (int64_t(1) << 31) ||
        L.Wr * Kp * 32 >= (int64_t(1) << 31))
      return FQT_E_SHAPE;
  }
  return FQT_OK;
}

}  // namespace fqt
