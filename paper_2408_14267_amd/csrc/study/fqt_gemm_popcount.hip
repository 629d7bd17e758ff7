// The two binary contractions of the 1-bit FQT backward on gfx950 (Section 5.3,
// SCQ; Appendix C, Alg. 1 binary products and dequantization, the {0,1} <-> {+-1}
// conversion and the Folder), popcount engine.
//
// A b-bit code line a = sum_p 2^p a_p (b packed planes) against a sign line t
// (bit 1 = +1, bit 0 = -1) contracts to
//     sum_j q_j s_j = sum_p 2^p (2 popcount(a_p & t) - popcount(a_p)),
// exact in int32.  The per-group rescale S * I + Z' * c (c = sum of the signs)
// is taken once per output in float32 without contraction.
#include "fqt_internal.hpp"

namespace fqt {
namespace {

constexpr int THREADS = 256;

// ----------------------------------------------------------------------------- dW

struct DwArgs {
  const uint64_t *pcq;     // [bits][D][Wr]
  const int32_t *kept;     // [D] kept ids ascending | pruned ids ascending
  const int32_t *count;    // [1]
  const float *scale, *offset;   // [D]
  const uint64_t *xsign;   // [K][Wr]
  const int32_t *xsum;     // [K]
  float *dW;               // [D][K]
  int32_t *I_out;          // [D][K] or null
  int64_t D, K, Wr;
};

constexpr int DW_TM = 32, DW_TN = 64, DW_KW = 8;

// Tile: 32 kept-channel slots x 64 columns of C*kh*kw; each thread 2 slots x 4 columns.
template <int BITS>
__global__ __launch_bounds__(THREADS) void k_gemm_dw(DwArgs a) {
  __shared__ uint64_t As[BITS][DW_TM][DW_KW + 1];
  __shared__ uint64_t Bs[DW_TN][DW_KW + 1];
  const int t = threadIdx.x, tr = t >> 4, tc = t & 15;
  const int64_t j0 = int64_t(blockIdx.y) * DW_TM, k0 = int64_t(blockIdx.x) * DW_TN;
  const int count = *a.count;

  int acc[BITS][2][4];
  int qsum[2] = {0, 0};
  for (int p = 0; p < BITS; ++p)
    for (int i = 0; i < 2; ++i)
      for (int c = 0; c < 4; ++c) acc[p][i][c] = 0;

  if (j0 < count) {
    for (int64_t w0 = 0; w0 < a.Wr; w0 += DW_KW) {
      for (int idx = t; idx < BITS * DW_TM * DW_KW; idx += THREADS) {
        const int p = idx / (DW_TM * DW_KW);
        const int jr = (idx / DW_KW) % DW_TM;
        const int ww = idx % DW_KW;
        const int64_t j = j0 + jr, w = w0 + ww;
        As[p][jr][ww] = (j < a.D && w < a.Wr) ? a.pcq[(int64_t(p) * a.D + j) * a.Wr + w] : 0ull;
      }
      for (int idx = t; idx < DW_TN * DW_KW; idx += THREADS) {
        const int kc = idx / DW_KW, ww = idx % DW_KW;
        const int64_t k = k0 + kc, w = w0 + ww;
        Bs[kc][ww] = (k < a.K && w < a.Wr) ? a.xsign[k * a.Wr + w] : 0ull;
      }
      __syncthreads();
#pragma unroll 2
      for (int ww = 0; ww < DW_KW; ++ww) {
        uint64_t bv[4];
        for (int c = 0; c < 4; ++c) bv[c] = Bs[tc + 16 * c][ww];
        for (int p = 0; p < BITS; ++p) {
          for (int i = 0; i < 2; ++i) {
            const uint64_t av = As[p][2 * tr + i][ww];
            qsum[i] += popc64(av) << p;
            for (int c = 0; c < 4; ++c) acc[p][i][c] += popc64(av & bv[c]);
          }
        }
      }
      __syncthreads();
    }
  }

  for (int i = 0; i < 2; ++i) {
    const int64_t j = j0 + 2 * tr + i;
    if (j >= a.D) continue;
    const int64_t d = a.kept[j];
    const bool live = j < count;
    const float S = live ? a.scale[d] : 0.0f;
    const float Zp = live ? a.offset[d] : 0.0f;
    for (int c = 0; c < 4; ++c) {
      const int64_t k = k0 + tc + 16 * c;
      if (k >= a.K) continue;
      int I = 0;
      if (live) {
        for (int p = 0; p < BITS; ++p) I += acc[p][i][c] << (p + 1);
        I -= qsum[i];
      }
      const float out = live ? __fadd_rn(__fmul_rn(S, float(I)), __fmul_rn(Zp, float(a.xsum[k])))
                             : 0.0f;
      a.dW[d * a.K + k] = out;
      if (a.I_out) a.I_out[d * a.K + k] = I;
    }
  }
}

// ----------------------------------------------------------------------------- dX

struct DxArgs {
  const uint64_t *psq;     // [bits][R][Wd]
  const int32_t *kept;     // [N]
  const int32_t *count;
  const float *scale, *offset;   // [N]
  const uint64_t *wsign;   // [K][Wd]
  const int32_t *wsum;     // [K]
  void *dX;                // [N][C][H][W]
  int32_t *I_out;
  int dx_t;
  int64_t N, C, H, W, HW, D, Ho, Wo, P, R, Wd, C8;
  int kh, kw, sh, sw, ph, pw;
};

constexpr int DX_CPT = 8;   // channels per thread

// One thread: one input pixel (h, w) of one sample slot and 8 channels.  Sums over the
// kernel taps that map an output pixel onto (h, w) (the Folder, in integers).
template <int BITS>
__global__ __launch_bounds__(THREADS) void k_gemm_dx(DxArgs a) {
  const int64_t item = int64_t(blockIdx.x) * THREADS + threadIdx.x;
  const int64_t jslot = blockIdx.y;
  if (item >= a.C8 * a.HW) return;
  const int64_t c8 = item / a.HW, pix = item - c8 * a.HW;
  const int64_t h = pix / a.W, w = pix - h * a.W;
  const int64_t cbase = c8 * DX_CPT;
  const int count = *a.count;
  const int64_t n = a.kept[jslot];
  const bool live = jslot < count;

  int acc[DX_CPT], csum[DX_CPT];
  for (int c = 0; c < DX_CPT; ++c) acc[c] = csum[c] = 0;
  if (live) {
    for (int i = 0; i < a.kh; ++i) {
      const int64_t th = h + a.ph - i;
      if (th < 0 || th % a.sh) continue;
      const int64_t ho = th / a.sh;
      if (ho >= a.Ho) continue;
      for (int j = 0; j < a.kw; ++j) {
        const int64_t tw = w + a.pw - j;
        if (tw < 0 || tw % a.sw) continue;
        const int64_t wo = tw / a.sw;
        if (wo >= a.Wo) continue;
        const int64_t row = jslot * a.P + ho * a.Wo + wo;
        const int tap = i * a.kw + j;
        for (int c = 0; c < DX_CPT; ++c) {
          const int64_t cc = cbase + c;
          if (cc < a.C) csum[c] += a.wsum[cc * a.kh * a.kw + tap];
        }
        for (int64_t wd = 0; wd < a.Wd; ++wd) {
          uint64_t av[BITS];
          int qs = 0;
          for (int p = 0; p < BITS; ++p) {
            av[p] = a.psq[(int64_t(p) * a.R + row) * a.Wd + wd];
            qs += popc64(av[p]) << p;
          }
          for (int c = 0; c < DX_CPT; ++c) {
            const int64_t cc = cbase + c;
            if (cc >= a.C) break;
            const uint64_t tv = a.wsign[(cc * a.kh * a.kw + tap) * a.Wd + wd];
            int v = 0;
            for (int p = 0; p < BITS; ++p) v += popc64(av[p] & tv) << (p + 1);
            acc[c] += v - qs;
          }
        }
      }
    }
  }
  const float S = live ? a.scale[n] : 0.0f;
  const float Zp = live ? a.offset[n] : 0.0f;
  for (int c = 0; c < DX_CPT; ++c) {
    const int64_t cc = cbase + c;
    if (cc >= a.C) break;
    const float out = live ? __fadd_rn(__fmul_rn(S, float(acc[c])), __fmul_rn(Zp, float(csum[c])))
                           : 0.0f;
    const int64_t o = ((n * a.C + cc) * a.H + h) * a.W + w;
    if (a.dx_t == FQT_BF16) static_cast<uint16_t *>(a.dX)[o] = f32_to_bf16(out);
    else static_cast<float *>(a.dX)[o] = out;
    if (a.I_out) a.I_out[o] = live ? acc[c] : 0;
  }
}

template <int B>
void launch_dw_b(const DwArgs &a, dim3 grid, hipStream_t s) {
  hipLaunchKernelGGL(k_gemm_dw<B>, grid, dim3(THREADS), 0, s, a);
}
template <int B>
void launch_dx_b(const DxArgs &a, dim3 grid, hipStream_t s) {
  hipLaunchKernelGGL(k_gemm_dx<B>, grid, dim3(THREADS), 0, s, a);
}

}  // namespace

int launch_gemm_dw(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                   const uint64_t *xsign, const int32_t *xsum, float *dW, int32_t *I_out,
                   hipStream_t s) {
  DwArgs a{q.pcq_planes, q.pcq_kept, q.pcq_count, q.pcq_scale, q.pcq_offset, xsign, xsum,
           dW, I_out, L.D, L.K, L.Wr};
  const dim3 grid(unsigned((L.K + DW_TN - 1) / DW_TN), unsigned((L.D + DW_TM - 1) / DW_TM));
  switch (cfg.bits) {
    case 1: launch_dw_b<1>(a, grid, s); break;
    case 2: launch_dw_b<2>(a, grid, s); break;
    case 3: launch_dw_b<3>(a, grid, s); break;
    case 4: launch_dw_b<4>(a, grid, s); break;
    case 5: launch_dw_b<5>(a, grid, s); break;
    case 6: launch_dw_b<6>(a, grid, s); break;
    case 7: launch_dw_b<7>(a, grid, s); break;
    default: launch_dw_b<8>(a, grid, s); break;
  }
  return last_launch_status();
}

int launch_gemm_dx(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                   const uint64_t *wsign, const int32_t *wsum, void *dX, int32_t *I_out,
                   hipStream_t s) {
  DxArgs a;
  a.psq = q.psq_planes; a.kept = q.psq_kept; a.count = q.psq_count;
  a.scale = q.psq_scale; a.offset = q.psq_offset; a.wsign = wsign; a.wsum = wsum;
  a.dX = dX; a.I_out = I_out; a.dx_t = L.dx_t;
  a.N = L.N; a.C = L.C; a.H = L.H; a.W = L.W; a.HW = L.HW; a.D = L.D; a.Ho = L.Ho; a.Wo = L.Wo;
  a.P = L.P; a.R = L.R; a.Wd = L.Wd; a.C8 = (L.C + DX_CPT - 1) / DX_CPT;
  a.kh = L.kh; a.kw = L.kw; a.sh = L.sh; a.sw = L.sw; a.ph = L.ph; a.pw = L.pw;
  const dim3 grid(unsigned((a.C8 * L.HW + THREADS - 1) / THREADS), unsigned(L.N));
  switch (cfg.bits) {
    case 1: launch_dx_b<1>(a, grid, s); break;
    case 2: launch_dx_b<2>(a, grid, s); break;
    case 3: launch_dx_b<3>(a, grid, s); break;
    case 4: launch_dx_b<4>(a, grid, s); break;
    case 5: launch_dx_b<5>(a, grid, s); break;
    case 6: launch_dx_b<6>(a, grid, s); break;
    case 7: launch_dx_b<7>(a, grid, s); break;
    default: launch_dx_b<8>(a, grid, s); break;
  }
  return last_launch_status();
}

}  // namespace fqt
