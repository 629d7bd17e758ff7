// The two binary contractions of the 1-bit FQT backward on gfx950, int8 MFMA engine
// (Section 5.3, SCQ; Appendix C, Alg. 1 binary products and dequantization, the
// {0,1} <-> {+-1} conversion and the Folder).
//
// Operands: the b-bit codes as bytes (written by the quantizer next to the bit planes)
// and the packed sign bits, unpacked in registers to {0,1} bytes t.  With s = 2t - 1,
//     I = sum_j q_j s_j = 2 * sum_j q_j t_j - sum_j q_j,
// so the MFMA computes sum q t (int32, exact), the row code sums come from v_dot4 on
// the same bytes, and the line popcounts T = sum t give the zero-point column sums
// c = 2T - len.  For b = 8 the codes do not fit a signed byte; the MFMA then takes
// q - 128 and adds 128 T back.  The rescale S * I + Z' * c is one float32 step per
// output without contraction.
//
// MFMA v_mfma_i32_32x32x32_i8: lane l feeds row (src0) / column (src1) l % 32 with 16
// bytes of the 32-deep contraction chosen by l / 32; both operands use the same
// (lane group, byte) -> k assignment, so each product pairs equal k.  Lane l then holds
// output column l % 32 at rows 8 (v / 4) + 4 (l / 32) + (v % 4), v = 0..15.
#include <algorithm>

#include "fqt_internal.hpp"

namespace fqt {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

// 16 sign bits (LSB first) -> 16 bytes of 0/1 (byte m of dword q holds bit 4q + m).
// A nibble times 0x00204081 places bit m at bit 8m without carries.
__device__ __forceinline__ v4i spread16(uint32_t bits) {
  v4i r;
  r.x = int((bits & 0xFu) * 0x00204081u & 0x01010101u);
  r.y = int(((bits >> 4) & 0xFu) * 0x00204081u & 0x01010101u);
  r.z = int(((bits >> 8) & 0xFu) * 0x00204081u & 0x01010101u);
  r.w = int(((bits >> 12) & 0xFu) * 0x00204081u & 0x01010101u);
  return r;
}

__device__ __forceinline__ uint32_t byte_sum16(v4i a) {
  uint32_t s = __builtin_amdgcn_udot4(uint32_t(a.x), 0x01010101u, 0u, false);
  s = __builtin_amdgcn_udot4(uint32_t(a.y), 0x01010101u, s, false);
  s = __builtin_amdgcn_udot4(uint32_t(a.z), 0x01010101u, s, false);
  return __builtin_amdgcn_udot4(uint32_t(a.w), 0x01010101u, s, false);
}

__device__ __forceinline__ v4i bias128(v4i a) {
  const int m = int(0x80808080u);
  return v4i{a.x ^ m, a.y ^ m, a.z ^ m, a.w ^ m};
}

__device__ __forceinline__ v16i mfma(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float rescale(float S, int I, float Zp, int c) {
  return __fadd_rn(__fmul_rn(S, float(I)), __fmul_rn(Zp, float(c)));
}

// Zero `count` elements of `esize` bytes starting at element `first` of `base`, by the
// `nthr` threads of a block: 16-byte stores where the run is 16-byte aligned, bytes of
// the ragged ends one element at a time.
__device__ void zero_run(void *base, size_t first, size_t count, int esize, int tid, int nthr) {
  char *p = static_cast<char *>(base) + first * esize;
  const size_t bytes = count * esize;
  const size_t head = (16 - (reinterpret_cast<uintptr_t>(p) & 15)) & 15;
  const size_t lead = head < bytes ? head : bytes;
  const size_t nvec = (bytes - lead) / 16;
  for (size_t e = tid; e * esize < lead; e += nthr) {
    if (esize == 4) reinterpret_cast<uint32_t *>(p)[e] = 0u;
    else reinterpret_cast<uint16_t *>(p)[e] = 0;
  }
  uint4 *v = reinterpret_cast<uint4 *>(p + lead);
  for (size_t e = tid; e < nvec; e += nthr) v[e] = make_uint4(0u, 0u, 0u, 0u);
  char *tail = p + lead + nvec * 16;
  const size_t rest = bytes - lead - nvec * 16;
  for (size_t e = tid; e * esize < rest; e += nthr) {
    if (esize == 4) reinterpret_cast<uint32_t *>(tail)[e] = 0u;
    else reinterpret_cast<uint16_t *>(tail)[e] = 0;
  }
}

// ----------------------------------------------------------------------------- dW

struct DwArgs {
  const uint8_t *codes;          // PCQ codes [D][Wr*64]
  const int32_t *kept, *count;   // [D], [1]
  const float *scale, *offset;   // [D]
  const uint64_t *xsign;         // [K][Wr]
  float *dW;                     // [D][K]
  int32_t *I_out;                // [D][K] or null
  uint32_t D, K, R, Wr, ktiles;
  int bits8;
};

constexpr int DW_WAVES = 16;
constexpr int DW_THREADS = DW_WAVES * 64;
constexpr int DW_BATCH = 4;        // 64-bit words of the contraction loaded per batch

// Grid: one block per 32x32 tile of (kept-channel slot, column of C*kh*kw) over the slot
// capacity D, plus a pool of extra blocks.  Blocks of the first ceil(count/32) slot tiles
// compute; all later blocks zero the dW rows of the pruned channels, each a contiguous
// run of K floats.
// A computing block is one 32x32 MFMA tile; sixteen waves split the contraction over
// N*Ho*Wo word by word (wave w takes words w, w+16, ...) and sum in LDS.
__global__ __launch_bounds__(DW_THREADS) void k_mfma_dw(DwArgs a) {
  __shared__ int32_t red[16][64];
  __shared__ int32_t qred[32];
  __shared__ int32_t tred[32];
  __shared__ int32_t rowd[32];
  __shared__ float rows_s[32], rows_z[32];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int i = lane & 31, g = lane >> 5;
  const int count = *a.count;
  const uint32_t live_blocks = uint32_t((count + 31) / 32) * a.ktiles;

  if (blockIdx.x >= live_blocks) {      // zero the rows of pruned channels, one row per block
    const uint32_t nz = gridDim.x - live_blocks;
    for (uint32_t row = blockIdx.x - live_blocks; row < a.D - uint32_t(count); row += nz) {
      const size_t d = size_t(a.kept[uint32_t(count) + row]);
      zero_run(a.dW, d * a.K, a.K, 4, t, DW_THREADS);
      if (a.I_out) zero_run(a.I_out, d * a.K, a.K, 4, t, DW_THREADS);
    }
    return;
  }
  const uint32_t j0 = (blockIdx.x / a.ktiles) * 32, k0 = (blockIdx.x % a.ktiles) * 32;

  (&red[0][0])[t] = 0;
  if (t < 32) {
    qred[t] = 0;
    tred[t] = 0;
    const uint32_t j = j0 + t;
    const int d = (int(j) < count) ? a.kept[j] : -1;
    rowd[t] = d;
    rows_s[t] = d >= 0 ? a.scale[d] : 0.0f;
    rows_z[t] = d >= 0 ? a.offset[d] : 0.0f;
  }
  __syncthreads();

  v16i acc = {0};
  uint32_t qpart = 0, tpart = 0;
  const uint32_t jr = j0 + i, kc = k0 + i;
  const bool a_ok = int(jr) < count, b_ok = kc < a.K;
  const uint8_t *arow = a.codes + size_t(a_ok ? jr : 0) * a.Wr * 64 + 16 * g;
  const uint64_t *brow = a.xsign + size_t(b_ok ? kc : 0) * a.Wr;
  for (uint32_t c0 = wave; c0 < a.Wr; c0 += DW_WAVES * DW_BATCH) {
    v4i av[DW_BATCH][2];
    uint64_t wb[DW_BATCH];
#pragma unroll
    for (int u = 0; u < DW_BATCH; ++u) {
      const uint32_t c = c0 + u * DW_WAVES;
      const bool live = c < a.Wr;
      av[u][0] = (live && a_ok) ? *reinterpret_cast<const v4i *>(arow + size_t(c) * 64)
                                : v4i{0, 0, 0, 0};
      av[u][1] = (live && a_ok) ? *reinterpret_cast<const v4i *>(arow + size_t(c) * 64 + 32)
                                : v4i{0, 0, 0, 0};
      wb[u] = (live && b_ok) ? brow[c] : 0ull;
    }
#pragma unroll
    for (int u = 0; u < DW_BATCH; ++u) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        v4i A = av[u][s];
        qpart += byte_sum16(A);
        if (a.bits8) A = bias128(A);
        const uint32_t bb = uint32_t(wb[u] >> (32 * s + 16 * g)) & 0xFFFFu;
        tpart += __popc(bb);
        acc = mfma(A, spread16(bb), acc);
      }
    }
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) atomicAdd(&red[v][lane], acc[v]);
  atomicAdd(&qred[i], int(qpart));
  atomicAdd(&tred[i], int(tpart));
  __syncthreads();

  const int row = t >> 5, col = t & 31;
  const int d = rowd[row];
  const uint32_t k = k0 + col;
  if (d < 0 || k >= a.K) return;          // rows past the count belong to the zero blocks
  const int T = tred[col];
  int Ip = red[4 * (row >> 3) + (row & 3)][col + 32 * ((row >> 2) & 1)];
  if (a.bits8) Ip += 128 * T;
  const int I = 2 * Ip - qred[row];
  const size_t idx = size_t(d) * a.K + k;
  a.dW[idx] = rescale(rows_s[row], I, rows_z[row], 2 * T - int(a.R));
  if (a.I_out) a.I_out[idx] = I;
}

// ----------------------------------------------------------------------------- dX

struct DxArgs {
  const uint8_t *codes;          // PSQ codes [N*Ho*Wo][Wd*64]
  const int32_t *kept, *count;   // [N], [1]
  const float *scale, *offset;   // [N]
  const uint64_t *wsign;         // [C*kh*kw][Wd]
  void *dX;                      // [N][C][H][W]
  int32_t *I_out;
  int dx_t;
  uint32_t N, C, H, W, HW, Ho, Wo, P, D, Wd, ctiles, CHW;
  int kh, kw, sh, sw, ph, pw;
  FastDiv divHW, divW, divWd;
  int bits8;
};

constexpr int DX_MAX_TAPS = 64;
constexpr int DX_WAVES = 8;
constexpr int DX_THREADS = DX_WAVES * 64;
constexpr int DX_BATCH = 4;        // contraction steps (tap, 64-bit word of D) per batch

// Grid: one block per 32x32 tile of (row m = (kept slot, h, w), channel) over the capacity
// N*H*W rows, plus a pool of extra blocks.  Blocks of the first ceil(count*H*W/32) row
// tiles compute; all later blocks zero the pruned samples of dX, each a contiguous run of
// C*H*W elements.
// A computing block is one 32x32 MFMA tile with the sign operand as src0 (rows =
// channels) so output lanes run along pixels.  Eight waves split the contraction steps
// (tap, word of D).  For tap (i, j) a pixel (h, w) reads the code row of the output pixel
// (ho, wo) with ho*sh - ph + i = h and wo*sw - pw + j = w, or nothing; the row of every
// (pixel, tap) is tabulated once per block.
__global__ __launch_bounds__(DX_THREADS) void k_mfma_dx(DxArgs a) {
  // Rows padded to DX_MAX_TAPS + 1 words: lanes reading column `tap` of 32 rows hit 32 banks.
  __shared__ int32_t rowtab[32][DX_MAX_TAPS + 1];   // code row of (pixel, tap), -1 if none
  __shared__ uint64_t vmask[32];                    // taps that reach each pixel
  __shared__ int32_t Tt[32][DX_MAX_TAPS + 1];       // popcount of sign(W) line (channel, tap)
  __shared__ int32_t red[16][64];
  __shared__ int32_t qred[32];                  // code sums of each pixel's rows
  __shared__ int32_t pix_out[32];               // NCHW offset of (sample, pixel) minus channel
  __shared__ float pix_s[32], pix_z[32];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int i = lane & 31, g = lane >> 5;
  const int count = *a.count;
  const uint32_t live_rows = uint32_t(count) * a.HW;
  const uint32_t live_blocks = ((live_rows + 31) / 32) * a.ctiles;
  const int taps = a.kh * a.kw;

  if (blockIdx.x >= live_blocks) {      // zero the pruned samples, one sample per block
    const uint32_t nz = gridDim.x - live_blocks;
    for (uint32_t slot = blockIdx.x - live_blocks; slot < a.N - uint32_t(count); slot += nz) {
      const size_t n = size_t(a.kept[uint32_t(count) + slot]);
      zero_run(a.dX, n * a.CHW, a.CHW, a.dx_t == FQT_BF16 ? 2 : 4, t, DX_THREADS);
      if (a.I_out) zero_run(a.I_out, n * a.CHW, a.CHW, 4, t, DX_THREADS);
    }
    return;
  }
  const uint32_t m0 = (blockIdx.x / a.ctiles) * 32, c0 = (blockIdx.x % a.ctiles) * 32;

  for (int e = t; e < 32 * taps; e += DX_THREADS) {
    const int p = e / taps, tap = e - p * taps;
    const int ti = tap / a.kw, tj = tap - ti * a.kw;
    const uint32_t m = m0 + p;
    int row = -1;
    if (m < live_rows) {
      const uint32_t slot = fdiv(m, a.divHW), pix = m - slot * a.HW;
      const uint32_t h = fdiv(pix, a.divW), w = pix - h * a.W;
      const int th = int(h) + a.ph - ti, tw = int(w) + a.pw - tj;
      if (th >= 0 && tw >= 0 && th % a.sh == 0 && tw % a.sw == 0) {
        const int ho = th / a.sh, wo = tw / a.sw;
        if (ho < int(a.Ho) && wo < int(a.Wo)) row = int(slot * a.P + ho * a.Wo + wo);
      }
    }
    rowtab[p][tap] = row;
    Tt[p][tap] = 0;
  }
  (&red[0][0])[t] = 0;
  (&red[0][0])[t + DX_THREADS] = 0;
  if (t < 32) {
    qred[t] = 0;
    const uint32_t m = m0 + t;
    int off = -1;
    float sc = 0.0f, zo = 0.0f;
    if (m < live_rows) {
      const uint32_t slot = fdiv(m, a.divHW), pix = m - slot * a.HW;
      const int n = a.kept[slot];
      off = int(uint32_t(n) * a.CHW + pix);
      sc = a.scale[n];
      zo = a.offset[n];
    }
    pix_out[t] = off;
    pix_s[t] = sc;
    pix_z[t] = zo;
  }
  __syncthreads();
  if (t < 32) {
    uint64_t mk = 0;
    for (int tap = 0; tap < taps; ++tap) mk |= uint64_t(rowtab[t][tap] >= 0) << tap;
    vmask[t] = mk;
  }

  // This lane: A row = channel c0 + i, B column = pixel m0 + i.
  const uint32_t ch = c0 + i;
  const bool ch_ok = ch < a.C;
  const uint64_t *wbase = a.wsign + size_t(ch_ok ? ch : 0) * taps * a.Wd;
  const uint8_t *cbase = a.codes + 16 * g;
  const uint32_t steps = uint32_t(taps) * a.Wd;
  v16i acc = {0};
  uint32_t qpart = 0;
  for (uint32_t s0 = wave; s0 < steps; s0 += DX_WAVES * DX_BATCH) {
    v4i bv[DX_BATCH][2];
    uint64_t sw[DX_BATCH];
    int tapu[DX_BATCH];
#pragma unroll
    for (int u = 0; u < DX_BATCH; ++u) {
      const uint32_t st = s0 + u * DX_WAVES;
      const bool live = st < steps;
      const uint32_t tap = live ? fdiv(st, a.divWd) : 0;
      const uint32_t dc = st - tap * a.Wd;
      const int row = live ? rowtab[i][tap] : -1;
      const uint8_t *p = cbase + (size_t(row < 0 ? 0 : row) * a.Wd + dc) * 64;
      bv[u][0] = row >= 0 ? *reinterpret_cast<const v4i *>(p) : v4i{0, 0, 0, 0};
      bv[u][1] = row >= 0 ? *reinterpret_cast<const v4i *>(p + 32) : v4i{0, 0, 0, 0};
      sw[u] = (live && ch_ok) ? wbase[st] : 0ull;
      tapu[u] = live ? int(tap) | (row >= 0 ? 0x10000 : 0) : -1;
    }
#pragma unroll
    for (int u = 0; u < DX_BATCH; ++u) {
      uint32_t tp = 0;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        v4i B = bv[u][s];
        qpart += byte_sum16(B);
        if (a.bits8 && (tapu[u] & 0x10000)) B = bias128(B);
        const uint32_t bits = uint32_t(sw[u] >> (32 * s + 16 * g)) & 0xFFFFu;
        tp += __popc(bits);
        acc = mfma(spread16(bits), B, acc);
      }
      if (tapu[u] >= 0) atomicAdd(&Tt[i][tapu[u] & 0xFFFF], int(tp));
    }
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) atomicAdd(&red[v][lane], acc[v]);
  atomicAdd(&qred[i], int(qpart));
  __syncthreads();

  // Epilogue: element e -> (channel row crow, pixel column pc).
  for (int e = t; e < 32 * 32; e += DX_THREADS) {
    const int pc = e & 31, crow = e >> 5;
    const uint32_t cc = c0 + crow;
    const int off = pix_out[pc];
    if (off < 0 || cc >= a.C) continue;   // rows past the count belong to the zero blocks
    uint64_t mk = vmask[pc];
    int T_valid = 0;
    const int nvalid = __popcll(mk);
    while (mk) {
      const int tap = __ffsll(static_cast<unsigned long long>(mk)) - 1;
      mk &= mk - 1;
      T_valid += Tt[crow][tap];
    }
    int Ip = red[4 * (crow >> 3) + (crow & 3)][pc + 32 * ((crow >> 2) & 1)];
    if (a.bits8) Ip += 128 * T_valid;
    const int I = 2 * Ip - qred[pc];
    const float out = rescale(pix_s[pc], I, pix_z[pc], 2 * T_valid - nvalid * int(a.D));
    const size_t o = size_t(off) + size_t(cc) * a.HW;
    if (a.dx_t == FQT_BF16) static_cast<uint16_t *>(a.dX)[o] = f32_to_bf16(out);
    else static_cast<float *>(a.dX)[o] = out;
    if (a.I_out) a.I_out[o] = I;
  }
}

}  // namespace

int launch_gemm_dw(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                   const uint64_t *xsign, float *dW, int32_t *I_out, hipStream_t s) {
  const uint32_t ktiles = uint32_t((L.K + 31) / 32);
  DwArgs a{q.pcq_codes, q.pcq_kept, q.pcq_count, q.pcq_scale, q.pcq_offset, xsign, dW, I_out,
           uint32_t(L.D), uint32_t(L.K), uint32_t(L.R), uint32_t(L.Wr), ktiles,
           cfg.bits == 8 ? 1 : 0};
  // Capacity tiles plus a pool of blocks that only zero pruned rows: whatever the device-side
  // count, at least `zb` blocks are left for the zeroing.
  const int64_t zb = std::min<int64_t>(256, L.D);
  const dim3 grid(unsigned(ktiles * ((L.D + 31) / 32) + zb));
  hipLaunchKernelGGL(k_mfma_dw, grid, dim3(DW_THREADS), 0, s, a);
  return last_launch_status();
}

int launch_gemm_dx(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                   const uint64_t *wsign, void *dX, int32_t *I_out, hipStream_t s) {
  if (L.kh * L.kw > DX_MAX_TAPS) return FQT_E_SHAPE;
  DxArgs a;
  a.codes = q.psq_codes; a.kept = q.psq_kept; a.count = q.psq_count;
  a.scale = q.psq_scale; a.offset = q.psq_offset; a.wsign = wsign;
  a.dX = dX; a.I_out = I_out; a.dx_t = L.dx_t;
  a.N = uint32_t(L.N); a.C = uint32_t(L.C); a.H = uint32_t(L.H); a.W = uint32_t(L.W);
  a.HW = uint32_t(L.HW); a.Ho = uint32_t(L.Ho); a.Wo = uint32_t(L.Wo); a.P = uint32_t(L.P);
  a.D = uint32_t(L.D); a.Wd = uint32_t(L.Wd);
  a.ctiles = uint32_t((L.C + 31) / 32);
  a.CHW = uint32_t(L.C * L.HW);
  a.kh = L.kh; a.kw = L.kw; a.sh = L.sh; a.sw = L.sw; a.ph = L.ph; a.pw = L.pw;
  a.divHW = make_fastdiv(uint32_t(L.HW)); a.divW = make_fastdiv(uint32_t(L.W));
  a.divWd = make_fastdiv(uint32_t(L.Wd));
  a.bits8 = cfg.bits == 8 ? 1 : 0;
  const int64_t zb = std::min<int64_t>(256, L.N);
  const dim3 grid(unsigned(((L.N * L.HW + 31) / 32) * a.ctiles + zb));
  hipLaunchKernelGGL(k_mfma_dx, grid, dim3(DX_THREADS), 0, s, a);
  return last_launch_status();
}

}  // namespace fqt
