// Sign-bit packing on gfx950 (Section 5.1 binarizer; Appendix C, Alg. 2 row
// encoder, column encoder and Unfolder).  One 64-lane wavefront produces one
// 64-bit word with a ballot: lane l contributes bit l.
#include "fqt_internal.hpp"

namespace fqt {
namespace {

constexpr int THREADS = 256;
constexpr int WAVES = THREADS / 64;

// Along the columns of a row-major [rows][cols] matrix: word w of row i.
template <int DT>
__global__ __launch_bounds__(THREADS) void k_pack_along_cols(const void *__restrict__ src,
                                                             int64_t rows,
                                                             int64_t cols, int64_t ld,
                                                             uint64_t *__restrict__ dst) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = (cols + 63) >> 6;
  const int64_t item = int64_t(blockIdx.x) * WAVES + (threadIdx.x >> 6);
  if (item >= rows * nw) return;
  const int64_t i = item / nw, w = item - i * nw;
  const int64_t j = (w << 6) + lane;
  const float v = j < cols ? load_elem<DT>(src, i * ld + j) : 0.0f;
  const bool bit = v > 0.0f;
  const uint64_t m = __ballot(bit);
  if (lane == 0) dst[i * nw + w] = m;
}

// Down the rows (transposing): 64x64 tile staged in LDS, read back column-wise.  WM: the
// output is word-major, word w of line c at w * cols + c (the layout the dW product reads).
template <int DT, bool WM>
__global__ __launch_bounds__(THREADS) void k_pack_along_rows(const void *__restrict__ src,
                                                             int64_t rows,
                                                             int64_t cols, int64_t ld,
                                                             uint64_t *__restrict__ dst) {
  __shared__ uint8_t bits[64][64 + 4];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t c0 = int64_t(blockIdx.x) * 64, r0 = int64_t(blockIdx.y) * 64;
  const int64_t nw = (rows + 63) >> 6;
  float v[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {   // unconditional loads (element 0 outside) issue back to back
    const int64_t r = r0 + wave + 4 * i, c = c0 + lane;
    v[i] = load_elem<DT>(src, (r < rows && c < cols) ? r * ld + c : 0);
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int64_t r = r0 + wave + 4 * i, c = c0 + lane;
    bits[wave + 4 * i][lane] = (r < rows && c < cols && v[i] > 0.0f) ? 1 : 0;
  }
  __syncthreads();
  for (int i = 0; i < 16; ++i) {
    const int cc = wave + 4 * i;
    const int64_t c = c0 + cc;
    if (c >= cols) break;
    const uint64_t m = __ballot(bits[lane][cc] != 0);
    if (lane == 0) dst[WM ? (r0 >> 6) * cols + c : c * nw + (r0 >> 6)] = m;
  }
}

struct Im2colGeom {
  uint32_t C, H, W, Wo, P, R, nw, cgroups;
  int kh, kw, sh, sw, ph, pw;
  FastDiv divP, divWo, divNw;
};

constexpr int IM2COL_CPW = 4;   // channels per wave sharing one index decomposition

// Bit-im2col: line (c, i, j), bit (n, ho, wo) = X[n][c][ho*sh - ph + i][wo*sw - pw + j] > 0;
// positions in the zero padding give bit 0 (sign -1).  One wave owns 64 consecutive
// (n, ho, wo) of IM2COL_CPW channels: one index decomposition per lane serves every
// channel and kernel tap.  The words of a channel's taps are gathered into lanes
// 0..taps-1 and stored by one instruction.  KH, KW > 0 fix the kernel size at compile
// time (fully unrolled); 0 reads it from the geometry.  WM: word-major output, word w of
// line l at w * C*kh*kw + l (the layout the dW product reads).
template <int DT, int KH, int KW, bool WM>
__global__ __launch_bounds__(THREADS) void k_pack_im2col(const void *__restrict__ x, Im2colGeom g,
                                                         uint64_t *__restrict__ dst) {
  const int lane = threadIdx.x & 63;
  const uint32_t item = blockIdx.x * WAVES + (threadIdx.x >> 6);
  if (item >= g.cgroups * g.nw) return;
  const uint32_t cg = fdiv(item, g.divNw), w = item - cg * g.nw;
  const uint32_t r0 = (w << 6) + lane;
  const bool valid = r0 < g.R;
  const uint32_t r = valid ? r0 : 0;
  const uint32_t n = fdiv(r, g.divP), pix = r - n * g.P;
  const uint32_t ho = fdiv(pix, g.divWo), wo = pix - ho * g.Wo;
  const int h0 = int(ho) * g.sh - g.ph, w0 = int(wo) * g.sw - g.pw;
  const int kh = KH > 0 ? KH : g.kh, kw = KW > 0 ? KW : g.kw;
  const int taps = kh * kw;
  uint32_t hok = 0, wok = 0;
  for (int i = 0; i < kh; ++i) hok |= uint32_t(valid && h0 + i >= 0 && h0 + i < int(g.H)) << i;
  for (int j = 0; j < kw; ++j) wok |= uint32_t(w0 + j >= 0 && w0 + j < int(g.W)) << j;
  const int plane = int(g.H * g.W);
  int base = (int(n * g.C + cg * IM2COL_CPW) * int(g.H) + h0) * int(g.W) + w0;
  for (int cc = 0; cc < IM2COL_CPW; ++cc, base += plane) {
    const uint32_t c = cg * IM2COL_CPW + cc;
    if (c >= g.C) break;
    uint64_t mine = 0;
    if constexpr (KH > 0) {
      float v[KH * KW];
#pragma unroll
      for (int i = 0; i < KH; ++i)
#pragma unroll
        for (int j = 0; j < KW; ++j) {
          const bool ok = (hok >> i) & (wok >> j) & 1u;
          v[i * KW + j] = load_elem<DT>(x, ok ? base + i * int(g.W) + j : 0);
        }
#pragma unroll
      for (int i = 0; i < KH; ++i)
#pragma unroll
        for (int j = 0; j < KW; ++j) {
          const bool ok = (hok >> i) & (wok >> j) & 1u;
          const uint64_t m = __ballot(ok && v[i * KW + j] > 0.0f);
          if (lane == i * KW + j) mine = m;
        }
      if (lane < KH * KW)
        dst[WM ? size_t(w) * g.C * (KH * KW) + size_t(c) * (KH * KW) + lane
               : (size_t(c) * (KH * KW) + lane) * g.nw + w] = mine;
    } else {
      for (int t0 = 0; t0 < taps; t0 += 16) {
        int ti = t0 / kw, tj = t0 - ti * kw;
        float v[16];
        uint32_t okm = 0;
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const bool ok = t0 + u < taps && ((hok >> ti) & (wok >> tj) & 1u);
          okm |= uint32_t(ok) << u;
          v[u] = load_elem<DT>(x, ok ? base + ti * int(g.W) + tj : 0);
          if (++tj == kw) {
            tj = 0;
            ++ti;
          }
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const uint64_t m = __ballot(((okm >> u) & 1u) && v[u] > 0.0f);
          if (lane == u) mine = m;
        }
        if (lane < 16 && t0 + lane < taps)
          dst[WM ? size_t(w) * g.C * taps + size_t(c) * taps + t0 + lane
                 : (size_t(c) * taps + t0 + lane) * g.nw + w] = mine;
      }
    }
  }
}

// Bit-im2col through LDS, word-major output, for layers whose output positions per sample
// are a multiple of 64 (every 64-position word lies in one sample) and whose rows are
// whole 16-byte quads (W % 4 == 0, pw <= 4).  A block takes one word w (output positions
// p0 .. p0 + 63 of sample n) and BAND_LG channels: it stages, per channel, the band of
// input rows those positions read as one byte per pixel (1 = positive), each band row
// framed by four zero bytes on either side and rows outside the image all zero; a lane
// loads one 16-byte quad and writes one LDS dword.  Then each (channel, tap) word is one
// LDS byte per lane and a ballot.  Lane l reads band row (ho - ho_lo) * sh + i, column
// wo * sw + j - pw + 4 for its position (ho, wo) and tap (i, j); band row 0 is image row
// ho_lo * sh - ph.
constexpr int BAND_LG = 16;            // channels per block (4 per wave)
struct BandGeom {
  uint32_t C, H, W, Wo, P, K, taps, BR, WL, plane;   // WL = W + 8, plane = BR * WL
  uint32_t qrow;                                     // dwords per band row, WL / 4
  int kw, sh, sw, ph, pw;
  FastDiv divWo, divP, divQrow, divBR, divKw;
};

template <int DT, int KH, int KW>
__global__ __launch_bounds__(THREADS) void k_pack_im2col_band(const void *__restrict__ x,
                                                              BandGeom g,
                                                              uint64_t *__restrict__ dst) {
  extern __shared__ uint32_t band[];             // [BAND_LG][BR][WL] bytes
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const uint32_t w = blockIdx.x;                 // word: output positions 64 w ...
  const uint32_t c0 = blockIdx.y * BAND_LG;
  const uint32_t nch = min(uint32_t(BAND_LG), g.C - c0);
  const uint32_t r0 = w * 64;
  const uint32_t n = fdiv(r0, g.divP), p0 = r0 - n * g.P;
  const uint32_t ho_lo = fdiv(p0, g.divWo);
  const int h_base = int(ho_lo) * g.sh - g.ph;   // image row of band row 0
  const size_t xbase = (size_t(n) * g.C + c0) * g.H * g.W;   // element (c0, 0, 0) of sample n

  // Stage: dword q of band row (c, br) holds image columns 4 (q - 1) .. 4 (q - 1) + 3.
  const uint32_t rows = nch * g.BR;
  const uint32_t items = rows * g.qrow;
  constexpr int SB = 4;
  for (uint32_t e0 = t; e0 < items; e0 += SB * THREADS) {
    float v[SB][4];
    bool in[SB];
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const uint32_t e = e0 + k * THREADS;
      const uint32_t row = fdiv(e, g.divQrow), q = e - row * g.qrow;
      const uint32_t c = fdiv(row, g.divBR), br = row - c * g.BR;
      const int h = h_base + int(br);
      in[k] = e < items && h >= 0 && h < int(g.H) && q >= 1 && q <= g.W / 4;
      const uint32_t off = (c * g.H + uint32_t(h)) * g.W + 4 * (q - 1);   // < C*H*W
      load_quad<DT>(x, in[k] ? int64_t(xbase + off) : 0, v[k]);
    }
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const uint32_t e = e0 + k * THREADS;
      if (e >= items) break;
      uint32_t b = 0;
      if (in[k])
        b = (v[k][0] > 0.0f ? 1u : 0u) | (v[k][1] > 0.0f ? 0x100u : 0u) |
            (v[k][2] > 0.0f ? 0x10000u : 0u) | (v[k][3] > 0.0f ? 0x1000000u : 0u);
      band[e] = b;
    }
  }
  __syncthreads();

  // This lane's output position and its band byte offset for tap (0, 0).
  const uint8_t *bb = reinterpret_cast<const uint8_t *>(band);
  const uint32_t p = p0 + lane;
  const uint32_t ho = fdiv(p, g.divWo), wo = p - ho * g.Wo;
  const uint32_t base = (ho - ho_lo) * g.sh * g.WL + wo * g.sw + 4 - g.pw;
  constexpr uint32_t per_wave = BAND_LG / WAVES;
  const uint32_t cl_lo = wave * per_wave, cl_hi = min(nch, cl_lo + per_wave);
  uint32_t mlo = 0, mhi = 0;                     // words gather in lanes 0 .. 63
  int filled = 0;
  uint64_t *out = dst + size_t(w) * g.K;
  auto put = [&](uint64_t m, uint32_t line_last) {
    mlo = writelane(uint32_t(m), filled, mlo);
    mhi = writelane(uint32_t(m >> 32), filled, mhi);
    if (++filled == 64) {                        // 64 words of consecutive lines
      out[line_last - 63 + lane] = (uint64_t(mhi) << 32) | mlo;
      filled = 0;
    }
  };
  for (uint32_t cl = cl_lo; cl < cl_hi; ++cl) {
    const uint8_t *pl = bb + cl * g.plane + base;
    if constexpr (KH > 0) {
      // Kernel size fixed at compile time: every tap's LDS read issues before the ballots.
      uint8_t b[KH * KW];
#pragma unroll
      for (int i = 0; i < KH; ++i)
#pragma unroll
        for (int j = 0; j < KW; ++j) b[i * KW + j] = pl[i * g.WL + j];
#pragma unroll
      for (int tap = 0; tap < KH * KW; ++tap)
        put(__ballot(b[tap] != 0), (c0 + cl) * (KH * KW) + tap);
    } else {
      for (uint32_t tap = 0; tap < g.taps; ++tap) {
        const uint32_t i = fdiv(tap, g.divKw), j = tap - i * g.kw;
        put(__ballot(pl[i * g.WL + j] != 0), (c0 + cl) * g.taps + tap);
      }
    }
  }
  if (filled > 0 && cl_hi > cl_lo) {
    // The words left end at the wave's last line.
    const uint32_t l_end = (c0 + cl_hi) * g.taps;
    if (lane < filled) out[l_end - filled + lane] = (uint64_t(mhi) << 32) | mlo;
  }
}

// linesum[l] = sum of the +-1 signs of line l = 2 * popcount - len.
__global__ __launch_bounds__(THREADS) void k_linesum(const uint64_t *__restrict__ words,
                                                     int64_t lines, int64_t nw, int64_t len,
                                                     int32_t *__restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int64_t l = int64_t(blockIdx.x) * WAVES + (threadIdx.x >> 6);
  if (l >= lines) return;
  int cnt = 0;
  for (int64_t w = lane; w < nw; w += 64) cnt += popc64(words[l * nw + w]);
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o);
  if (lane == 0) out[l] = int32_t(2 * int64_t(cnt) - len);
}

unsigned blocks_for(int64_t items) { return unsigned((items + WAVES - 1) / WAVES); }

// sign(W) as signed bytes for the int8 dX product (Section 5.1 binarizer; the +-1 form of
// Appendix C's {0,1} <-> {+-1} conversion).  W is viewed as [D][K] (K = C*kh*kw, line
// l = (c, tap)); byte d of line l is +1 if W[d][l] > 0 else -1 for d < D, 0 for
// D <= d < Dp, stored chunk-major at ((d/32 * taps + tap) * C + c) * 32 + d % 32 so that the
// 32-byte chunks of consecutive channels are adjacent; lsum[l] = sum over d < D of the
// line.  One block of 1024 threads per 64 lines walks D in passes of 256 rows (one pass
// for D <= 256): each thread loads 16 rows of its line back to back, the pass is
// transposed through LDS (pitch 260 bytes = 65 dwords: the column writes of a wave spread
// over the banks) and written as 16-byte pieces of the 32-byte chunks.
constexpr int WB_THREADS = 1024;
constexpr int WB_ROWS = 256;                  // rows of D per pass: 16 per thread
constexpr int WB_PITCH = WB_ROWS + 4;
template <int DT>
__global__ __launch_bounds__(WB_THREADS) void k_pack_w_i8(const void *__restrict__ w, uint32_t D,
                                                          uint32_t K, uint32_t Dp, uint32_t C,
                                                          uint32_t taps, FastDiv div_taps,
                                                          int8_t *__restrict__ dst,
                                                          int32_t *__restrict__ lsum) {
  constexpr int Q = WB_THREADS / 64;          // row phases per pass
  __shared__ __align__(16) int8_t tile[64][WB_PITCH];
  __shared__ int32_t pos[64];
  const int t = threadIdx.x, line = t & 63, q = t >> 6;
  const uint32_t l0 = blockIdx.x * 64, l = l0 + line;
  if (t < 64) pos[t] = 0;
  int mine = 0;
  for (uint32_t d0 = 0; d0 < Dp; d0 += WB_ROWS) {
    float v[WB_ROWS / Q];
#pragma unroll
    for (int k = 0; k < WB_ROWS / Q; ++k) {   // unconditional loads (element 0 outside) issue back to back
      const uint32_t d = d0 + Q * k + q;
      v[k] = load_elem<DT>(w, (d < D && l < K) ? int64_t(d) * K + l : 0);
    }
#pragma unroll
    for (int k = 0; k < WB_ROWS / Q; ++k) {
      const uint32_t d = d0 + Q * k + q;
      const bool in = d < D && l < K;
      const bool pos_sign = in && v[k] > 0.0f;
      mine += pos_sign ? 1 : 0;
      tile[line][Q * k + q] = in ? (pos_sign ? int8_t(1) : int8_t(-1)) : int8_t(0);
    }
    __syncthreads();
    // 64 lines x 16 pieces of 16 bytes; pieces past Dp (last pass of a short D) are not stored.
    const int wl = t >> 4, part = t & 15;
    if (l0 + wl < K && d0 + 16 * part < Dp) {
      const uint32_t lw = l0 + wl, c = fdiv(lw, div_taps), tap = lw - c * taps;
      const uint32_t chunk = (d0 >> 5) + (part >> 1);
      const uint32_t *src = reinterpret_cast<const uint32_t *>(&tile[wl][16 * part]);
      *reinterpret_cast<uint4 *>(dst + ((size_t(chunk) * taps + tap) * C + c) * 32 +
                                 16 * (part & 1)) = make_uint4(src[0], src[1], src[2], src[3]);
    }
    __syncthreads();
  }
  atomicAdd(&pos[line], mine);
  __syncthreads();
  if (t < 64 && l0 + t < K) lsum[l0 + t] = 2 * pos[t] - int(D);
}

}  // namespace

int launch_pack_w_i8(const void *W, const Layer &L, int8_t *dst, int32_t *lsum, hipStream_t s) {
  const uint32_t D = uint32_t(L.D), K = uint32_t(L.K), Dp = uint32_t(L.Wd * 64);
  const uint32_t taps = uint32_t(L.kh * L.kw);
  dispatch_dtype(L.w_t, [&]<int DT>() {
    hipLaunchKernelGGL(k_pack_w_i8<DT>, dim3(unsigned((L.K + 63) / 64)), dim3(WB_THREADS), 0, s, W,
                       D, K, Dp, uint32_t(L.C), taps, make_fastdiv(taps), dst, lsum);
  });
  return last_launch_status();
}

int launch_pack_bits(const void *src, int dtype, int64_t rows, int64_t cols, int64_t ld, int axis,
                     const Layer *conv, uint64_t *dst, int32_t *linesum, hipStream_t s,
                     bool word_major) {
  int64_t lines, nw, len;
  if (axis == FQT_PACK_ALONG_COLS) {
    nw = (cols + 63) / 64;
    lines = rows;
    len = cols;
    dispatch_dtype(dtype, [&]<int DT>() {
      hipLaunchKernelGGL(k_pack_along_cols<DT>, dim3(blocks_for(rows * nw)), dim3(THREADS), 0, s,
                         src, rows, cols, ld, dst);
    });
  } else if (axis == FQT_PACK_ALONG_ROWS) {
    nw = (rows + 63) / 64;
    lines = cols;
    len = rows;
    dispatch_dtype(dtype, [&]<int DT>() {
      const dim3 grid(unsigned((cols + 63) / 64), unsigned(nw));
      if (word_major)
        hipLaunchKernelGGL((k_pack_along_rows<DT, true>), grid, dim3(THREADS), 0, s, src, rows,
                           cols, ld, dst);
      else
        hipLaunchKernelGGL((k_pack_along_rows<DT, false>), grid, dim3(THREADS), 0, s, src, rows,
                           cols, ld, dst);
    });
  } else {
    const Layer &L = *conv;
    const uint32_t cgroups = uint32_t((L.C + IM2COL_CPW - 1) / IM2COL_CPW);
    Im2colGeom g{uint32_t(L.C), uint32_t(L.H), uint32_t(L.W), uint32_t(L.Wo), uint32_t(L.P),
                 uint32_t(L.R), uint32_t(L.Wr), cgroups, L.kh, L.kw, L.sh, L.sw, L.ph, L.pw,
                 make_fastdiv(uint32_t(L.P)), make_fastdiv(uint32_t(L.Wo)),
                 make_fastdiv(uint32_t(L.Wr))};
    nw = L.Wr;
    lines = L.K;
    len = L.R;
    // (Quad loads: X must be aligned to four elements.)
    const bool quads_ok = reinterpret_cast<uintptr_t>(src) % (dtype == FQT_BF16 ? 8 : 16) == 0;
    if (word_major && quads_ok && L.P % 64 == 0 && L.W % 4 == 0 && L.pw <= 4) {
      // Band of input rows read by one word: its output rows times the stride plus the
      // kernel height; rows framed by four zero bytes on either side.
      const int64_t orows = (64 + L.Wo - 1) / L.Wo + 1;
      const int64_t BR = (orows - 1) * L.sh + L.kh;
      const int64_t WL = L.W + 8;
      const int64_t plane = BR * WL;
      if (plane * BAND_LG <= 48 * 1024 && L.kh * L.kw <= 64) {
        BandGeom bg{uint32_t(L.C), uint32_t(L.H), uint32_t(L.W), uint32_t(L.Wo), uint32_t(L.P),
                    uint32_t(L.K), uint32_t(L.kh * L.kw), uint32_t(BR), uint32_t(WL),
                    uint32_t(plane), uint32_t(WL / 4), L.kw, L.sh, L.sw, L.ph, L.pw,
                    make_fastdiv(uint32_t(L.Wo)), make_fastdiv(uint32_t(L.P)),
                    make_fastdiv(uint32_t(WL / 4)), make_fastdiv(uint32_t(BR)),
                    make_fastdiv(uint32_t(L.kw))};
        const dim3 bgrid(unsigned(L.Wr), unsigned((L.C + BAND_LG - 1) / BAND_LG));
        const size_t lds = size_t(plane * BAND_LG);
        dispatch_dtype(dtype, [&]<int DT>() {
          if (L.kh == 3 && L.kw == 3)
            hipLaunchKernelGGL((k_pack_im2col_band<DT, 3, 3>), bgrid, dim3(THREADS), lds, s,
                               src, bg, dst);
          else if (L.kh == 1 && L.kw == 1)
            hipLaunchKernelGGL((k_pack_im2col_band<DT, 1, 1>), bgrid, dim3(THREADS), lds, s,
                               src, bg, dst);
          else
            hipLaunchKernelGGL((k_pack_im2col_band<DT, 0, 0>), bgrid, dim3(THREADS), lds, s,
                               src, bg, dst);
        });
        return last_launch_status();
      }
    }
    const dim3 grid(blocks_for(int64_t(cgroups) * L.Wr));
    auto go = [&]<int DT, bool WM>() {
      if (L.kh == 1 && L.kw == 1)
        hipLaunchKernelGGL((k_pack_im2col<DT, 1, 1, WM>), grid, dim3(THREADS), 0, s, src, g, dst);
      else if (L.kh == 3 && L.kw == 3)
        hipLaunchKernelGGL((k_pack_im2col<DT, 3, 3, WM>), grid, dim3(THREADS), 0, s, src, g, dst);
      else if (L.kh == 7 && L.kw == 7)
        hipLaunchKernelGGL((k_pack_im2col<DT, 7, 7, WM>), grid, dim3(THREADS), 0, s, src, g, dst);
      else
        hipLaunchKernelGGL((k_pack_im2col<DT, 0, 0, WM>), grid, dim3(THREADS), 0, s, src, g, dst);
    };
    dispatch_dtype(dtype, [&]<int DT>() {
      if (word_major) go.template operator()<DT, true>();
      else go.template operator()<DT, false>();
    });
  }
  if (last_launch_status() != FQT_OK) return FQT_E_HIP;
  if (linesum && !word_major) {
    hipLaunchKernelGGL(k_linesum, dim3(blocks_for(lines)), dim3(THREADS), 0, s, dst, lines, nw,
                       len, linesum);
    return last_launch_status();
  }
  return FQT_OK;
}

}  // namespace fqt
