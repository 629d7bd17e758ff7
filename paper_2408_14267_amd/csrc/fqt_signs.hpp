// Device bodies of the sign packers that feed the MFMA products (Section 5.1 binarizer;
// Appendix C, Alg. 2 encoders, the Unfolder and the {0,1} <-> {+-1} conversion):
//   band, bit-level and wave im2col   sign(unfold(X)) as word-major bits, the dW operand
//                 (rows: the same for a linear layer's X);
//   weight bytes  sign(W) as +-1 bytes with per-line sums, the dX operand.
// fqt_pack.hip launches them on their own; the layer backward runs them in spare blocks
// of the AGP selection launch, whose two selection workgroups leave the chip idle.
#pragma once

#include <algorithm>

#include "fqt_internal.hpp"

namespace fqt {

// ----------------------------------------------------------------------------- band im2col
// Bit-im2col through LDS, word-major output, for layers whose output positions per sample
// are a multiple of 64 (every 64-position word lies in one sample) and whose rows are
// whole 16-byte quads (W % 4 == 0, pw <= 4).  A block takes up to wpb consecutive words of
// one sample (output positions p0 .. p0 + 64 wpb - 1) and BAND_CPW channels per wave: it
// stages, per channel, the band of input rows those positions read as one byte per pixel
// (1 = positive), each band row framed by four zero bytes on either side and rows outside
// the image all zero; a lane loads one 16-byte quad and writes one LDS dword.  Then each
// (word, channel, tap) is one LDS byte per lane and a ballot.  Lane l of word j reads band
// row (ho - ho_lo) * sh + i, column wo * sw + j' - pw + 4 for its position (ho, wo) and tap
// (i, j'); band row 0 is image row ho_lo * sh - ph.  Several words per block keep wide
// images from staging whole rows for a fraction of their columns.
constexpr int BAND_CPW = 4;            // channels per wave
struct BandGeom {
  uint32_t C, H, W, Wo, P, K, taps, BR, WL, plane;   // WL = W + 8, plane = BR * WL
  uint32_t qrow;                                     // dwords per band row, WL / 4
  uint32_t wps, wpb, wgroups;    // words per sample, per block, word groups per sample
  int kw, sh, sw, ph, pw;
  FastDiv divWo, divP, divQrow, divBR, divKw, divWg;
};

// Geometry of the band im2col for blocks of `nt` threads (BAND_CPW * nt / 64 channels),
// or false when the layer does not fit it or its band exceeds `lds_max` bytes.  Up to 16
// words per block, as many as the band for them fits while the grid keeps about 2048
// blocks.
inline bool band_geom(const Layer &L, const void *x, int dtype, int nt, size_t lds_max,
                      BandGeom *bg, size_t *lds) {
  const bool quads_ok = reinterpret_cast<uintptr_t>(x) % (dtype == FQT_BF16 ? 8 : 16) == 0;
  if (L.kind != FQT_CONV2D || !quads_ok || L.P % 64 != 0 || L.W % 4 != 0 || L.pw > 4 ||
      L.kh * L.kw > 64)
    return false;
  const int64_t wps = L.P / 64;
  const int64_t WL = L.W + 8;
  const int64_t chans = int64_t(BAND_CPW) * (nt / 64);
  const int64_t cgroups = (L.C + chans - 1) / chans;
  const int64_t wmax = std::max<int64_t>(1, L.N * wps * cgroups / 2048);
  for (int64_t wpb = std::min<int64_t>({wps, 16, wmax}); wpb >= 1; --wpb) {
    // Band of input rows read by wpb words: the output rows they can span times the
    // stride plus the kernel height.
    const int64_t orows = (64 * wpb - 1 + L.Wo - 1) / L.Wo + 1;
    const int64_t BR = (orows - 1) * L.sh + L.kh;
    const int64_t plane = BR * WL;
    const size_t bytes = size_t(plane * std::min<int64_t>(chans, L.C));   // channels staged
    if (bytes > lds_max) continue;
    const int64_t wgroups = (wps + wpb - 1) / wpb;
    *bg = BandGeom{uint32_t(L.C), uint32_t(L.H), uint32_t(L.W), uint32_t(L.Wo), uint32_t(L.P),
                   uint32_t(L.K), uint32_t(L.kh * L.kw), uint32_t(BR), uint32_t(WL),
                   uint32_t(plane), uint32_t(WL / 4), uint32_t(wps), uint32_t(wpb),
                   uint32_t(wgroups), L.kw, L.sh, L.sw, L.ph, L.pw,
                   make_fastdiv(uint32_t(L.Wo)), make_fastdiv(uint32_t(L.P)),
                   make_fastdiv(uint32_t(WL / 4)), make_fastdiv(uint32_t(BR)),
                   make_fastdiv(uint32_t(L.kw)), make_fastdiv(uint32_t(wgroups))};
    *lds = bytes;
    return true;
  }
  return false;
}
// Blocks along the words: samples x word groups.
inline uint32_t band_word_blocks(const Layer &L, const BandGeom &bg) {
  return uint32_t(L.N) * bg.wgroups;
}

// One block of NT threads: word group `wb` (sample wb / wgroups), channels
// [cblk * BAND, (cblk + 1) * BAND).  band: the block's LDS, BAND * plane bytes.
template <int DT, int KH, int KW, int NT>
__device__ __forceinline__ void band_im2col_body(const void *__restrict__ x, const BandGeom &g,
                                                 uint64_t *__restrict__ dst, uint32_t wb,
                                                 uint32_t cblk, uint32_t *band) {
  constexpr int NW = NT / 64, BAND = BAND_CPW * NW;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const uint32_t c0 = cblk * BAND;
  const uint32_t nch = min(uint32_t(BAND), g.C - c0);
  const uint32_t n = fdiv(wb, g.divWg), wg = wb - n * g.wgroups;
  const uint32_t wfirst = wg * g.wpb;                       // first word within the sample
  const uint32_t nwords = min(g.wpb, g.wps - wfirst);
  const uint32_t p0 = wfirst * 64;
  const uint32_t ho_lo = fdiv(p0, g.divWo);
  const int h_base = int(ho_lo) * g.sh - g.ph;   // image row of band row 0
  const size_t xbase = (size_t(n) * g.C + c0) * g.H * g.W;   // element (c0, 0, 0) of sample n

  // Stage: dword q of band row (c, br) holds image columns 4 (q - 1) .. 4 (q - 1) + 3.
  const uint32_t rows = nch * g.BR;
  const uint32_t items = rows * g.qrow;
  constexpr int SB = 4;
  for (uint32_t e0 = t; e0 < items; e0 += SB * NT) {
    float v[SB][4];
    bool in[SB];
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const uint32_t e = e0 + k * NT;
      const uint32_t row = fdiv(e, g.divQrow), q = e - row * g.qrow;
      const uint32_t c = fdiv(row, g.divBR), br = row - c * g.BR;
      const int h = h_base + int(br);
      in[k] = e < items && h >= 0 && h < int(g.H) && q >= 1 && q <= g.W / 4;
      const uint32_t off = (c * g.H + uint32_t(h)) * g.W + 4 * (q - 1);   // < C*H*W
      load_quad<DT>(x, in[k] ? int64_t(xbase + off) : 0, v[k]);
    }
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const uint32_t e = e0 + k * NT;
      if (e >= items) break;
      uint32_t b = 0;
      if (in[k])
        b = (v[k][0] > 0.0f ? 1u : 0u) | (v[k][1] > 0.0f ? 0x100u : 0u) |
            (v[k][2] > 0.0f ? 0x10000u : 0u) | (v[k][3] > 0.0f ? 0x1000000u : 0u);
      band[e] = b;
    }
  }
  __syncthreads();

  const uint8_t *bb = reinterpret_cast<const uint8_t *>(band);
  // KH > 0: BAND_CPW channels per wave.  KH = 0: the block's nch * taps lines split evenly
  // over the waves, so that a block of few channels (a 3-channel stem) keeps every wave busy.
  const uint32_t nl = nch * g.taps, lpw = (nl + NW - 1) / NW;
  const uint32_t cl_lo = wave * BAND_CPW, cl_hi = min(nch, cl_lo + BAND_CPW);
  const uint32_t l_lo = min(nl, wave * lpw), l_hi = min(nl, l_lo + lpw);
  if (KH > 0 ? cl_hi <= cl_lo : l_hi <= l_lo) return;
  for (uint32_t j = 0; j < nwords; ++j) {
    // This lane's output position in word j and its band byte offset for tap (0, 0).
    const uint32_t p = p0 + 64 * j + lane;
    const uint32_t ho = fdiv(p, g.divWo), wo = p - ho * g.Wo;
    const uint32_t base = (ho - ho_lo) * g.sh * g.WL + wo * g.sw + 4 - g.pw;
    uint32_t mlo = 0, mhi = 0;                   // words gather in lanes 0 .. 63
    int filled = 0;
    uint64_t *out = dst + size_t(n * g.wps + wfirst + j) * g.K;
    auto put = [&](uint64_t m, uint32_t line_last) {
      mlo = writelane(uint32_t(m), filled, mlo);
      mhi = writelane(uint32_t(m >> 32), filled, mhi);
      if (++filled == 64) {                      // 64 words of consecutive lines
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
          for (int jj = 0; jj < KW; ++jj) b[i * KW + jj] = pl[i * g.WL + jj];
#pragma unroll
        for (int tap = 0; tap < KH * KW; ++tap)
          put(__ballot(b[tap] != 0), (c0 + cl) * (KH * KW) + tap);
      }
    }
    if constexpr (KH == 0) {
      uint32_t cl = l_lo / g.taps, tap = l_lo - cl * g.taps;
      for (uint32_t l = l_lo; l < l_hi; ++l) {
        const uint32_t i = fdiv(tap, g.divKw), jj = tap - i * g.kw;
        put(__ballot(bb[cl * g.plane + base + i * g.WL + jj] != 0), c0 * g.taps + l);
        if (++tap == g.taps) {
          tap = 0;
          ++cl;
        }
      }
    }
    if (filled > 0) {
      // The words left end at the wave's last line.
      const uint32_t l_end = KH > 0 ? (c0 + cl_hi) * g.taps : c0 * g.taps + l_hi;
      if (lane < filled) out[l_end - filled + lane] = (uint64_t(mhi) << 32) | mlo;
    }
  }
}

// ----------------------------------------------------------------------------- bit im2col
// Bit-level im2col for stride-1 convolutions with "same" padding (2 ph = kh - 1,
// 2 pw = kw - 1, so Ho = H and Wo = W and an output position and the input position a tap
// reads differ by a constant offset in the row-major order of N*H*W).  Let s_c be the
// string of sign bits of channel c over all N*H*W positions (bit r = X[n][c][h][w] > 0 at
// r = (n H + h) W + w).  Output word w of line (c, tap) (positions 64 w .. 64 w + 63) is
// then the 64 bits of s_c from bit 64 w + off(tap), off = (i - ph) W + (j - pw), with the
// positions whose tap falls outside the image (row ho + i - ph or column wo + j - pw out
// of range) cleared by a row mask and a column mask of the word.  A block builds s_c for
// its CB channels over its WB words plus the halo words the offsets reach, one ballot per
// word, in LDS; every output word is then one funnel shift and two masks, 64 lines per
// wave instruction.  Compared with a ballot per output word this takes the VALU work of
// the packing from once per (position, tap) to once per position.
struct BitGeom {
  uint32_t N, C, H, W, P, R, Wr, K, taps;
  int kh, kw, ph, pw;
  uint32_t CB, WB;            // channels and output words per block
  uint32_t dlo, span;         // staged words below the block's first word; words staged
  uint32_t jl0, jl1;          // staged words [jl0, jl1) are loaded, the others are zero
  uint32_t own;               // 1: only the block's own words are loaded (whole samples)
  uint32_t cgroups, wgroups;
  FastDiv divP, divW, divTaps, divKw, divWB, divWg;
  uint32_t vec;               // 1: X is 16-byte aligned and every word lies in one sample,
                              //    so a lane loads 8 consecutive elements at once
};

constexpr int BIT_U = 8;        // sign words a wave loads back to back

// Geometry for blocks of `nt` threads.  The words staged per channel are dlo + WB + dhi:
// the WB output words of the block and the words the tap offsets reach below and above
// them.  When a sample is a whole number of words, at most 16 (P % 64 == 0, P <= 1024), WB
// is a whole number of samples and only the block's own words are loaded: every tap a
// mask keeps reads its own sample, so the reached words of other samples are staged as
// zeros.  Otherwise the reached words are loaded too, and WB is large enough that they are
// at most a sixteenth of the loads (whole-sample blocks of larger samples would be many
// serial batches per wave).  CB channels, a power of two, at least enough for one batch of BIT_U
// words per wave and then doubled up to 64 while the grid has more than about
// `target_blocks` blocks, and halved while the staging exceeds `lds_max` bytes.  False
// when the layer is not a stride-1 same-padded convolution or one channel's staging does
// not fit.
inline bool bit_geom(const Layer &L, int nt, int64_t target_blocks, size_t lds_max,
                     BitGeom *g, size_t *lds) {
  if (L.kind != FQT_CONV2D || L.sh != 1 || L.sw != 1 || 2 * L.ph != L.kh - 1 ||
      2 * L.pw != L.kw - 1 || L.kh * L.kw > 64)
    return false;
  const int64_t reach = int64_t(L.ph) * L.W + L.pw;     // largest |offset| of a tap, bits
  const int64_t dlo = (reach + 63) / 64, dhi = reach / 64 + 1;
  const bool own = L.P % 64 == 0 && L.P <= 1024;
  int64_t WB, jl0, jl1, span;
  if (own) {
    const int64_t wps = L.P / 64;
    WB = wps * std::max<int64_t>(1, BIT_U / wps);
    jl0 = dlo;
    jl1 = dlo + (WB + BIT_U - 1) / BIT_U * BIT_U;
    span = jl1 + dhi;
  } else {
    span = BIT_U;
    while (span < 16 * (dlo + dhi)) span += BIT_U;
    // No more staged words than the layer has (plus its halo), in whole batches.
    const int64_t need = (L.Wr + dlo + dhi + BIT_U - 1) / BIT_U * BIT_U;
    if (span > need) span = need;
    WB = span - dlo - dhi;
    jl0 = 0;
    jl1 = span;
  }
  const int64_t batches = (jl1 - jl0) / BIT_U;
  const int64_t wgroups = (L.Wr + WB - 1) / WB;
  int64_t CB = 1;
  while (CB < 64 && CB * batches < nt / 64) CB *= 2;
  while (CB < 64 && CB < L.C && ((L.C + CB - 1) / CB) * wgroups > target_blocks) CB *= 2;
  auto lds_bytes = [&](int64_t cb) { return size_t(8) * size_t(cb * span + WB * (L.kh + L.kw)); };
  while (CB > 1 && lds_bytes(CB) > lds_max) CB /= 2;
  const size_t bytes = lds_bytes(CB);
  if (bytes > lds_max) return false;
  const int64_t cgroups = (L.C + CB - 1) / CB;
  *g = BitGeom{uint32_t(L.N), uint32_t(L.C), uint32_t(L.H), uint32_t(L.W), uint32_t(L.P),
               uint32_t(L.R), uint32_t(L.Wr), uint32_t(L.K), uint32_t(L.kh * L.kw),
               L.kh, L.kw, L.ph, L.pw, uint32_t(CB), uint32_t(WB), uint32_t(dlo),
               uint32_t(span), uint32_t(jl0), uint32_t(jl1), own ? 1u : 0u,
               uint32_t(cgroups), uint32_t(wgroups),
               make_fastdiv(uint32_t(L.P)), make_fastdiv(uint32_t(L.W)),
               make_fastdiv(uint32_t(L.kh * L.kw)), make_fastdiv(uint32_t(L.kw)),
               make_fastdiv(uint32_t(WB)), make_fastdiv(uint32_t(wgroups)), 0u};
  *lds = bytes;
  return true;
}
// The 8-elements-per-lane staging: words that never straddle samples and a 16-byte aligned X.
inline void bit_geom_vec(BitGeom *g, const void *x) {
  g->vec = (g->P % 64 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0) ? 1u : 0u;
}
inline uint32_t bit_blocks(const BitGeom &g) { return g.cgroups * g.wgroups; }

// One block of NT threads: block index `blk` = channel group * wgroups + word group.
// sm: 8 * (CB * span + WB * (kh + kw)) bytes of LDS.
template <int DT, int NT>
__device__ __forceinline__ void bit_im2col_body(const void *__restrict__ x, const BitGeom &g,
                                                uint64_t *__restrict__ dst, uint32_t blk,
                                                uint64_t *sm) {
  constexpr int NW = NT / 64, U = BIT_U;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const uint32_t cg = fdiv(blk, g.divWg), wg = blk - cg * g.wgroups;
  const uint32_t c0 = cg * g.CB, nch = min(g.CB, g.C - c0);
  const uint32_t w0 = wg * g.WB, nw = min(g.WB, g.Wr - w0);
  uint64_t *bits = sm;                               // [CB][span]: word w0 - dlo + j of s_c
  uint64_t *rowm = sm + g.CB * g.span;               // [WB][kh]
  uint64_t *colm = rowm + g.WB * g.kh;               // [WB][kw]

  // Staged words [0, jl0) and [jl1, span) of every channel are zero.
  const uint32_t pad = g.span - (g.jl1 - g.jl0);
  for (uint32_t e = t; e < nch * pad; e += NT) {
    const uint32_t c = e / pad, k = e - c * pad;
    bits[c * g.span + (k < g.jl0 ? k : g.jl1 + (k - g.jl0))] = 0;
  }
  // Sign words [jl0, jl1) in items (channel c, batch of U consecutive words), item i to
  // wave i % NW, the U loads of an item back to back: every load is in bounds (words
  // outside the loaded range read the nearest word of it, and a flag clears the bit).
  // Whole-sample words step a wave-uniform element index through X; others take each
  // lane's (sample, position).
  const bool whole = (g.P & 63) == 0;      // every word lies in one sample
  const uint32_t wps = g.P >> 6;
  const uint32_t nb = (g.jl1 - g.jl0) / U; // batches per channel
  // Words the block loads: its own [w0, w0 + nw), or everything in the layer.
  const int32_t lo_w = g.own ? int32_t(w0) : 0;
  const int32_t hi_w = g.own ? int32_t(w0 + nw) : int32_t(g.Wr);
  if (g.vec) {
    // Lane l takes positions 8 (l % 8) .. 8 (l % 8) + 7 of word l / 8 of the item with one
    // 16-byte load (bf16; two for float32) and stores their 8 sign bits as one byte of the
    // staged word: byte m of a word holds its positions 8 m .. 8 m + 7, least significant
    // bit first, the same bits the per-position ballots give.
    static_assert(U == 8, "one word per 8 lanes");
    uint8_t *bytes = reinterpret_cast<uint8_t *>(bits);
    const uint32_t k = uint32_t(lane) >> 3, m = uint32_t(lane) & 7u;
    for (uint32_t it = wave; it < nch * nb; it += NW) {
      const uint32_t c = it / nb, j0 = g.jl0 + (it - c * nb) * U;
      const int32_t wa = int32_t(w0 + j0 + k) - int32_t(g.dlo);
      const bool inw = wa >= lo_w && wa < hi_w;
      const uint32_t u = uint32_t(min(max(wa, lo_w), hi_w - 1));
      const uint32_t n = fdiv(u * 64, g.divP);
      const int64_t e = (int64_t(n) * g.C + c0 + c) * g.P + int64_t(u - n * wps) * 64 + 8 * m;
      float v[8];
      load_oct<DT>(x, e, v);
      uint32_t b = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) b |= (v[i] > 0.0f ? 1u : 0u) << i;
      bytes[size_t(c * g.span + j0 + k) * 8 + m] = uint8_t(inw ? b : 0u);
    }
  }
  for (uint32_t it = g.vec ? nch * nb : uint32_t(wave); it < nch * nb; it += NW) {
    const uint32_t c = it / nb, j0 = g.jl0 + (it - c * nb) * U;
    const int32_t wa0 = int32_t(w0 + j0) - int32_t(g.dlo);
    float v[U];
    if (whole) {
      // Word u = clamp(wa): sample u / wps, positions (u % wps) * 64 onwards.
      const uint32_t u0 = uint32_t(min(max(wa0, lo_w), hi_w - 1));
      const uint32_t n0 = fdiv(u0 * 64, g.divP);
      uint32_t q = u0 - n0 * wps;                          // word within the sample
      int64_t e = (int64_t(n0) * g.C + c0 + c) * g.P + int64_t(q) * 64;
      const int64_t skip = int64_t(g.C - 1) * g.P;      // to the next sample's plane
#pragma unroll
      for (int k = 0; k < U; ++k) {
        v[k] = load_elem<DT>(x, e + lane);
        // Step to the next word when it is a new one (selects, no branch).
        const int32_t wa = wa0 + k;
        const bool step = wa >= lo_w && wa + 1 < hi_w;
        const bool wrap = step && q + 1 == wps;
        e += step ? (wrap ? 64 + skip : int64_t(64)) : int64_t(0);
        q = wrap ? 0u : (step ? q + 1 : q);
      }
    } else {
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const int32_t wa = wa0 + k;
        const uint32_t r = min(uint32_t(max(wa, 0)) * 64 + lane, g.R - 1);
        const uint32_t n = fdiv(r, g.divP), p = r - n * g.P;
        v[k] = load_elem<DT>(x, (int64_t(n) * g.C + c0 + c) * g.P + p);
      }
    }
    uint64_t mine = 0;
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int32_t wa = wa0 + k;
      const bool in = wa >= lo_w && wa < hi_w && uint32_t(wa) * 64 + lane < g.R;
      const uint64_t m = __ballot(in && v[k] > 0.0f);
      if (lane == k) mine = m;
    }
    if (lane < U) bits[c * g.span + j0 + lane] = mine;
  }
  // Row and column masks of each output word.
  for (uint32_t j = wave; j < nw; j += NW) {
    const uint32_t r = (w0 + j) * 64 + lane;
    const bool in = r < g.R;
    const uint32_t n = fdiv(r, g.divP), p = r - n * g.P;
    const uint32_t ho = fdiv(p, g.divW), wo = p - ho * g.W;
    uint64_t mr = 0, mc = 0;
    for (int i = 0; i < g.kh; ++i) {
      const int h = int(ho) + i - g.ph;
      const uint64_t m = __ballot(in && h >= 0 && h < int(g.H));
      if (lane == i) mr = m;
    }
    for (int i = 0; i < g.kw; ++i) {
      const int w = int(wo) + i - g.pw;
      const uint64_t m = __ballot(in && w >= 0 && w < int(g.W));
      if (lane == i) mc = m;
    }
    if (lane < g.kh) rowm[j * g.kh + lane] = mr;
    if (lane < g.kw) colm[j * g.kw + lane] = mc;
  }
  __syncthreads();

  // Output words: item o = (line chunk lc, word j), 64 lines (c, tap) per chunk.
  const uint32_t nl = nch * g.taps, nlc = (nl + 63) / 64;
  for (uint32_t o = wave; o < nlc * g.WB; o += NW) {
    const uint32_t lc = fdiv(o, g.divWB), j = o - lc * g.WB;
    if (j >= nw) continue;
    const uint32_t ll = lc * 64 + lane;
    if (ll >= nl) continue;
    const uint32_t c = fdiv(ll, g.divTaps), tap = ll - c * g.taps;
    const uint32_t i = fdiv(tap, g.divKw), jj = tap - i * g.kw;
    const int off = (int(i) - g.ph) * int(g.W) + int(jj) - g.pw;
    const uint32_t bp = uint32_t(int((j + g.dlo) * 64) + off);     // >= 0 by dlo
    const uint32_t q = bp >> 6, sh = bp & 63;
    const uint64_t lo = bits[c * g.span + q], hi = bits[c * g.span + q + 1];
    uint64_t v = sh ? (lo >> sh) | (hi << (64 - sh)) : lo;
    v &= rowm[j * g.kh + i] & colm[j * g.kw + jj];
    dst[size_t(w0 + j) * g.K + size_t(c0) * g.taps + ll] = v;
  }
}

// ----------------------------------------------------------------------------- wave im2col
struct Im2colGeom {
  uint32_t C, H, W, Wo, P, R, nw, cgroups;
  int kh, kw, sh, sw, ph, pw;
  FastDiv divP, divWo, divNw;
};

constexpr int IM2COL_CPW = 4;   // channels per wave sharing one index decomposition
inline Im2colGeom im2col_geom(const Layer &L) {
  return Im2colGeom{uint32_t(L.C), uint32_t(L.H), uint32_t(L.W), uint32_t(L.Wo), uint32_t(L.P),
                    uint32_t(L.R), uint32_t(L.Wr), uint32_t((L.C + IM2COL_CPW - 1) / IM2COL_CPW),
                    L.kh, L.kw, L.sh, L.sw, L.ph, L.pw, make_fastdiv(uint32_t(L.P)),
                    make_fastdiv(uint32_t(L.Wo)), make_fastdiv(uint32_t(L.Wr))};
}


// Bit-im2col: line (c, i, j), bit (n, ho, wo) = X[n][c][ho*sh - ph + i][wo*sw - pw + j] > 0;
// positions in the zero padding give bit 0 (sign -1).  One wave owns 64 consecutive
// (n, ho, wo) of IM2COL_CPW channels (work item `item` = channel group * nw + word): one
// index decomposition per lane serves every
// channel and kernel tap.  The words of a channel's taps are gathered into lanes
// 0..taps-1 and stored by one instruction.  KH, KW > 0 fix the kernel size at compile
// time (fully unrolled); 0 reads it from the geometry.  WM: word-major output, word w of
// line l at w * C*kh*kw + l (the layout the dW product reads).
template <int DT, int KH, int KW, bool WM>
__device__ __forceinline__ void wave_im2col_body(const void *__restrict__ x, const Im2colGeom &g,
                                                 uint64_t *__restrict__ dst, uint32_t item) {
  const int lane = threadIdx.x & 63;
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

// ----------------------------------------------------------------------------- rows
// sign(X) of a linear layer's input X[N][C] down the rows, word-major: bit l of word w of
// column c is X[64 w + l][c] > 0, at dst[w * C + c] (the layout the dW product reads).  One
// wave per work item (word w, 16 columns c0 .. c0 + 15; column groups fastest): lane l
// loads its row's 16 elements back to back and one ballot per column gives that column's
// word, kept by lane k for column c0 + k.
__device__ __forceinline__ uint32_t rows_items(uint32_t N, uint32_t C) {
  return ((N + 63) / 64) * ((C + 15) / 16);
}
template <int DT>
__device__ __forceinline__ void rows_wave_body(const void *__restrict__ x, uint32_t N, uint32_t C,
                                               uint64_t *__restrict__ dst, uint32_t item) {
  const int lane = threadIdx.x & 63;
  const uint32_t ncg = (C + 15) / 16;
  if (item >= rows_items(N, C)) return;
  const uint32_t w = item / ncg, c0 = (item - w * ncg) * 16;
  const uint32_t r = w * 64 + uint32_t(lane);
  const bool rin = r < N;
  float v[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) {   // element 0 outside X, so the loads issue back to back
    const uint32_t c = c0 + k;
    v[k] = load_elem<DT>(x, (rin && c < C) ? int64_t(r) * C + c : 0);
  }
  uint64_t mine = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const uint64_t m = __ballot(rin && c0 + k < C && v[k] > 0.0f);
    if (lane == k) mine = m;
  }
  if (lane < 16 && c0 + uint32_t(lane) < C) dst[size_t(w) * C + c0 + lane] = mine;
}

// ----------------------------------------------------------------------------- weight bytes
// sign(W) as signed bytes for the int8 dX product.  W is viewed as [D][K] (K = C*kh*kw,
// line l = (c, tap)); byte d of line l is +1 if W[d][l] > 0 else -1 for d < D, 0 for
// D <= d < Dp, stored chunk-major at ((d/32 * taps + tap) * C + c) * 32 + d % 32 so that the
// 32-byte chunks of consecutive channels are adjacent; lsum[l] = sum over d < D of the
// line.  One block of 1024 threads per 64 lines walks D in passes of 256 rows (one pass
// for D <= 256): each thread loads 16 rows of its line back to back, the pass is
// transposed through LDS (pitch 260 bytes = 65 dwords: the column writes of a wave spread
// over the banks) and written as 16-byte pieces of the 32-byte chunks.
constexpr int WB_THREADS = 1024;
constexpr int WB_ROWS = 256;                  // rows of D per pass: 16 per thread
constexpr int WB_PITCH = WB_ROWS + 4;
struct PackWGeom {
  uint32_t D, K, Dp, C, taps;
  FastDiv div_taps;
};
struct alignas(16) PackWLds {
  int8_t tile[64][WB_PITCH];
  int32_t pos[64];
};

template <int DT>
__device__ __forceinline__ void pack_w_body(const void *__restrict__ w, const PackWGeom &g,
                                            int8_t *__restrict__ dst, int32_t *__restrict__ lsum,
                                            uint32_t bid, PackWLds &sm) {
  constexpr int Q = WB_THREADS / 64;          // row phases per pass
  const int t = threadIdx.x, line = t & 63, q = t >> 6;
  const uint32_t l0 = bid * 64, l = l0 + line;
  if (t < 64) sm.pos[t] = 0;
  int mine = 0;
  for (uint32_t d0 = 0; d0 < g.Dp; d0 += WB_ROWS) {
    float v[WB_ROWS / Q];
#pragma unroll
    for (int k = 0; k < WB_ROWS / Q; ++k) {   // unconditional loads (element 0 outside) issue back to back
      const uint32_t d = d0 + Q * k + q;
      v[k] = load_elem<DT>(w, (d < g.D && l < g.K) ? int64_t(d) * g.K + l : 0);
    }
#pragma unroll
    for (int k = 0; k < WB_ROWS / Q; ++k) {
      const uint32_t d = d0 + Q * k + q;
      const bool in = d < g.D && l < g.K;
      const bool pos_sign = in && v[k] > 0.0f;
      mine += pos_sign ? 1 : 0;
      sm.tile[line][Q * k + q] = in ? (pos_sign ? int8_t(1) : int8_t(-1)) : int8_t(0);
    }
    __syncthreads();
    // 64 lines x 16 pieces of 16 bytes; pieces past Dp (last pass of a short D) are not stored.
    const int wl = t >> 4, part = t & 15;
    if (l0 + wl < g.K && d0 + 16 * part < g.Dp) {
      const uint32_t lw = l0 + wl, c = fdiv(lw, g.div_taps), tap = lw - c * g.taps;
      const uint32_t chunk = (d0 >> 5) + (part >> 1);
      const uint32_t *src = reinterpret_cast<const uint32_t *>(&sm.tile[wl][16 * part]);
      *reinterpret_cast<uint4 *>(dst + ((size_t(chunk) * g.taps + tap) * g.C + c) * 32 +
                                 16 * (part & 1)) = make_uint4(src[0], src[1], src[2], src[3]);
    }
    __syncthreads();
  }
  atomicAdd(&sm.pos[line], mine);
  __syncthreads();
  if (t < 64 && l0 + t < g.K) lsum[l0 + t] = 2 * sm.pos[t] - int(g.D);
}

inline PackWGeom pack_w_geom(const Layer &L) {
  const uint32_t taps = uint32_t(L.kh * L.kw);
  return PackWGeom{uint32_t(L.D), uint32_t(L.K), uint32_t(L.Wd * 64), uint32_t(L.C), taps,
                   make_fastdiv(taps)};
}
inline uint32_t pack_w_blocks(const Layer &L) { return uint32_t((L.K + 63) / 64); }

}  // namespace fqt
