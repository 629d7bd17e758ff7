// The two binary contractions of the 1-bit FQT backward on gfx950, int8 MFMA engine
// (Section 5.3, SCQ; Appendix C, Alg. 1 binary products and dequantization, the
// {0,1} <-> {+-1} conversion and the Folder).
//
// Both products contract b-bit codes q (one byte each, written by the quantizer next to
// the bit planes) with signs s = +-1 held as signed bytes, so one v_mfma_i32_32x32x32_i8
// chain gives I = sum_j q_j s_j exactly in int32.  For b = 8 the codes do not fit a
// signed byte: the MFMA takes q - 128 and 128 * (sum of the signs it saw) is added back.
//   dX: the weight signs arrive expanded to +-1 bytes (fqt_pack_weight_signs), so the
//       inner loop is 16-byte buffer loads and MFMAs.  The zero-point term c = sum over
//       the valid taps of the per-(channel, tap) sign sums is summed per output in the
//       split form and, in the register-tile form, is one float16 (D <= 2048) or a few
//       float32 MFMAs of the sign sums against the 0/1 reach flags (exact either way).
//   dW: the X signs stay packed; each 16-bit piece is expanded in registers to +-1
//       bytes once and feeds up to four MFMAs (128 kept channels).  c = 2 popcount - len.
// The rescale S * I + Z' * c is one float32 step per output without contraction.
//
// MFMA layouts (32 x 32 outputs, 16 accumulators per lane): lane l feeds row (src0) and
// column (src1) l % 32; in the i8 form its 16 bytes are contraction positions
// 16 (l / 32) .. 16 (l / 32) + 15, in the f32 32x32x2 form its one value is position
// l / 32, in the f16 32x32x16 form its 8 values are 8 of the 16 positions (the same
// ones in both operands).  Lane l then holds column l % 32 at rows
// 8 (v / 4) + 4 (l / 32) + (v % 4).
//
// Operands are read through buffer resources: a lane whose row does not exist (padding
// tap, pruned slot, channel past the end) gets the offset BUF_NONE, past every buffer,
// and loads zeros without touching memory.  Every operand layout puts the 32-byte
// contraction chunks of consecutive MFMA rows next to each other (chunk-major codes,
// word-major X signs, chunk-major weight bytes), so one operand load of a wave reads
// about 1 KB of contiguous memory instead of one cache line per lane.
#include <algorithm>
#include <type_traits>

#include "fqt_internal.hpp"

namespace fqt {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// The wave index as a scalar, so that per-wave loop bounds and strides stay in SGPRs.
__device__ __forceinline__ uint32_t wave_id() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

// 16 sign bits (LSB first) -> 16 signed bytes, +1 for a set bit and -1 for a clear one
// (byte m of dword k holds bit 4k + m).  A nibble times 0x00408102 puts bit m at bit
// 8m + 1 without carries; per byte 2t + 0x7F is 0x7F or 0x81, and flipping bit 7 gives
// 0xFF (-1) or 0x01 (+1).
__device__ __forceinline__ v4i signs16(uint32_t bits) {
  v4i r;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t t2 = (((bits >> (4 * k)) & 0xFu) * 0x00408102u) & 0x02020202u;
    r[k] = int((t2 + 0x7F7F7F7Fu) ^ 0x80808080u);
  }
  return r;
}

__device__ __forceinline__ v4i bias128(v4i a) {
  const int m = int(0x80808080u);
  return v4i{a.x ^ m, a.y ^ m, a.z ^ m, a.w ^ m};
}

__device__ __forceinline__ v16i mfma_i8(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float rescale(float S, int I, float Zp, float c) {
  return __fadd_rn(__fmul_rn(S, float(I)), __fmul_rn(Zp, c));
}

// The dispatcher hands the workgroups of a launch to the eight XCDs in turn (block b to
// XCD b % 8), and each XCD has its own L2.  xcd_tile maps the s-th block of a segment of n
// blocks to a tile index so that every XCD walks runs of RUN consecutive tiles: its k-th
// run (in dispatch order) is tiles [RUN (8 k + x), RUN (8 k + x + 1)) for x = s % 8, and
// neighbouring tiles, which read the same operand rows, share one L2.  A bijection of
// [0, n): blocks past the last whole round of 8 runs keep their own index.  (Any other
// dispatch order changes only which L2 a tile's operands go through.)
constexpr uint32_t XCDS = 8;
template <uint32_t RUN>
__device__ __forceinline__ uint32_t xcd_tile(uint32_t s, uint32_t n) {
  constexpr uint32_t ROUND = XCDS * RUN;
  if (s >= n / ROUND * ROUND) return s;
  const uint32_t x = s % XCDS, i = s / XCDS;
  return ((i / RUN) * XCDS + x) * RUN + i % RUN;
}

// Output row (0..31) of accumulator v of a lane in half-wave g.
__device__ __forceinline__ int acc_row(int v, int g) { return 8 * (v >> 2) + 4 * g + (v & 3); }

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
  const uint8_t *codes;          // PCQ codes [2*Wr][D][32], chunk-major
  const int32_t *kept, *count;   // [D], [1]
  const float *scale, *offset;   // [D]
  const float2 *slot_sz;         // [D] (scale, offset) by kept slot, or null (read via kept)
  const uint64_t *xsign;         // [Wr][K], word-major
  float *dW;                     // [D][K]
  int32_t *I_out;                // [D][K] or null
  int32_t *part;                 // [S][D][Kp] partial sums of each split (slots < count)
  int32_t *partT;                // [S][Kp] set bits of each split of each sign line
  uint32_t D, K, Kp, R, Rp, Wr, ktiles, kgroups, codes_bytes, xsign_bytes, S, wps;
  uint32_t wpw;                  // in-block reduction form: words of the contraction per wave
  FastDiv divS, divKg, divQ;    // divQ: Kp / 4
  FastDiv divKt;                 // ktiles
};

constexpr int DW_WAVES = 4;                 // column tiles per block, one per wave
constexpr int DW_THREADS = DW_WAVES * 64;
constexpr int DW_PREF = 4;                  // 64-bit words of the contraction per batch

// One batch of a wave's operands: PREF words of its sign column and the two 32-byte
// code chunks of each word.
template <int PREF>
struct DwBatch {
  uint64_t word[PREF];
  v4i A[PREF][2];
};
template <int PREF>
__device__ __forceinline__ void dw_issue(const DwArgs &a, __amdgpu_buffer_rsrc_t crs,
                                         __amdgpu_buffer_rsrc_t xrs, uint32_t aoff,
                                         uint32_t boff, uint32_t c0, uint32_t w_end,
                                         DwBatch<PREF> &b) {
  const uint32_t chunk_bytes = a.D * 32;      // one 32-position chunk of every PCQ row
#pragma unroll
  for (int u = 0; u < PREF; ++u) {
    const uint32_t c = c0 + u < w_end ? c0 + u : c0;   // past the end: word c0 again
    b.word[u] = load8(xrs, boff, c * a.K * 8);
#pragma unroll
    for (int h = 0; h < 2; ++h) b.A[u][h] = load16(crs, aoff, (2 * c + h) * chunk_bytes);
  }
}
template <bool B8, int PREF>
__device__ __forceinline__ void dw_consume(const DwBatch<PREF> &b, uint32_t c0, uint32_t w_end,
                                           int g, v16i &acc, uint32_t &tpart) {
#pragma unroll
  for (int u = 0; u < PREF; ++u) {
    if (c0 + u >= w_end) break;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t bits = uint32_t(b.word[u] >> (32 * h + 16 * g)) & 0xFFFFu;
      tpart += __popc(bits);
      acc = mfma_i8(B8 ? bias128(b.A[u][h]) : b.A[u][h], signs16(bits), acc);
    }
  }
}

// The contraction of one wave's 32x32 tile over the words [c_first, w_end) of its split,
// double-buffered: the loads of batch i + 1 issue before the products of batch i (a
// sched_barrier keeps the compiler from sinking them), so a long contraction costs one
// exposed memory latency.
template <bool B8, int PREF = DW_PREF>
__device__ __forceinline__ void dw_accumulate(const DwArgs &a, __amdgpu_buffer_rsrc_t crs,
                                              __amdgpu_buffer_rsrc_t xrs, uint32_t aoff,
                                              uint32_t boff, uint32_t c_first, uint32_t w_end,
                                              int g, v16i &acc, uint32_t &tpart) {
  if (c_first >= w_end) return;
  DwBatch<PREF> b0, b1;
  uint32_t c0 = c_first;
  dw_issue<PREF>(a, crs, xrs, aoff, boff, c0, w_end, b0);
  for (;;) {
    if (c0 + PREF < w_end) dw_issue<PREF>(a, crs, xrs, aoff, boff, c0 + PREF, w_end, b1);
    __builtin_amdgcn_sched_barrier(0);
    dw_consume<B8, PREF>(b0, c0, w_end, g, acc, tpart);
    c0 += PREF;
    if (c0 >= w_end) break;
    if (c0 + PREF < w_end) dw_issue<PREF>(a, crs, xrs, aoff, boff, c0 + PREF, w_end, b0);
    __builtin_amdgcn_sched_barrier(0);
    dw_consume<B8, PREF>(b1, c0, w_end, g, acc, tpart);
    c0 += PREF;
    if (c0 >= w_end) break;
  }
}
// Words per batch of the in-block reduction form (8 was measured slower at the 256 -> 256
// conv on 8x8 maps: the products launch it shares with the dX blocks lost occupancy).
constexpr int DW_KRED_PREF = 4;

// dW rows of the slot tile [j0, j0 + 32) of one wave's 32 columns written directly (one
// split, S = 1): I, T, the rescale S_d I + Z'_d (2T - N*Ho*Wo) (b = 8 adds back
// 128 (2T - Rp)), zero rows for pruned slots.  acc: the wave's tile (rows
// acc_row(v, g) of column lane % 32); T: set bits of this lane's column.
template <bool B8>
__device__ __forceinline__ void dw_write_direct(const DwArgs &a, uint32_t j0, uint32_t kc,
                                                int count, const v16i &acc, int T) {
  const int g = (threadIdx.x & 63) >> 5;
  if (kc >= a.K) return;
  // The rows' kept ids, scales and offsets first, all loads together (after a row's dW
  // store the next row's loads could not move ahead of it).
  uint32_t dv[16];
  float2 szv[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const uint32_t j = j0 + uint32_t(acc_row(v, g));
    dv[v] = j < a.D ? uint32_t(a.kept[j]) : 0u;
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const uint32_t j = j0 + uint32_t(acc_row(v, g));
    szv[v] = make_float2(0.0f, 0.0f);
    if (int(j) < count)
      szv[v] = a.slot_sz ? a.slot_sz[j] : make_float2(a.scale[dv[v]], a.offset[dv[v]]);
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const uint32_t j = j0 + uint32_t(acc_row(v, g));
    if (j >= a.D) continue;
    const size_t d = dv[v];
    int I = 0;
    float out = 0.0f;
    if (int(j) < count) {
      I = acc[v] + (B8 ? 128 * (2 * T - int(a.Rp)) : 0);
      out = rescale(szv[v].x, I, szv[v].y, float(2 * T - int(a.R)));
    }
    a.dW[d * a.K + kc] = out;
    if (a.I_out) a.I_out[d * a.K + kc] = I;
  }
}

// Split-R partial products.  Grid: S splits x ceil(ceil(K/32) / 4) column groups x
// ceil(D/32) slot tiles over the slot capacity, the split index fastest (consecutive
// blocks land on different XCDs, so each XCD reads its own slices of the codes and of the
// signs) and the slot tile slowest.  Wave w of a block computes the 32x32 MFMA tile (slot
// tile, column tile 4 * group + w) over the words [s * wps, (s + 1) * wps) of the
// contraction over N*Ho*Wo: the four waves read the same code rows (one fetch from L2)
// and their own sign columns, and each writes its tile and the set-bit counts of its
// columns to the split's slice.  No LDS, no barrier.
// DIRECT (S = 1): the wave writes dW itself, and slot tiles past the kept channels zero
// their rows; otherwise those blocks exit at once and the finish pass writes dW.
template <bool B8, bool DIRECT>
__device__ __forceinline__ void dw_part_body(const DwArgs &a, uint32_t bid) {
  const int lane = threadIdx.x & 63;
  const uint32_t wave = wave_id();
  const int i = lane & 31, g = lane >> 5;
  const int count = *a.count;
  const uint32_t rest = fdiv(bid, a.divS);
  const uint32_t sp = bid - rest * a.S;
  const uint32_t rt = fdiv(rest, a.divKg);
  const uint32_t kt = (rest - rt * a.kgroups) * DW_WAVES + wave;
  const uint32_t j0 = rt * 32;
  if (kt >= a.ktiles) return;                   // past the columns
  const uint32_t kc = kt * 32 + i;
  if (int(j0) >= count) {                       // past the kept channels
    if (DIRECT) dw_write_direct<B8>(a, j0, kc, count, v16i{0}, 0);
    return;
  }

  const __amdgpu_buffer_rsrc_t crs = buffer_of(a.codes, a.codes_bytes);
  const __amdgpu_buffer_rsrc_t xrs = buffer_of(a.xsign, a.xsign_bytes);
  const uint32_t j = j0 + i;
  const uint32_t aoff = int(j) < count ? j * 32 + 16 * g : BUF_NONE;
  const bool b_ok = kc < a.K;
  const uint32_t boff = b_ok ? kc * 8 : BUF_NONE;
  const uint32_t w_end = min(a.Wr, (sp + 1) * a.wps);
  v16i acc = v16i{0};
  uint32_t tpart = 0;
  dw_accumulate<B8>(a, crs, xrs, aoff, boff, sp * a.wps, w_end, g, acc, tpart);

  // Set bits of column kc in this split: lanes i and i + 32 counted the two halves of
  // every 32-bit piece.
  const uint32_t T = tpart + lane_xor<32>(tpart);
  if (DIRECT) {
    dw_write_direct<B8>(a, j0, kc, count, acc, int(T));
    return;
  }
  if (!b_ok) return;
  if (rt == 0 && g == 0) a.partT[size_t(sp) * a.Kp + kc] = int32_t(T);
  int32_t *out = a.part + (size_t(sp) * a.D + j0) * a.Kp + kc;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int row = acc_row(v, g);
    if (int(j0) + row < count) out[size_t(row) * a.Kp] = acc[v];
  }
}

// dW with the contraction split over the four waves of a block and reduced in LDS (no
// partial sums leave the workgroup, no finish pass).  Grid: ceil(D/32) slot tiles x
// ceil(K/32) column tiles over the slot capacity, column tiles fastest (a column tile keeps
// its XCD across slot tiles when the number of column tiles is a multiple of eight, so its
// sign words are fetched into one L2).  Wave w contracts the 32 x 32 tile over the words
// [w wpw, (w + 1) wpw) of N*Ho*Wo; the four partial tiles and set-bit counts meet in LDS,
// and wave w finishes accumulator registers 4w .. 4w + 3 (slot rows 8w + 4g + u): the sum
// over the waves, the b = 8 bias term, the rescale and the dW stores.  Slot tiles past the
// kept channels write their rows of zeros.
struct DwRedLds {
  int32_t red[DW_WAVES][16][64];
  uint32_t tred[DW_WAVES][32];
};
template <bool B8>
__device__ __forceinline__ void dw_kred_body(const DwArgs &a, uint32_t bid, DwRedLds &sm) {
  const int lane = threadIdx.x & 63;
  const uint32_t wave = wave_id();
  const int i = lane & 31, g = lane >> 5;
  const int count = *a.count;
  const uint32_t rt = fdiv(bid, a.divKt);
  const uint32_t kt = bid - rt * a.ktiles;
  const uint32_t j0 = rt * 32, kc = kt * 32 + uint32_t(i);
  const bool live = int(j0) < count;            // uniform over the block
  if (live) {
    const __amdgpu_buffer_rsrc_t crs = buffer_of(a.codes, a.codes_bytes);
    const __amdgpu_buffer_rsrc_t xrs = buffer_of(a.xsign, a.xsign_bytes);
    const uint32_t j = j0 + uint32_t(i);
    const uint32_t aoff = int(j) < count ? j * 32 + 16 * g : BUF_NONE;
    const uint32_t boff = kc < a.K ? kc * 8 : BUF_NONE;
    const uint32_t cb = wave * a.wpw;
    const uint32_t ce = min(a.Wr, cb + a.wpw);
    v16i acc = v16i{0};
    uint32_t tpart = 0;
    dw_accumulate<B8, DW_KRED_PREF>(a, crs, xrs, aoff, boff, cb, ce, g, acc, tpart);
    const uint32_t T = tpart + lane_xor<32>(tpart);
#pragma unroll
    for (int v = 0; v < 16; ++v) sm.red[wave][v][lane] = acc[v];
    if (g == 0) sm.tred[wave][i] = T;
  }
  __syncthreads();
  int T = 0;
  if (live) T = int(sm.tred[0][i] + sm.tred[1][i] + sm.tred[2][i] + sm.tred[3][i]);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int v = 4 * int(wave) + u;
    const uint32_t j = j0 + uint32_t(acc_row(v, g));
    if (j >= a.D) continue;
    const size_t d = size_t(a.kept[j]);
    int I = 0;
    float out = 0.0f;
    if (int(j) < count) {
      I = sm.red[0][v][lane] + sm.red[1][v][lane] + sm.red[2][v][lane] + sm.red[3][v][lane];
      if (B8) I += 128 * (2 * T - int(a.Rp));
      const float2 sz = a.slot_sz ? a.slot_sz[j] : make_float2(a.scale[d], a.offset[d]);
      out = rescale(sz.x, I, sz.y, float(2 * T - int(a.R)));
    }
    if (kc < a.K) {
      a.dW[d * a.K + kc] = out;
      if (a.I_out) a.I_out[d * a.K + kc] = I;
    }
  }
}

// Large dW outputs in one split (DIRECT): each wave holds a (32 RT) x (32 CT) block of
// the output in RT x CT MFMA tiles, and a block's four waves take four adjacent column
// blocks of the same slots (the code rows come from L2 once).  Grid: ceil(D / (32 RT))
// slot blocks x ceil(K / (128 CT)) column groups, slots slowest.
// Here the X signs enter the MFMA as 0/1 bytes b (three VALU operations per four signs,
// shared by the row tiles) instead of +-1, and the signed sum comes back per output as
// sum q s = 2 sum q b - sum q (s = 2b - 1; b = 0 on the zero tail of the last word, where
// q = 0 too).  The code sums sum q of the rows are taken from the A fragments with
// v_dot4_u32_u8 (four per fragment, shared by the column tiles).  For b = 8 the codes
// enter as q - 128: sum q b = acc + 128 T.  The words of the contraction stream through a
// ring of ST register batches.
// Shapes (row tiles RT, column tiles CT, ring depth ST): long contractions take 2 x 4
// tiles and a four-word ring at two waves per SIMD; short ones (a few words, where the
// dW stores dominate) 2 x 2 tiles and two words at the occupancy the registers allow.
constexpr int DWB_LONG_WORDS = 8;     // contractions of at least this many words: long form
template <int RT, int CT>
struct DwBigBatch {
  uint64_t word[CT];
  v4i A[2][RT];                           // [half][row tile]
};
template <int RT, int CT>
__device__ __forceinline__ void dwb_issue(const DwArgs &a, __amdgpu_buffer_rsrc_t crs,
                                          __amdgpu_buffer_rsrc_t xrs, const uint32_t (&aoff)[RT],
                                          const uint32_t (&boff)[CT], uint32_t c,
                                          DwBigBatch<RT, CT> &b) {
  // Word offsets as scalars (kept out of any vector induction variable).
  const uint32_t xs = __builtin_amdgcn_readfirstlane(c * a.K * 8);
  const uint32_t cs0 = __builtin_amdgcn_readfirstlane(2 * c * a.D * 32);
  const uint32_t cs1 = __builtin_amdgcn_readfirstlane((2 * c + 1) * a.D * 32);
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) b.word[ct] = load8(xrs, boff[ct], xs);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    b.A[0][rt] = load16(crs, aoff[rt], cs0);
    b.A[1][rt] = load16(crs, aoff[rt], cs1);
  }
}
// Four sign bits of `half` from bit `off` (LSB first) as four 0/1 bytes: a nibble times
// 0x00204081 puts bit m at bit 8m (the cross terms land on other bits, without carries)
// and the mask keeps those.
__device__ __forceinline__ int bits01x4(uint32_t half, uint32_t off) {
  return int((__builtin_amdgcn_ubfe(half, off, 4) * 0x00204081u) & 0x01010101u);
}
template <bool B8, int RT, int CT>
__device__ __forceinline__ void dwb_consume(const DwBigBatch<RT, CT> &b, const uint32_t (&off)[4],
                                            v16i (&acc)[RT][CT], uint32_t (&tcnt)[CT],
                                            uint32_t (&qsum)[RT]) {
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
    tcnt[ct] += __popc(uint32_t(b.word[ct])) + __popc(uint32_t(b.word[ct] >> 32));
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    // For b = 8 the sums are taken of the biased bytes q - 128 (signed), the only form
    // kept in registers; the epilogue adds 128 per position back.
    v4i A[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      A[rt] = B8 ? bias128(b.A[h][rt]) : b.A[h][rt];
#pragma unroll
      for (int k = 0; k < 4; ++k)
        qsum[rt] = B8 ? uint32_t(__builtin_amdgcn_sdot4(A[rt][k], 0x01010101, int(qsum[rt]), false))
                      : __builtin_amdgcn_udot4(uint32_t(A[rt][k]), 0x01010101u, qsum[rt], false);
    }
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const uint32_t half = uint32_t(b.word[ct] >> (32 * h));
      const v4i B = v4i{bits01x4(half, off[0]), bits01x4(half, off[1]), bits01x4(half, off[2]),
                        bits01x4(half, off[3])};
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt][ct] = mfma_i8(A[rt], B, acc[rt][ct]);
    }
  }
}
// SPLIT: the same tiles over the word slice [s wps, (s + 1) wps) of a split-R product,
// writing the slice's partial sums (in the split kernel's form, sum over the slice of
// A_r s_r with A_r the MFMA code byte: 2 sum A b - sum A) and its set-bit counts for the
// finish pass.  Grid: S slices (fastest) x slot blocks x column groups.
template <bool B8, int RT, int CT, int ST, bool SPLIT = false>
__device__ __forceinline__ void dw_big_body(const DwArgs &a, uint32_t bid) {
  const int lane = threadIdx.x & 63;
  const uint32_t wave = wave_id();
  const int i = lane & 31, g = lane >> 5;
  const int count = *a.count;
  const uint32_t kgroups = (a.K + DW_WAVES * 32 * CT - 1) / (DW_WAVES * 32 * CT);
  uint32_t sp = 0;
  if (SPLIT) {
    const uint32_t rest = fdiv(bid, a.divS);
    sp = bid - rest * a.S;
    bid = rest;
  }
  const uint32_t cb = SPLIT ? sp * a.wps : 0u;
  const uint32_t ce = SPLIT ? min(a.Wr, cb + a.wps) : a.Wr;
  const uint32_t rb = bid / kgroups;
  const uint32_t j0 = rb * (32 * RT);
  const uint32_t k0 = ((bid - rb * kgroups) * DW_WAVES + wave) * (32 * CT);
  if (k0 >= a.K) return;
  v16i acc[RT][CT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = v16i{0};
  uint32_t tcnt[CT], qsum[RT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) tcnt[ct] = 0u;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) qsum[rt] = 0u;
  if (int(j0) < count && ce > cb) {
    const __amdgpu_buffer_rsrc_t crs = buffer_of(a.codes, a.codes_bytes);
    const __amdgpu_buffer_rsrc_t xrs = buffer_of(a.xsign, a.xsign_bytes);
    uint32_t aoff[RT], boff[CT], off[4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const uint32_t j = j0 + 32 * rt + i;
      aoff[rt] = int(j) < count ? j * 32 + 16 * g : BUF_NONE;
    }
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const uint32_t kc = k0 + 32 * ct + i;
      boff[ct] = kc < a.K ? kc * 8 : BUF_NONE;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) off[k] = uint32_t(16 * g + 4 * k);
    // A ring of ST words: word c + ST is requested as soon as word c has
    // been used, so ST - 1 words are in flight during each word's products.  Every
    // step issues the same loads (a word past the end re-reads the last one), so the
    // waits count exactly.
    DwBigBatch<RT, CT> bs[ST];
    const uint32_t last = ce - 1;
#pragma unroll
    for (int u = 0; u < ST; ++u) dwb_issue(a, crs, xrs, aoff, boff, min(cb + uint32_t(u), last), bs[u]);
    for (uint32_t c = cb; c < ce; c += ST) {
#pragma unroll
      for (int u = 0; u < ST; ++u) {
        if (c + u >= ce) break;
        dwb_consume<B8, RT, CT>(bs[u], off, acc, tcnt, qsum);
        __builtin_amdgcn_sched_barrier(0);
        dwb_issue(a, crs, xrs, aoff, boff, min(c + u + ST, last), bs[u]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  // Lane i (and i + 32) holds half of the code sum of row i of each row tile; the
  // accumulator rows of a lane are acc_row(v, g), fetched from their lanes.
  if (SPLIT) {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const uint32_t kc = k0 + 32 * ct + i;
      if (rb == 0 && g == 0 && kc < a.K) a.partT[size_t(sp) * a.Kp + kc] = int32_t(tcnt[ct]);
    }
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int qrow = int(qsum[rt] + lane_xor<32>(qsum[rt]));   // sum of A over the slice
      int qv[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) qv[v] = __shfl(qrow, acc_row(v, g));
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const uint32_t kc = k0 + 32 * ct + i;
        if (kc >= a.K) continue;
        int32_t *out = a.part + (size_t(sp) * a.D + j0 + 32 * rt) * a.Kp + kc;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = acc_row(v, g);
          if (int(j0) + 32 * rt + row < count) out[size_t(row) * a.Kp] = 2 * acc[rt][ct][v] - qv[v];
        }
      }
    }
    return;
  }
  // The 32 x 32 tiles go out through a row-major LDS copy per wave, each lane storing 16
  // consecutive columns of one kept row in 16-byte pieces (the integer debug output takes
  // the element stores below).
  if constexpr (!SPLIT) {
    if (!a.I_out) {
      __shared__ float stage[DW_WAVES][32 * 32];
      float *st = stage[wave];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int qrow = int(qsum[rt] + lane_xor<32>(qsum[rt])) + (B8 ? 128 * int(a.Rp) : 0);
        int qv[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) qv[v] = __shfl(qrow, acc_row(v, g));
        const uint32_t jt = j0 + 32 * rt;
        // The rows' scales and offsets and this lane's store row, loaded once per row tile,
        // all at once (inside the column-tile loop they would follow each tile's dW stores,
        // which the compiler cannot move them across: a dependent round trip per tile).
        float2 szv[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const uint32_t j = jt + uint32_t(acc_row(v, g));
          szv[v] = make_float2(0.0f, 0.0f);
          if (int(j) < count)
            szv[v] = a.slot_sz ? a.slot_sz[j] : make_float2(a.scale[a.kept[j]], a.offset[a.kept[j]]);
        }
        const uint32_t jrow = jt + uint32_t(lane >> 1);
        const size_t drow = jrow < a.D ? size_t(a.kept[jrow]) : 0;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          const int T = int(tcnt[ct]);
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const uint32_t j = jt + uint32_t(acc_row(v, g));
            float out = 0.0f;
            if (int(j) < count) {
              const int I = 2 * (acc[rt][ct][v] + (B8 ? 128 * T : 0)) - qv[v];
              out = rescale(szv[v].x, I, szv[v].y, float(2 * T - int(a.R)));
            }
            st[acc_row(v, g) * 32 + i] = out;
          }
          __builtin_amdgcn_wave_barrier();    // LDS operations of a wave run in order
          const uint32_t j = jrow;
          const uint32_t c0 = k0 + 32 * ct + 16 * uint32_t(lane & 1);
          if (j < a.D && c0 < a.K) {
            const float *src = st + (lane >> 1) * 32 + 16 * (lane & 1);
            float *dst = a.dW + drow * a.K + c0;
            if (c0 + 16 <= a.K && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
              const uint4 *s4 = reinterpret_cast<const uint4 *>(src);
              uint4 *d4 = reinterpret_cast<uint4 *>(dst);
#pragma unroll
              for (int k = 0; k < 4; ++k) d4[k] = s4[k];
            } else {
              for (uint32_t e = 0; e < 16 && c0 + e < a.K; ++e) dst[e] = src[e];
            }
          }
          __builtin_amdgcn_wave_barrier();    // the next tile's copy waits for these reads
        }
      }
      return;
    }
  }
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    // Sum of the codes of row i of the tile (b = 8: of q - 128 over all Rp positions).
    const int qrow = int(qsum[rt] + lane_xor<32>(qsum[rt])) + (B8 ? 128 * int(a.Rp) : 0);
    int qv[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) qv[v] = __shfl(qrow, acc_row(v, g));
    const uint32_t jt = j0 + 32 * rt;
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const uint32_t kc = k0 + 32 * ct + i;
      if (kc >= a.K) continue;
      const int T = int(tcnt[ct]);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const uint32_t j = jt + uint32_t(acc_row(v, g));
        if (j >= a.D) continue;
        const size_t d = size_t(a.kept[j]);
        int I = 0;
        float out = 0.0f;
        if (int(j) < count) {
          const float2 sz = a.slot_sz ? a.slot_sz[j] : make_float2(a.scale[d], a.offset[d]);
          I = 2 * (acc[rt][ct][v] + (B8 ? 128 * T : 0)) - qv[v];
          out = rescale(sz.x, I, sz.y, float(2 * T - int(a.R)));
        }
        a.dW[d * a.K + kc] = out;
        if (a.I_out) a.I_out[d * a.K + kc] = I;
      }
    }
  }
}
// Blocks of the big form with RT row tiles and CT column tiles per wave.
uint32_t dw_big_blocks(uint32_t D, uint32_t K, int rt, int ct) {
  return ((D + 32 * rt - 1) / (32 * rt)) * ((K + DW_WAVES * 32 * ct - 1) / (DW_WAVES * 32 * ct));
}

// Split-R partials in the big form (long slices of the contraction, wide outputs): two row
// tiles per wave, or one when the kept channels are expected to fit 32 rows (a second
// row tile would multiply zeros).  A four-word ring (163 registers for two row tiles, 96
// for one) was measured 2-5 % faster than two words on VGG-16's layers at 224.
template <bool B8, int RT>
__global__ __launch_bounds__(DW_THREADS) __attribute__((amdgpu_waves_per_eu(3, 3))) void k_mfma_dw_split(DwArgs a) {
  dw_big_body<B8, RT, 2, 4, true>(a, blockIdx.x);
}
uint32_t dw_split_blocks(const DwArgs &a, int rt) {
  return a.S * dw_big_blocks(a.D, a.K, rt, 2);
}

// Long contractions: two waves per SIMD (the accumulators and the word ring fit 256
// registers).
template <bool B8>
__global__ __launch_bounds__(DW_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_mfma_dw_big(DwArgs a) {
  dw_big_body<B8, 2, 4, 4>(a, blockIdx.x);
}
// Short contractions: three waves per SIMD, for the stores.
template <bool B8>
__global__ __launch_bounds__(DW_THREADS) __attribute__((amdgpu_waves_per_eu(3, 3))) void k_mfma_dw_short(DwArgs a) {
  dw_big_body<B8, 2, 2, 2>(a, blockIdx.x);
}

template <bool B8, bool DIRECT>
__global__ __launch_bounds__(DW_THREADS) void k_mfma_dw_part(DwArgs a) {
  dw_part_body<B8, DIRECT>(a, blockIdx.x);
}

template <bool B8>
__global__ __launch_bounds__(DW_THREADS) void k_mfma_dw_kred(DwArgs a) {
  __shared__ DwRedLds sm;
  dw_kred_body<B8>(a, blockIdx.x, sm);
}

// dW from the split partials: one thread per 4 columns (slot, k .. k + 3) of the slot
// capacity, reading 16 bytes of each partial row.  A kept slot sums its S partials,
// I = sum (+ 128 (2T - Rp) for b = 8, whose codes entered as q - 128 against every sign
// including the zero tail of the last word) and writes S_d * I + Z'_d * (2T - N*Ho*Wo) to
// row d = kept[slot]; a pruned slot zeroes its row.
template <bool B8>
__global__ __launch_bounds__(256) void k_dw_finish(DwArgs a) {
  const uint32_t e = blockIdx.x * 256 + threadIdx.x;
  const uint32_t qrow = a.Kp / 4;
  if (e >= a.D * qrow) return;
  const uint32_t slot = fdiv(e, a.divQ), k = 4 * (e - slot * qrow);
  if (k >= a.K) return;
  const int count = *a.count;
  const size_t d = size_t(a.kept[slot]);
  int I[4] = {0, 0, 0, 0};
  float out[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (int(slot) < count) {
    int4 acc = make_int4(0, 0, 0, 0), T4 = make_int4(0, 0, 0, 0);
    // Eight slices' loads issue together (a slice past S re-reads the last one and is not
    // added), so the sum costs one memory latency per eight slices.
    constexpr uint32_t U = 8;
    for (uint32_t s0 = 0; s0 < a.S; s0 += U) {
      int4 v[U], t4[U];
#pragma unroll
      for (uint32_t u = 0; u < U; ++u) {
        const uint32_t s = min(s0 + u, a.S - 1);
        v[u] = *reinterpret_cast<const int4 *>(a.part + (size_t(s) * a.D + slot) * a.Kp + k);
        t4[u] = *reinterpret_cast<const int4 *>(a.partT + size_t(s) * a.Kp + k);
      }
#pragma unroll
      for (uint32_t u = 0; u < U; ++u) {
        const int m = s0 + u < a.S ? 1 : 0;
        acc.x += m * v[u].x; acc.y += m * v[u].y; acc.z += m * v[u].z; acc.w += m * v[u].w;
        T4.x += m * t4[u].x; T4.y += m * t4[u].y; T4.z += m * t4[u].z; T4.w += m * t4[u].w;
      }
    }
    const int T[4] = {T4.x, T4.y, T4.z, T4.w};
    I[0] = acc.x; I[1] = acc.y; I[2] = acc.z; I[3] = acc.w;
    const float2 sz = a.slot_sz ? a.slot_sz[slot] : make_float2(a.scale[d], a.offset[d]);
    const float Sd = sz.x, Zd = sz.y;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (B8) I[u] += 128 * (2 * T[u] - int(a.Rp));
      out[u] = rescale(Sd, I[u], Zd, float(2 * T[u] - int(a.R)));
    }
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (k + u >= a.K) break;
    a.dW[d * a.K + k + u] = out[u];
    if (a.I_out) a.I_out[d * a.K + k + u] = I[u];
  }
}

// The same for many splits: one block per (slot, 64 columns); thread t sums every 16th
// split of column quad t % 16 from split t / 16, and the 16 partial sums of each quad
// meet in LDS.
constexpr int DWF_CHUNKS = 16;
template <bool B8>
__global__ __launch_bounds__(256) void k_dw_finish_wide(DwArgs a) {
  __shared__ int4 red[DWF_CHUNKS][16], tred[DWF_CHUNKS][16];
  const int t = threadIdx.x, quad = t & 15, chunk = t >> 4;
  const uint32_t qblocks = a.Kp / 64 + (a.Kp % 64 ? 1 : 0);
  const uint32_t slot = blockIdx.x / qblocks;
  const uint32_t k = (blockIdx.x - slot * qblocks) * 64 + 4 * quad;
  const int count = *a.count;
  const bool live = int(slot) < count && k < a.Kp;
  int4 acc = make_int4(0, 0, 0, 0), T4 = make_int4(0, 0, 0, 0);
  if (live) {
    // Four of this chunk's slices load together (a slice past S re-reads the last one and
    // is not added).
    constexpr uint32_t U = 4;
    for (uint32_t s0 = chunk; s0 < a.S; s0 += U * DWF_CHUNKS) {
      int4 v[U], t4[U];
#pragma unroll
      for (uint32_t u = 0; u < U; ++u) {
        const uint32_t s = min(s0 + u * DWF_CHUNKS, a.S - 1);
        v[u] = *reinterpret_cast<const int4 *>(a.part + (size_t(s) * a.D + slot) * a.Kp + k);
        t4[u] = *reinterpret_cast<const int4 *>(a.partT + size_t(s) * a.Kp + k);
      }
#pragma unroll
      for (uint32_t u = 0; u < U; ++u) {
        const int m = s0 + u * DWF_CHUNKS < a.S ? 1 : 0;
        acc.x += m * v[u].x; acc.y += m * v[u].y; acc.z += m * v[u].z; acc.w += m * v[u].w;
        T4.x += m * t4[u].x; T4.y += m * t4[u].y; T4.z += m * t4[u].z; T4.w += m * t4[u].w;
      }
    }
  }
  red[chunk][quad] = acc;
  tred[chunk][quad] = T4;
  __syncthreads();
  if (chunk != 0 || k >= a.K) return;
#pragma unroll
  for (int c = 1; c < DWF_CHUNKS; ++c) {
    const int4 v = red[c][quad], t4 = tred[c][quad];
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    T4.x += t4.x; T4.y += t4.y; T4.z += t4.z; T4.w += t4.w;
  }
  const size_t d = size_t(a.kept[slot]);
  int I[4] = {0, 0, 0, 0};
  float out[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (live) {
    const int T[4] = {T4.x, T4.y, T4.z, T4.w};
    I[0] = acc.x; I[1] = acc.y; I[2] = acc.z; I[3] = acc.w;
    const float2 sz = a.slot_sz ? a.slot_sz[slot] : make_float2(a.scale[d], a.offset[d]);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (B8) I[u] += 128 * (2 * T[u] - int(a.Rp));
      out[u] = rescale(sz.x, I[u], sz.y, float(2 * T[u] - int(a.R)));
    }
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (k + u >= a.K) break;
    a.dW[d * a.K + k + u] = out[u];
    if (a.I_out) a.I_out[d * a.K + k + u] = I[u];
  }
}
// Splits above which the finish takes a block per (slot, 64 columns).
constexpr uint32_t DWF_WIDE = 32;

// ----------------------------------------------------------------------------- dX

struct DxArgs {
  const uint8_t *codes;          // PSQ codes [Dp/32][N*Ho*Wo][32], chunk-major
  const int32_t *kept, *count;   // [N], [1]
  const float *scale, *offset;   // [N]
  const float2 *slot_sz;         // [N] (scale, offset) by kept slot, or null (read via kept)
  const int8_t *wsb;             // sign(W) bytes [Dp/32][kh*kw][C][32]: +-1, 0 past D
  const int32_t *wlsum;          // [C*kh*kw] sum over d of the signs of each line
  void *dX;                      // [N][C][H][W]
  int32_t *I_out;
  int dx_t;
  uint32_t N, C, H, W, HW, Ho, Wo, P, R, Dp, ctiles, CHW, taps, nch;   // nch = Dp / 32
  uint32_t codes_bytes, wsb_bytes;
  int kh, kw, sh, sw, ph, pw;
  FastDiv divHW, divW, divKw, divNch, divCt, divSh, divSw;
  uint32_t nblocks;              // blocks of the dX grid (compute tiles + zero pool)
  uint32_t zpieces;              // pieces of DX_ZCHUNK elements per pruned sample
  uint32_t wide;                 // 0: split form; CT >= 1: register tiles, CT channel tiles
  uint32_t cblocks;              // register-tile form: channel blocks of 32 CT channels
  FastDiv divCb;
};

constexpr int DX_MAX_TAPS = 64;
constexpr uint32_t DX_ZCHUNK = 65536;    // elements of a pruned sample one block zeroes
constexpr int DX_WAVES = 4;
constexpr int DX_THREADS = DX_WAVES * 64;
// Tiles (channel tiles fastest, then pixel tiles) of one XCD run: 16 split-form tiles of
// 32 x 32, 32 register-form tiles of 256 pixels x 32 CT channels.
constexpr uint32_t DX_XCD_RUN = 16, DXW_XCD_RUN = 32;

// NB: contraction steps (tap, 32 bytes of D) a wave loads at once, sized on the host so
// that the common shapes take one batch: the loads of a wave then cost one memory latency.
// Grid: one block per 32x32 tile of (channel, row m = (kept slot, h, w)) over the capacity
// N*H*W rows, plus a pool of extra blocks.  Blocks of the first ceil(count*H*W/32) row
// tiles compute; all later blocks zero the pruned samples of dX (each a contiguous run of
// C*H*W elements) in pieces of DX_ZCHUNK elements.
// A computing block is one 32x32 MFMA tile with the sign operand as src0 (rows =
// channels) so output lanes run along pixels.  Its four waves take every fourth
// contraction step (tap, 32 bytes of D).  For tap (i, j) a pixel (h, w) reads the code row
// of the output pixel (ho, wo) with ho*sh - ph + i = h and wo*sw - pw + j = w, or nothing;
// the byte offset of every (tap, pixel) row is tabulated once per block, next to the sign
// sums of the block's channels per tap.  The four partial tiles meet in LDS and wave w
// finishes accumulator registers 4w .. 4w + 3 (channel rows 8w + 4g + u): their integer
// sums, the zero-point term c = sum of the channel's sign sums over the taps that reach
// the pixel (exact integers), the rescale and the stores.
struct alignas(16) DxLds {
  uint32_t rowoff[DX_MAX_TAPS][32];     // 32 * code row, BUF_NONE if none
  int32_t wl[DX_MAX_TAPS][32];          // sign sum of line (channel c0 + k, tap), 0 past C
  int32_t red[DX_WAVES][16][64];        // partial tiles of the four waves
  int32_t pix_out[32];                  // NCHW offset of (sample, pixel) minus channel
  float pix_s[32], pix_z[32];
};

// Zeroing of the pruned samples by the blocks of the zero pool: task t of
// (N - count) * zpieces is piece t % zpieces of pruned slot t / zpieces.
__device__ __forceinline__ void dx_zero_pool(const DxArgs &a, uint32_t zb, uint32_t nz,
                                             int count) {
  const int t = threadIdx.x;
  const uint32_t tasks = (a.N - uint32_t(count)) * a.zpieces;
  for (uint32_t task = zb; task < tasks; task += nz) {
    const uint32_t slot = task / a.zpieces, piece = task - slot * a.zpieces;
    const size_t n = size_t(a.kept[uint32_t(count) + slot]);
    const size_t first = size_t(piece) * DX_ZCHUNK;
    const size_t len = min(size_t(DX_ZCHUNK), size_t(a.CHW) - first);
    zero_run(a.dX, n * a.CHW + first, len, a.dx_t == FQT_BF16 ? 2 : 4, t, DX_THREADS);
    if (a.I_out) zero_run(a.I_out, n * a.CHW + first, len, 4, t, DX_THREADS);
  }
}

// The code-row offsets of a block's BP pixel rows m0 .. m0 + BP - 1 over the taps:
// rowoff[tap][p] = 32 * (code row of the output pixel that pixel m0 + p meets through the
// tap), BUF_NONE where the tap falls between strides or outside dY, or past the live rows.
// Thread t decodes pixel p = t % BP once and walks the taps t / BP, t / BP + NT / BP, ...
// (a pixel's taps differ only in the tap's (i, j)).
template <uint32_t BP, int NT>
__device__ __forceinline__ void dx_row_table(const DxArgs &a, uint32_t m0, uint32_t live_rows,
                                             uint32_t (*rowoff)[BP]) {
  static_assert(NT % BP == 0, "whole pixel sets per pass");
  constexpr uint32_t STEP = NT / BP;
  const uint32_t p = uint32_t(threadIdx.x) % BP;
  const uint32_t m = m0 + p;
  const bool live = m < live_rows;
  uint32_t slot = 0, h = 0, w = 0;
  if (live) {
    slot = fdiv(m, a.divHW);
    const uint32_t pix = m - slot * a.HW;
    h = fdiv(pix, a.divW);
    w = pix - h * a.W;
  }
  uint32_t tap = uint32_t(threadIdx.x) / BP;
  uint32_t ti = fdiv(tap, a.divKw), tj = tap - ti * uint32_t(a.kw);
  for (; tap < a.taps; tap += STEP) {
    uint32_t off = BUF_NONE;
    const int th = int(h) + a.ph - int(ti), tw = int(w) + a.pw - int(tj);
    if (live && th >= 0 && tw >= 0) {
      const uint32_t ho = fdiv(uint32_t(th), a.divSh), wo = fdiv(uint32_t(tw), a.divSw);
      if (ho * uint32_t(a.sh) == uint32_t(th) && wo * uint32_t(a.sw) == uint32_t(tw) &&
          ho < a.Ho && wo < a.Wo)
        off = (slot * a.P + ho * a.Wo + wo) * 32;
    }
    rowoff[tap][p] = off;
    tj += STEP;
    while (tj >= uint32_t(a.kw)) {
      tj -= uint32_t(a.kw);
      ++ti;
    }
  }
}

template <bool B8, int NB>
__device__ __forceinline__ void dx_body(const DxArgs &a, uint32_t bid, DxLds &sm) {
  bid = xcd_tile<DX_XCD_RUN>(bid, a.nblocks);
  const int t = threadIdx.x, lane = t & 63;
  const uint32_t wave = wave_id();
  const int i = lane & 31, g = lane >> 5;
  const int count = *a.count;
  // Loads that do not depend on the count issue with it: the pixel parameters and the
  // line sign sums this block needs were it a computing block (indices clamped into the
  // arrays for the zeroing blocks past the capacity tiles).
  const uint32_t mt = fdiv(bid, a.divCt);
  const uint32_t m0 = mt * 32, c0 = (bid - mt * a.ctiles) * 32;
  const int taps = int(a.taps);
  int kn = 0;
  float2 sz = make_float2(0.0f, 0.0f);
  uint32_t pslot = 0, ppix = 0;
  if (t < 32) {
    const uint32_t m = min(m0 + uint32_t(t), a.N * a.HW - 1);
    pslot = fdiv(m, a.divHW);
    ppix = m - pslot * a.HW;
    kn = a.kept[pslot];
    if (a.slot_sz) sz = a.slot_sz[pslot];
  }
  constexpr int WLT = DX_MAX_TAPS * 32 / DX_THREADS;   // sign sums per thread, at most
  int wlv[WLT];
#pragma unroll
  for (int k = 0; k < WLT; ++k) {
    const int e = t + k * DX_THREADS, p = e & 31, tap = e >> 5;
    const uint32_t ch = c0 + uint32_t(p);
    wlv[k] = (e < 32 * taps && ch < a.C) ? a.wlsum[ch * a.taps + uint32_t(tap)] : 0;
  }
  const uint32_t live_rows = uint32_t(count) * a.HW;
  const uint32_t live_blocks = ((live_rows + 31) / 32) * a.ctiles;

  if (bid >= live_blocks) {      // zero the pruned samples, a piece of one per block
    dx_zero_pool(a, bid - live_blocks, a.nblocks - live_blocks, count);
    return;
  }

  if (t < 32) {
    const bool live = m0 + uint32_t(t) < live_rows;
    if (!a.slot_sz && live) sz = make_float2(a.scale[kn], a.offset[kn]);
    sm.pix_out[t] = live ? int(uint32_t(kn) * a.CHW + ppix) : -1;
    sm.pix_s[t] = live ? sz.x : 0.0f;
    sm.pix_z[t] = live ? sz.y : 0.0f;
  }
#pragma unroll
  for (int k = 0; k < WLT; ++k) {
    const int e = t + k * DX_THREADS;
    if (e < 32 * taps) sm.wl[e >> 5][e & 31] = wlv[k];
  }
  dx_row_table<32, DX_THREADS>(a, m0, live_rows, sm.rowoff);
  __syncthreads();

  // This lane: A row = channel c0 + i, B column = pixel m0 + i.
  const uint32_t ch = c0 + i;
  const uint32_t abase = ch < a.C ? ch * 32 + 16 * g : BUF_NONE;
  const __amdgpu_buffer_rsrc_t ars = buffer_of(a.wsb, a.wsb_bytes);
  const __amdgpu_buffer_rsrc_t brs = buffer_of(a.codes, a.codes_bytes);
  const uint32_t steps = a.taps * a.nch;
  v16i acc = {0};
  for (uint32_t s0 = wave; s0 < steps; s0 += DX_WAVES * NB) {
    // All NB steps' loads issue before the first product (one memory latency per batch);
    // a step past the end reads zeros through its A operand and adds nothing.
    v4i A[NB], B[NB];
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const uint32_t st0 = s0 + u * DX_WAVES;
      const bool live = st0 < steps;
      const uint32_t st = live ? st0 : 0;
      const uint32_t tap = fdiv(st, a.divNch);
      const uint32_t kc = st - tap * a.nch;
      A[u] = load16(ars, live ? abase : BUF_NONE, (kc * a.taps + tap) * a.C * 32);
      B[u] = load16(brs, sm.rowoff[tap][i] + 16 * g, kc * a.R * 32);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < NB; ++u) acc = mfma_i8(A[u], B8 ? bias128(B[u]) : B[u], acc);
  }

#pragma unroll
  for (int v = 0; v < 16; ++v) sm.red[wave][v][lane] = acc[v];
  __syncthreads();
  const int off = sm.pix_out[i];
  if (off < 0) return;                    // rows past the count belong to the zero blocks
  const float S = sm.pix_s[i], Z = sm.pix_z[i];
  const int r0 = 8 * int(wave) + 4 * g;   // channel rows r0 .. r0 + 3 of this lane
  int I[4], c[4] = {0, 0, 0, 0}, lt[4] = {0, 0, 0, 0};
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int v = 4 * int(wave) + u;
    I[u] = sm.red[0][v][lane] + sm.red[1][v][lane] + sm.red[2][v][lane] + sm.red[3][v][lane];
  }
  for (int tap = 0; tap < taps; ++tap) {
    const bool reach = sm.rowoff[tap][i] != BUF_NONE;
    const int4 w4 = *reinterpret_cast<const int4 *>(&sm.wl[tap][r0]);
    c[0] += reach ? w4.x : 0; c[1] += reach ? w4.y : 0;
    c[2] += reach ? w4.z : 0; c[3] += reach ? w4.w : 0;
    if (B8) { lt[0] += w4.x; lt[1] += w4.y; lt[2] += w4.z; lt[3] += w4.w; }
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const uint32_t cc = c0 + uint32_t(r0 + u);
    if (cc >= a.C) continue;
    const int Iu = I[u] + (B8 ? 128 * lt[u] : 0);
    const float out = rescale(S, Iu, Z, float(c[u]));
    const size_t o = size_t(off) + size_t(cc) * a.HW;
    if (a.dx_t == FQT_BF16) static_cast<uint16_t *>(a.dX)[o] = f32_to_bf16(out);
    else static_cast<float *>(a.dX)[o] = out;
    if (a.I_out) a.I_out[o] = Iu;
  }
}

// Large layers (many row tiles, at most DXW_MAX_TAPS taps): register tiles.  A block
// holds 4 * DXT_RT pixel tiles of 32 rows and CT channel tiles; wave w runs the whole
// contraction of pixel tiles DXT_RT w .. DXT_RT (w + 1) - 1 against all CT channel tiles
// (no split over the waves, no reduction), so each loaded sign fragment feeds DXT_RT
// MFMAs and each code fragment CT of them: (DXT_RT + CT) 1 KB loads per DXT_RT * CT
// products instead of two per product.  The per-(tap, pixel) code row
// offsets of the block's pixels and the channel sign sums are tabulated in LDS as in the
// split form.  CT = 2 unless the layer has a single channel tile.
constexpr int DXW_MAX_TAPS = 16;
constexpr int DXT_RT = 2;                            // pixel tiles per wave
constexpr int DXT_NB = 4;                            // contraction steps per load batch
constexpr uint32_t DXT_BP = DX_WAVES * DXT_RT * 32;  // pixel rows per block
template <int CT>
struct alignas(16) DxTileLds {
  uint32_t rowoff[DXW_MAX_TAPS][DXT_BP];
  int32_t wl[DXW_MAX_TAPS][CT * 32];
  int32_t pix_out[DXT_BP];
  float pix_s[DXT_BP], pix_z[DXT_BP];
  // A wave's output tile, [channel row][pixel] (two channel tiles: full 32-channel tiles;
  // one channel tile has C <= 32 and stores element by element).
  uint32_t stage[CT == 2 ? DX_WAVES : 1][CT == 2 ? 32 * 32 : 1];
};

// Stores of one wave's 32 x 32 output tile (channels c0t .. c0t + 31 x the 32 pixels from
// block pixel p0) from its row-major copy in LDS: lane L writes half h = L % 2 (16
// pixels) of channel row L / 2, as 16-byte stores when those 16 pixels are live, in one
// sample (consecutive offsets) and 16-byte aligned in dX; else element by element.
template <typename T>
__device__ __forceinline__ void dx_store_tile(const DxArgs &a, const int32_t *pix_out,
                                              const T *stage, uint32_t c0t, uint32_t p0,
                                              int lane) {
  constexpr int PER16 = 16 / sizeof(T);            // elements per 16-byte store
  static_assert(16 % PER16 == 0, "whole 16-byte pieces");
  const int rr = lane >> 1, h = lane & 1;
  const uint32_t cc = c0t + uint32_t(rr);
  if (cc >= a.C) return;
  const uint32_t pb = p0 + 16 * h;
  const int o0 = pix_out[pb], o15 = pix_out[pb + 15];
  const T *src = stage + rr * 32 + 16 * h;
  T *dst = static_cast<T *>(a.dX);
  const size_t base = size_t(o0) + size_t(cc) * a.HW;
  // (o15 = o0 + 15 with both live: the 16 offsets are consecutive, also where a sample
  // boundary falls inside, which only C = 1 allows.)
  if (o0 >= 0 && o15 == o0 + 15 && (reinterpret_cast<uintptr_t>(dst + base) & 15) == 0) {
    const uint4 *s4 = reinterpret_cast<const uint4 *>(src);
    uint4 *d4 = reinterpret_cast<uint4 *>(dst + base);
#pragma unroll
    for (int k = 0; k < 16 / PER16; ++k) d4[k] = s4[k];
  } else {
    for (int j = 0; j < 16; ++j) {
      const int o = pix_out[pb + j];
      if (o >= 0) dst[size_t(o) + size_t(cc) * a.HW] = src[j];
    }
  }
}

template <bool B8, int CT>
__device__ __forceinline__ void dx_body_tiles(const DxArgs &a, uint32_t bid, DxTileLds<CT> &sm) {
  static_assert(DXT_BP == DX_THREADS, "one pixel row per thread");
  bid = xcd_tile<DXW_XCD_RUN>(bid, a.nblocks);
  constexpr uint32_t BP = DXT_BP;
  constexpr int CW = CT * 32;                    // channels per block
  const int t = threadIdx.x, lane = t & 63;
  const uint32_t wave = wave_id();
  const int i = lane & 31, g = lane >> 5;
  const int count = *a.count;
  const uint32_t mt = fdiv(bid, a.divCb);
  const uint32_t m0 = mt * BP, c0 = (bid - mt * a.cblocks) * CW;
  const int taps = int(a.taps);
  // Loads that do not depend on the count issue with it (clamped indices).
  const uint32_t m = min(m0 + uint32_t(t), a.N * a.HW - 1);
  const uint32_t pslot = fdiv(m, a.divHW);
  const uint32_t ppix = m - pslot * a.HW;
  const int kn = a.kept[pslot];
  float2 sz = a.slot_sz ? a.slot_sz[pslot] : make_float2(0.0f, 0.0f);
  constexpr int WLT = DXW_MAX_TAPS * CW / DX_THREADS;
  int wlv[WLT];
#pragma unroll
  for (int k = 0; k < WLT; ++k) {
    const int e = t + k * DX_THREADS, p = e % CW, tap = e / CW;
    const uint32_t ch = c0 + uint32_t(p);
    wlv[k] = (tap < taps && ch < a.C) ? a.wlsum[ch * a.taps + uint32_t(tap)] : 0;
  }
  const uint32_t live_rows = uint32_t(count) * a.HW;
  const uint32_t live_blocks = ((live_rows + BP - 1) / BP) * a.cblocks;
  if (bid >= live_blocks) {
    dx_zero_pool(a, bid - live_blocks, a.nblocks - live_blocks, count);
    return;
  }
  {
    const bool live = m0 + uint32_t(t) < live_rows;
    if (!a.slot_sz && live) sz = make_float2(a.scale[kn], a.offset[kn]);
    sm.pix_out[t] = live ? int(uint32_t(kn) * a.CHW + ppix) : -1;
    sm.pix_s[t] = live ? sz.x : 0.0f;
    sm.pix_z[t] = live ? sz.y : 0.0f;
  }
#pragma unroll
  for (int k = 0; k < WLT; ++k) {
    const int e = t + k * DX_THREADS;
    if (e / CW < taps) sm.wl[e / CW][e % CW] = wlv[k];
  }
  dx_row_table<BP, DX_THREADS>(a, m0, live_rows, sm.rowoff);
  __syncthreads();

  // This lane: A rows = channels c0 + 32 ct + i, B columns = pixels 32 (DXT_RT wave + rt) + i.
  uint32_t px[DXT_RT], abase[CT];
#pragma unroll
  for (int rt = 0; rt < DXT_RT; ++rt) px[rt] = (wave * DXT_RT + uint32_t(rt)) * 32 + uint32_t(i);
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) {
    const uint32_t ch = c0 + uint32_t(32 * ct + i);
    abase[ct] = ch < a.C ? ch * 32 + 16 * g : BUF_NONE;
  }
  const __amdgpu_buffer_rsrc_t ars = buffer_of(a.wsb, a.wsb_bytes);
  const __amdgpu_buffer_rsrc_t brs = buffer_of(a.codes, a.codes_bytes);
  const uint32_t steps = a.taps * a.nch;
  v16i acc[DXT_RT][CT];
#pragma unroll
  for (int rt = 0; rt < DXT_RT; ++rt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = v16i{0};
  for (uint32_t s0 = 0; s0 < steps; s0 += DXT_NB) {
    // A batch's loads all issue before its first product; a step past the end reads zeros
    // through its A operands and adds nothing.
    v4i A[DXT_NB][CT], B[DXT_NB][DXT_RT];
#pragma unroll
    for (int u = 0; u < DXT_NB; ++u) {
      const uint32_t st0 = s0 + u;
      const bool live = st0 < steps;
      const uint32_t st = live ? st0 : 0;
      const uint32_t tap = fdiv(st, a.divNch);
      const uint32_t kc = st - tap * a.nch;
      const uint32_t aoff = (kc * a.taps + tap) * a.C * 32;
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) A[u][ct] = load16(ars, live ? abase[ct] : BUF_NONE, aoff);
#pragma unroll
      for (int rt = 0; rt < DXT_RT; ++rt)
        B[u][rt] = load16(brs, sm.rowoff[tap][px[rt]] + 16 * g, kc * a.R * 32);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < DXT_NB; ++u)
#pragma unroll
      for (int rt = 0; rt < DXT_RT; ++rt) {
        const v4i b = B8 ? bias128(B[u][rt]) : B[u][rt];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = mfma_i8(A[u][ct], b, acc[rt][ct]);
      }
  }

#pragma unroll
  for (int rt = 0; rt < DXT_RT; ++rt) {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      // Zero-point term of each output, c = sum over the taps that reach the pixel of the
      // channel's line sign sum: the 32 x 32 product [channel][tap] x [tap][pixel] of the
      // sign sums and the 0/1 reach flags in the accumulator layout of the tile.  Exact:
      // with D <= 2048 every sign sum is a float16 integer and all taps go into one f16
      // MFMA (lane half g holds taps 8 g .. 8 g + 7); else two taps per float32 MFMA.
      v16f cz = v16f{0};
      if (a.Dp <= 2048) {
        f16x8 wa, rb;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int tap = 8 * g + k;
          const bool in = tap < taps;
          wa[k] = in ? _Float16(sm.wl[tap][32 * ct + i]) : _Float16(0.0f);
          rb[k] = in && sm.rowoff[tap][px[rt]] != BUF_NONE ? _Float16(1.0f) : _Float16(0.0f);
        }
        cz = __builtin_amdgcn_mfma_f32_32x32x16_f16(wa, rb, cz, 0, 0, 0);
      } else {
        for (int j = 0; 2 * j < taps; ++j) {
          const int tap = 2 * j + g;
          const bool in = tap < taps;
          const float wv = in ? float(sm.wl[tap][32 * ct + i]) : 0.0f;
          const float rv = in && sm.rowoff[tap][px[rt]] != BUF_NONE ? 1.0f : 0.0f;
          cz = __builtin_amdgcn_mfma_f32_32x32x2f32(wv, rv, cz, 0, 0, 0);
        }
      }
      const int off = sm.pix_out[px[rt]];
      const float S = sm.pix_s[px[rt]], Z = sm.pix_z[px[rt]];
      if constexpr (CT == 2) {
        if (!a.I_out && c0 + uint32_t(32 * ct + 32) <= a.C) {
          // A whole tile of 32 channels goes through the wave's LDS copy (row-major), then
          // out in 16-byte pieces along the pixels: 2-byte stores scattered over 32 channel
          // rows were the slowest part of the kernel.
          uint32_t *st = sm.stage[wave];
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int row = acc_row(v, g);
            int lt = 0;
            if (B8)
              for (int tap = 0; tap < taps; ++tap) lt += sm.wl[tap][32 * ct + row];
            const float out = rescale(S, acc[rt][ct][v] + (B8 ? 128 * lt : 0), Z, cz[v]);
            if (a.dx_t == FQT_BF16)
              reinterpret_cast<uint16_t *>(st)[row * 32 + i] = f32_to_bf16(out);
            else
              reinterpret_cast<float *>(st)[row * 32 + i] = out;
          }
          __builtin_amdgcn_wave_barrier();    // LDS operations of a wave run in order
          const uint32_t p0 = (wave * DXT_RT + uint32_t(rt)) * 32;
          if (a.dx_t == FQT_BF16)
            dx_store_tile<uint16_t>(a, sm.pix_out, reinterpret_cast<const uint16_t *>(st),
                                    c0 + uint32_t(32 * ct), p0, lane);
          else
            dx_store_tile<float>(a, sm.pix_out, reinterpret_cast<const float *>(st),
                                 c0 + uint32_t(32 * ct), p0, lane);
          __builtin_amdgcn_wave_barrier();    // the next tile's copy waits for these reads
          continue;
        }
      }
      if (off < 0) continue;               // rows past the count belong to the zero blocks
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = 32 * ct + acc_row(v, g);
        const uint32_t cc = c0 + uint32_t(row);
        if (cc >= a.C) continue;
        int lt = 0;
        if (B8)
          for (int tap = 0; tap < taps; ++tap) lt += sm.wl[tap][row];
        const int Iv = acc[rt][ct][v] + (B8 ? 128 * lt : 0);
        const float out = rescale(S, Iv, Z, cz[v]);
        const size_t o = size_t(off) + size_t(cc) * a.HW;
        if (a.dx_t == FQT_BF16) static_cast<uint16_t *>(a.dX)[o] = f32_to_bf16(out);
        else static_cast<float *>(a.dX)[o] = out;
        if (a.I_out) a.I_out[o] = Iv;
      }
    }
  }
}

// WT: 0 for the split form, CT (1 or 2 channel tiles per wave) for the register-tile form.
template <int WT>
using DxLdsOf = std::conditional_t<WT != 0, DxTileLds<WT == 0 ? 1 : WT>, DxLds>;

// The register-tile forms (WT != 0) are held to three waves per SIMD (at most 170
// registers; the compiler's own choice, 182, leaves two).
template <bool B8, int NB, int WT>
__global__ __launch_bounds__(DX_THREADS) __attribute__((amdgpu_waves_per_eu(WT != 0 ? 3 : 1)))
void k_mfma_dx(DxArgs a) {
  __shared__ DxLdsOf<WT> sm;
  if constexpr (WT != 0) dx_body_tiles<B8, WT>(a, blockIdx.x, sm);
  else dx_body<B8, NB>(a, blockIdx.x, sm);
}

// How the dW blocks of the products launch run: split-R partials summed by a finish pass
// (PARTS), one split writing dW itself (DIRECT), or the contraction split over a block's
// waves and reduced in LDS (KRED).
enum DwForm { DWF_PARTS = 0, DWF_DIRECT = 1, DWF_KRED = 2 };

// Both products in one launch (the layer backward): blocks [0, ndw) are dW blocks, the rest
// dX blocks; the two share one LDS allocation.
template <int WT>
union ProductsLds {
  DxLdsOf<WT> dx;
  DwRedLds dw;
};
template <bool B8, int NB, int DWF, int WT>
__global__ __launch_bounds__(DX_THREADS) __attribute__((amdgpu_waves_per_eu(WT != 0 ? 3 : 1)))
void k_products(DxArgs dxa, DwArgs dwa, uint32_t ndw) {
  __shared__ ProductsLds<WT> sm;
  if (blockIdx.x < ndw) {
    if constexpr (DWF == DWF_KRED) dw_kred_body<B8>(dwa, blockIdx.x, sm.dw);
    else dw_part_body<B8, DWF == DWF_DIRECT>(dwa, blockIdx.x);
  } else {
    if constexpr (WT != 0) dx_body_tiles<B8, WT>(dxa, blockIdx.x - ndw, sm.dx);
    else dx_body<B8, NB>(dxa, blockIdx.x - ndw, sm.dx);
  }
}


// ----------------------------------------------------------------------------- forward

// Binary forward product (Section 5.1; Appendix C, Alg. 1 forward and the Unfolder):
// I[r][d] = sum_k sign(X_u)[r][k] sign(W)[d][k] over k < Kp, and Y = gamma_d * I.
// Operands: sign(W) as +-1 bytes in 32-line chunks [Kp/32][Dp][32] (0 past D and K), the
// MFMA's src0 (rows = output channels; a wave's 32 rows of one chunk are 1 KB contiguous); sign(X_u) as bits, k-block-major [Kw][Rp] (word (kb, r) holds
// lines 64 kb .. 64 kb + 63 of row r), expanded in registers 16 bits at a time into the
// src1 bytes (columns = rows r of the unfolded input, so output lanes run along pixels).
// Lines past K are -1 in X and 0 in W, so they add nothing.  A tile is 64 channels x 32
// rows (two MFMA tiles sharing one expanded X operand); a block's four waves take
// consecutive row tiles of the same 64 channels, WPT waves per tile splitting its
// contraction.  Grid: ceil(Dp/64) x ceil(R/(32 * 4 / WPT)), channel blocks fastest.
struct FwdArgs {
  const int8_t *wb;              // [Kp/32][Dp][32]
  const uint64_t *xr;            // [Kw][Rp]
  const float *gamma;            // [D]
  void *Y;                       // [N][D][P]
  int32_t *I_out;
  int y_t;
  uint32_t D, Dp, Kp, R, Rp, P, dblocks;
  uint32_t wb_bytes, xr_bytes;
  FastDiv divP, divDb;
};
constexpr int FWD_WAVES = 4;
constexpr int FWD_THREADS = FWD_WAVES * 64;

// One batch of a forward wave's operands: FWD_PREF words of its X rows (two 32-line steps
// each) and, per step, the 16-byte pieces of its two W row tiles.
constexpr int FWD_PREF = 4;
struct FwdBatch {
  uint64_t word[FWD_PREF];
  v4i A0[FWD_PREF][2], A1[FWD_PREF][2];
};
__device__ __forceinline__ void fwd_issue(const FwdArgs &a, __amdgpu_buffer_rsrc_t wrs,
                                          __amdgpu_buffer_rsrc_t xrs, uint32_t aoff0,
                                          uint32_t aoff1, uint32_t boff, uint32_t kb0,
                                          uint32_t kstride, uint32_t kw, FwdBatch &b) {
#pragma unroll
  for (int u = 0; u < FWD_PREF; ++u) {
    const uint32_t kb1 = kb0 + u * kstride;
    const uint32_t kb = kb1 < kw ? kb1 : kb0;            // past the end: word kb0 again
    b.word[u] = load8(xrs, boff, kb * a.Rp * 8);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      b.A0[u][h] = load16(wrs, aoff0, (2 * kb + h) * a.Dp * 32);
      b.A1[u][h] = load16(wrs, aoff1, (2 * kb + h) * a.Dp * 32);
    }
  }
}
__device__ __forceinline__ void fwd_consume(const FwdBatch &b, uint32_t kb0, uint32_t kstride,
                                            uint32_t kw, int g, v16i &acc0, v16i &acc1) {
#pragma unroll
  for (int u = 0; u < FWD_PREF; ++u) {
    if (kb0 + u * kstride >= kw) break;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const v4i x = signs16(uint32_t(b.word[u] >> (32 * h + 16 * g)) & 0xFFFFu);
      acc0 = mfma_i8(b.A0[u][h], x, acc0);
      acc1 = mfma_i8(b.A1[u][h], x, acc1);
    }
  }
}

// A block's four waves: WPT waves per 64 x 32 tile, each taking every WPT-th word of X
// (the contraction split over the waves for more waves in flight), 4 / WPT row tiles.
// The split partial tiles meet in LDS.
template <int WPT>
struct FwdLds {
  int32_t red[WPT > 1 ? FWD_WAVES : 1][2][16][64];
};
template <int WPT>
__global__ __launch_bounds__(FWD_THREADS) void k_mfma_fwd(FwdArgs a) {
  constexpr int TPB = FWD_WAVES / WPT;                 // row tiles per block
  __shared__ FwdLds<WPT> sm;
  const int lane = threadIdx.x & 63;
  const uint32_t wave = wave_id();
  const int i = lane & 31, g = lane >> 5;
  const uint32_t rb = fdiv(blockIdx.x, a.divDb), db = blockIdx.x - rb * a.dblocks;
  const uint32_t tile = wave / WPT, part = wave - tile * WPT;
  const uint32_t d0 = db * 64, r0 = (rb * TPB + tile) * 32;
  const bool live = r0 < a.R;                          // wave-uniform
  const __amdgpu_buffer_rsrc_t wrs = buffer_of(a.wb, a.wb_bytes);
  const __amdgpu_buffer_rsrc_t xrs = buffer_of(a.xr, a.xr_bytes);
  // src0 rows d0 + i and d0 + 32 + i (always inside Dp), bytes 16 g .. 16 g + 15 of a step.
  const uint32_t aoff0 = (d0 + uint32_t(i)) * 32 + 16 * g, aoff1 = aoff0 + 32 * 32;
  const uint32_t boff = (r0 + uint32_t(i)) * 8;        // word (kb, r0 + i) at kb * Rp * 8
  const uint32_t kw = a.Kp / 64;                       // X words per row
  constexpr uint32_t kstride = WPT;
  v16i acc0 = {0}, acc1 = {0};
  if (live && part < kw) {
    // Double-buffered: batch i + 1's loads issue before batch i's products.
    FwdBatch b0, b1;
    uint32_t kb0 = part;
    const uint32_t step = FWD_PREF * kstride;
    fwd_issue(a, wrs, xrs, aoff0, aoff1, boff, kb0, kstride, kw, b0);
    for (;;) {
      if (kb0 + step < kw) fwd_issue(a, wrs, xrs, aoff0, aoff1, boff, kb0 + step, kstride, kw, b1);
      __builtin_amdgcn_sched_barrier(0);
      fwd_consume(b0, kb0, kstride, kw, g, acc0, acc1);
      kb0 += step;
      if (kb0 >= kw) break;
      if (kb0 + step < kw) fwd_issue(a, wrs, xrs, aoff0, aoff1, boff, kb0 + step, kstride, kw, b0);
      __builtin_amdgcn_sched_barrier(0);
      fwd_consume(b1, kb0, kstride, kw, g, acc0, acc1);
      kb0 += step;
      if (kb0 >= kw) break;
    }
  }
  uint32_t vlo = 0, vhi = 16;                          // accumulator registers this wave ends
  if constexpr (WPT > 1) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      sm.red[wave][0][v][lane] = acc0[v];
      sm.red[wave][1][v][lane] = acc1[v];
    }
    __syncthreads();
    // Part p of the tile sums registers [16 p / WPT, 16 (p + 1) / WPT) over the parts.
    vlo = 16 * part / WPT;
    vhi = 16 * (part + 1) / WPT;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      if (uint32_t(v) < vlo || uint32_t(v) >= vhi) continue;
      int s0 = 0, s1 = 0;
#pragma unroll
      for (int q = 0; q < WPT; ++q) {
        s0 += sm.red[tile * WPT + q][0][v][lane];
        s1 += sm.red[tile * WPT + q][1][v][lane];
      }
      acc0[v] = s0;
      acc1[v] = s1;
    }
  }
  const uint32_t r = r0 + uint32_t(i);
  if (!live || r >= a.R) return;
  const uint32_t n = fdiv(r, a.divP), p = r - n * a.P;
  const size_t base = size_t(n) * a.D * a.P + p;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      if (uint32_t(v) < vlo || uint32_t(v) >= vhi) continue;
      const uint32_t d = d0 + 32 * t + uint32_t(acc_row(v, g));
      if (d >= a.D) continue;
      const int I = t ? acc1[v] : acc0[v];
      const float y = __fmul_rn(a.gamma[d], float(I));
      const size_t o = base + size_t(d) * a.P;
      if (a.y_t == FQT_BF16) static_cast<uint16_t *>(a.Y)[o] = f32_to_bf16(y);
      else static_cast<float *>(a.Y)[o] = y;
      if (a.I_out) a.I_out[o] = I;
    }
  }
}

}  // namespace

// Splits of the dW contraction over N*Ho*Wo: enough 32x32 wave tiles of the expected
// kept channels (all of them without AGP, about D / b with it) to give about 1024 waves
// while every split keeps at least 16 words (1024 positions), and at most 256 words per
// split (about 64 in the long split form, below), within at most DW_MAX_SPLITS splits,
// 128 MB of partials and one batch of words per split.
constexpr int64_t DW_TARGET_WAVES = 1024;
constexpr int64_t DW_MIN_WORDS = 16;
constexpr int64_t DW_MAX_WORDS = 256;
constexpr int64_t DW_MAX_SPLITS = 4096;
constexpr int64_t DW_MAX_PART_BYTES = int64_t(128) << 20;
constexpr int64_t DW_SPLIT_WORDS = 64;
constexpr int64_t DW_SPLIT_MIN = 768;         // contraction words of the split form, at least
int gemm_dw_splits(const Layer &L, const fqt_quant_cfg &cfg) {
  const int64_t dkeep =
      cfg.agp_mode == FQT_AGP_OFF ? L.D : std::max<int64_t>(1, (L.D + cfg.bits - 1) / cfg.bits);
  const int64_t tiles = ((dkeep + 31) / 32) * ((L.K + 31) / 32);
  int64_t S = std::max(std::min((DW_TARGET_WAVES + tiles - 1) / tiles,
                                (L.Wr + DW_MIN_WORDS - 1) / DW_MIN_WORDS),
                       (L.Wr + DW_MAX_WORDS - 1) / DW_MAX_WORDS);
  const int64_t kp = ((L.K + 31) / 32) * 32;
  const int64_t part_cap = std::max<int64_t>(1, DW_MAX_PART_BYTES / (L.D * kp * 4));
  S = std::min(S, part_cap);
  S = std::min(S, DW_MAX_SPLITS);
  S = std::min(S, (L.Wr + DW_PREF - 1) / DW_PREF);
  // Long contractions in the split form (their own launch: at least DW_SPLIT_MIN words,
  // slices of at least 16): slices of about DW_SPLIT_WORDS words, so that each wave's chain
  // of loads is short, while the many-split finish keeps at most 4 splits per block of its
  // D x ceil(Kp / 64) blocks (its reduction over the splits is serial per thread).
  if (S > 1 && L.Wr >= DW_SPLIT_MIN && (L.Wr + S - 1) / S >= 16) {
    int64_t Sb = std::min((L.Wr + DW_SPLIT_WORDS - 1) / DW_SPLIT_WORDS,
                          4 * L.D * ((kp + 63) / 64));
    Sb = std::min(std::min(Sb, part_cap), DW_MAX_SPLITS);
    S = std::max(S, Sb);
  }
  return int(std::max<int64_t>(S, 1));
}

// Contractions of at most this many words that would need split-R partials run in the
// in-block reduction form instead (four waves of at most 64 words each).
constexpr int64_t DW_KRED_MAX_WORDS = 256;
bool dw_kred_form(const Layer &L, int64_t S) { return S > 1 && L.Wr <= DW_KRED_MAX_WORDS; }

// dW workspace: partials [S][D][Kp] and set-bit counts [S][Kp] (Kp = K rounded up to 32);
// none when one split or the in-block reduction writes dW directly.
static size_t dw_kp(const Layer &L) { return size_t((L.K + 31) / 32) * 32; }
size_t gemm_dw_ws_bytes(const Layer &L, const fqt_quant_cfg &cfg) {
  const size_t S = size_t(gemm_dw_splits(L, cfg));
  if (S == 1 || dw_kred_form(L, int64_t(S))) return 256;
  return align256(S * size_t(L.D) * dw_kp(L) * 4) + align256(S * dw_kp(L) * 4);
}

namespace {

DwArgs make_dw_args(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                    const uint64_t *xsign, float *dW, int32_t *I_out, void *ws) {
  const uint32_t ktiles = uint32_t((L.K + 31) / 32);
  const uint32_t S = uint32_t(gemm_dw_splits(L, cfg));
  DwArgs a;
  a.codes = q.pcq_codes; a.kept = q.pcq_kept; a.count = q.pcq_count;
  a.scale = q.pcq_scale; a.offset = q.pcq_offset; a.slot_sz = nullptr; a.xsign = xsign;
  a.dW = dW; a.I_out = I_out;
  a.part = S > 1 ? static_cast<int32_t *>(ws) : nullptr;
  a.partT = S > 1 ? reinterpret_cast<int32_t *>(static_cast<char *>(ws) +
                                                align256(size_t(S) * L.D * dw_kp(L) * 4))
                  : nullptr;
  a.D = uint32_t(L.D); a.K = uint32_t(L.K); a.Kp = uint32_t(dw_kp(L)); a.R = uint32_t(L.R);
  a.Rp = uint32_t(L.Wr * 64); a.Wr = uint32_t(L.Wr); a.ktiles = ktiles;
  a.codes_bytes = uint32_t(L.D * L.Wr * 64);
  a.xsign_bytes = uint32_t(L.Wr * L.K * 8);
  a.kgroups = (ktiles + DW_WAVES - 1) / DW_WAVES;
  a.S = S; a.wps = uint32_t((L.Wr + S - 1) / S);
  a.wpw = uint32_t((L.Wr + DW_WAVES - 1) / DW_WAVES);
  a.divS = make_fastdiv(S); a.divKg = make_fastdiv(a.kgroups); a.divQ = make_fastdiv(uint32_t(dw_kp(L) / 4));
  a.divKt = make_fastdiv(ktiles);
  return a;
}
// Blocks of the in-block reduction form: every (slot tile, column tile) of the capacity.
uint32_t dw_kred_blocks(const Layer &L, const DwArgs &a) {
  return a.ktiles * uint32_t((L.D + 31) / 32);
}
// Split-R partial blocks over the slot capacity: S x ceil(ceil(K/32) / 4) x ceil(D/32).
uint32_t dw_part_blocks(const Layer &L, const DwArgs &a) {
  return a.S * a.kgroups * uint32_t((L.D + 31) / 32);
}

DxArgs make_dx_args(const Layer &L, const fqt_qgrad &q, const int8_t *wsb,
                    const int32_t *wlsum, void *dX, int32_t *I_out) {
  DxArgs a;
  a.codes = q.psq_codes; a.kept = q.psq_kept; a.count = q.psq_count;
  a.scale = q.psq_scale; a.offset = q.psq_offset; a.slot_sz = nullptr; a.wsb = wsb;
  a.wlsum = wlsum;
  a.dX = dX; a.I_out = I_out; a.dx_t = L.dx_t;
  a.N = uint32_t(L.N); a.C = uint32_t(L.C); a.H = uint32_t(L.H); a.W = uint32_t(L.W);
  a.HW = uint32_t(L.HW); a.Ho = uint32_t(L.Ho); a.Wo = uint32_t(L.Wo); a.P = uint32_t(L.P);
  a.R = uint32_t(L.R); a.Dp = uint32_t(L.Wd * 64);
  a.ctiles = uint32_t((L.C + 31) / 32);
  a.CHW = uint32_t(L.C * L.HW);
  a.taps = uint32_t(L.kh * L.kw);
  a.nch = a.Dp / 32;
  a.codes_bytes = uint32_t(L.R * L.Wd * 64);
  a.wsb_bytes = uint32_t(L.K * L.Wd * 64);
  a.kh = L.kh; a.kw = L.kw; a.sh = L.sh; a.sw = L.sw; a.ph = L.ph; a.pw = L.pw;
  a.divHW = make_fastdiv(uint32_t(L.HW)); a.divW = make_fastdiv(uint32_t(L.W));
  a.divKw = make_fastdiv(uint32_t(L.kw)); a.divNch = make_fastdiv(a.nch);
  a.divCt = make_fastdiv(a.ctiles);
  a.divSh = make_fastdiv(uint32_t(L.sh)); a.divSw = make_fastdiv(uint32_t(L.sw));
  // Capacity tiles plus a pool of blocks that only zero pruned samples, a piece of at most
  // DX_ZCHUNK elements each: whatever the device-side count, at least
  // min(2048, N * pieces) blocks are left for the zeroing.
  a.zpieces = uint32_t((int64_t(a.CHW) + DX_ZCHUNK - 1) / DX_ZCHUNK);
  // Four pixel tiles per block once the capacity has 16384 tiles (with few taps).
  const int64_t tiles = ((L.N * L.HW + 31) / 32) * a.ctiles;
  a.wide = (a.taps <= uint32_t(DXW_MAX_TAPS) && tiles >= 16384) ? (a.ctiles > 1 ? 2u : 1u) : 0u;
  a.cblocks = a.wide ? (a.ctiles + a.wide - 1) / a.wide : a.ctiles;
  a.divCb = make_fastdiv(a.cblocks);
  const int64_t rows = a.wide ? DXT_BP : 32;
  a.nblocks = uint32_t(((L.N * L.HW + rows - 1) / rows) * a.cblocks +
                       std::min<int64_t>(2048, L.N * int64_t(a.zpieces)));
  return a;
}
// Contraction steps of one dX wave, rounded to the instantiated batch depths (10 steps
// per batch still leaves four resident blocks per CU; 18 steps in one batch was measured
// slower at the 256 -> 256 conv on 8x8 maps).
int dx_batch(const DxArgs &a) {
  const uint32_t per_wave = a.wide ? a.taps * a.nch : (a.taps * a.nch + DX_WAVES - 1) / DX_WAVES;
  return per_wave <= 4 ? 4 : per_wave <= 8 ? 8 : 10;
}

// One split and at least 1024 waves of 64 x 64: the 2 x 2-tile form.
bool dw_big(const Layer &L, const DwArgs &a) {
  return a.S == 1 && ((L.D + 63) / 64) * ((L.K + 63) / 64) >= 1024;
}

// Split-R products over long contractions (N*Ho*Wo of DW_SPLIT_MIN words and more, slices
// of 16 words and more): the partials in the big form's wave tiles, in a launch of their
// own.  Shorter ones stay in the products launch, where their partial blocks overlap the dX
// blocks.
bool dw_split_big(const Layer &L, const DwArgs &a) {
  return a.S > 1 && L.Wr >= DW_SPLIT_MIN && a.wps >= 16;
}
// Row tiles of the split form: one when the expected kept channels (D, or D / b with AGP)
// fit 32 rows.
int dw_split_rt(const Layer &L, const fqt_quant_cfg &cfg) {
  const int64_t dkeep =
      cfg.agp_mode == FQT_AGP_OFF ? L.D : (L.D + cfg.bits - 1) / std::max(cfg.bits, 1);
  return dkeep <= 32 ? 1 : 2;
}
template <bool B8>
void launch_dw_split(const DwArgs &a, int rt, hipStream_t s) {
  if (rt == 1)
    hipLaunchKernelGGL((k_mfma_dw_split<B8, 1>), dim3(dw_split_blocks(a, 1)), dim3(DW_THREADS), 0,
                       s, a);
  else
    hipLaunchKernelGGL((k_mfma_dw_split<B8, 2>), dim3(dw_split_blocks(a, 2)), dim3(DW_THREADS), 0,
                       s, a);
}

template <bool B8>
void launch_dw_big(const DwArgs &a, hipStream_t s) {
  if (a.Wr >= uint32_t(DWB_LONG_WORDS))
    hipLaunchKernelGGL(k_mfma_dw_big<B8>, dim3(dw_big_blocks(a.D, a.K, 2, 4)), dim3(DW_THREADS),
                       0, s, a);
  else
    hipLaunchKernelGGL(k_mfma_dw_short<B8>, dim3(dw_big_blocks(a.D, a.K, 2, 2)), dim3(DW_THREADS),
                       0, s, a);
}

template <bool B8>
void launch_dw_finish(const Layer &L, const DwArgs &a, hipStream_t s) {
  if (a.S > DWF_WIDE) {
    const uint32_t qblocks = uint32_t((dw_kp(L) + 63) / 64);
    hipLaunchKernelGGL(k_dw_finish_wide<B8>, dim3(unsigned(L.D) * qblocks), dim3(256), 0, s, a);
  } else {
    const dim3 fgrid(unsigned((L.D * (dw_kp(L) / 4) + 255) / 256));
    hipLaunchKernelGGL(k_dw_finish<B8>, fgrid, dim3(256), 0, s, a);
  }
}

}  // namespace

int launch_gemm_dw(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                   const uint64_t *xsign, float *dW, int32_t *I_out, void *ws, hipStream_t s) {
  const DwArgs a = make_dw_args(L, cfg, q, xsign, dW, I_out, ws);
  const dim3 grid(dw_part_blocks(L, a));
  auto go = [&]<bool B8>() {
    if (dw_big(L, a)) {
      launch_dw_big<B8>(a, s);
    } else if (dw_kred_form(L, a.S) && !dw_split_big(L, a)) {
      hipLaunchKernelGGL(k_mfma_dw_kred<B8>, dim3(dw_kred_blocks(L, a)), dim3(DW_THREADS), 0, s,
                         a);
    } else if (dw_split_big(L, a)) {
      launch_dw_split<B8>(a, dw_split_rt(L, cfg), s);
      launch_dw_finish<B8>(L, a, s);
    } else if (a.S == 1) {
      hipLaunchKernelGGL((k_mfma_dw_part<B8, true>), grid, dim3(DW_THREADS), 0, s, a);
    } else {
      hipLaunchKernelGGL((k_mfma_dw_part<B8, false>), grid, dim3(DW_THREADS), 0, s, a);
      launch_dw_finish<B8>(L, a, s);
    }
  };
  if (cfg.bits == 8) go.template operator()<true>();
  else go.template operator()<false>();
  return last_launch_status();
}

int launch_gemm_dx(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                   const int8_t *wsb, const int32_t *wlsum, void *dX, int32_t *I_out,
                   hipStream_t s) {
  if (L.kh * L.kw > DX_MAX_TAPS) return FQT_E_SHAPE;
  const DxArgs a = make_dx_args(L, q, wsb, wlsum, dX, I_out);
  const dim3 grid(a.nblocks);
  const int nb = dx_batch(a);
  auto go = [&]<bool B8, int WT>() {
    if constexpr (WT != 0)      // the register-tile form batches DXT_NB steps itself
      hipLaunchKernelGGL((k_mfma_dx<B8, 4, WT>), grid, dim3(DX_THREADS), 0, s, a);
    else if (nb == 4) hipLaunchKernelGGL((k_mfma_dx<B8, 4, 0>), grid, dim3(DX_THREADS), 0, s, a);
    else if (nb == 8) hipLaunchKernelGGL((k_mfma_dx<B8, 8, 0>), grid, dim3(DX_THREADS), 0, s, a);
    else hipLaunchKernelGGL((k_mfma_dx<B8, 10, 0>), grid, dim3(DX_THREADS), 0, s, a);
  };
  auto go2 = [&]<bool B8>() {
    if (a.wide == 2) go.template operator()<B8, 2>();
    else if (a.wide == 1) go.template operator()<B8, 1>();
    else go.template operator()<B8, 0>();
  };
  if (cfg.bits == 8) go2.template operator()<true>();
  else go2.template operator()<false>();
  return last_launch_status();
}

int launch_products(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                    const uint64_t *xsign, const int8_t *wsb, const int32_t *wlsum, void *dX,
                    float *dW, void *dw_ws, const float2 *sslot, const float2 *cslot,
                    hipStream_t s) {
  if (L.kh * L.kw > DX_MAX_TAPS) return FQT_E_SHAPE;
  DwArgs dwa = make_dw_args(L, cfg, q, xsign, dW, nullptr, dw_ws);
  DxArgs dxa = make_dx_args(L, q, wsb, wlsum, dX, nullptr);
  dwa.slot_sz = cslot;
  dxa.slot_sz = sslot;
  // A large one-split dW runs as its own launch in the 2 x 2-tile form; the products
  // launch then holds only dX blocks.
  // Long split-R contractions likewise run their partials as their own launch.
  const bool big = dw_big(L, dwa);
  const bool split_big = !big && dw_split_big(L, dwa);
  const bool kred = !big && !split_big && dw_kred_form(L, dwa.S);
  if (big) {
    if (cfg.bits == 8) launch_dw_big<true>(dwa, s);
    else launch_dw_big<false>(dwa, s);
  } else if (split_big) {
    if (cfg.bits == 8) launch_dw_split<true>(dwa, dw_split_rt(L, cfg), s);
    else launch_dw_split<false>(dwa, dw_split_rt(L, cfg), s);
  }
  const uint32_t ndw = (big || split_big) ? 0u
                      : kred ? dw_kred_blocks(L, dwa) : dw_part_blocks(L, dwa);
  const dim3 grid(ndw + dxa.nblocks);
  const int nb = dx_batch(dxa);
  auto go = [&]<bool B8, int DWF, int WT>() {
    if constexpr (WT != 0)
      hipLaunchKernelGGL((k_products<B8, 4, DWF, WT>), grid, dim3(DX_THREADS), 0, s, dxa, dwa,
                         ndw);
    else if (nb == 4)
      hipLaunchKernelGGL((k_products<B8, 4, DWF, 0>), grid, dim3(DX_THREADS), 0, s, dxa, dwa,
                         ndw);
    else if (nb == 8)
      hipLaunchKernelGGL((k_products<B8, 8, DWF, 0>), grid, dim3(DX_THREADS), 0, s, dxa, dwa,
                         ndw);
    else
      hipLaunchKernelGGL((k_products<B8, 10, DWF, 0>), grid, dim3(DX_THREADS), 0, s, dxa, dwa,
                         ndw);
    if (DWF == DWF_PARTS) launch_dw_finish<B8>(L, dwa, s);
  };
  auto go2 = [&]<bool B8, int DWF>() {
    if (dxa.wide == 2) go.template operator()<B8, DWF, 2>();
    else if (dxa.wide == 1) go.template operator()<B8, DWF, 1>();
    else go.template operator()<B8, DWF, 0>();
  };
  auto go3 = [&]<bool B8>() {
    // With the dW product in its own launch the products launch has no dW blocks: the big
    // form (one split) needs no finish, the split_big partials do.
    if (split_big) go2.template operator()<B8, DWF_PARTS>();
    else if (big || dwa.S == 1) go2.template operator()<B8, DWF_DIRECT>();
    else if (kred) go2.template operator()<B8, DWF_KRED>();
    else go2.template operator()<B8, DWF_PARTS>();
  };
  if (cfg.bits == 8) go3.template operator()<true>();
  else go3.template operator()<false>();
  return last_launch_status();
}

int launch_forward_gemm(const Layer &L, const int8_t *wrows, int64_t Dp, int64_t Kp,
                        const uint64_t *xrows, const float *gamma, void *Y, int32_t *I_out,
                        hipStream_t s) {
  FwdArgs a;
  a.wb = wrows; a.xr = xrows; a.gamma = gamma; a.Y = Y; a.I_out = I_out; a.y_t = L.dy_t;
  a.D = uint32_t(L.D); a.Dp = uint32_t(Dp); a.Kp = uint32_t(Kp); a.R = uint32_t(L.R);
  a.Rp = uint32_t(L.Wr * 64); a.P = uint32_t(L.P);
  a.dblocks = uint32_t(Dp / 64);
  a.wb_bytes = uint32_t(Dp * Kp);
  a.xr_bytes = uint32_t((Kp / 64) * L.Wr * 64 * 8);
  a.divP = make_fastdiv(uint32_t(L.P)); a.divDb = make_fastdiv(a.dblocks);
  // Row tiles per block: four (one wave each, the contraction whole) when the grid still
  // has four waves per SIMD that way, else fewer with the contraction split over the waves.
  const int64_t tiles = ((L.R + 31) / 32) * a.dblocks;
  const int wpt = tiles >= 4096 ? 1 : tiles >= 1024 ? 2 : 4;
  const uint32_t tpb = uint32_t(FWD_WAVES / wpt);
  const dim3 grid(a.dblocks * uint32_t((L.R + 32 * tpb - 1) / (32 * tpb)));
  if (wpt == 1) hipLaunchKernelGGL(k_mfma_fwd<1>, grid, dim3(FWD_THREADS), 0, s, a);
  else if (wpt == 2) hipLaunchKernelGGL(k_mfma_fwd<2>, grid, dim3(FWD_THREADS), 0, s, a);
  else hipLaunchKernelGGL(k_mfma_fwd<4>, grid, dim3(FWD_THREADS), 0, s, a);
  return last_launch_status();
}

}  // namespace fqt
