// Sign-bit packing on gfx950 (Section 5.1 binarizer; Appendix C, Alg. 2 row
// encoder, column encoder and Unfolder).  One 64-lane wavefront produces one
// 64-bit word with a ballot: lane l contributes bit l.
#include "fqt_internal.hpp"
#include "fqt_signs.hpp"

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

// Bit-im2col, one wave per 64 positions of IM2COL_CPW channels (the body is shared with the
// layer backward's selection launch).
template <int DT, int KH, int KW, bool WM>
__global__ __launch_bounds__(THREADS) void k_pack_im2col(const void *__restrict__ x, Im2colGeom g,
                                                         uint64_t *__restrict__ dst) {
  wave_im2col_body<DT, KH, KW, WM>(x, g, dst, blockIdx.x * WAVES + (threadIdx.x >> 6));
}

// Bit-im2col through an LDS band of sign bytes (the body is shared with the layer
// backward's selection launch): 256 threads, 16 channels per block.
template <int DT, int KH, int KW>
__global__ __launch_bounds__(THREADS) void k_pack_im2col_band(const void *__restrict__ x,
                                                              BandGeom g,
                                                              uint64_t *__restrict__ dst) {
  extern __shared__ uint32_t band[];             // [16][BR][WL] bytes
  band_im2col_body<DT, KH, KW, THREADS>(x, g, dst, blockIdx.x, blockIdx.y, band);
}

// Bit-level im2col of a stride-1 same-padded convolution (the body is shared with the
// layer backward's selection launch): 1024 threads per block, so that a block stages
// several channels and the grid still spreads the loads of X over every CU.
constexpr int BITS_THREADS = 1024;
template <int DT>
__global__ __launch_bounds__(BITS_THREADS) void k_pack_im2col_bits(const void *__restrict__ x,
                                                                   BitGeom g,
                                                                   uint64_t *__restrict__ dst) {
  extern __shared__ uint64_t bsm[];
  bit_im2col_body<DT, BITS_THREADS>(x, g, dst, blockIdx.x, bsm);
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

// sign(W) as +-1 bytes with line sums (the body is shared with the layer backward's
// selection launch): one 1024-thread block per 64 lines.
template <int DT>
__global__ __launch_bounds__(WB_THREADS) void k_pack_w_i8(const void *__restrict__ w, PackWGeom g,
                                                          int8_t *__restrict__ dst,
                                                          int32_t *__restrict__ lsum) {
  __shared__ PackWLds sm;
  pack_w_body<DT>(w, g, dst, lsum, blockIdx.x, sm);
}

// 64 x 64 bit transpose, one wave per block (w, kb): lane l loads word (w, 64 kb + l) and
// ends with word (kb, 64 w + l).  Six stages swap the off-diagonal S x S sub-blocks
// (S = 32, 16, ..., 1) between lanes l and l ^ S: the lane with bit S of its index clear
// keeps the bits b with bit S of b clear and takes its partner's, shifted up by S; the
// other lane keeps the bits with bit S set and takes its partner's, shifted down.
template <int S>
__device__ __forceinline__ uint64_t transpose_stage(uint64_t x, int lane) {
  constexpr uint64_t m = S == 32 ? 0x00000000FFFFFFFFull : S == 16 ? 0x0000FFFF0000FFFFull
                       : S == 8 ? 0x00FF00FF00FF00FFull : S == 4 ? 0x0F0F0F0F0F0F0F0Full
                       : S == 2 ? 0x3333333333333333ull : 0x5555555555555555ull;
  const uint64_t y = lane_xor64<S>(x);
  return (lane & S) == 0 ? (x & m) | ((y & m) << S) : (x & ~m) | ((y & ~m) >> S);
}
__global__ __launch_bounds__(THREADS) void k_transpose_bits(const uint64_t *__restrict__ src,
                                                            uint32_t Wr, uint32_t K,
                                                            uint32_t Kw,
                                                            uint64_t *__restrict__ dst) {
  const int lane = threadIdx.x & 63;
  const uint32_t blk = blockIdx.x * WAVES + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (blk >= Wr * Kw) return;
  const uint32_t kb = blk / Wr, w = blk - kb * Wr;     // consecutive waves: consecutive w
  const uint32_t line = kb * 64 + uint32_t(lane);
  uint64_t x = line < K ? src[size_t(w) * K + line] : 0ull;
  x = transpose_stage<32>(x, lane);
  x = transpose_stage<16>(x, lane);
  x = transpose_stage<8>(x, lane);
  x = transpose_stage<4>(x, lane);
  x = transpose_stage<2>(x, lane);
  x = transpose_stage<1>(x, lane);
  dst[size_t(kb) * Wr * 64 + size_t(w) * 64 + lane] = x;
}

// sign(W) as +-1 bytes in 32-line chunks, chunk-major: byte (d, k) at
// ((k / 32) * Dp + d) * 32 + k % 32, so that the 32-byte pieces of consecutive channels
// are adjacent.  16 bytes per thread: channel d, lines [16 q, 16 q + 16).
template <int DT>
__global__ __launch_bounds__(THREADS) void k_pack_w_rows(const void *__restrict__ w, uint32_t D,
                                                         uint32_t K, uint32_t Kp, uint32_t Dp,
                                                         int8_t *__restrict__ dst) {
  const uint32_t qpr = Kp / 16;                          // 16-byte pieces per channel
  const uint32_t e = blockIdx.x * THREADS + threadIdx.x;
  if (e >= Dp * qpr) return;
  const uint32_t d = e / qpr, k0 = (e - d * qpr) * 16;
  uint32_t word[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const uint32_t k = k0 + uint32_t(j);
    uint32_t b = 0u;                                     // 0 past D or K
    if (d < D && k < K) b = load_elem<DT>(w, int64_t(d) * K + k) > 0.0f ? 0x01u : 0xFFu;
    word[j >> 2] |= b << (8 * (j & 3));
  }
  const size_t o = (size_t(k0 / 32) * Dp + d) * 32 + k0 % 32;
  *reinterpret_cast<uint4 *>(dst + o) = make_uint4(word[0], word[1], word[2], word[3]);
}

}  // namespace

int launch_transpose_bits(const uint64_t *src, int64_t Wr, int64_t K, uint64_t *dst,
                          hipStream_t s) {
  const int64_t Kw = (K + 63) / 64;
  hipLaunchKernelGGL(k_transpose_bits, dim3(blocks_for(Wr * Kw)), dim3(THREADS), 0, s, src,
                     uint32_t(Wr), uint32_t(K), uint32_t(Kw), dst);
  return last_launch_status();
}

int launch_pack_w_rows(const void *W, const Layer &L, int64_t Dp, int64_t Kp, int8_t *dst,
                       hipStream_t s) {
  const int64_t items = Dp * (Kp / 16);
  dispatch_dtype(L.w_t, [&]<int DT>() {
    hipLaunchKernelGGL(k_pack_w_rows<DT>, dim3(unsigned((items + THREADS - 1) / THREADS)),
                       dim3(THREADS), 0, s, W, uint32_t(L.D), uint32_t(L.K), uint32_t(Kp),
                       uint32_t(Dp), dst);
  });
  return last_launch_status();
}

int launch_pack_w_i8(const void *W, const Layer &L, int8_t *dst, int32_t *lsum, hipStream_t s) {
  const PackWGeom g = pack_w_geom(L);
  dispatch_dtype(L.w_t, [&]<int DT>() {
    hipLaunchKernelGGL(k_pack_w_i8<DT>, dim3(pack_w_blocks(L)), dim3(WB_THREADS), 0, s, W, g, dst,
                       lsum);
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
    const Im2colGeom g = im2col_geom(L);
    const uint32_t cgroups = g.cgroups;
    nw = L.Wr;
    lines = L.K;
    len = L.R;
    BitGeom bt;
    BandGeom bg;
    size_t lds = 0;
    if (word_major && bit_geom(L, BITS_THREADS, 512, 48 * 1024, &bt, &lds)) {
      bit_geom_vec(&bt, src);
      dispatch_dtype(dtype, [&]<int DT>() {
        hipLaunchKernelGGL(k_pack_im2col_bits<DT>, dim3(bit_blocks(bt)), dim3(BITS_THREADS), lds,
                           s, src, bt, dst);
      });
      return last_launch_status();
    }
    if (word_major && band_geom(L, src, dtype, THREADS, 48 * 1024, &bg, &lds)) {
      const dim3 bgrid(band_word_blocks(L, bg),
                       unsigned((L.C + BAND_CPW * WAVES - 1) / (BAND_CPW * WAVES)));
      dispatch_dtype(dtype, [&]<int DT>() {
        if (L.kh == 3 && L.kw == 3)
          hipLaunchKernelGGL((k_pack_im2col_band<DT, 3, 3>), bgrid, dim3(THREADS), lds, s, src,
                             bg, dst);
        else if (L.kh == 1 && L.kw == 1)
          hipLaunchKernelGGL((k_pack_im2col_band<DT, 1, 1>), bgrid, dim3(THREADS), lds, s, src,
                             bg, dst);
        else
          hipLaunchKernelGGL((k_pack_im2col_band<DT, 0, 0>), bgrid, dim3(THREADS), lds, s, src,
                             bg, dst);
      });
      return last_launch_status();
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
