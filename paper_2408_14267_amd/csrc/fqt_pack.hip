// Sign-bit packing on gfx950 (Section 5.1 binarizer; Appendix C, Alg. 2 row
// encoder, column encoder and Unfolder).  One 64-lane wavefront produces one
// 64-bit word with a ballot: lane l contributes bit l.
#include "fqt_internal.hpp"

namespace fqt {
namespace {

constexpr int THREADS = 256;
constexpr int WAVES = THREADS / 64;

// Along the columns of a row-major [rows][cols] matrix: word w of row i.
__global__ __launch_bounds__(THREADS) void k_pack_along_cols(const void *__restrict__ src,
                                                             int dtype, int64_t rows,
                                                             int64_t cols, int64_t ld,
                                                             uint64_t *__restrict__ dst) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = (cols + 63) >> 6;
  const int64_t item = int64_t(blockIdx.x) * WAVES + (threadIdx.x >> 6);
  if (item >= rows * nw) return;
  const int64_t i = item / nw, w = item - i * nw;
  const int64_t j = (w << 6) + lane;
  const bool bit = j < cols && load_elem(src, dtype, i * ld + j) > 0.0f;
  const uint64_t m = __ballot(bit);
  if (lane == 0) dst[i * nw + w] = m;
}

// Down the rows (transposing): 64x64 tile staged in LDS, read back column-wise.
__global__ __launch_bounds__(THREADS) void k_pack_along_rows(const void *__restrict__ src,
                                                             int dtype, int64_t rows,
                                                             int64_t cols, int64_t ld,
                                                             uint64_t *__restrict__ dst) {
  __shared__ uint8_t bits[64][64 + 4];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t c0 = int64_t(blockIdx.x) * 64, r0 = int64_t(blockIdx.y) * 64;
  const int64_t nw = (rows + 63) >> 6;
  for (int i = 0; i < 16; ++i) {
    const int rr = wave + 4 * i;
    const int64_t r = r0 + rr, c = c0 + lane;
    bits[rr][lane] = (r < rows && c < cols && load_elem(src, dtype, r * ld + c) > 0.0f) ? 1 : 0;
  }
  __syncthreads();
  for (int i = 0; i < 16; ++i) {
    const int cc = wave + 4 * i;
    const int64_t c = c0 + cc;
    if (c >= cols) break;
    const uint64_t m = __ballot(bits[lane][cc] != 0);
    if (lane == 0) dst[c * nw + (r0 >> 6)] = m;
  }
}

struct Im2colGeom {
  int64_t N, C, H, W, Ho, Wo, P, R, K, nw;
  int kh, kw, sh, sw, ph, pw;
};

// Bit-im2col: line (c, i, j), bit (n, ho, wo) = X[n][c][ho*sh - ph + i][wo*sw - pw + j] > 0;
// positions in the zero padding give bit 0 (sign -1).
__global__ __launch_bounds__(THREADS) void k_pack_im2col(const void *__restrict__ x, int dtype,
                                                         Im2colGeom g,
                                                         uint64_t *__restrict__ dst) {
  const int lane = threadIdx.x & 63;
  const int64_t item = int64_t(blockIdx.x) * WAVES + (threadIdx.x >> 6);
  if (item >= g.K * g.nw) return;
  const int64_t line = item / g.nw, w = item - line * g.nw;
  const int64_t c = line / (g.kh * g.kw);
  const int tap = int(line - c * g.kh * g.kw);
  const int i = tap / g.kw, j = tap - (tap / g.kw) * g.kw;
  const int64_t r = (w << 6) + lane;
  bool bit = false;
  if (r < g.R) {
    const int64_t n = r / g.P, pix = r - n * g.P;
    const int64_t ho = pix / g.Wo, wo = pix - ho * g.Wo;
    const int64_t h = ho * g.sh - g.ph + i, ww = wo * g.sw - g.pw + j;
    if (h >= 0 && h < g.H && ww >= 0 && ww < g.W)
      bit = load_elem(x, dtype, ((n * g.C + c) * g.H + h) * g.W + ww) > 0.0f;
  }
  const uint64_t m = __ballot(bit);
  if (lane == 0) dst[line * g.nw + w] = m;
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

}  // namespace

int launch_pack_bits(const void *src, int dtype, int64_t rows, int64_t cols, int64_t ld, int axis,
                     const Layer *conv, uint64_t *dst, int32_t *linesum, hipStream_t s) {
  int64_t lines, nw, len;
  if (axis == FQT_PACK_ALONG_COLS) {
    nw = (cols + 63) / 64;
    lines = rows;
    len = cols;
    hipLaunchKernelGGL(k_pack_along_cols, dim3(blocks_for(rows * nw)), dim3(THREADS), 0, s, src,
                       dtype, rows, cols, ld, dst);
  } else if (axis == FQT_PACK_ALONG_ROWS) {
    nw = (rows + 63) / 64;
    lines = cols;
    len = rows;
    hipLaunchKernelGGL(k_pack_along_rows, dim3(unsigned((cols + 63) / 64), unsigned(nw)),
                       dim3(THREADS), 0, s, src, dtype, rows, cols, ld, dst);
  } else {
    const Layer &L = *conv;
    Im2colGeom g{L.N, L.C, L.H, L.W, L.Ho, L.Wo, L.P, L.R, L.K, L.Wr,
                 L.kh, L.kw, L.sh, L.sw, L.ph, L.pw};
    nw = L.Wr;
    lines = L.K;
    len = L.R;
    hipLaunchKernelGGL(k_pack_im2col, dim3(blocks_for(L.K * L.Wr)), dim3(THREADS), 0, s, src,
                       dtype, g, dst);
  }
  if (last_launch_status() != FQT_OK) return FQT_E_HIP;
  if (linesum) {
    hipLaunchKernelGGL(k_linesum, dim3(blocks_for(lines)), dim3(THREADS), 0, s, dst, lines, nw,
                       len, linesum);
    return last_launch_status();
  }
  return FQT_OK;
}

}  // namespace fqt
