// Internal declarations of libfqt: validated layer geometry, workspace carving,
// kernel launchers and the device helpers shared by the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <climits>
#include <stdint.h>

#include "fqt.h"

namespace fqt {

// ----------------------------------------------------------------------------- host side

// Layer geometry after validation; every derived size the kernels need.
struct Layer {
  int kind;
  int dy_t, x_t, w_t, dx_t;
  int64_t N, C, H, W, D;
  int kh, kw, sh, sw, ph, pw;
  int64_t Ho, Wo;
  int64_t P;    // output pixels per sample, Ho*Wo
  int64_t R;    // rows of the unfolded gradient, N*P
  int64_t K;    // unfolded weight width, C*kh*kw
  int64_t HW;   // input pixels per sample, H*W
  int64_t Wd;   // 64-bit words of a line packed along D
  int64_t Wr;   // 64-bit words of a line packed along R
};

// Per-group parameters the quantize kernel reads (written by the select kernel).
struct GroupParam {
  float z;        // zero point Z (the group minimum)
  float inv;      // B / R in float32, 0 when R == 0
  int32_t rank;   // position among the kept groups (ascending ids), -1 if pruned
  int32_t pad;
};

// Quantize workspace: per-tile partial min/max keys, the reduced keys of both group
// sets, and the per-group parameters of the quantizer.
// Merged group keys: (min, max) keys of every sample and channel combined by atomics while
// the statistics run (both stored so that 0 is the identity of an unsigned max), at the
// start of the quantizer's workspace.  MKEY_REP replicas of each key, written by different
// workgroups, cut the number of atomics that meet at one address.  They are zero between
// calls: the workspace is zero-filled once before its first use and each selection clears
// the entries it reads.
constexpr int MKEY_GROUPS = 2 * 1024;
constexpr int MKEY_REP = 8;
constexpr int MKEY_SLOTS = MKEY_GROUPS * MKEY_REP;
struct QuantWs {
  uint2 *mkeys;            // [MKEY_REP][MKEY_GROUPS]: samples at [0, N), channels at
                           //   [N, N + D) of each replica
  int2 *part_c;            // [stats_row_blocks][D]  channel partials of each row block
  int2 *part_s;            // [ceil(D/64)][ceil(R/64)][stats_slots]  sample partials of
                           //   each 64 x 64 tile, one slot per sample the tile meets
                           //   (P = 1: [R][ceil(D/64)], one per sample and tile)
  int2 *skey;              // [N] (min, max) ordered-int keys of each sample
  int2 *ckey;              // [D] (min, max) keys of each output channel
  GroupParam *sp;          // [N]
  GroupParam *cp;          // [D]
  float2 *sslot;           // [N] (scale, offset) of the kept sample in slot j (j < count)
  float2 *cslot;           // [D] the same for the kept channels
};

// Division by a fixed divisor for numerators below 2^31:
// q = (n * m) >> s with l = ceil(log2 d), m = ceil(2^(32+l) / d), s = 32 + l.
// The rounding error of m is below d, so n * (m*d - 2^s) / (d 2^s) < 1/(2d) never
// carries the quotient past the next integer.
struct FastDiv {
  uint64_t m;
  uint32_t s;
  uint32_t d;
};
inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((uint64_t(1) << l) < d) ++l;
  FastDiv f;
  f.m = ((uint64_t(1) << (32 + l)) + d - 1) / d;
  f.s = 32 + l;
  f.d = d;
  return f;
}
__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f) {
  return static_cast<uint32_t>((uint64_t(n) * f.m) >> f.s);
}

int make_layer(const fqt_layer_desc *d, Layer *L);
int check_cfg(const fqt_quant_cfg *c, const Layer &L);
size_t quant_ws_bytes(const Layer &L);
uint32_t stats_slots(const Layer &L);       // sample slots of a 64-row tile
int64_t stats_row_blocks(const Layer &L);   // row blocks of the stats kernel
void carve_quant_ws(void *ws, const Layer &L, QuantWs *q);
inline size_t align256(size_t b) { return (b + 255) & ~size_t(255); }
inline bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Launchers (stream-ordered, no synchronisation).  They return an fqt_status.
// The sign operands of the products, packed in spare blocks of the selection launch when
// the layer allows it (launch_quantize then sets *done).
struct SignJob {
  const void *X, *W;
  uint64_t *xsign;       // word-major sign(unfold(X))
  int8_t *wsb;           // sign(W) bytes
  int32_t *wlsum;
  bool done;
};
// Zero-fills the FQT_WS_STATE_BYTES of state at the start of a quantize / layer workspace.
int launch_state_clear(void *state, hipStream_t s);
// planes = false: the codes one byte each only (what the products read), no bit planes.
int launch_quantize(const Layer &L, const fqt_quant_cfg &cfg, const void *dY, const fqt_qgrad &q,
                    const QuantWs &w, hipStream_t s, SignJob *signs = nullptr,
                    bool planes = true);
int launch_pack_bits(const void *src, int dtype, int64_t rows, int64_t cols, int64_t ld, int axis,
                     const Layer *conv, uint64_t *dst, int32_t *linesum, hipStream_t s,
                     bool word_major = false);
size_t gemm_dw_ws_bytes(const Layer &L, const fqt_quant_cfg &cfg);
int launch_gemm_dw(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                   const uint64_t *xsign, float *dW, int32_t *I_out, void *ws, hipStream_t s);
int launch_pack_w_i8(const void *W, const Layer &L, int8_t *dst, int32_t *lsum, hipStream_t s);
int launch_gemm_dx(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                   const int8_t *wsb, const int32_t *wlsum, void *dX, int32_t *I_out,
                   hipStream_t s);
// Both products of the layer backward in one launch, then the dW finish pass.
// sslot / cslot: the selection's slot-ordered (scale, offset) pairs (QuantWs).
int launch_products(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                    const uint64_t *xsign, const int8_t *wsb, const int32_t *wlsum, void *dX,
                    float *dW, void *dw_ws, const float2 *sslot, const float2 *cslot,
                    hipStream_t s);

// The dW product from the code planes and line-major sign bits (popcount or fp4 engine).
size_t engine_ws_bytes(const Layer &L, const fqt_quant_cfg &cfg, int engine);
int check_engine(const Layer &L, const fqt_quant_cfg &cfg, int engine);
int launch_gemm_dw_planes(const Layer &L, const fqt_quant_cfg &cfg, const fqt_qgrad &q,
                          const uint64_t *xbits, const int32_t *xsum, float *dW, int32_t *I_out,
                          int engine, void *ws, hipStream_t s);

// Binary forward (Section 5.1): the operands and the product.
// Word-major sign words [Wr][K] -> k-block-major [Kw][Wr * 64] (bit b of word (kb, r) is
// line 64 kb + b of row r; lines past K are 0).
int launch_transpose_bits(const uint64_t *src, int64_t Wr, int64_t K, uint64_t *dst,
                          hipStream_t s);
// sign(W) as +-1 bytes in 32-line chunks [Kp/32][Dp][32], lines in W's own [D][C*kh*kw]
// order, 0 past D and past K.
int launch_pack_w_rows(const void *W, const Layer &L, int64_t Dp, int64_t Kp, int8_t *dst,
                       hipStream_t s);
// Y[n][d][p] = gamma[d] * sum_k sign(X_u)[r][k] sign(W)[d][k] from the two packed operands.
int launch_forward_gemm(const Layer &L, const int8_t *wrows, int64_t Dp, int64_t Kp,
                        const uint64_t *xrows, const float *gamma, void *Y, int32_t *I_out,
                        hipStream_t s);

inline int hip_status(hipError_t e) { return e == hipSuccess ? FQT_OK : FQT_E_HIP; }
inline int last_launch_status() { return hip_status(hipGetLastError()); }

// ----------------------------------------------------------------------------- device side

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of the 4x32 S-box
// with multipliers M0 = 0xD2511F53, M1 = 0xCD9E8D57 and Weyl key increments
// W0 = 0x9E3779B9, W1 = 0xBB67AE85 between rounds.
struct Ctr4 {
  uint32_t v[4];
};

// Word j (0..3, known only at run time) of a Philox block, by selects: indexing the
// array with a run-time value would move it to scratch memory.
__device__ __forceinline__ uint32_t ctr_word(const Ctr4 &c, uint32_t j) {
  const uint32_t lo = (j & 1u) ? c.v[1] : c.v[0];
  const uint32_t hi = (j & 1u) ? c.v[3] : c.v[2];
  return (j & 2u) ? hi : lo;
}

__device__ __forceinline__ Ctr4 philox4x32_10(Ctr4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    // One 32 x 32 -> 64-bit product gives both halves.
    const uint64_t p0 = uint64_t(0xD2511F53u) * c.v[0];
    const uint64_t p1 = uint64_t(0xCD9E8D57u) * c.v[2];
    Ctr4 n;
    if (r < 2) {
      // Counter words that are the same across a wave (stream, layer, step) keep the
      // first rounds partly on the scalar unit; plain XORs leave the compiler that choice.
      n.v[0] = uint32_t(p1 >> 32) ^ c.v[1] ^ k0;
      n.v[2] = uint32_t(p0 >> 32) ^ c.v[3] ^ k1;
    } else {
      // Both XORs in one instruction (bitop3 with truth table 0x96 = a ^ b ^ c).
      n.v[0] = __builtin_amdgcn_bitop3_b32(uint32_t(p1 >> 32), c.v[1], k0, 0x96);
      n.v[2] = __builtin_amdgcn_bitop3_b32(uint32_t(p0 >> 32), c.v[3], k1, 0x96);
    }
    n.v[1] = uint32_t(p1);
    n.v[3] = uint32_t(p0);
    c = n;
  }
  return c;
}

enum : uint32_t { STREAM_ELEM = 0, STREAM_SAMPLE = 1, STREAM_CHANNEL = 2 };

// The four words of the Philox block holding items 4*blk .. 4*blk+3 of a stream.
__device__ __forceinline__ Ctr4 philox_block(uint64_t blk, uint32_t stream, uint64_t seed,
                                             uint32_t step, uint32_t layer) {
  Ctr4 c;
  c.v[0] = static_cast<uint32_t>(blk);
  c.v[1] = (static_cast<uint32_t>(blk >> 32) & 0x3FFFFFFFu) | (stream << 30);
  c.v[2] = layer;
  c.v[3] = step;
  return philox4x32_10(c, static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32));
}

// Order-preserving map float -> int32 (for atomicMin/atomicMax on float values).
__device__ __forceinline__ int32_t f2key(float f) {
  const int32_t i = __float_as_int(f);
  return i >= 0 ? i : (i ^ 0x7FFFFFFF);
}
__device__ __forceinline__ float key2f(int32_t k) {
  return __int_as_float(k >= 0 ? k : (k ^ 0x7FFFFFFF));
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}
// float32 -> bfloat16, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Load one element of a float32 (DT = FQT_F32) or bfloat16 (FQT_BF16) tensor as float32.
// The dtype is a template parameter so that a load carries no branch and a run of
// loads issues back to back before the first use.
template <int DT>
__device__ __forceinline__ float load_elem(const void *p, int64_t i) {
  if (DT == FQT_BF16) return bf16_to_f32(static_cast<const uint16_t *>(p)[i]);
  return static_cast<const float *>(p)[i];
}

// Load four consecutive elements starting at i (i % 4 == 0, base 16-byte aligned).
template <int DT>
__device__ __forceinline__ void load_quad(const void *p, int64_t i, float out[4]) {
  if (DT == FQT_BF16) {
    const uint2 v = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(p) + i);
    out[0] = __uint_as_float(v.x << 16);
    out[1] = __uint_as_float(v.x & 0xFFFF0000u);
    out[2] = __uint_as_float(v.y << 16);
    out[3] = __uint_as_float(v.y & 0xFFFF0000u);
  } else {
    const float4 v = *reinterpret_cast<const float4 *>(static_cast<const float *>(p) + i);
    out[0] = v.x;
    out[1] = v.y;
    out[2] = v.z;
    out[3] = v.w;
  }
}

// Load eight consecutive elements starting at i (i % 8 == 0, base 16-byte aligned): one
// 16-byte load for bfloat16, two for float32.
template <int DT>
__device__ __forceinline__ void load_oct(const void *p, int64_t i, float out[8]) {
  if (DT == FQT_BF16) {
    const uint4 v = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(p) + i);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      out[2 * k] = __uint_as_float(w[k] << 16);
      out[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
    }
  } else {
    load_quad<DT>(p, i, out);
    load_quad<DT>(p, i + 4, out + 4);
  }
}

// Calls F.template operator()<DT>() with DT the compile-time dtype code of `dt`.
template <typename F>
__host__ void dispatch_dtype(int dt, F &&f) {
  if (dt == FQT_BF16) f.template operator()<FQT_BF16>();
  else f.template operator()<FQT_F32>();
}

__device__ __forceinline__ int popc64(uint64_t v) { return __popcll(v); }

// ----------------------------------------------------------------------------- buffer loads
// Raw buffer resources: a lane whose offset is BUF_NONE (past every buffer here, all
// shorter than 2^31 bytes) loads zeros without touching memory.  The bounds check covers
// the per-lane offset only; the wave-uniform offset (an SGPR) must keep in-bounds lanes in
// bounds by construction.
typedef int v4i __attribute__((ext_vector_type(4)));
constexpr uint32_t BUF_NONE = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void *p, uint32_t bytes) {
  // Raw buffer (stride 0) of `bytes` bytes; 0x00020000 is the gfx9 32-bit data format.
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), static_cast<short>(0),
                                           static_cast<int>(bytes), 0x00020000);
}
// 16 / 8 bytes at byte offset voff + soff of buffer r (soff wave-uniform).
__device__ __forceinline__ v4i load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ uint64_t load8(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
}

// ----------------------------------------------------------------------------- cross-lane
// Wave-level exchanges on the VALU data path (DPP row operations and the gfx950 lane
// swaps) instead of ds_bpermute, whose LDS round trip dominates short dependency chains.
// DPP row operations act within rows of 16 lanes: row_shr:n (0x110 + n) reads lane
// i - n of the row (lanes without a source keep `old`), row_ror:8 (0x128) swaps the row's
// halves, row_bcast:15 / :31 (0x142 / 0x143, rows 1,3 / 2,3 enabled) read the last lane
// of the preceding row / of row 1.
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ int dpp(int old, int v) {
  return __builtin_amdgcn_update_dpp(old, v, CTRL, ROWS, 0xF, false);
}

// v of lane (lane ^ M), M in {1, 2, 4, 8, 16, 32}.
template <int M>
__device__ __forceinline__ uint32_t lane_xor(uint32_t v) {
  const int x = int(v);
  if constexpr (M == 1) return uint32_t(dpp<0xB1>(0, x));          // quad_perm [1,0,3,2]
  else if constexpr (M == 2) return uint32_t(dpp<0x4E>(0, x));     // quad_perm [2,3,0,1]
  else if constexpr (M == 4) return uint32_t(dpp<0x141>(0, dpp<0x1B>(0, x)));  // i^3, then i^7
  else if constexpr (M == 8) return uint32_t(dpp<0x128>(0, x));    // row_ror:8
  else if constexpr (M == 16) {
    // permlane16_swap(v, v): .x holds the even rows twice, .y the odd rows twice.
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    return uint32_t((__lane_id() & 16) ? r[0] : r[1]);
  } else {
    static_assert(M == 32, "lane_xor: M must be a power of two below 64");
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return uint32_t((__lane_id() & 32) ? r[0] : r[1]);
  }
}
template <int M>
__device__ __forceinline__ uint64_t lane_xor64(uint64_t v) {
  return (uint64_t(lane_xor<M>(uint32_t(v >> 32))) << 32) | lane_xor<M>(uint32_t(v));
}

// Write the wave-uniform value v into lane `l` of `old` (v_writelane_b32; the LLVM
// intrinsic has no clang builtin here).
extern "C" __device__ int fqt_llvm_writelane(int v, int l, int old) __asm("llvm.amdgcn.writelane.i32");
__device__ __forceinline__ uint32_t writelane(uint32_t v, int l, uint32_t old) {
  return uint32_t(fqt_llvm_writelane(int(v), l, int(old)));
}

// 8 x 8 bit-matrix transpose of x, byte k = row k, LSB first: byte p of the result holds
// bit p of every byte k of x at bit k (three delta swaps).
__device__ __forceinline__ uint64_t bit_transpose8(uint64_t x) {
  uint64_t t = (x ^ (x >> 7)) & 0x00AA00AA00AA00AAull;
  x ^= t ^ (t << 7);
  t = (x ^ (x >> 14)) & 0x0000CCCC0000CCCCull;
  x ^= t ^ (t << 14);
  t = (x ^ (x >> 28)) & 0x00000000F0F0F0F0ull;
  x ^= t ^ (t << 28);
  return x;
}

// Inclusive scan of v over the wave's lanes under `op` with identity `id` (lane 63 ends
// with the whole wave's result).
template <typename Op>
__device__ __forceinline__ int wave_scan_i32(int v, int id, Op op) {
  v = op(v, dpp<0x111>(id, v));
  v = op(v, dpp<0x112>(id, v));
  v = op(v, dpp<0x114>(id, v));
  v = op(v, dpp<0x118>(id, v));
  v = op(v, dpp<0x142, 0xA>(id, v));
  v = op(v, dpp<0x143, 0xC>(id, v));
  return v;
}
__device__ __forceinline__ int wave_min_all(int v) {
  return __builtin_amdgcn_readlane(wave_scan_i32(v, INT_MAX, [](int a, int b) { return min(a, b); }), 63);
}
__device__ __forceinline__ int wave_max_all(int v) {
  return __builtin_amdgcn_readlane(wave_scan_i32(v, INT_MIN, [](int a, int b) { return max(a, b); }), 63);
}
// Inclusive prefix sum over the wave for 64-bit values (carries through the high word).
__device__ __forceinline__ uint64_t wave_scan_add_u64(uint64_t v) {
#define FQT_DPP_ADD64(CTRL, ROWS)                                                    \
  do {                                                                               \
    const uint32_t lo = uint32_t(dpp<CTRL, ROWS>(0, int(uint32_t(v))));              \
    const uint32_t hi = uint32_t(dpp<CTRL, ROWS>(0, int(uint32_t(v >> 32))));        \
    v += (uint64_t(hi) << 32) | lo;                                                  \
  } while (0)
  FQT_DPP_ADD64(0x111, 0xF);
  FQT_DPP_ADD64(0x112, 0xF);
  FQT_DPP_ADD64(0x114, 0xF);
  FQT_DPP_ADD64(0x118, 0xF);
  FQT_DPP_ADD64(0x142, 0xA);
  FQT_DPP_ADD64(0x143, 0xC);
#undef FQT_DPP_ADD64
  return v;
}
// Sum of v over the wave, in every lane (the scan's last lane, read as two scalars).
__device__ __forceinline__ uint64_t wave_total_u64(uint64_t v) {
  const uint64_t s = wave_scan_add_u64(v);
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(s)), 63));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(s >> 32)), 63));
  return (uint64_t(hi) << 32) | lo;
}

}  // namespace fqt
