/*
 * fqt.h -- C ABI of libfqt, the MI355X (gfx950) backward pass of binary linear and
 * convolution layers under 1-bit fully quantized training with Activation
 * Gradient Pruning (AGP) and Sample-Channel joint Quantization (SCQ).
 *
 * Method: Gao et al., "1-Bit FQT: Pushing the Limit of Fully Quantized Training
 * to 1-bit" (arXiv 2408.14267).  Section 5.2 defines AGP and the lossless
 * bit-plane decomposition, Section 5.3 SCQ (per-sample codes feed the
 * activation gradient dX, per-channel codes feed the weight gradient dW),
 * Appendix C Alg. 1 the backward sequence (pruner, PSQ/PCQ, encoders, binary
 * products, dequantization), Alg. 2 the row encoder, and the Unfolder/Folder
 * for convolutions.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensors are NCHW, torch layout: X [N][C][H][W], W [D][C][kh][kw],
 *    dY [N][D][Ho][Wo], dX like X, dW like W (fp32).  A linear layer is the
 *    case H = W = kh = kw = 1 (X [N][C], W [D][C], dY [N][D]).
 *  - Every tensor pointer is a DEVICE pointer on the current HIP device; the
 *    caller owns all memory; the library never allocates and never synchronizes
 *    the stream.  It keeps no host-side state; the only state that outlives a
 *    call is the zeroed first FQT_WS_STATE_BYTES of a quantize or layer
 *    workspace (see fqt_workspace_init).  Work is enqueued on
 *    `hip_stream` (a hipStream_t; NULL = the null stream); outputs are valid
 *    once that stream has reached the enqueued work.
 *  - Descriptor structs are HOST pointers, read during the call only.
 *  - Arguments are validated on the host before anything is launched; a
 *    failing validation returns a negative fqt_status and launches nothing.
 *    A failed launch returns FQT_E_HIP.  No C++ exception crosses the ABI.
 *  - Alignment: dY 16 bytes, other float/bf16 tensors their element size, uint64 bit
 *    arrays 8 bytes, byte-code arrays 16 bytes, int32 and float32 arrays 4 bytes,
 *    workspaces 256 bytes (FQT_E_ALIGN otherwise).
 *  - Bit packing: bit j of a packed line is bit (j % 64) of 64-bit word j / 64,
 *    least significant bit first; ragged tails are zero.  A set bit is +1, a
 *    clear bit -1 (sign(x) = -1 for x <= 0, Section 5.1), or a code bit.
 *  - Inputs must be finite; NaN/Inf gradients give unspecified codes.
 */
#ifndef FQT_H
#define FQT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FQT_OK = 0,
  FQT_E_INVAL = -1,     /* scalar argument out of range (kind, bits, agp_mode, axis, ...)   */
  FQT_E_DTYPE = -2,     /* unsupported dtype or dtype combination                           */
  FQT_E_SHAPE = -3,     /* non-positive or inconsistent dims, or a size limit exceeded      */
  FQT_E_WORKSPACE = -4, /* workspace smaller than fqt_workspace_size() reports              */
  FQT_E_ALIGN = -5,     /* a pointer violates the alignment rule above                      */
  FQT_E_NULL = -6,      /* a required pointer is NULL                                       */
  FQT_E_HIP = -7        /* a HIP runtime call or kernel launch failed                       */
} fqt_status;

typedef enum { FQT_F32 = 0, FQT_BF16 = 1 } fqt_dtype;

typedef enum { FQT_LINEAR = 0, FQT_CONV2D = 1 } fqt_layer_kind;

typedef enum {
  FQT_AGP_BERNOULLI = 0, /* Section 5.2: p_i proportional to the group range, sum p_i = G/b,
                            capped at 1 (water-filling), masks m_i ~ Bern(p_i), 1/p rescale */
  FQT_AGP_TOPK = 1,      /* Appendix B.2's limit p in {0,1}: keep the max(1, G/b) largest
                            ranges, no rescale (biased; provided for study)                */
  FQT_AGP_OFF = 2        /* plain b-bit PSQ/PCQ (Section 5.2): every group kept, p = 1      */
} fqt_agp_mode;

/* Limits.  The AGP sort of one group set runs in one workgroup's LDS. */
#define FQT_MAX_BITS 8
#define FQT_MAX_AGP_GROUPS 16384   /* N and D bound for BERNOULLI / TOPK               */

/* Layer geometry (Section 3, Eq. 1-3; Appendix C Unfolder: X_u is NHW x CK^2).
 * Ho = (H + 2 ph - kh) / sh + 1 and Wo likewise must be >= 1.
 * dy_dtype, x_dtype, dx_dtype: FQT_F32 or FQT_BF16; w_dtype: FQT_F32 or FQT_BF16.
 * N*Ho*Wo, N*C*H*W, N*D*Ho*Wo and D*C*kh*kw must stay below 2^31, and so must the
 * byte sizes of the code arrays and of the weight-sign bytes: N*Ho*Wo * 64*ceil(D/64),
 * D * 64*ceil(N*Ho*Wo/64) and C*kh*kw * 64*ceil(D/64) (FQT_E_SHAPE otherwise). */
typedef struct {
  int32_t kind;                       /* fqt_layer_kind                                  */
  int32_t dy_dtype, x_dtype, w_dtype, dx_dtype;
  int64_t N, C, H, W, D;              /* linear: H = W = 1, C = in features, D = out     */
  int32_t kh, kw, sh, sw, ph, pw;     /* linear: 1, 1, 1, 1, 0, 0                        */
} fqt_layer_desc;

/* Quantizer configuration (Section 3.2 quantizer; Section 5.2 AGP keep ratio 1/b).
 * The random words come from Philox4x32-10 (Salmon et al., SC'11) with key = seed
 * and counter (lo32(i >> 2), hi32(i >> 2) | stream << 30, layer_id, step), word i & 3,
 * where i is the element's NCHW index of dY (stream 0), the sample id (stream 1)
 * or the output-channel id (stream 2). */
typedef struct {
  int32_t bits;                       /* b in [1, FQT_MAX_BITS]: code width of kept groups  */
  int32_t agp_mode;                   /* fqt_agp_mode                                       */
  uint64_t seed;
  uint32_t step;
  uint32_t layer_id;
} fqt_quant_cfg;

/* Quantized output gradient (Section 5.3, SCQ; Appendix C Alg. 1 quantization and
 * encoding).  All members are device pointers sized to capacity; the caller owns
 * them.  With P = Ho*Wo, R = N*P, Wd = ceil(D/64), Wr = ceil(R/64), b = bits:
 *   psq_planes  uint64 [b][R][Wd]   PSQ code planes, plane k = bit k of the code; row
 *                                   j*P + p holds pixel p of the j-th kept sample
 *                                   (kept samples in ascending order), packed along D.
 *                                   Rows >= count*P are left untouched.
 *   pcq_planes  uint64 [b][D][Wr]   PCQ code planes; row j holds the j-th kept channel,
 *                                   packed along (n, ho, wo).  Rows >= count untouched.
 *   psq_codes   uint8 [2*Wd][R][32] the same PSQ codes one byte each (the operand of the
 *                                   int8 products), chunk-major: code d of row r (rows as
 *                                   in psq_planes) at ((d/32)*R + r)*32 + d%32; codes past
 *                                   D are 0.  The 32-byte chunks of consecutive rows are
 *                                   adjacent, so the product's operand loads coalesce.
 *   pcq_codes   uint8 [2*Wr][D][32] the PCQ codes one byte each, chunk-major: code r of
 *                                   row j at ((r/32)*D + j)*32 + r%32; codes past R are 0
 *   psq_kept    int32 [N]           kept sample ids ascending, then pruned ids ascending
 *   psq_count   int32 [1]           number of kept samples
 *   psq_scale   float [N]           S_n = R_n / (B p_n) if kept, else 0
 *   psq_offset  float [N]           Z'_n = Z_n / p_n if kept, else 0
 *   psq_prob    float [N]           keep probability p_n
 *   pcq_*       the same for the D output channels. */
typedef struct {
  uint64_t *psq_planes;
  uint64_t *pcq_planes;
  uint8_t *psq_codes;                 /* 16-byte aligned */
  uint8_t *pcq_codes;                 /* 16-byte aligned */
  int32_t *psq_kept, *psq_count, *pcq_kept, *pcq_count;
  float *psq_scale, *psq_offset, *psq_prob;
  float *pcq_scale, *pcq_offset, *pcq_prob;
} fqt_qgrad;

/* Element counts of the plane arrays (uint64 words) and the code arrays (bytes) of
 * fqt_qgrad (host call, no device work). */
int fqt_qgrad_words(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg,
                    int64_t *psq_words, int64_t *pcq_words, int64_t *psq_code_bytes,
                    int64_t *pcq_code_bytes);

/* Workspace sizes (host call).  which = FQT_WS_QUANTIZE for fqt_agp_scq_quantize,
 * FQT_WS_GEMM_DW for fqt_binary_gemm_dw (its split partial sums), FQT_WS_LAYER for
 * fqt_layer_backward (which holds an fqt_qgrad, the packed signs and the partial sums
 * inside it).  The library carves the workspace.  A FQT_WS_QUANTIZE or FQT_WS_LAYER
 * workspace keeps state between calls in its first 128 KiB (FQT_WS_STATE_BYTES): the group
 * keys that the statistics combine with atomics.  Those bytes must be zero when a call
 * starts: run fqt_workspace_init on the workspace once, after allocating it and before its
 * first use; every call that returns FQT_OK leaves them zero again (and the rest of the
 * workspace garbage).  A call that fails after its first launch clears them itself on the
 * same stream; if that clearing launch fails too, the call returns FQT_E_HIP and the
 * caller runs fqt_workspace_init again before reusing the workspace.  An uninitialised
 * workspace gives wrong group ranges, undetected.  Such a workspace may serve layers of
 * any shape, one call at a time, but nothing else may write its first 128 KiB (do not
 * share it with a FQT_WS_GEMM_DW workspace).  A FQT_WS_GEMM_DW or FQT_WS_FORWARD
 * workspace needs no initialisation. */
#define FQT_WS_STATE_BYTES 131072
#define FQT_WS_QUANTIZE 0
#define FQT_WS_LAYER 1
#define FQT_WS_GEMM_DW 2
#define FQT_WS_FORWARD 3   /* fqt_binary_forward; cfg may be NULL for this one */
#define FQT_WS_DW_POPCOUNT 4   /* fqt_binary_gemm_dw_planes, FQT_ENGINE_POPCOUNT */
#define FQT_WS_DW_FP4 5        /* fqt_binary_gemm_dw_planes, FQT_ENGINE_FP4 */
int fqt_workspace_size(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, int32_t which,
                       size_t *bytes);

/* Prepares a FQT_WS_QUANTIZE or FQT_WS_LAYER workspace for use: zero-fills its first
 * FQT_WS_STATE_BYTES with one small kernel on hip_stream (no memset node, so it may be
 * captured in a HIP graph).  ws: device pointer, 256-byte aligned; ws_bytes >=
 * FQT_WS_STATE_BYTES (FQT_E_WORKSPACE otherwise).  Not a statement of the paper: the
 * statistics combine group keys with atomics, which need a zeroed target. */
int fqt_workspace_init(void *ws, size_t ws_bytes, void *hip_stream);

/* AGP + SCQ quantization of dY (Section 5.2 AGP; Section 5.3 SCQ; Appendix C Alg. 1
 * pruner, PSQ/PCQ, row/column encoders).  Per-sample and per-channel range R = max - min
 * and zero point Z = min (float32); AGP keep probabilities and Bernoulli masks for both
 * group sets; for every element of a kept sample (kept channel) a b-bit stochastic
 * rounding code q = floor(v) + [u24 < frac(v) 2^24], v = clamp((x - Z) * (B / R), 0, B)
 * in float32, B = 2^b - 1, one Philox word per element shared by its PSQ and PCQ code;
 * codes split into b bit planes and packed (row encoder along D for PSQ, column encoder
 * along N*Ho*Wo for PCQ), and the same codes as bytes.  dY has desc->dy_dtype.  Writes
 * every member of *out.
 * ws: >= fqt_workspace_size(FQT_WS_QUANTIZE) bytes. */
int fqt_agp_scq_quantize(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, const void *dY,
                         const fqt_qgrad *out, void *ws, size_t ws_bytes, void *hip_stream);

/* Sign-bit packing (Section 5.1 binarizer; Appendix C Alg. 2 row/column encoders and
 * the Unfolder).  src has dtype `dtype` (FQT_F32 / FQT_BF16).
 *   axis = FQT_PACK_ALONG_COLS: src is a row-major [rows][cols] matrix with leading
 *          dimension ld (elements); dst is uint64 [rows][ceil(cols/64)], bit j of line i
 *          = src[i][j] > 0.
 *   axis = FQT_PACK_ALONG_ROWS: same src; dst is uint64 [cols][ceil(rows/64)], bit i of
 *          line j = src[i][j] > 0 (the column encoder; W [D][C*kh*kw] packed along D).
 *   axis = FQT_PACK_IM2COL: src is the conv input X of `conv`; rows/cols/ld are ignored;
 *          dst is uint64 [C*kh*kw][ceil(N*Ho*Wo/64)], bit (n, ho, wo) of line (c, i, j)
 *          = X[n][c][ho*sh - ph + i][wo*sw - pw + j] > 0, and 0 (sign -1) where that
 *          position lies in the zero padding.
 * linesum (optional, int32 [lines]) receives sum over the line of the +-1 signs,
 * 2 * popcount - length.  conv must be non-NULL exactly for FQT_PACK_IM2COL. */
#define FQT_PACK_ALONG_ROWS 0
#define FQT_PACK_ALONG_COLS 1
#define FQT_PACK_IM2COL 2
int fqt_pack_bits(const void *src, int32_t dtype, int64_t rows, int64_t cols, int64_t ld,
                  int32_t axis, const fqt_layer_desc *conv, uint64_t *dst, int32_t *linesum,
                  void *hip_stream);

/* Weight-gradient product with PCQ codes (Section 5.3, SCQ; Appendix C Alg. 1 binary
 * product and dequantization; {0,1} <-> {+-1} conversion):
 *   I[d][k]  = sum_r q_pcq[d][r] * s_X[r][k]   (k over C*kh*kw, r over N*Ho*Wo);
 *   dW[d][k] = S_d * I[d][k] + Z'_d * c_X[k] in float32 for kept channels, 0 for pruned,
 *   with c_X[k] = sum_r s_X[r][k] (the zero-point term).
 * Computed on int8 MFMA from q->pcq_codes and the packed signs, which are expanded to
 * +-1 bytes in registers, in slices of N*Ho*Wo whose partial sums meet in the workspace.
 * xsign: the output of fqt_pack_input_signs for the layer's X.  dW: float [D][C*kh*kw].
 * I_out (optional): int32 [D][C*kh*kw] receives I (0 in pruned rows).
 * ws: >= fqt_workspace_size(FQT_WS_GEMM_DW) bytes, 256-byte aligned.
 * I is exact in int32 only while (2^b - 1) * N*Ho*Wo < 2^31: larger layers return
 * FQT_E_SHAPE (here and in fqt_layer_backward). */
int fqt_binary_gemm_dw(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg,
                       const fqt_qgrad *q, const uint64_t *xsign, float *dW, int32_t *I_out,
                       void *ws, size_t ws_bytes, void *hip_stream);

/* The weight-gradient product from the paper's packed operands (Section 5.2's bit-plane
 * decomposition; Appendix C, binary multiplication, average 1-bit and the {0,1} <-> {+-1}
 * conversion): the same I and dW as fqt_binary_gemm_dw, from
 *   q->pcq_planes  the PCQ code planes written by fqt_agp_scq_quantize, and
 *   xbits          sign(unfold(X)) packed along N*Ho*Wo, uint64 [C*kh*kw][ceil(N*Ho*Wo/64)]
 *                  (fqt_pack_bits FQT_PACK_IM2COL for a convolution, FQT_PACK_ALONG_ROWS of
 *                  X [N][C] for a linear layer), with
 *   xbits_linesum  its line sums, int32 [C*kh*kw] (fqt_pack_bits' linesum),
 * I = sum_p 2^p (2 popcount(q_p & t) - popcount(q_p)) over the words.  engine:
 *   FQT_ENGINE_POPCOUNT  AND + popcount on the vector ALUs (the paper's engine), any b;
 *   FQT_ENGINE_FP4       both operands expanded once to e2m1 (a set bit 1.0, a clear one 0)
 *                        and contracted by gfx950's scaled fp4 MFMA, one per plane with
 *                        the plane weight 2^p as its scale; float32 sums are exact, so
 *                        b <= 4 and (2^b - 1) * N*Ho*Wo < 2^24 (FQT_E_INVAL / FQT_E_SHAPE
 *                        otherwise).
 * ws: >= fqt_workspace_size(FQT_WS_DW_POPCOUNT or FQT_WS_DW_FP4) bytes, 256-byte aligned,
 * no initialisation.  dW: float [D][C*kh*kw]; I_out (optional) int32 [D][C*kh*kw]. */
#define FQT_ENGINE_POPCOUNT 1
#define FQT_ENGINE_FP4 2
int fqt_binary_gemm_dw_planes(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg,
                              const fqt_qgrad *q, const uint64_t *xbits,
                              const int32_t *xbits_linesum, float *dW, int32_t *I_out,
                              int32_t engine, void *ws, size_t ws_bytes, void *hip_stream);

/* sign(X) in the operand form of the dW product (Section 5.1 binarizer; Appendix C Alg. 2
 * and the Unfolder): the bits of fqt_pack_bits IM2COL for a convolution (ALONG_ROWS of X
 * [N][C] for a linear layer) stored word-major, dst uint64 [ceil(N*Ho*Wo/64)][C*kh*kw] with
 * word w of line l at w * C*kh*kw + l, so that the words of consecutive lines are
 * adjacent.  X has desc->x_dtype. */
int fqt_pack_input_signs(const fqt_layer_desc *desc, const void *X, uint64_t *dst,
                         void *hip_stream);

/* sign(W) in the operand form of the int8 dX product (Section 5.1 binarizer; the +-1 form
 * of Appendix C's {0,1} <-> {+-1} conversion).  W [D][C][kh][kw] of desc->w_dtype is
 * viewed as [D][C*kh*kw]; with Dp = 64*ceil(D/64), taps = kh*kw, line l = (c, tap):
 *   dst      int8 [Dp/32][taps][C][32]   byte d of line (c, tap) at
 *                                 ((d/32 * taps + tap) * C + c) * 32 + d%32: +1 if
 *                                 W[d][c][tap] > 0, -1 otherwise, for d < D; 0 for
 *                                 D <= d < Dp.  16-byte aligned.
 *   linesum  int32 [C*kh*kw]      sum over d < D of dst[l][d] (2 * positives - D). */
int fqt_pack_weight_signs(const fqt_layer_desc *desc, const void *W, int8_t *dst,
                          int32_t *linesum, void *hip_stream);

/* Activation-gradient product with PSQ codes (Section 5.3, SCQ; Appendix C Alg. 1, and
 * the Folder for convolutions):
 *   I[n][c][h][w] = sum over kernel taps (i, j) that map an output pixel (ho, wo) onto
 *                   (h, w) of sum_d q_psq[n][d][ho][wo] * s_W[d][c][i][j];
 *   c[c][h][w]    = sum over the same taps of sum_d s_W[d][c][i][j];
 *   dX            = S_n * I + Z'_n * c in float32 (rounded to bf16 if dx_dtype is bf16)
 *                   for kept samples, 0 for pruned samples.
 * This is the unfolded product followed by the folder, taken in integers, on int8 MFMA
 * from q->psq_codes.  wsign, wsign_linesum: the outputs of fqt_pack_weight_signs for the
 * layer's W.  kh*kw <= 64.  dX: [N][C][H][W] of dx_dtype.  I_out (optional):
 * int32 [N][C][H][W]. */
int fqt_binary_gemm_dx(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg,
                       const fqt_qgrad *q, const int8_t *wsign, const int32_t *wsign_linesum,
                       void *dX, int32_t *I_out, void *hip_stream);

/* Both products of the layer backward from one quantized gradient (Section 5.3, SCQ;
 * Appendix C Alg. 1 binary products, dequantization and Folder): the dW of
 * fqt_binary_gemm_dw and the dX of fqt_binary_gemm_dx, computed in one launch whose dW and
 * dX workgroups run side by side (the form fqt_layer_backward uses).  Arguments as in those
 * two calls: q from fqt_agp_scq_quantize, xsign from fqt_pack_input_signs, wsign and
 * wsign_linesum from fqt_pack_weight_signs; ws >= fqt_workspace_size(FQT_WS_GEMM_DW), 256-byte
 * aligned, no initialisation.  Layers whose dW contraction needs split partials over many
 * rows add a second launch that sums them. */
int fqt_binary_products(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, const fqt_qgrad *q,
                        const uint64_t *xsign, const int8_t *wsign, const int32_t *wsign_linesum,
                        void *dX, float *dW, void *ws, size_t ws_bytes, void *hip_stream);

/* Whole layer backward (Appendix C Alg. 1 backward; Section 5.3's final form):
 * quantize dY, pack sign(X) (im2col for conv), expand sign(W) to bytes, then both
 * products.
 * X: x_dtype, W: w_dtype, dY: dy_dtype, dX: dx_dtype, dW: float32.
 * ws: >= fqt_workspace_size(FQT_WS_LAYER) bytes, 256-byte aligned. */
int fqt_layer_backward(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, const void *X,
                       const void *W, const void *dY, void *dX, float *dW, void *ws,
                       size_t ws_bytes, void *hip_stream);

/* fqt_layer_backward for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same computation and
 * results, with the library's own workspace, a static device array of
 * FQT_NOALLOC_SCRATCH_BYTES that every GPU the library runs on holds until the process
 * ends.  The call allocates and frees nothing.  Layers whose FQT_WS_LAYER workspace exceeds
 * that size return FQT_E_WORKSPACE before any launch (at 64 MiB: the 256 -> 256 3x3 conv on
 * 8x8 maps at batch 128, every ResNet-18 layer at batch 128, VGG-16 conv11-13 and fc7/fc8 at
 * batch 64 fit; VGG-16 conv1-10 and fc6 at batch 64 do not).  Each call first clears the
 * array's state bytes with a fill kernel on hip_stream.  All calls on one GPU share its
 * array: calls that overlap on one GPU (other streams, other host threads) race and give
 * wrong results; serialise them.  Other arguments, layouts and errors as in
 * fqt_layer_backward; FQT_E_HIP if the array's device address cannot be obtained. */
#define FQT_NOALLOC_SCRATCH_BYTES (64u << 20)
int fqt_layer_backward_noalloc(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg,
                               const void *X, const void *W, const void *dY, void *dX, float *dW,
                               void *hip_stream);

/* Binary layer forward (Section 5.1: the output is sign(H_prev) times sign(Theta), scaled
 * per output channel by the learnable Gamma; Appendix C, Alg. 1 forward, with the Unfolder
 * for convolutions):
 *   I[n][d][ho][wo] = sum over (c, i, j) of sign(X)[n][c][ho*sh - ph + i][wo*sw - pw + j]
 *                     * sign(W)[d][c][i][j],   sign(x) = -1 for x <= 0 (NaN too), +1 else,
 *   Y = gamma[d] * I (one float32 rounding; bf16 Y rounds that to nearest even).
 * Padded positions of X count as sign -1 (the unfold is zero-padded, then binarized).
 * X: x_dtype [N][C][H][W] (linear [N][C]); W: w_dtype [D][C][kh][kw] ([D][C]); gamma:
 * float32 [D]; Y: dy_dtype, the layout of dY ([N][D][Ho][Wo], linear [N][D]); I_out
 * (optional, NULL to skip): int32 in Y's layout.  ws: >= fqt_workspace_size(FQT_WS_FORWARD)
 * bytes, 256-byte aligned, no initialisation needed (it holds the packed operands:
 * sign(X_u) bits and sign(W) bytes).  All pointers are device pointers; stream-ordered on
 * hip_stream; returns FQT_E_SHAPE when an operand exceeds 2 GiB. */
int fqt_binary_forward(const fqt_layer_desc *desc, const void *X, const void *W,
                       const float *gamma, void *Y, int32_t *I_out, void *ws, size_t ws_bytes,
                       void *hip_stream);

/* Static description of a status code. */
const char *fqt_status_string(int status);

#ifdef __cplusplus
}
#endif
#endif /* FQT_H */
