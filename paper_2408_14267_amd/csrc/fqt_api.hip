// C ABI of libfqt: argument validation, workspace carving and the entry points.
// Every check runs on the host before anything is launched.
#include <mutex>

#include "fqt_internal.hpp"

namespace fqt {

namespace {
constexpr int64_t LIMIT31 = (int64_t(1) << 31) - 1;

bool dtype_ok(int t) { return t == FQT_F32 || t == FQT_BF16; }
size_t dtype_size(int t) { return t == FQT_BF16 ? 2 : 4; }

// Sub-allocator over a caller-provided workspace: 256-byte aligned slices.
struct Carver {
  char *base;
  size_t off = 0;
  template <typename T>
  T *take(size_t count) {
    T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
    off += align256(count * sizeof(T));
    return p;
  }
};

struct LayerWs {
  QuantWs qws;
  fqt_qgrad q;
  uint64_t *xsign;
  int8_t *wsb;
  int32_t *wlsum;
  void *dw_ws;
};

void carve_quant_ws(Carver *c, const Layer &L, QuantWs *q) {
  static_assert(MKEY_SLOTS * sizeof(uint2) == FQT_WS_STATE_BYTES, "state bytes");
  q->mkeys = c->take<uint2>(MKEY_SLOTS);            // first: a fixed place in every layout
  q->part_c = c->take<int2>(size_t(L.D) * stats_row_blocks(L));
  q->part_s = c->take<int2>(size_t(L.Wd) * L.Wr * stats_slots(L));
  q->skey = c->take<int2>(L.N);
  q->ckey = c->take<int2>(L.D);
  q->sp = c->take<GroupParam>(L.N);
  q->cp = c->take<GroupParam>(L.D);
  q->sslot = c->take<float2>(L.N);
  q->cslot = c->take<float2>(L.D);
}

size_t carve_layer_ws(void *ws, const Layer &L, const fqt_quant_cfg &cfg, LayerWs *out) {
  const int bits = cfg.bits;
  Carver c{static_cast<char *>(ws)};
  LayerWs w{};
  carve_quant_ws(&c, L, &w.qws);
  w.q.psq_planes = c.take<uint64_t>(size_t(bits) * L.R * L.Wd);
  w.q.pcq_planes = c.take<uint64_t>(size_t(bits) * L.D * L.Wr);
  w.q.psq_codes = c.take<uint8_t>(size_t(L.R) * L.Wd * 64);
  w.q.pcq_codes = c.take<uint8_t>(size_t(L.D) * L.Wr * 64);
  w.q.psq_kept = c.take<int32_t>(L.N);
  w.q.psq_count = c.take<int32_t>(1);
  w.q.pcq_kept = c.take<int32_t>(L.D);
  w.q.pcq_count = c.take<int32_t>(1);
  w.q.psq_scale = c.take<float>(L.N);
  w.q.psq_offset = c.take<float>(L.N);
  w.q.psq_prob = c.take<float>(L.N);
  w.q.pcq_scale = c.take<float>(L.D);
  w.q.pcq_offset = c.take<float>(L.D);
  w.q.pcq_prob = c.take<float>(L.D);
  w.xsign = c.take<uint64_t>(size_t(L.K) * L.Wr);
  w.wsb = c.take<int8_t>(size_t(L.K) * L.Wd * 64);
  w.wlsum = c.take<int32_t>(L.K);
  w.dw_ws = c.take<char>(gemm_dw_ws_bytes(L, cfg));
  if (out) *out = w;
  return c.off;
}

// Forward workspace: sign(X_u) word-major [Wr][K], the same bits k-block-major [Kw][Wr*64]
// and sign(W) as +-1 bytes [Dp][Kp] (Dp, Kp: D and K rounded up to 64).
struct ForwardWs {
  uint64_t *xwm, *xrows;
  int8_t *wrows;
  int64_t Dp, Kp;
};
size_t carve_forward_ws(void *ws, const Layer &L, ForwardWs *out) {
  Carver c{static_cast<char *>(ws)};
  ForwardWs f;
  f.Dp = (L.D + 63) / 64 * 64;
  f.Kp = (L.K + 63) / 64 * 64;
  f.xwm = c.take<uint64_t>(size_t(L.Wr) * L.K);
  f.xrows = c.take<uint64_t>(size_t(f.Kp / 64) * L.Wr * 64);
  f.wrows = c.take<int8_t>(size_t(f.Dp) * f.Kp);
  if (out) *out = f;
  return c.off;
}

int check_qgrad(const fqt_qgrad *q, bool psq, bool pcq) {
  if (!q) return FQT_E_NULL;
  if (psq) {
    if (!q->psq_planes || !q->psq_codes || !q->psq_kept || !q->psq_count || !q->psq_scale ||
        !q->psq_offset || !q->psq_prob)
      return FQT_E_NULL;
    if (!aligned(q->psq_planes, 8) || !aligned(q->psq_codes, 16) || !aligned(q->psq_kept, 4) ||
        !aligned(q->psq_count, 4) ||
        !aligned(q->psq_scale, 4) || !aligned(q->psq_offset, 4) || !aligned(q->psq_prob, 4))
      return FQT_E_ALIGN;
  }
  if (pcq) {
    if (!q->pcq_planes || !q->pcq_codes || !q->pcq_kept || !q->pcq_count || !q->pcq_scale ||
        !q->pcq_offset || !q->pcq_prob)
      return FQT_E_NULL;
    if (!aligned(q->pcq_planes, 8) || !aligned(q->pcq_codes, 16) || !aligned(q->pcq_kept, 4) ||
        !aligned(q->pcq_count, 4) ||
        !aligned(q->pcq_scale, 4) || !aligned(q->pcq_offset, 4) || !aligned(q->pcq_prob, 4))
      return FQT_E_ALIGN;
  }
  return FQT_OK;
}

#define FQT_TRY(expr)              \
  do {                             \
    const int st__ = (expr);       \
    if (st__ != FQT_OK) return st__; \
  } while (0)

}  // namespace

int make_layer(const fqt_layer_desc *d, Layer *L) {
  if (!d) return FQT_E_NULL;
  if (d->kind != FQT_LINEAR && d->kind != FQT_CONV2D) return FQT_E_INVAL;
  if (!dtype_ok(d->dy_dtype) || !dtype_ok(d->x_dtype) || !dtype_ok(d->w_dtype) ||
      !dtype_ok(d->dx_dtype))
    return FQT_E_DTYPE;
  if (d->N <= 0 || d->C <= 0 || d->H <= 0 || d->W <= 0 || d->D <= 0) return FQT_E_SHAPE;
  if (d->kh <= 0 || d->kw <= 0 || d->sh <= 0 || d->sw <= 0 || d->ph < 0 || d->pw < 0)
    return FQT_E_SHAPE;
  if (d->kind == FQT_LINEAR &&
      (d->H != 1 || d->W != 1 || d->kh != 1 || d->kw != 1 || d->sh != 1 || d->sw != 1 ||
       d->ph != 0 || d->pw != 0))
    return FQT_E_SHAPE;
  if (d->H + 2 * int64_t(d->ph) < d->kh || d->W + 2 * int64_t(d->pw) < d->kw) return FQT_E_SHAPE;
  if (d->N > FQT_MAX_AGP_GROUPS || d->D > FQT_MAX_AGP_GROUPS) return FQT_E_SHAPE;
  Layer l;
  l.kind = d->kind;
  l.dy_t = d->dy_dtype; l.x_t = d->x_dtype; l.w_t = d->w_dtype; l.dx_t = d->dx_dtype;
  l.N = d->N; l.C = d->C; l.H = d->H; l.W = d->W; l.D = d->D;
  l.kh = d->kh; l.kw = d->kw; l.sh = d->sh; l.sw = d->sw; l.ph = d->ph; l.pw = d->pw;
  l.Ho = (l.H + 2 * l.ph - l.kh) / l.sh + 1;
  l.Wo = (l.W + 2 * l.pw - l.kw) / l.sw + 1;
  if (l.C > LIMIT31 || l.H > LIMIT31 || l.W > LIMIT31) return FQT_E_SHAPE;
  l.P = l.Ho * l.Wo;
  l.HW = l.H * l.W;
  l.K = l.C * l.kh * l.kw;
  if (l.P > LIMIT31 || l.HW > LIMIT31 || l.K > LIMIT31) return FQT_E_SHAPE;
  l.R = l.N * l.P;
  if (l.R > LIMIT31 || l.N * l.C > LIMIT31 / l.HW || l.N * l.D > LIMIT31 / l.P) return FQT_E_SHAPE;
  if (l.D * l.K > LIMIT31) return FQT_E_SHAPE;
  l.Wd = (l.D + 63) / 64;
  l.Wr = (l.R + 63) / 64;
  // Byte sizes of the code arrays and of the weight-sign bytes: the products address
  // them with 32-bit buffer offsets.
  if (l.R * l.Wd * 64 > LIMIT31 || l.D * l.Wr * 64 > LIMIT31 || l.K * l.Wd * 64 > LIMIT31 ||
      l.K * l.Wr * 8 > LIMIT31)
    return FQT_E_SHAPE;
  *L = l;
  return FQT_OK;
}

int check_cfg(const fqt_quant_cfg *c, const Layer &) {
  if (!c) return FQT_E_NULL;
  if (c->bits < 1 || c->bits > FQT_MAX_BITS) return FQT_E_INVAL;
  if (c->agp_mode != FQT_AGP_BERNOULLI && c->agp_mode != FQT_AGP_TOPK &&
      c->agp_mode != FQT_AGP_OFF)
    return FQT_E_INVAL;
  return FQT_OK;
}

// The dW product keeps I = sum_r q s in int32 (MFMA accumulators, code sums, the b = 8
// bias term): |I| <= (2^b - 1) * N*Ho*Wo must stay below 2^31.
int check_dw_range(const Layer &L, const fqt_quant_cfg &c) {
  return int64_t((1 << c.bits) - 1) * L.R > LIMIT31 ? FQT_E_SHAPE : FQT_OK;
}

size_t quant_ws_bytes(const Layer &L) {
  Carver c{nullptr};
  QuantWs q;
  carve_quant_ws(&c, L, &q);
  return c.off;
}

void carve_quant_ws(void *ws, const Layer &L, QuantWs *q) {
  Carver c{static_cast<char *>(ws)};
  carve_quant_ws(&c, L, q);
}

namespace {

int layer_backward_run(const Layer &L, const fqt_quant_cfg &cfg, const void *X, const void *W,
                       const void *dY, void *dX, float *dW, void *ws, hipStream_t s);

// Validation shared by the layer backward entry points (everything but the workspace).
int check_layer_backward(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, const void *X,
                         const void *W, const void *dY, const void *dX, const float *dW,
                         Layer *L) {
  FQT_TRY(make_layer(desc, L));
  FQT_TRY(check_cfg(cfg, *L));
  FQT_TRY(check_dw_range(*L, *cfg));
  if (!X || !W || !dY || !dX || !dW) return FQT_E_NULL;
  if (!aligned(dY, 16) || !aligned(X, dtype_size(L->x_t)) || !aligned(W, dtype_size(L->w_t)) ||
      !aligned(dX, dtype_size(L->dx_t)) || !aligned(dW, 4))
    return FQT_E_ALIGN;
  if (L->kh * L->kw > 64) return FQT_E_SHAPE;
  return FQT_OK;
}

// The workspace of fqt_layer_backward_noalloc: one array per GPU, held until the process
// ends.  In host code `scratch` names a host-side stand-in, not device memory: its device
// address comes from hipGetSymbolAddress, once per device with that device current, and
// only that address is ever handed to a kernel.
static __device__ __align__(256) unsigned char scratch[FQT_NOALLOC_SCRATCH_BYTES];

constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex scratch_mutex;
void *scratch_ptr[SCRATCH_MAX_DEVICES] = {};

int scratch_of_current_device(void **out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return FQT_E_HIP;
  if (dev < 0 || dev >= SCRATCH_MAX_DEVICES) return FQT_E_HIP;
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (!scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FQT_E_HIP;
    scratch_ptr[dev] = p;
  }
  *out = scratch_ptr[dev];
  return FQT_OK;
}

}  // namespace

}  // namespace fqt

using namespace fqt;

extern "C" {

const char *fqt_status_string(int status) {
  switch (status) {
    case FQT_OK: return "FQT_OK: success";
    case FQT_E_INVAL: return "FQT_E_INVAL: scalar argument out of range";
    case FQT_E_DTYPE: return "FQT_E_DTYPE: unsupported dtype or dtype combination";
    case FQT_E_SHAPE: return "FQT_E_SHAPE: invalid or unsupported shape";
    case FQT_E_WORKSPACE: return "FQT_E_WORKSPACE: workspace too small";
    case FQT_E_ALIGN: return "FQT_E_ALIGN: pointer misaligned";
    case FQT_E_NULL: return "FQT_E_NULL: required pointer is NULL";
    case FQT_E_HIP: return "FQT_E_HIP: HIP runtime or launch failure";
    default: return "unknown fqt status";
  }
}

int fqt_qgrad_words(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, int64_t *psq_words,
                    int64_t *pcq_words, int64_t *psq_code_bytes, int64_t *pcq_code_bytes) {
  Layer L;
  FQT_TRY(make_layer(desc, &L));
  FQT_TRY(check_cfg(cfg, L));
  if (!psq_words || !pcq_words || !psq_code_bytes || !pcq_code_bytes) return FQT_E_NULL;
  *psq_words = int64_t(cfg->bits) * L.R * L.Wd;
  *pcq_words = int64_t(cfg->bits) * L.D * L.Wr;
  *psq_code_bytes = L.R * L.Wd * 64;
  *pcq_code_bytes = L.D * L.Wr * 64;
  return FQT_OK;
}

int fqt_workspace_size(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, int32_t which,
                       size_t *bytes) {
  Layer L;
  FQT_TRY(make_layer(desc, &L));
  if (!bytes) return FQT_E_NULL;
  if (which == FQT_WS_FORWARD) {          // the forward takes no quantizer configuration
    *bytes = carve_forward_ws(nullptr, L, nullptr);
    return FQT_OK;
  }
  FQT_TRY(check_cfg(cfg, L));
  if (which == FQT_WS_QUANTIZE) *bytes = quant_ws_bytes(L);
  else if (which == FQT_WS_LAYER) *bytes = carve_layer_ws(nullptr, L, *cfg, nullptr);
  else if (which == FQT_WS_GEMM_DW) *bytes = gemm_dw_ws_bytes(L, *cfg);
  else if (which == FQT_WS_DW_POPCOUNT) *bytes = engine_ws_bytes(L, *cfg, FQT_ENGINE_POPCOUNT);
  else if (which == FQT_WS_DW_FP4) *bytes = engine_ws_bytes(L, *cfg, FQT_ENGINE_FP4);
  else return FQT_E_INVAL;
  return FQT_OK;
}

int fqt_workspace_init(void *ws, size_t ws_bytes, void *hip_stream) {
  if (!ws) return FQT_E_NULL;
  if (!aligned(ws, 256)) return FQT_E_ALIGN;
  if (ws_bytes < FQT_WS_STATE_BYTES) return FQT_E_WORKSPACE;
  return launch_state_clear(ws, static_cast<hipStream_t>(hip_stream));
}

int fqt_agp_scq_quantize(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, const void *dY,
                         const fqt_qgrad *out, void *ws, size_t ws_bytes, void *hip_stream) {
  Layer L;
  FQT_TRY(make_layer(desc, &L));
  FQT_TRY(check_cfg(cfg, L));
  FQT_TRY(check_qgrad(out, true, true));
  if (!dY || !ws) return FQT_E_NULL;
  if (!aligned(dY, 16) || !aligned(ws, 256)) return FQT_E_ALIGN;
  if (ws_bytes < quant_ws_bytes(L)) return FQT_E_WORKSPACE;
  QuantWs q;
  carve_quant_ws(ws, L, &q);
  return launch_quantize(L, *cfg, dY, *out, q, static_cast<hipStream_t>(hip_stream));
}

int fqt_pack_bits(const void *src, int32_t dtype, int64_t rows, int64_t cols, int64_t ld,
                  int32_t axis, const fqt_layer_desc *conv, uint64_t *dst, int32_t *linesum,
                  void *hip_stream) {
  if (!src || !dst) return FQT_E_NULL;
  if (!dtype_ok(dtype)) return FQT_E_DTYPE;
  if (!aligned(src, dtype_size(dtype)) || !aligned(dst, 8) || (linesum && !aligned(linesum, 4)))
    return FQT_E_ALIGN;
  const hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (axis == FQT_PACK_IM2COL) {
    if (!conv) return FQT_E_NULL;
    Layer L;
    FQT_TRY(make_layer(conv, &L));
    if (int64_t(L.K) * L.Wr > LIMIT31 * 4) return FQT_E_SHAPE;
    return launch_pack_bits(src, dtype, 0, 0, 0, axis, &L, dst, linesum, s);
  }
  if (axis != FQT_PACK_ALONG_ROWS && axis != FQT_PACK_ALONG_COLS) return FQT_E_INVAL;
  if (conv) return FQT_E_INVAL;
  if (rows <= 0 || cols <= 0 || ld < cols) return FQT_E_SHAPE;
  if (axis == FQT_PACK_ALONG_ROWS && ((rows + 63) / 64 > 65535 || (cols + 63) / 64 > LIMIT31))
    return FQT_E_SHAPE;
  if (axis == FQT_PACK_ALONG_COLS && rows * ((cols + 63) / 64) > LIMIT31 * 4) return FQT_E_SHAPE;
  if (rows > LIMIT31 || cols > LIMIT31) return FQT_E_SHAPE;
  return launch_pack_bits(src, dtype, rows, cols, ld, axis, nullptr, dst, linesum, s);
}

int fqt_binary_gemm_dw(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, const fqt_qgrad *q,
                       const uint64_t *xsign, float *dW, int32_t *I_out, void *ws,
                       size_t ws_bytes, void *hip_stream) {
  Layer L;
  FQT_TRY(make_layer(desc, &L));
  FQT_TRY(check_cfg(cfg, L));
  FQT_TRY(check_qgrad(q, false, true));
  FQT_TRY(check_dw_range(L, *cfg));
  if (!xsign || !dW || !ws) return FQT_E_NULL;
  if (!aligned(xsign, 8) || !aligned(dW, 4) || (I_out && !aligned(I_out, 4)) ||
      !aligned(ws, 256))
    return FQT_E_ALIGN;
  if (ws_bytes < gemm_dw_ws_bytes(L, *cfg)) return FQT_E_WORKSPACE;
  return launch_gemm_dw(L, *cfg, *q, xsign, dW, I_out, ws, static_cast<hipStream_t>(hip_stream));
}

int fqt_binary_gemm_dw_planes(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg,
                              const fqt_qgrad *q, const uint64_t *xbits,
                              const int32_t *xbits_linesum, float *dW, int32_t *I_out,
                              int32_t engine, void *ws, size_t ws_bytes, void *hip_stream) {
  Layer L;
  FQT_TRY(make_layer(desc, &L));
  FQT_TRY(check_cfg(cfg, L));
  FQT_TRY(check_qgrad(q, false, true));
  FQT_TRY(check_dw_range(L, *cfg));
  FQT_TRY(check_engine(L, *cfg, engine));
  if (!xbits || !xbits_linesum || !dW || !ws) return FQT_E_NULL;
  if (!aligned(xbits, 8) || !aligned(xbits_linesum, 4) || !aligned(dW, 4) ||
      (I_out && !aligned(I_out, 4)) || !aligned(ws, 256))
    return FQT_E_ALIGN;
  if (ws_bytes < engine_ws_bytes(L, *cfg, engine)) return FQT_E_WORKSPACE;
  return launch_gemm_dw_planes(L, *cfg, *q, xbits, xbits_linesum, dW, I_out, engine, ws,
                               static_cast<hipStream_t>(hip_stream));
}

int fqt_pack_input_signs(const fqt_layer_desc *desc, const void *X, uint64_t *dst,
                         void *hip_stream) {
  Layer L;
  FQT_TRY(make_layer(desc, &L));
  if (!X || !dst) return FQT_E_NULL;
  if (!aligned(X, dtype_size(L.x_t)) || !aligned(dst, 8)) return FQT_E_ALIGN;
  const hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (L.kind == FQT_LINEAR)
    return launch_pack_bits(X, L.x_t, L.N, L.C, L.C, FQT_PACK_ALONG_ROWS, nullptr, dst, nullptr,
                            s, true);
  return launch_pack_bits(X, L.x_t, 0, 0, 0, FQT_PACK_IM2COL, &L, dst, nullptr, s, true);
}

int fqt_pack_weight_signs(const fqt_layer_desc *desc, const void *W, int8_t *dst,
                          int32_t *linesum, void *hip_stream) {
  Layer L;
  FQT_TRY(make_layer(desc, &L));
  if (!W || !dst || !linesum) return FQT_E_NULL;
  if (!aligned(W, dtype_size(L.w_t)) || !aligned(dst, 16) || !aligned(linesum, 4))
    return FQT_E_ALIGN;
  return launch_pack_w_i8(W, L, dst, linesum, static_cast<hipStream_t>(hip_stream));
}

int fqt_binary_gemm_dx(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, const fqt_qgrad *q,
                       const int8_t *wsign, const int32_t *wsign_linesum, void *dX,
                       int32_t *I_out, void *hip_stream) {
  Layer L;
  FQT_TRY(make_layer(desc, &L));
  FQT_TRY(check_cfg(cfg, L));
  FQT_TRY(check_qgrad(q, true, false));
  if (!wsign || !wsign_linesum || !dX) return FQT_E_NULL;
  if (!aligned(wsign, 16) || !aligned(wsign_linesum, 4) || !aligned(dX, dtype_size(L.dx_t)) ||
      (I_out && !aligned(I_out, 4)))
    return FQT_E_ALIGN;
  if (L.kh * L.kw > 64) return FQT_E_SHAPE;
  return launch_gemm_dx(L, *cfg, *q, wsign, wsign_linesum, dX, I_out,
                        static_cast<hipStream_t>(hip_stream));
}

int fqt_binary_products(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, const fqt_qgrad *q,
                        const uint64_t *xsign, const int8_t *wsign, const int32_t *wsign_linesum,
                        void *dX, float *dW, void *ws, size_t ws_bytes, void *hip_stream) {
  Layer L;
  FQT_TRY(make_layer(desc, &L));
  FQT_TRY(check_cfg(cfg, L));
  FQT_TRY(check_qgrad(q, true, true));
  FQT_TRY(check_dw_range(L, *cfg));
  if (!xsign || !wsign || !wsign_linesum || !dX || !dW || !ws) return FQT_E_NULL;
  if (!aligned(xsign, 8) || !aligned(wsign, 16) || !aligned(wsign_linesum, 4) ||
      !aligned(dX, dtype_size(L.dx_t)) || !aligned(dW, 4) || !aligned(ws, 256))
    return FQT_E_ALIGN;
  if (L.kh * L.kw > 64) return FQT_E_SHAPE;
  if (ws_bytes < gemm_dw_ws_bytes(L, *cfg)) return FQT_E_WORKSPACE;
  return launch_products(L, *cfg, *q, xsign, wsign, wsign_linesum, dX, dW, ws, nullptr, nullptr,
                         static_cast<hipStream_t>(hip_stream));
}

int fqt_layer_backward(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg, const void *X,
                       const void *W, const void *dY, void *dX, float *dW, void *ws,
                       size_t ws_bytes, void *hip_stream) {
  Layer L;
  FQT_TRY(check_layer_backward(desc, cfg, X, W, dY, dX, dW, &L));
  if (!ws) return FQT_E_NULL;
  if (!aligned(ws, 256)) return FQT_E_ALIGN;
  if (ws_bytes < carve_layer_ws(nullptr, L, *cfg, nullptr)) return FQT_E_WORKSPACE;
  return layer_backward_run(L, *cfg, X, W, dY, dX, dW, ws, static_cast<hipStream_t>(hip_stream));
}

int fqt_layer_backward_noalloc(const fqt_layer_desc *desc, const fqt_quant_cfg *cfg,
                               const void *X, const void *W, const void *dY, void *dX, float *dW,
                               void *hip_stream) {
  Layer L;
  FQT_TRY(check_layer_backward(desc, cfg, X, W, dY, dX, dW, &L));
  if (carve_layer_ws(nullptr, L, *cfg, nullptr) > FQT_NOALLOC_SCRATCH_BYTES)
    return FQT_E_WORKSPACE;
  void *ws = nullptr;
  FQT_TRY(scratch_of_current_device(&ws));
  const hipStream_t s = static_cast<hipStream_t>(hip_stream);
  // The array keeps whatever the last call on this GPU left in it: clear the state bytes
  // (the merged group keys) before the statistics combine into them.
  FQT_TRY(launch_state_clear(ws, s));
  return layer_backward_run(L, *cfg, X, W, dY, dX, dW, ws, s);
}

}  // extern "C"

namespace fqt {
namespace {
int layer_backward_run(const Layer &L, const fqt_quant_cfg &cfg_, const void *X, const void *W,
                       const void *dY, void *dX, float *dW, void *ws, hipStream_t s) {
  const fqt_quant_cfg *cfg = &cfg_;
  LayerWs w;
  carve_layer_ws(ws, L, *cfg, &w);
  // Statistics, then the selection (whose launch also packs the sign operands when the
  // layer allows), the quantizer, both products.
  SignJob sj{X, W, w.xsign, w.wsb, w.wlsum, false};
  // The products read the byte codes; the bit planes (the paper's packed form) are left to
  // fqt_agp_scq_quantize callers.
  FQT_TRY(launch_quantize(L, *cfg, dY, w.q, w.qws, s, &sj, false));
  if (!sj.done) {
    if (L.kind == FQT_LINEAR)
      FQT_TRY(launch_pack_bits(X, L.x_t, L.N, L.C, L.C, FQT_PACK_ALONG_ROWS, nullptr, w.xsign,
                               nullptr, s, true));
    else
      FQT_TRY(launch_pack_bits(X, L.x_t, 0, 0, 0, FQT_PACK_IM2COL, &L, w.xsign, nullptr, s,
                               true));
    FQT_TRY(launch_pack_w_i8(W, L, w.wsb, w.wlsum, s));
  }
  return launch_products(L, *cfg, w.q, w.xsign, w.wsb, w.wlsum, dX, dW, w.dw_ws, w.qws.sslot,
                         w.qws.cslot, s);
}
}  // namespace
}  // namespace fqt

extern "C" {

int fqt_binary_forward(const fqt_layer_desc *desc, const void *X, const void *W,
                       const float *gamma, void *Y, int32_t *I_out, void *ws, size_t ws_bytes,
                       void *hip_stream) {
  Layer L;
  FQT_TRY(make_layer(desc, &L));
  if (!X || !W || !gamma || !Y || !ws) return FQT_E_NULL;
  if (!aligned(X, dtype_size(L.x_t)) || !aligned(W, dtype_size(L.w_t)) || !aligned(gamma, 4) ||
      !aligned(Y, dtype_size(L.dy_t)) || (I_out && !aligned(I_out, 4)) || !aligned(ws, 256))
    return FQT_E_ALIGN;
  ForwardWs f;
  const size_t need = carve_forward_ws(ws, L, &f);
  if (ws_bytes < need) return FQT_E_WORKSPACE;
  // Byte offsets the kernels form stay below 2^31.
  if (f.Dp * f.Kp > LIMIT31 || (f.Kp / 64) * L.Wr * 64 * 8 > LIMIT31 ||
      int64_t(L.N) * L.D * L.P > LIMIT31)
    return FQT_E_SHAPE;
  const hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (L.kind == FQT_LINEAR)
    FQT_TRY(launch_pack_bits(X, L.x_t, L.N, L.C, L.C, FQT_PACK_ALONG_ROWS, nullptr, f.xwm,
                             nullptr, s, true));
  else
    FQT_TRY(launch_pack_bits(X, L.x_t, 0, 0, 0, FQT_PACK_IM2COL, &L, f.xwm, nullptr, s, true));
  FQT_TRY(launch_transpose_bits(f.xwm, L.Wr, L.K, f.xrows, s));
  FQT_TRY(launch_pack_w_rows(W, L, f.Dp, f.Kp, f.wrows, s));
  return launch_forward_gemm(L, f.wrows, f.Dp, f.Kp, f.xrows, gamma, Y, I_out, s);
}

}  // extern "C"
