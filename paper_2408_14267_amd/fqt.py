"""ctypes binding of libfqt (the C ABI declared in include/fqt.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels of libfqt.so.  Functions keep the C names; tensors are torch tensors
on the current HIP device (their data pointers are passed through) and
`stream` defaults to torch's current stream.  A non-zero status raises
FqtError.  Importing this module raises if libfqt.so has not been built --
there is no fallback path.
"""
import ctypes
import os
from ctypes import POINTER, Structure, c_char_p, c_int, c_int32, c_int64, c_size_t, c_uint32, c_uint64, c_void_p

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfqt.so")

FQT_OK = 0
FQT_E_INVAL, FQT_E_DTYPE, FQT_E_SHAPE, FQT_E_WORKSPACE, FQT_E_ALIGN, FQT_E_NULL, FQT_E_HIP = range(-1, -8, -1)
FQT_F32, FQT_BF16 = 0, 1
FQT_LINEAR, FQT_CONV2D = 0, 1
FQT_AGP_BERNOULLI, FQT_AGP_TOPK, FQT_AGP_OFF = 0, 1, 2
FQT_PACK_ALONG_ROWS, FQT_PACK_ALONG_COLS, FQT_PACK_IM2COL = 0, 1, 2
FQT_WS_QUANTIZE, FQT_WS_LAYER, FQT_WS_GEMM_DW, FQT_WS_FORWARD = 0, 1, 2, 3
FQT_WS_DW_POPCOUNT, FQT_WS_DW_FP4 = 4, 5
FQT_ENGINE_POPCOUNT, FQT_ENGINE_FP4 = 1, 2
FQT_WS_STATE_BYTES = 131072    # zeroed state at the start of quantize and layer workspaces
FQT_MAX_BITS = 8
FQT_NOALLOC_SCRATCH_BYTES = 64 << 20   # static workspace of fqt_layer_backward_noalloc
FQT_MAX_AGP_GROUPS = 16384
EXPORTED = ("fqt_status_string", "fqt_qgrad_words", "fqt_workspace_size", "fqt_agp_scq_quantize",
            "fqt_pack_bits", "fqt_pack_input_signs", "fqt_binary_gemm_dw", "fqt_pack_weight_signs",
            "fqt_binary_gemm_dx",
            "fqt_layer_backward", "fqt_binary_forward", "fqt_workspace_init",
            "fqt_layer_backward_noalloc", "fqt_binary_products", "fqt_binary_gemm_dw_planes")


class FqtError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {fqt_status_string(status)} ({status})")


class fqt_layer_desc(Structure):
    _fields_ = [("kind", c_int32), ("dy_dtype", c_int32), ("x_dtype", c_int32),
                ("w_dtype", c_int32), ("dx_dtype", c_int32),
                ("N", c_int64), ("C", c_int64), ("H", c_int64), ("W", c_int64), ("D", c_int64),
                ("kh", c_int32), ("kw", c_int32), ("sh", c_int32), ("sw", c_int32),
                ("ph", c_int32), ("pw", c_int32)]


class fqt_quant_cfg(Structure):
    _fields_ = [("bits", c_int32), ("agp_mode", c_int32), ("seed", c_uint64),
                ("step", c_uint32), ("layer_id", c_uint32)]


class fqt_qgrad(Structure):
    _fields_ = [("psq_planes", c_void_p), ("pcq_planes", c_void_p),
                ("psq_codes", c_void_p), ("pcq_codes", c_void_p),
                ("psq_kept", c_void_p), ("psq_count", c_void_p),
                ("pcq_kept", c_void_p), ("pcq_count", c_void_p),
                ("psq_scale", c_void_p), ("psq_offset", c_void_p), ("psq_prob", c_void_p),
                ("pcq_scale", c_void_p), ("pcq_offset", c_void_p), ("pcq_prob", c_void_p)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                           "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(LIB_PATH)
    D, Q, G = POINTER(fqt_layer_desc), POINTER(fqt_quant_cfg), POINTER(fqt_qgrad)
    sig = {
        "fqt_status_string": (c_char_p, [c_int]),
        "fqt_qgrad_words": (c_int, [D, Q, POINTER(c_int64), POINTER(c_int64), POINTER(c_int64),
                                    POINTER(c_int64)]),
        "fqt_workspace_size": (c_int, [D, Q, c_int32, POINTER(c_size_t)]),
        "fqt_workspace_init": (c_int, [c_void_p, c_size_t, c_void_p]),
        "fqt_agp_scq_quantize": (c_int, [D, Q, c_void_p, G, c_void_p, c_size_t, c_void_p]),
        "fqt_pack_bits": (c_int, [c_void_p, c_int32, c_int64, c_int64, c_int64, c_int32, D,
                                  c_void_p, c_void_p, c_void_p]),
        "fqt_binary_gemm_dw": (c_int, [D, Q, G, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                       c_void_p]),
        "fqt_pack_input_signs": (c_int, [D, c_void_p, c_void_p, c_void_p]),
        "fqt_pack_weight_signs": (c_int, [D, c_void_p, c_void_p, c_void_p, c_void_p]),
        "fqt_binary_gemm_dx": (c_int, [D, Q, G, c_void_p, c_void_p, c_void_p, c_void_p,
                                       c_void_p]),
        "fqt_layer_backward": (c_int, [D, Q, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                       c_void_p, c_size_t, c_void_p]),
        "fqt_binary_gemm_dw_planes": (c_int, [D, Q, G, c_void_p, c_void_p, c_void_p, c_void_p,
                                              c_int32, c_void_p, c_size_t, c_void_p]),
        "fqt_binary_products": (c_int, [D, Q, G, c_void_p, c_void_p, c_void_p, c_void_p,
                                        c_void_p, c_void_p, c_size_t, c_void_p]),
        "fqt_layer_backward_noalloc": (c_int, [D, Q, c_void_p, c_void_p, c_void_p, c_void_p,
                                               c_void_p, c_void_p]),
        "fqt_binary_forward": (c_int, [D, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                       c_void_p, c_size_t, c_void_p]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


# ----------------------------------------------------------------------------- marshalling helpers

def _ptr(t):
    return None if t is None else c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(status, where):
    if status != FQT_OK:
        raise FqtError(status, where)


_TORCH_OF = {FQT_F32: torch.float32, FQT_BF16: torch.bfloat16}


def _sizes(desc):
    """Element counts of the layer's tensors and its packed-operand sizes: X, W, dY, the X
    sign words (Wr * K) and the weight sign bytes (K * 64 * Wd)."""
    if desc.kind == FQT_LINEAR:
        P, K = 1, desc.C
    else:
        Ho = (desc.H + 2 * desc.ph - desc.kh) // desc.sh + 1
        Wo = (desc.W + 2 * desc.pw - desc.kw) // desc.sw + 1
        P, K = Ho * Wo, desc.C * desc.kh * desc.kw
    HW = 1 if desc.kind == FQT_LINEAR else desc.H * desc.W
    R = desc.N * P
    return {"X": desc.N * desc.C * HW, "W": desc.D * K, "dY": R * desc.D,
            "xsign": (R + 63) // 64 * K, "wsign": K * 64 * ((desc.D + 63) // 64), "K": K}


def _need(where, *specs):
    """Raise before any launch when a tensor cannot hold what the descriptor describes (a
    kernel would read or write past it): specs are (tensor, dtype, elements, name[,
    optional]); every shape check runs before the device check."""
    for t, dtype, numel, name, *opt in specs:
        what = f"{where}: {name}"
        if t is None:
            if opt and opt[0]:
                continue
            raise ValueError(f"{what}: a tensor is required")
        if dtype is not None and t.dtype != dtype:
            raise ValueError(f"{what}: dtype {t.dtype} does not match the descriptor's {dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{what}: tensor must be contiguous")
        if t.numel() < numel:
            raise ValueError(f"{what}: {t.numel()} elements, the descriptor needs {numel}")
    for t, _, _, name, *opt in specs:
        if t is not None and not t.is_cuda:
            raise ValueError(f"{where}: {name}: expected a device tensor, got one on {t.device}")


def dtype_code(dt):
    if dt in (torch.float32, "f32"):
        return FQT_F32
    if dt in (torch.bfloat16, "bf16"):
        return FQT_BF16
    raise ValueError(f"unsupported dtype {dt}")


def layer_desc(shape, dy_dtype=FQT_F32, x_dtype=FQT_F32, w_dtype=FQT_F32, dx_dtype=FQT_F32):
    """fqt_layer_desc from an object with kind/N/C/H/W/D/kh/kw/sh/sw/ph/pw attributes."""
    return fqt_layer_desc(FQT_LINEAR if shape.kind == "linear" else FQT_CONV2D,
                          dy_dtype, x_dtype, w_dtype, dx_dtype,
                          shape.N, shape.C, shape.H, shape.W, shape.D,
                          shape.kh, shape.kw, shape.sh, shape.sw, shape.ph, shape.pw)


def quant_cfg(bits, agp_mode=FQT_AGP_BERNOULLI, seed=0, step=0, layer_id=0):
    return fqt_quant_cfg(bits, agp_mode, seed, step, layer_id)


# ----------------------------------------------------------------------------- C entry points

def fqt_status_string(status):
    return _lib.fqt_status_string(status).decode()


def fqt_qgrad_words(desc, cfg):
    """(psq plane words, pcq plane words, psq code bytes, pcq code bytes)."""
    v = [c_int64() for _ in range(4)]
    _check(_lib.fqt_qgrad_words(desc, cfg, *(ctypes.byref(x) for x in v)), "fqt_qgrad_words")
    return tuple(x.value for x in v)


def fqt_workspace_size(desc, cfg, which=FQT_WS_LAYER):
    n = c_size_t()
    _check(_lib.fqt_workspace_size(desc, cfg, which, ctypes.byref(n)), "fqt_workspace_size")
    return n.value


def fqt_workspace_init(ws, stream=None):
    _check(_lib.fqt_workspace_init(_ptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "fqt_workspace_init")


def fqt_agp_scq_quantize(desc, cfg, dY, qgrad, ws, stream=None):
    _need("fqt_agp_scq_quantize",
          (dY, _TORCH_OF.get(desc.dy_dtype), _sizes(desc)["dY"], "dY"))
    _check(_lib.fqt_agp_scq_quantize(desc, cfg, _ptr(dY), ctypes.byref(qgrad.struct), _ptr(ws),
                                     ws.numel() * ws.element_size(), _stream(stream)),
           "fqt_agp_scq_quantize")


def fqt_pack_bits(src, dtype, rows, cols, ld, axis, conv, dst, linesum=None, stream=None):
    _check(_lib.fqt_pack_bits(_ptr(src), dtype, rows, cols, ld, axis,
                              ctypes.byref(conv) if conv is not None else None,
                              _ptr(dst), _ptr(linesum), _stream(stream)), "fqt_pack_bits")


def fqt_binary_gemm_dw(desc, cfg, qgrad, xsign, dW, ws, I_out=None, stream=None):
    z = _sizes(desc)
    _need("fqt_binary_gemm_dw",
          (xsign, torch.int64, z["xsign"], "xsign"),
          (dW, torch.float32, z["W"], "dW"),
          (I_out, torch.int32, z["W"], "I_out", True))
    _check(_lib.fqt_binary_gemm_dw(desc, cfg, ctypes.byref(qgrad.struct), _ptr(xsign), _ptr(dW),
                                   _ptr(I_out), _ptr(ws), ws.numel() * ws.element_size(),
                                   _stream(stream)), "fqt_binary_gemm_dw")


def fqt_binary_gemm_dw_planes(desc, cfg, qgrad, xbits, xbits_linesum, dW, engine, ws, I_out=None,
                              stream=None):
    z = _sizes(desc)
    _need("fqt_binary_gemm_dw_planes",
          (xbits, torch.int64, z["xsign"], "xbits"),
          (xbits_linesum, torch.int32, z["K"], "xbits_linesum"),
          (dW, torch.float32, z["W"], "dW"),
          (I_out, torch.int32, z["W"], "I_out", True))
    _check(_lib.fqt_binary_gemm_dw_planes(desc, cfg, ctypes.byref(qgrad.struct), _ptr(xbits),
                                          _ptr(xbits_linesum), _ptr(dW), _ptr(I_out), engine,
                                          _ptr(ws), ws.numel() * ws.element_size(),
                                          _stream(stream)), "fqt_binary_gemm_dw_planes")


def fqt_pack_input_signs(desc, X, dst, stream=None):
    z = _sizes(desc)
    _need("fqt_pack_input_signs",
          (X, _TORCH_OF.get(desc.x_dtype), z["X"], "X"),
          (dst, torch.int64, z["xsign"], "dst"))
    _check(_lib.fqt_pack_input_signs(desc, _ptr(X), _ptr(dst), _stream(stream)),
           "fqt_pack_input_signs")


def fqt_pack_weight_signs(desc, W, dst, linesum, stream=None):
    z = _sizes(desc)
    _need("fqt_pack_weight_signs",
          (W, _TORCH_OF.get(desc.w_dtype), z["W"], "W"),
          (dst, torch.int8, z["wsign"], "dst"),
          (linesum, torch.int32, z["K"], "linesum"))
    _check(_lib.fqt_pack_weight_signs(desc, _ptr(W), _ptr(dst), _ptr(linesum), _stream(stream)),
           "fqt_pack_weight_signs")


def fqt_binary_gemm_dx(desc, cfg, qgrad, wsign, wsign_linesum, dX, I_out=None, stream=None):
    z = _sizes(desc)
    _need("fqt_binary_gemm_dx",
          (wsign, torch.int8, z["wsign"], "wsign"),
          (wsign_linesum, torch.int32, z["K"], "wsign_linesum"),
          (dX, _TORCH_OF.get(desc.dx_dtype), z["X"], "dX"),
          (I_out, torch.int32, z["X"], "I_out", True))
    _check(_lib.fqt_binary_gemm_dx(desc, cfg, ctypes.byref(qgrad.struct), _ptr(wsign),
                                   _ptr(wsign_linesum), _ptr(dX), _ptr(I_out), _stream(stream)),
           "fqt_binary_gemm_dx")


def fqt_binary_products(desc, cfg, qgrad, xsign, wsign, wsign_linesum, dX, dW, ws, stream=None):
    z = _sizes(desc)
    _need("fqt_binary_products",
          (xsign, torch.int64, z["xsign"], "xsign"),
          (wsign, torch.int8, z["wsign"], "wsign"),
          (wsign_linesum, torch.int32, z["K"], "wsign_linesum"),
          (dX, _TORCH_OF.get(desc.dx_dtype), z["X"], "dX"),
          (dW, torch.float32, z["W"], "dW"))
    _check(_lib.fqt_binary_products(desc, cfg, ctypes.byref(qgrad.struct), _ptr(xsign),
                                    _ptr(wsign), _ptr(wsign_linesum), _ptr(dX), _ptr(dW),
                                    _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "fqt_binary_products")


def fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws, stream=None):
    z = _sizes(desc)
    _need("fqt_layer_backward",
          (X, _TORCH_OF.get(desc.x_dtype), z["X"], "X"),
          (W, _TORCH_OF.get(desc.w_dtype), z["W"], "W"),
          (dY, _TORCH_OF.get(desc.dy_dtype), z["dY"], "dY"),
          (dX, _TORCH_OF.get(desc.dx_dtype), z["X"], "dX"),
          (dW, torch.float32, z["W"], "dW"))
    _check(_lib.fqt_layer_backward(desc, cfg, _ptr(X), _ptr(W), _ptr(dY), _ptr(dX), _ptr(dW),
                                   _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "fqt_layer_backward")


def fqt_layer_backward_noalloc(desc, cfg, X, W, dY, dX, dW, stream=None):
    z = _sizes(desc)
    _need("fqt_layer_backward_noalloc",
          (X, _TORCH_OF.get(desc.x_dtype), z["X"], "X"),
          (W, _TORCH_OF.get(desc.w_dtype), z["W"], "W"),
          (dY, _TORCH_OF.get(desc.dy_dtype), z["dY"], "dY"),
          (dX, _TORCH_OF.get(desc.dx_dtype), z["X"], "dX"),
          (dW, torch.float32, z["W"], "dW"))
    _check(_lib.fqt_layer_backward_noalloc(desc, cfg, _ptr(X), _ptr(W), _ptr(dY), _ptr(dX),
                                           _ptr(dW), _stream(stream)),
           "fqt_layer_backward_noalloc")


def fqt_binary_forward(desc, X, W, gamma, Y, I_out, ws, stream=None):
    z = _sizes(desc)
    _need("fqt_binary_forward",
          (X, _TORCH_OF.get(desc.x_dtype), z["X"], "X"),
          (W, _TORCH_OF.get(desc.w_dtype), z["W"], "W"),
          (gamma, torch.float32, desc.D, "gamma"),
          (Y, _TORCH_OF.get(desc.dy_dtype), z["dY"], "Y"),
          (I_out, torch.int32, z["dY"], "I_out", True))
    _check(_lib.fqt_binary_forward(desc, _ptr(X), _ptr(W), _ptr(gamma), _ptr(Y), _ptr(I_out),
                                   _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "fqt_binary_forward")


# ----------------------------------------------------------------------------- buffers

class QGrad:
    """Device buffers of one fqt_qgrad (allocated with torch), plus the ctypes struct."""

    def __init__(self, desc, cfg, device="cuda"):
        psq_words, pcq_words, psq_bytes, pcq_bytes = fqt_qgrad_words(desc, cfg)
        N, D = desc.N, desc.D
        i32 = dict(dtype=torch.int32, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        self.psq_planes = torch.empty(psq_words, dtype=torch.int64, device=device)
        self.pcq_planes = torch.empty(pcq_words, dtype=torch.int64, device=device)
        self.psq_codes = torch.empty(psq_bytes, dtype=torch.uint8, device=device)
        self.pcq_codes = torch.empty(pcq_bytes, dtype=torch.uint8, device=device)
        self.psq_kept, self.psq_count = torch.empty(N, **i32), torch.empty(1, **i32)
        self.pcq_kept, self.pcq_count = torch.empty(D, **i32), torch.empty(1, **i32)
        self.psq_scale, self.psq_offset, self.psq_prob = (torch.empty(N, **f32) for _ in range(3))
        self.pcq_scale, self.pcq_offset, self.pcq_prob = (torch.empty(D, **f32) for _ in range(3))
        self.struct = fqt_qgrad(*(t.data_ptr() for t in (
            self.psq_planes, self.pcq_planes, self.psq_codes, self.pcq_codes,
            self.psq_kept, self.psq_count, self.pcq_kept,
            self.pcq_count, self.psq_scale, self.psq_offset, self.psq_prob, self.pcq_scale,
            self.pcq_offset, self.pcq_prob)))


def workspace(desc, cfg, which=FQT_WS_LAYER, device="cuda", stream=None):
    """A 256-byte aligned uint8 workspace tensor of the size the library asks for; quantize
    and layer workspaces go through fqt_workspace_init (their first bytes hold zeroed state
    between calls)."""
    n = fqt_workspace_size(desc, cfg, which)
    ws = torch.empty(max(n, 1), dtype=torch.uint8, device=device)
    if which in (FQT_WS_QUANTIZE, FQT_WS_LAYER):
        fqt_workspace_init(ws, stream)
    return ws
