"""Thin ctypes binding of libfp8lin.so (include/fp8lin.h).

Argument marshalling only: every function passes device pointers, sizes and
the current HIP stream to the C entry point of the same name and raises
Fp8Error on a non-zero status.  All arithmetic happens in the HIP kernels.
PyTorch provides device memory and streams.  If the shared library has not
been built the first call raises; nothing here falls back to another
implementation.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfp8lin.so")

E4M3, E5M2 = 0, 1
E4_A, E5_A = 2, 3   # the paper's formats (Table 7 rows "(a)"); bias and cast calls only
DT_BF16, DT_F32 = 0, 1
FLAG_NONFINITE, FLAG_ZERO, FLAG_SATURATED = 1, 2, 4
OK, EINVAL, ENOTSUP, EHIP = 0, 1, 2, 3

# Every symbol declared in include/fp8lin.h.
EXPORTS = (
    "fp8_status_string", "fp8_abi_version", "fp8_scale_bias_ws_bytes", "fp8_scale_bias",
    "fp8_bias_from_amax", "fp8_cast_e4", "fp8_cast_e5", "fp8_cast", "fp8_quantise_ws_bytes",
    "fp8_quantise", "fp8_quantise_noalloc", "fp8_quantise_delayed",
    "fp8_quantise_batch",
    "fp8_linear_fwd", "fp8_linear_bwd_dx", "fp8_linear_bias_ws_bytes", "fp8_linear_fwd_bias",
    "fp8_linear_bwd_dx_bias", "fp8_linear_quantise_ws_bytes",
    "fp8_linear_fwd_quantise", "fp8_linear_bwd_dx_quantise",
    "fp8_linear_bwd_dw", "ptq_quantise_weights",
    "fp8_quantise_segments", "fp8_linear_fwd_rows", "fp8_bias_mode",
    "llama_rmsnorm_ws_bytes", "llama_rmsnorm_quantise", "llama_rope_table", "llama_rope",
    "llama_attention_ws_bytes", "llama_attention", "llama_swiglu_ws_bytes", "llama_swiglu_quantise",
    "llama_residual_add",
)


class Fp8Error(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2309_17224_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.fp8_status_string.restype = ctypes.c_char_p
        L.fp8_status_string.argtypes = [i32]
        L.fp8_abi_version.restype = i32
        L.fp8_abi_version.argtypes = []
        L.fp8_scale_bias_ws_bytes.restype = sz
        L.fp8_scale_bias_ws_bytes.argtypes = [i64]
        L.fp8_scale_bias.restype = i32
        L.fp8_scale_bias.argtypes = [vp, i32, i64, i32, i32, vp, vp, vp, vp, sz, vp]
        L.fp8_bias_from_amax.restype = i32
        L.fp8_bias_from_amax.argtypes = [vp, i32, i32, vp, vp, vp]
        for name in ("fp8_cast_e4", "fp8_cast_e5"):
            f = getattr(L, name)
            f.restype = i32
            f.argtypes = [vp, i32, i64, i64, i64, vp, vp, i64, vp, i64, vp]
        L.fp8_cast.restype = i32
        L.fp8_cast.argtypes = [vp, i32, i64, i64, i64, i32, vp, vp, i64, vp, i64, vp]
        L.fp8_quantise_ws_bytes.restype = sz
        L.fp8_quantise_ws_bytes.argtypes = [i64, i64]
        L.fp8_quantise.restype = i32
        L.fp8_quantise.argtypes = [vp, i32, i64, i64, i64, i32, i32, vp, vp, vp, vp, vp, i64, vp,
                                   i64, vp, sz, vp]
        L.fp8_quantise_noalloc.restype = i32
        L.fp8_quantise_noalloc.argtypes = [vp, i32, i64, i64, i64, i32, i32, vp, vp, vp, vp, vp, i64, vp,
                                           i64, vp]
        L.fp8_quantise_delayed.restype = i32
        L.fp8_quantise_delayed.argtypes = [vp, i32, i64, i64, i64, i32, i32, vp, vp, i64, vp, vp, vp, vp, i64,
                                           vp, i64, vp, sz, vp]
        L.fp8_quantise_batch.argtypes = [i32, vp, i32, i32, i32, vp]
        L.fp8_quantise_batch.restype = i32
        for name in ("fp8_linear_fwd", "fp8_linear_bwd_dx"):
            f = getattr(L, name)
            f.restype = i32
            f.argtypes = [vp, vp, vp, vp, vp, i32, i64, i64, i64, vp, vp]
        L.fp8_linear_bias_ws_bytes.restype = sz
        L.fp8_linear_bias_ws_bytes.argtypes = []
        for name in ("fp8_linear_fwd_bias", "fp8_linear_bwd_dx_bias"):
            f = getattr(L, name)
            f.restype = i32
            f.argtypes = [vp, vp, vp, vp, vp, i32, i64, i64, i64, i32, i32, vp, vp, vp, vp, sz, vp]
        L.fp8_linear_quantise_ws_bytes.restype = sz
        L.fp8_linear_quantise_ws_bytes.argtypes = [i64, i64]
        for name in ("fp8_linear_fwd_quantise", "fp8_linear_bwd_dx_quantise"):
            f = getattr(L, name)
            f.restype = i32
            f.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i32, i32, vp, vp, vp, vp, vp, i64, vp,
                          i64, vp, sz, vp]
        L.fp8_linear_bwd_dw.restype = i32
        L.fp8_linear_bwd_dw.argtypes = [vp, vp, vp, vp, vp, i32, i64, i64, i64, vp]
        L.fp8_quantise_segments.restype = i32
        L.fp8_quantise_segments.argtypes = [vp, i32, i64, i64, i64, i32, i32, vp, i64, vp, vp, vp, vp, vp, i64,
                                            vp, i64, vp]
        L.fp8_linear_fwd_rows.restype = i32
        L.fp8_linear_fwd_rows.argtypes = [vp, vp, vp, vp, vp, i32, i64, i64, i64, vp, vp]
        L.fp8_bias_mode.restype = i32
        L.fp8_bias_mode.argtypes = [vp, i64, vp, i64, vp, vp]
        f32, f64 = ctypes.c_float, ctypes.c_double
        L.llama_rmsnorm_ws_bytes.restype = sz
        L.llama_rmsnorm_ws_bytes.argtypes = [i64]
        L.llama_rmsnorm_quantise.restype = i32
        L.llama_rmsnorm_quantise.argtypes = [vp, i64, vp, i64, vp, i64, i64, f32, vp, i64, vp, i64, i32, i32,
                                             vp, vp, vp, vp, vp, i64, vp, sz, vp]
        L.llama_rope_table.restype = i32
        L.llama_rope_table.argtypes = [i64, i32, f64, vp, vp]
        L.llama_rope.restype = i32
        L.llama_rope.argtypes = [vp, i64, i64, i32, i32, i64, vp, vp]
        L.llama_attention_ws_bytes.restype = sz
        L.llama_attention_ws_bytes.argtypes = [i64, i64, i32]
        L.llama_attention.restype = i32
        L.llama_attention.argtypes = [vp, i64, i64, i64, i32, i32, i32, vp, i64, i32, i32, vp, vp, vp, vp, vp,
                                      i64, vp, sz, vp]
        L.llama_swiglu_ws_bytes.restype = sz
        L.llama_swiglu_ws_bytes.argtypes = []
        L.llama_swiglu_quantise.restype = i32
        L.llama_swiglu_quantise.argtypes = [vp, i64, i64, i64, vp, i64, i32, i32, vp, vp, vp, vp, vp, i64, vp,
                                            sz, vp]
        L.llama_residual_add.restype = i32
        L.llama_residual_add.argtypes = [vp, vp, vp, i64, vp]
        L.ptq_quantise_weights.restype = i32
        L.ptq_quantise_weights.argtypes = [vp, i32, i64, i64, vp, vp, vp, vp, vp, sz, vp]
        _lib = L
    return _lib


def _check(fn: str, status: int) -> None:
    if status != OK:
        raise Fp8Error(fn, status, lib().fp8_status_string(status).decode())


def _p(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return DT_BF16
    if t.dtype == torch.float32:
        return DT_F32
    raise TypeError(f"expected bfloat16 or float32, got {t.dtype}")


def _ld(t: torch.Tensor) -> int:
    """Row stride (elements) of a 2-D tensor whose rows are contiguous."""
    if t.dim() != 2 or (t.stride(1) != 1 and t.size(1) > 1):
        raise ValueError("expected a 2-D tensor with contiguous rows")
    return t.stride(0) if t.size(0) > 1 else max(t.size(1), 1)


def _i32(dev):
    return torch.empty(1, dtype=torch.int32, device=dev)


# ------------------------------------------------------------------ calls
def fp8_scale_bias_ws_bytes(n: int) -> int:
    return int(lib().fp8_scale_bias_ws_bytes(int(n)))


def workspace(n: int, device) -> torch.Tensor:
    return torch.empty(max(fp8_scale_bias_ws_bytes(n), 4), dtype=torch.uint8, device=device)


def fp8_scale_bias(x: torch.Tensor, fmt: int, margin: int = 0, bias=None, amax_bits=None,
                   flags=None, ws=None, stream=None):
    """amax + Eq. 3 bias of a whole tensor.  Returns (bias, amax_bits, flags),
    each a one-element device tensor (int32 / int32 holding uint32 bits)."""
    if not x.is_contiguous():
        raise ValueError("fp8_scale_bias needs a contiguous tensor")
    dev = x.device
    bias = _i32(dev) if bias is None else bias
    amax_bits = _i32(dev) if amax_bits is None else amax_bits
    flags = _i32(dev) if flags is None else flags
    n = x.numel()
    ws = workspace(n, dev) if ws is None else ws
    st = lib().fp8_scale_bias(_p(x), _dt(x), n, fmt, margin, _p(bias), _p(amax_bits), _p(flags),
                              _p(ws), ws.numel() * ws.element_size(), _stream(stream))
    _check("fp8_scale_bias", st)
    return bias, amax_bits, flags


def fp8_bias_from_amax(amax_bits: torch.Tensor, fmt: int, margin: int = 0, bias=None, flags=None,
                       stream=None):
    dev = amax_bits.device
    bias = _i32(dev) if bias is None else bias
    flags = _i32(dev) if flags is None else flags
    st = lib().fp8_bias_from_amax(_p(amax_bits), fmt, margin, _p(bias), _p(flags), _stream(stream))
    _check("fp8_bias_from_amax", st)
    return bias, flags


def _cast(name: str, x: torch.Tensor, bias: torch.Tensor, q=None, qT=None, want_q=True,
          want_qT=False, stream=None):
    x2 = x if x.dim() == 2 else x.reshape(1, -1)
    rows, cols = x2.shape
    if want_q and q is None:
        q = torch.empty((rows, cols), dtype=torch.uint8, device=x.device)
    if want_qT and qT is None:
        qT = torch.empty((cols, rows), dtype=torch.uint8, device=x.device)
    st = getattr(lib(), name)(_p(x2), _dt(x2), rows, cols, _ld(x2), _p(bias),
                              _p(q), _ld(q) if q is not None else 0,
                              _p(qT), _ld(qT) if qT is not None else 0, _stream(stream))
    _check(name, st)
    return q, qT


def fp8_cast_e4(x, bias, q=None, qT=None, want_q=True, want_qT=False, stream=None):
    """Scale by 2^bias and cast to E4M3; returns (q, qT)."""
    return _cast("fp8_cast_e4", x, bias, q, qT, want_q, want_qT, stream)


def fp8_cast_e5(x, bias, q=None, qT=None, want_q=True, want_qT=False, stream=None):
    """Scale by 2^bias and cast to E5M2; returns (q, qT)."""
    return _cast("fp8_cast_e5", x, bias, q, qT, want_q, want_qT, stream)


def fp8_cast(x, fmt, bias, q=None, qT=None, want_q=True, want_qT=False, stream=None):
    """Scale by 2^bias and cast to any of E4M3, E5M2, E4_A, E5_A; returns (q, qT)."""
    x2 = x if x.dim() == 2 else x.reshape(1, -1)
    rows, cols = x2.shape
    if want_q and q is None:
        q = torch.empty((rows, cols), dtype=torch.uint8, device=x.device)
    if want_qT and qT is None:
        qT = torch.empty((cols, rows), dtype=torch.uint8, device=x.device)
    st = lib().fp8_cast(_p(x2), _dt(x2), rows, cols, _ld(x2), fmt, _p(bias),
                        _p(q), _ld(q) if q is not None else 0,
                        _p(qT), _ld(qT) if qT is not None else 0, _stream(stream))
    _check("fp8_cast", st)
    return q, qT


def fp8_quantise_ws_bytes(rows: int, cols: int) -> int:
    return int(lib().fp8_quantise_ws_bytes(rows, cols))


def quantise_workspace(rows: int, cols: int, device) -> torch.Tensor:
    return torch.empty(max(fp8_quantise_ws_bytes(rows, cols), 4), dtype=torch.uint8, device=device)


def fp8_quantise(x: torch.Tensor, fmt: int, margin: int = 0, bias_pred=None, bias=None,
                 amax_bits=None, flags=None, q=None, qT=None, want_q=True, want_qT=False, ws=None,
                 stream=None):
    """amax + Eq. 3 bias + cast of a whole 2-D tensor (codes and/or transposed
    codes).  bias_pred: optional one-element device tensor with a predicted
    bias (may be `bias` itself).  Returns (q, qT, bias, amax_bits, flags)."""
    x2 = x if x.dim() == 2 else x.reshape(1, -1)
    rows, cols = x2.shape
    dev = x.device
    bias = _i32(dev) if bias is None else bias
    amax_bits = _i32(dev) if amax_bits is None else amax_bits
    flags = _i32(dev) if flags is None else flags
    if want_q and q is None:
        q = torch.empty((rows, cols), dtype=torch.uint8, device=dev)
    if want_qT and qT is None:
        qT = torch.empty((cols, rows), dtype=torch.uint8, device=dev)
    ws = quantise_workspace(rows, cols, dev) if ws is None else ws
    st = lib().fp8_quantise(_p(x2), _dt(x2), rows, cols, _ld(x2), fmt, margin, _p(bias_pred),
                            _p(bias), _p(amax_bits), _p(flags), _p(q),
                            _ld(q) if q is not None else 0, _p(qT),
                            _ld(qT) if qT is not None else 0, _p(ws),
                            ws.numel() * ws.element_size(), _stream(stream))
    _check("fp8_quantise", st)
    return q, qT, bias, amax_bits, flags


def fp8_quantise_delayed(x: torch.Tensor, fmt: int, bias: torch.Tensor, history: torch.Tensor,
                         count: torch.Tensor, margin: int = 0, amax_bits=None, flags=None, q=None, qT=None,
                         want_q=True, want_qT=False, ws=None, stream=None):
    """Delayed scaling: cast with *bias, append amax(x) to the history ring
    and write the next call's bias (Eq. 3 of the history maximum) into bias.
    history: int32 device tensor of history_len words (zeros at first);
    count: one int32 device word.  Returns (q, qT, bias, amax_bits, flags)."""
    x2 = x if x.dim() == 2 else x.reshape(1, -1)
    rows, cols = x2.shape
    dev = x.device
    amax_bits = _i32(dev) if amax_bits is None else amax_bits
    flags = _i32(dev) if flags is None else flags
    if want_q and q is None:
        q = torch.empty((rows, cols), dtype=torch.uint8, device=dev)
    if want_qT and qT is None:
        qT = torch.empty((cols, rows), dtype=torch.uint8, device=dev)
    ws = quantise_workspace(rows, cols, dev) if ws is None else ws
    st = lib().fp8_quantise_delayed(_p(x2), _dt(x2), rows, cols, _ld(x2), fmt, margin, _p(bias), _p(history),
                                    history.numel(), _p(count), _p(amax_bits), _p(flags), _p(q),
                                    _ld(q) if q is not None else 0, _p(qT), _ld(qT) if qT is not None else 0,
                                    _p(ws), ws.numel() * ws.element_size(), _stream(stream))
    _check("fp8_quantise_delayed", st)
    return q, qT, bias, amax_bits, flags


NOALLOC_SCRATCH_BYTES = 1048576
NOALLOC_MAX_TILES = 262143


def fp8_quantise_noalloc(x: torch.Tensor, fmt: int, margin: int = 0, bias_pred=None, bias=None,
                         amax_bits=None, flags=None, q=None, qT=None, want_q=True, want_qT=False,
                         stream=None):
    """fp8_quantise with the library's static scratch instead of a workspace
    (nothing allocated by the library; outputs are allocated here only when
    not given).  Returns (q, qT, bias, amax_bits, flags)."""
    x2 = x if x.dim() == 2 else x.reshape(1, -1)
    rows, cols = x2.shape
    dev = x.device
    bias = _i32(dev) if bias is None else bias
    amax_bits = _i32(dev) if amax_bits is None else amax_bits
    flags = _i32(dev) if flags is None else flags
    if want_q and q is None:
        q = torch.empty((rows, cols), dtype=torch.uint8, device=dev)
    if want_qT and qT is None:
        qT = torch.empty((cols, rows), dtype=torch.uint8, device=dev)
    st = lib().fp8_quantise_noalloc(_p(x2), _dt(x2), rows, cols, _ld(x2), fmt, margin, _p(bias_pred),
                                    _p(bias), _p(amax_bits), _p(flags), _p(q),
                                    _ld(q) if q is not None else 0, _p(qT),
                                    _ld(qT) if qT is not None else 0, _stream(stream))
    _check("fp8_quantise_noalloc", st)
    return q, qT, bias, amax_bits, flags


class QuantiseArgs(ctypes.Structure):
    """fp8_quantise_args of the C header (device pointers, sizes)."""
    _fields_ = [("x", ctypes.c_void_p), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("ldx", ctypes.c_int64), ("bias_pred", ctypes.c_void_p), ("bias", ctypes.c_void_p),
                ("amax_bits", ctypes.c_void_p), ("flags", ctypes.c_void_p), ("q", ctypes.c_void_p),
                ("ldq", ctypes.c_int64), ("qT", ctypes.c_void_p), ("ldqT", ctypes.c_int64),
                ("ws", ctypes.c_void_p), ("ws_bytes", ctypes.c_size_t)]


QUANTISE_BATCH_MAX = 4


def fp8_quantise_batch(items, fmt: int, margin: int = 0, stream=None):
    """fp8_quantise of several 2-D tensors of one dtype in two launches (same
    bits as separate calls).  items: dicts with x, bias, ws and optionally
    bias_pred, amax_bits, flags, q, qT (outputs are not allocated here)."""
    arr = (QuantiseArgs * max(len(items), 1))()
    dt = _dt(items[0]["x"]) if items else DT_BF16
    for a, it in zip(arr, items):
        x = it["x"]
        q, qT, ws = it.get("q"), it.get("qT"), it["ws"]
        a.x, a.rows, a.cols, a.ldx = _p(x), x.shape[0], x.shape[1], _ld(x)
        a.bias_pred, a.bias = _p(it.get("bias_pred")), _p(it["bias"])
        a.amax_bits, a.flags = _p(it.get("amax_bits")), _p(it.get("flags"))
        a.q, a.ldq = _p(q), _ld(q) if q is not None else 0
        a.qT, a.ldqT = _p(qT), _ld(qT) if qT is not None else 0
        a.ws, a.ws_bytes = _p(ws), ws.numel() * ws.element_size()
    st = lib().fp8_quantise_batch(len(items), ctypes.cast(arr, ctypes.c_void_p), dt, fmt, margin,
                                  _stream(stream))
    _check("fp8_quantise_batch", st)


def _out(shape, out_dt, dev, out):
    if out is not None:
        return out
    return torch.empty(shape, dtype=torch.bfloat16 if out_dt == DT_BF16 else torch.float32,
                       device=dev)


def _odt(out_dt: int, out) -> int:
    return out_dt if out is None else _dt(out)


def fp8_linear_fwd(x8, bx, w8t, bw, out_dt=DT_BF16, y=None, y_amax_bits=None, stream=None):
    """Y [M,N] = 2^-(bx+bw) X8 [M,K] . W8T [N,K]^T."""
    M, K = x8.shape
    N = w8t.shape[0]
    y = _out((M, N), out_dt, x8.device, y)
    st = lib().fp8_linear_fwd(_p(x8), _p(bx), _p(w8t), _p(bw), _p(y), _odt(out_dt, y), M, N, K,
                              _p(y_amax_bits), _stream(stream))
    _check("fp8_linear_fwd", st)
    return y


def fp8_linear_bwd_dx(dy8, bg, w8, bw, out_dt=DT_BF16, dx=None, dx_amax_bits=None, stream=None):
    """dX [M,K] = 2^-(bg+bw) dY8 [M,N] . W8 [K,N]^T."""
    M, N = dy8.shape
    K = w8.shape[0]
    dx = _out((M, K), out_dt, dy8.device, dx)
    st = lib().fp8_linear_bwd_dx(_p(dy8), _p(bg), _p(w8), _p(bw), _p(dx), _odt(out_dt, dx), M, N, K,
                                 _p(dx_amax_bits), _stream(stream))
    _check("fp8_linear_bwd_dx", st)
    return dx


def bias_workspace(device) -> torch.Tensor:
    """Workspace of fp8_linear_fwd_bias / fp8_linear_bwd_dx_bias: zeros, and
    left zero by every completed call (one per stream of concurrent calls)."""
    return torch.zeros(int(lib().fp8_linear_bias_ws_bytes()) // 4, dtype=torch.int32, device=device)


def _gemm_bias(name, a8, ba, b8, bb, out, out_dt, rows, cols, kc, fmt, margin, bias, amax_bits, flags,
               ws, stream):
    dev = a8.device
    out = _out((rows, cols), out_dt, dev, out)
    bias = _i32(dev) if bias is None else bias
    amax_bits = _i32(dev) if amax_bits is None else amax_bits
    flags = _i32(dev) if flags is None else flags
    ws = bias_workspace(dev) if ws is None else ws
    st = getattr(lib(), name)(_p(a8), _p(ba), _p(b8), _p(bb), _p(out), _odt(out_dt, out), *(
        (rows, cols, kc) if name == "fp8_linear_fwd_bias" else (rows, kc, cols)),
        fmt, margin, _p(bias), _p(amax_bits), _p(flags), _p(ws), ws.numel() * ws.element_size(),
        _stream(stream))
    _check(name, st)
    return out, bias, amax_bits, flags


def fp8_linear_fwd_bias(x8, bx, w8t, bw, fmt=E4M3, margin=0, out_dt=DT_BF16, y=None, bias=None,
                        amax_bits=None, flags=None, ws=None, stream=None):
    """Y = fp8_linear_fwd(...) with the Eq. 3 bias of Y (format fmt) from the
    same launch.  Returns (y, bias, amax_bits, flags)."""
    M, K = x8.shape
    N = w8t.shape[0]
    return _gemm_bias("fp8_linear_fwd_bias", x8, bx, w8t, bw, y, out_dt, M, N, K, fmt, margin, bias,
                      amax_bits, flags, ws, stream)


def fp8_linear_bwd_dx_bias(dy8, bg, w8, bw, fmt=E5M2, margin=0, out_dt=DT_BF16, dx=None, bias=None,
                           amax_bits=None, flags=None, ws=None, stream=None):
    """dX = fp8_linear_bwd_dx(...) with the Eq. 3 bias of dX from the same
    launch.  Returns (dx, bias, amax_bits, flags)."""
    M, N = dy8.shape
    K = w8.shape[0]
    return _gemm_bias("fp8_linear_bwd_dx_bias", dy8, bg, w8, bw, dx, out_dt, M, K, N, fmt, margin, bias,
                      amax_bits, flags, ws, stream)


def _gemm_quantise(name, a8, ba, b8, bb, out, rows, cols, kc, fmt, margin, bias_pred, bias,
                   amax_bits, flags, q, qT, want_qT, ws, stream):
    dev = a8.device
    out = _out((rows, cols), DT_BF16, dev, out)
    bias = _i32(dev) if bias is None else bias
    amax_bits = _i32(dev) if amax_bits is None else amax_bits
    flags = _i32(dev) if flags is None else flags
    if q is None:
        q = torch.empty((rows, cols), dtype=torch.uint8, device=dev)
    if want_qT and qT is None:
        qT = torch.empty((cols, rows), dtype=torch.uint8, device=dev)
    if ws is None:
        ws = torch.empty(max(int(lib().fp8_linear_quantise_ws_bytes(rows, cols)), 4), dtype=torch.uint8,
                         device=dev)
    st = getattr(lib(), name)(_p(a8), _p(ba), _p(b8), _p(bb), _p(out), *(
        (rows, cols, kc) if name == "fp8_linear_fwd_quantise" else (rows, kc, cols)),
        fmt, margin, _p(bias_pred), _p(bias), _p(amax_bits), _p(flags), _p(q), _ld(q), _p(qT),
        _ld(qT) if qT is not None else 0, _p(ws), ws.numel() * ws.element_size(), _stream(stream))
    _check(name, st)
    return out, q, qT, bias, amax_bits, flags


def fp8_linear_fwd_quantise(x8, bx, w8t, bw, fmt=E4M3, margin=0, bias_pred=None, y=None, bias=None,
                            amax_bits=None, flags=None, y8=None, y8t=None, want_y8t=False, ws=None,
                            stream=None):
    """Y = fp8_linear_fwd(...) (bf16) and its FP8 codes, bias, amax, flags from
    the epilogue.  Returns (y, y8, y8t, bias, amax_bits, flags)."""
    M, K = x8.shape
    N = w8t.shape[0]
    return _gemm_quantise("fp8_linear_fwd_quantise", x8, bx, w8t, bw, y, M, N, K, fmt, margin,
                          bias_pred, bias, amax_bits, flags, y8, y8t, want_y8t, ws, stream)


def fp8_linear_bwd_dx_quantise(dy8, bg, w8, bw, fmt=E5M2, margin=0, bias_pred=None, dx=None,
                               bias=None, amax_bits=None, flags=None, dx8=None, dx8t=None,
                               want_dx8t=False, ws=None, stream=None):
    """dX = fp8_linear_bwd_dx(...) (bf16) and its FP8 codes etc.  Returns
    (dx, dx8, dx8t, bias, amax_bits, flags)."""
    M, N = dy8.shape
    K = w8.shape[0]
    return _gemm_quantise("fp8_linear_bwd_dx_quantise", dy8, bg, w8, bw, dx, M, K, N, fmt, margin,
                          bias_pred, bias, amax_bits, flags, dx8, dx8t, want_dx8t, ws, stream)


def fp8_linear_bwd_dw(x8t, bx, dy8t, bg, out_dt=DT_F32, dw=None, stream=None):
    """dW [K,N] = 2^-(bx+bg) X8T [K,M] . dY8T [N,M]^T."""
    K, M = x8t.shape
    N = dy8t.shape[0]
    dw = _out((K, N), out_dt, x8t.device, dw)
    st = lib().fp8_linear_bwd_dw(_p(x8t), _p(bx), _p(dy8t), _p(bg), _p(dw), _odt(out_dt, dw), M, N, K,
                                 _stream(stream))
    _check("fp8_linear_bwd_dw", st)
    return dw


def ptq_quantise_weights(w, want_w8=True, want_w8t=True, w8=None, w8t=None, bw=None, flags=None,
                         ws=None, stream=None):
    """Post-training quantisation of a [K, N] weight: returns (w8, w8t, bw, flags)."""
    if not w.is_contiguous():
        raise ValueError("ptq_quantise_weights needs a contiguous weight")
    K, N = w.shape
    dev = w.device
    if want_w8 and w8 is None:
        w8 = torch.empty((K, N), dtype=torch.uint8, device=dev)
    if want_w8t and w8t is None:
        w8t = torch.empty((N, K), dtype=torch.uint8, device=dev)
    bw = _i32(dev) if bw is None else bw
    flags = _i32(dev) if flags is None else flags
    ws = workspace(K * N, dev) if ws is None else ws
    st = lib().ptq_quantise_weights(_p(w), _dt(w), K, N, _p(w8), _p(w8t), _p(bw), _p(flags), _p(ws),
                                    ws.numel() * ws.element_size(), _stream(stream))
    _check("ptq_quantise_weights", st)
    return w8, w8t, bw, flags


def fp8_quantise_segments(x: torch.Tensor, offsets: torch.Tensor, fmt: int, margin: int = 0, bias=None,
                          amax_bits=None, flags=None, row_bias=None, q=None, qT=None, want_q=True,
                          want_qT=False, stream=None):
    """amax + Eq. 3 bias + cast per row segment (rows offsets[s] .. offsets[s+1]-1,
    offsets a device int32 [nseg + 1]).  Returns (q, qT, bias[nseg],
    amax_bits[nseg], flags[nseg], row_bias[rows])."""
    rows, cols = x.shape
    dev = x.device
    nseg = offsets.numel() - 1
    i32 = dict(dtype=torch.int32, device=dev)
    bias = torch.empty(nseg, **i32) if bias is None else bias
    amax_bits = torch.empty(nseg, **i32) if amax_bits is None else amax_bits
    flags = torch.empty(nseg, **i32) if flags is None else flags
    row_bias = torch.empty(max(rows, 1), **i32) if row_bias is None else row_bias
    if want_q and q is None:
        q = torch.empty((rows, cols), dtype=torch.uint8, device=dev)
    if want_qT and qT is None:
        qT = torch.empty((cols, rows), dtype=torch.uint8, device=dev)
    st = lib().fp8_quantise_segments(_p(x), _dt(x), rows, cols, _ld(x), fmt, margin, _p(offsets), nseg,
                                     _p(bias), _p(amax_bits), _p(flags), _p(row_bias), _p(q),
                                     _ld(q) if q is not None else 0, _p(qT), _ld(qT) if qT is not None else 0,
                                     _stream(stream))
    _check("fp8_quantise_segments", st)
    return q, qT, bias, amax_bits, flags, row_bias[:rows]


def fp8_linear_fwd_rows(x8, bx_rows, w8t, bw, out_dt=DT_BF16, y=None, y_amax_bits=None, stream=None):
    """Y [M,N] = 2^-(bx_rows[m]+bw) X8 [M,K] . W8T [N,K]^T (one activation bias per row)."""
    M, K = x8.shape
    N = w8t.shape[0]
    y = _out((M, N), out_dt, x8.device, y)
    st = lib().fp8_linear_fwd_rows(_p(x8), _p(bx_rows), _p(w8t), _p(bw), _p(y), _odt(out_dt, y), M, N, K,
                                   _p(y_amax_bits), _stream(stream))
    _check("fp8_linear_fwd_rows", st)
    return y


def fp8_bias_mode(bias: torch.Tensor, ring: torch.Tensor, count: torch.Tensor, stream=None):
    """Append the mode of `bias` to the device ring buffer `ring` at
    count % capacity and increment `count` (one-element int32), on the device."""
    st = lib().fp8_bias_mode(_p(bias), bias.numel(), _p(ring), ring.numel(), _p(count), _stream(stream))
    _check("fp8_bias_mode", st)


# ------------------------------------------------------------------ decoder-layer glue
class FusedQuant:
    """Arguments of a quantise fused into a glue call: codes q [rows, cols]
    (uint8), the format and margin, an optional predicted bias, and one-element
    int32 device tensors for the bias, amax bits and flags; ws is the op's
    workspace (uint8 tensor)."""

    def __init__(self, q, bias, ws, fmt=E4M3, margin=0, bias_pred=None, amax_bits=None, flags=None):
        self.q, self.bias, self.ws = q, bias, ws
        self.fmt, self.margin, self.bias_pred = fmt, margin, bias_pred
        self.amax_bits, self.flags = amax_bits, flags

    def args(self):
        return (self.fmt, self.margin, _p(self.bias_pred), _p(self.bias), _p(self.amax_bits), _p(self.flags),
                _p(self.q), _ld(self.q), _p(self.ws), self.ws.numel() * self.ws.element_size())


_NO_QUANT = (E4M3, 0, None, None, None, None, None, 0, None, 0)


def _bf16(t: torch.Tensor, name: str) -> None:
    if t.dtype != torch.bfloat16:
        raise TypeError(f"{name}: expected bfloat16, got {t.dtype}")


def llama_rmsnorm_ws_bytes(rows: int) -> int:
    return int(lib().llama_rmsnorm_ws_bytes(int(rows)))


def llama_rmsnorm_quantise(x, g, eps=1e-5, res=None, h=None, y=None, fq: FusedQuant | None = None, stream=None):
    """y = RMSNorm(x [+ res]) * g (and h = x + res), optionally with the fused
    quantise of y.  Returns y."""
    _bf16(x, "x")
    rows, cols = x.shape
    y = torch.empty((rows, cols), dtype=torch.bfloat16, device=x.device) if y is None else y
    st = lib().llama_rmsnorm_quantise(_p(x), _ld(x), _p(res), _ld(res) if res is not None else 0, _p(g), rows,
                                      cols, float(eps), _p(h), _ld(h) if h is not None else 0, _p(y), _ld(y),
                                      *(fq.args() if fq else _NO_QUANT), _stream(stream))
    _check("llama_rmsnorm_quantise", st)
    return y


def llama_rope_table(seq_len: int, d_head: int, theta: float = 10000.0, table=None, device=None, stream=None):
    if table is None:
        table = torch.empty(seq_len * d_head, dtype=torch.float32, device=device)
    st = lib().llama_rope_table(int(seq_len), int(d_head), float(theta), _p(table), _stream(stream))
    _check("llama_rope_table", st)
    return table


def llama_rope(x, n_heads: int, d_head: int, seq_len: int, table, stream=None):
    """Rotary embedding in place on the first n_heads heads of x (a 2-D view
    whose rows are contiguous, e.g. the Q and K columns of the QKV output)."""
    _bf16(x, "x")
    rows = x.shape[0]
    ld = x.stride(0)
    st = lib().llama_rope(_p(x), rows, ld, int(n_heads), int(d_head), int(seq_len), _p(table), _stream(stream))
    _check("llama_rope", st)
    return x


def llama_attention_ws_bytes(rows: int, seq_len: int, n_heads: int) -> int:
    return int(lib().llama_attention_ws_bytes(int(rows), int(seq_len), int(n_heads)))


def llama_attention(qkv, seq_len: int, n_heads: int, n_kv_heads: int, d_head: int = 128, o=None,
                    fq: FusedQuant | None = None, stream=None):
    """Causal grouped-query attention over the QKV output; returns o."""
    _bf16(qkv, "qkv")
    rows = qkv.shape[0]
    o = torch.empty((rows, n_heads * d_head), dtype=torch.bfloat16, device=qkv.device) if o is None else o
    st = lib().llama_attention(_p(qkv), rows, _ld(qkv), int(seq_len), int(n_heads), int(n_kv_heads), int(d_head),
                               _p(o), _ld(o), *(fq.args() if fq else _NO_QUANT), _stream(stream))
    _check("llama_attention", st)
    return o


def llama_swiglu_ws_bytes() -> int:
    return int(lib().llama_swiglu_ws_bytes())


def llama_swiglu_quantise(gu, ffn: int, a=None, fq: FusedQuant | None = None, stream=None):
    """a = silu(gate) * up over the fused gate+up output; returns a."""
    _bf16(gu, "gu")
    rows = gu.shape[0]
    a = torch.empty((rows, ffn), dtype=torch.bfloat16, device=gu.device) if a is None else a
    st = lib().llama_swiglu_quantise(_p(gu), _ld(gu), rows, int(ffn), _p(a), _ld(a),
                                     *(fq.args() if fq else _NO_QUANT), _stream(stream))
    _check("llama_swiglu_quantise", st)
    return a


def llama_residual_add(a, b, out=None, stream=None):
    _bf16(a, "a")
    out = torch.empty_like(a) if out is None else out
    st = lib().llama_residual_add(_p(a), _p(b), _p(out), a.numel(), _stream(stream))
    _check("llama_residual_add", st)
    return out
