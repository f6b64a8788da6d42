"""CPU oracle for the FP8 linear layer with per-tensor power-of-two scaling biases.

TEST INFRASTRUCTURE ONLY.  Plain, slow, obviously correct statement of what the
GPU path computes (Perez et al., arXiv 2309.17224).  Only the tests, the smoke
check and the benchmark's CPU-baseline leg may import this package; the library
and its Python binding never do.  The arithmetic lives in ``fp8_oracle.c``
(plain C, fp64); this module compiles it with gcc and wraps it with ctypes over
numpy arrays (host memory, synchronous).

Paper passages (section / equation / table):
  * formats: App. A Eq. 4, Table 7, App. B special values
  * ``amax`` and ``bias_from_amax``: Sec. 2.3 Eq. 3; margin Sec. 3.2
  * ``cast``: Sec. 2.1 Eq. 1 (scale = x * 2^b), App. A (clip on overflow)
  * ``gemm_nt``: Sec. 2 and 2.2 (FP8 x FP8, high-precision accumulate),
    Sec. 2.1 Eq. 2 (unscale by -(b_a + b_b))
  * ``ptq_quantise_weights``: Sec. 3.1
  * ``quantise_segments``, ``gemm_nt_rows``: one bias per micro batch / data or
    tensor replica (Sec. 4) and per data sample at inference (App. D): each
    row segment is an independent tensor for ``scale_bias`` and ``cast``
  * ``bias_mode``: the statistical mode of per-sample biases (App. D, App. F)
  * ``quantise_delayed``: delayed scaling, the amax-history remedy Sec. 3 cites
    for the second pass over a tensor: the bias of a call is Eq. 3 of the
    largest amax recorded by the previous calls, used as it is
  * ``oracle.decoder``: the higher-precision glue of the Llama 2 decoder layer
    (RMSNorm, RoPE, causal grouped-query attention, SwiGLU, residual adds)
    around its four FP8 linears (App. E), and the layer as a chain (numpy, fp64)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "fp8_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

# format ids: E4M3 / E5M2 are the OCP formats, Table 7 rows "(b)";
# E4_A / E5_A are the paper's default formats, Table 7 rows "(a)".
E4M3, E5M2, E4_A, E5_A = 0, 1, 2, 3
BF16, F32 = 0, 1
FLAG_NONFINITE, FLAG_ZERO = 1, 2

_lib = None


def build(force: bool = True) -> str:
    """Compile fp8_oracle.c into liboracle.so with gcc (plain -O2, OpenMP)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB)
    return LIB


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build(force=True)
        L = ctypes.CDLL(LIB)
        vp, i32, i64, u32p = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.POINTER(ctypes.c_uint32)
        L.oracle_fp8_decode.restype = ctypes.c_double
        L.oracle_fp8_decode.argtypes = [ctypes.c_int, ctypes.c_int]
        L.oracle_fp8_encode.restype = ctypes.c_int
        L.oracle_fp8_encode.argtypes = [ctypes.c_int, ctypes.c_double]
        L.oracle_fp8_max_num.restype = ctypes.c_double
        L.oracle_fp8_max_num.argtypes = [ctypes.c_int]
        L.oracle_amax.restype = None
        L.oracle_amax.argtypes = [vp, ctypes.c_int, i64, u32p]
        L.oracle_bias_from_amax.restype = i32
        L.oracle_bias_from_amax.argtypes = [ctypes.c_uint32, ctypes.c_int, i32, u32p]
        L.oracle_fp8_scale_bias.restype = i32
        L.oracle_fp8_scale_bias.argtypes = [vp, ctypes.c_int, i64, ctypes.c_int, i32,
                                            ctypes.POINTER(i32), u32p, u32p]
        L.oracle_fp8_cast.restype = i32
        L.oracle_fp8_cast.argtypes = [vp, ctypes.c_int, i64, i64, i64, ctypes.c_int, i32,
                                      vp, i64, vp, i64]
        L.oracle_gemm_nt.restype = i32
        L.oracle_gemm_nt.argtypes = [vp, ctypes.c_int, i32, i64, vp, ctypes.c_int, i32, i64,
                                     i64, i64, i64, vp, vp, ctypes.c_int, i64]
        L.oracle_ptq_quantise_weights.restype = i32
        L.oracle_ptq_quantise_weights.argtypes = [vp, ctypes.c_int, i64, i64, vp, vp,
                                                  ctypes.POINTER(i32), u32p]
        L.oracle_num_threads.restype = ctypes.c_int
        L.oracle_set_num_threads.argtypes = [ctypes.c_int]
        L.oracle_bf16_to_double.restype = ctypes.c_double
        L.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
        L.oracle_round_bf16.restype = ctypes.c_uint16
        L.oracle_round_bf16.argtypes = [ctypes.c_double]
        _lib = L
    return _lib


# ---------------------------------------------------------------- helpers
def _hp(x: np.ndarray) -> tuple[np.ndarray, int]:
    """Accept bf16 bit patterns (uint16) or float32; return (contiguous array, dtype id)."""
    if x.dtype == np.uint16:
        return np.ascontiguousarray(x), BF16
    if x.dtype == np.float32:
        return np.ascontiguousarray(x), F32
    raise TypeError("oracle inputs are bf16 bit patterns (uint16) or float32, got %s" % x.dtype)


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def decode(fmt: int, code: int) -> float:
    return lib().oracle_fp8_decode(fmt, int(code))


def decode_table(fmt: int) -> np.ndarray:
    return np.array([decode(fmt, c) for c in range(256)], dtype=np.float64)


def encode(fmt: int, v: float) -> int:
    return lib().oracle_fp8_encode(fmt, float(v))


def max_num(fmt: int) -> float:
    return lib().oracle_fp8_max_num(fmt)


def amax_bits(x: np.ndarray) -> int:
    x, dt = _hp(x)
    out = ctypes.c_uint32(0)
    lib().oracle_amax(_ptr(x), dt, x.size, ctypes.byref(out))
    return out.value


def bias_from_amax(amax_f32_bits: int, fmt: int, margin: int = 0) -> tuple[int, int]:
    """Returns (bias, flags)."""
    fl = ctypes.c_uint32(0)
    b = lib().oracle_bias_from_amax(ctypes.c_uint32(amax_f32_bits), fmt, margin, ctypes.byref(fl))
    return int(b), int(fl.value)


def scale_bias(x: np.ndarray, fmt: int, margin: int = 0) -> tuple[int, int, int]:
    """compute_bias of the paper: returns (bias, amax fp32 bits, flags)."""
    x, dt = _hp(x)
    b = ctypes.c_int32(0)
    a = ctypes.c_uint32(0)
    fl = ctypes.c_uint32(0)
    st = lib().oracle_fp8_scale_bias(_ptr(x), dt, x.size, fmt, margin, ctypes.byref(b),
                                     ctypes.byref(a), ctypes.byref(fl))
    if st:
        raise ValueError("oracle_fp8_scale_bias failed")
    return int(b.value), int(a.value), int(fl.value)


def cast(x: np.ndarray, fmt: int, bias: int, transpose: bool = False):
    """Scale by 2^bias and cast to FP8 codes.  x is [rows, cols] (or 1-D).
    Returns q (uint8, same shape) and, if transpose, qT ([cols, rows])."""
    x, dt = _hp(x)
    shp = x.shape if x.ndim == 2 else (1, x.size)
    rows, cols = shp
    q = np.empty(shp, dtype=np.uint8)
    qT = np.empty((cols, rows), dtype=np.uint8) if transpose else None
    st = lib().oracle_fp8_cast(_ptr(x), dt, rows, cols, cols, fmt, int(bias), _ptr(q), cols,
                               _ptr(qT), rows)
    if st:
        raise ValueError("oracle_fp8_cast failed")
    q = q.reshape(x.shape)
    return (q, qT) if transpose else q


def gemm_nt(a8: np.ndarray, fmt_a: int, ba: int, b8: np.ndarray, fmt_b: int, bb: int,
            out_dt: int = F32, rows: np.ndarray | None = None) -> np.ndarray:
    """out[r, j] = round(2^-(ba+bb) * sum_k dec(a8[i, k]) * dec(b8[j, k])), fp64 sum.
    a8 is [M, K], b8 is [N, K] (uint8 codes).  If rows is given, only those rows
    of a8 are used.  Returns float32, or bf16 bit patterns (uint16)."""
    a8 = np.ascontiguousarray(a8, dtype=np.uint8)
    b8 = np.ascontiguousarray(b8, dtype=np.uint8)
    M, K = a8.shape
    N, K2 = b8.shape
    if K != K2:
        raise ValueError("contraction sizes differ")
    rr = None
    if rows is not None:
        rr = np.ascontiguousarray(rows, dtype=np.int64)
        M = rr.size
    out = np.empty((M, N), dtype=np.float32 if out_dt == F32 else np.uint16)
    st = lib().oracle_gemm_nt(_ptr(a8), fmt_a, int(ba), K, _ptr(b8), fmt_b, int(bb), K,
                              M, N, K, _ptr(rr), _ptr(out), out_dt, N)
    if st:
        raise ValueError("oracle_gemm_nt failed")
    return out


def ptq_quantise_weights(w: np.ndarray):
    """Post-training quantisation of one [K, N] weight: returns (w8, w8t, bias, flags)."""
    w, dt = _hp(w)
    K, N = w.shape
    w8 = np.empty((K, N), dtype=np.uint8)
    w8t = np.empty((N, K), dtype=np.uint8)
    b = ctypes.c_int32(0)
    fl = ctypes.c_uint32(0)
    st = lib().oracle_ptq_quantise_weights(_ptr(w), dt, K, N, _ptr(w8), _ptr(w8t),
                                           ctypes.byref(b), ctypes.byref(fl))
    if st:
        raise ValueError("oracle_ptq_quantise_weights failed")
    return w8, w8t, int(b.value), int(fl.value)


def quantise_segments(x: np.ndarray, offsets, fmt: int, margin: int = 0):
    """Rows offsets[s] .. offsets[s+1]-1 of x form segment s, quantised as a
    tensor of its own: returns (q, qT, biases, amax bits, flags, row_bias)."""
    x, dt = _hp(x)
    rows, cols = x.shape
    q = np.zeros((rows, cols), dtype=np.uint8)
    qT = np.zeros((cols, rows), dtype=np.uint8)
    row_bias = np.zeros(rows, dtype=np.int32)
    biases, amaxes, flags = [], [], []
    for s in range(len(offsets) - 1):
        lo, hi = int(offsets[s]), int(offsets[s + 1])
        seg = x[lo:hi]
        b, a, fl = scale_bias(seg.reshape(-1), fmt, margin)
        biases.append(b)
        amaxes.append(a)
        flags.append(fl)
        row_bias[lo:hi] = b
        if hi > lo and cols > 0:
            q[lo:hi] = cast(seg, fmt, b)
            qT[:, lo:hi] = q[lo:hi].T
    return q, qT, biases, amaxes, flags, row_bias


def gemm_nt_rows(a8: np.ndarray, fmt_a: int, ba_rows, b8: np.ndarray, fmt_b: int, bb: int,
                 out_dt: int = F32) -> np.ndarray:
    """gemm_nt with one bias per row of a8: row m unscaled by 2^-(ba_rows[m] + bb)."""
    ba_rows = np.asarray(ba_rows, dtype=np.int64)
    M, N = a8.shape[0], b8.shape[0]
    out = np.empty((M, N), dtype=np.float32 if out_dt == F32 else np.uint16)
    for v in np.unique(ba_rows):
        rows = np.nonzero(ba_rows == v)[0]
        out[rows] = gemm_nt(a8, fmt_a, int(v), b8, fmt_b, bb, out_dt=out_dt, rows=rows)
    return out


def bias_mode(biases) -> int:
    """The most frequent bias, the smallest of equally frequent ones; a bias is
    counted clamped to [-1024, 1023] (the range the library's histogram holds)."""
    counts: dict[int, int] = {}
    for b in biases:
        v = max(-1024, min(1023, int(b)))
        counts[v] = counts.get(v, 0) + 1
    top = max(counts.values())
    return min(v for v, c in counts.items() if c == top)


FLAG_SATURATED = 4


def _f32(bits: int) -> float:
    return float(np.array([bits], dtype=np.uint32).view(np.float32)[0])


def history_max(history) -> int:
    """The largest of a list of amax values given as fp32 bit patterns (sign
    clear): the pattern of the largest value, or the canonical NaN 0x7FC00000
    when one of them is NaN.  An empty list gives 0."""
    vals = [_f32(h) for h in history]
    if any(np.isnan(v) for v in vals):
        return 0x7FC00000
    if not vals:
        return 0
    best = max(range(len(vals)), key=lambda i: vals[i])
    return int(history[best])


def quantise_delayed(xs, fmt: int, margin: int = 0, history_len: int = 16, bias0: int = 0):
    """Delayed scaling over a sequence of tensors (one call each).

    Call t casts its tensor with bias b_t, computed before the tensor is read:
    b_0 = bias0, and b_{t+1} is Eq. 3 (minus the margin) of the largest amax
    among the last history_len calls (calls 0..t); the history starts as
    history_len zeros.  So each tensor is read once: its own amax only enters
    the biases of later calls.  When a tensor's amax * 2^b_t exceeds the
    format's largest value its codes clip (App. A) and the call reports
    FLAG_SATURATED.  Flags otherwise describe the tensor's own amax (NaN or
    infinite: FLAG_NONFINITE; zero: FLAG_ZERO).

    Returns a list of dicts per call: q (codes), bias (b_t), amax (bit
    pattern of the tensor's amax), flags, next_bias (b_{t+1}); and the final
    history (list of bit patterns, slot t % history_len written by call t).
    """
    if history_len < 1:
        raise ValueError("history_len must be at least 1")
    hist = [0] * history_len
    b = int(bias0)
    out = []
    mx = max_num(fmt)
    for t, x in enumerate(xs):
        q = cast(x, fmt, b)
        a = amax_bits(x)
        av = _f32(a)
        if np.isnan(av) or np.isinf(av):
            fl = FLAG_NONFINITE
        elif av == 0.0:
            fl = FLAG_ZERO
        else:
            fl = FLAG_SATURATED if av * 2.0 ** b > mx else 0
        hist[t % history_len] = a
        nb, _ = bias_from_amax(history_max(hist), fmt, margin)
        out.append(dict(q=q, bias=b, amax=a, flags=fl, next_bias=nb))
        b = nb
    return out, hist


def bf16_to_f64(h: int) -> float:
    return lib().oracle_bf16_to_double(int(h))


def round_bf16(y: float) -> int:
    return int(lib().oracle_round_bf16(float(y)))


def num_threads() -> int:
    return int(lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    lib().oracle_set_num_threads(int(n))
