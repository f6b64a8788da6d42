"""CPU oracle for the Llama 2 decoder layer around the FP8 linears.

TEST INFRASTRUCTURE ONLY: plain, slow, obviously correct statements of what
the GPU path computes, in fp64 with numpy.  Only the tests, the smoke check and
the benchmark's CPU-baseline leg may import this module; the library and its
binding never do.

The paper quantises the four linear layers of each decoder layer to FP8 (the
Q/K/V projection, the attention output projection, and the two feed-forward
layers; App. E) and keeps everything else in higher precision.  The Llama 2
decoder it evaluates uses RMSNorm pre-normalisation, SwiGLU and rotary
position embeddings, and grouped-query attention in the 70B model (Sec. 4.3,
Table 1).  This module states that higher-precision glue, and the layer as a
chain of it with the FP8-AMAX linears of the main oracle (Sec. 2.3 Eq. 3 bias,
Sec. 2.1 Eq. 1 cast, Sec. 2 matmul), for post-training-quantised weights
(Sec. 3.1).

Readings where the paper is silent (each also listed in the design notes):
  * every glue output is rounded once, to nearest even, to bf16 (the
    higher-precision type of the path): RMSNorm y = x / sqrt(mean(x^2) + eps) * g
    with one rounding (eps = 1e-5); SwiGLU a = g * sigmoid(g) * u; the residual
    sum a + b; RoPE and attention outputs;
  * RoPE pairs element i with element i + d_head/2 ("rotate half") at angle
    pos * theta^(-2i/d_head), theta = 10000, pos = position in the sequence;
  * attention is causal within each sequence of seq_len consecutive rows,
    scores scaled by 1/sqrt(d_head); query head h reads key/value head
    h // (n_heads / n_kv_heads);
  * the fused QKV projection's output holds Q heads, then K heads, then V
    heads, each head's d_head columns contiguous; the fused gate+up output
    holds gate columns [0, ffn), then up columns [ffn, 2 ffn).
"""
from __future__ import annotations

import numpy as np

from . import BF16, E4M3, cast, decode_table, scale_bias  # noqa: F401

LLAMA_EPS = 1e-5
ROPE_THETA = 10000.0


# ---------------------------------------------------------------- bf16
def bf16_to_f64(h: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> fp64 values (exact)."""
    h = np.asarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def round_bf16(y: np.ndarray) -> np.ndarray:
    """fp64 -> bf16 bit patterns, one rounding to nearest, ties to even.
    bf16 keeps 8 significant bits, smallest normal 2^-126 (subnormals keep the
    quantum 2^-133), largest finite (2 - 2^-7) * 2^127; beyond that: infinity.
    NaN -> 0x7FC0 with the sign cleared."""
    y = np.asarray(y, dtype=np.float64)
    a = np.abs(y)
    finite = np.isfinite(a) & (a > 0)
    _, e = np.frexp(np.where(finite, a, 1.0))      # a = f * 2^e, f in [0.5, 1)
    ex = np.maximum(e - 1, -126)                     # floor(log2 a), clamped to the normal range
    quantum = np.ldexp(1.0, ex - 7)
    r = np.where(finite, np.rint(a / quantum) * quantum, a)   # rint: ties to even
    r = np.where(r >= 2.0 ** 128, np.inf, r)
    f = np.where(np.signbit(y), -r, r).astype(np.float32)    # exact: r has <= 8 significant bits
    bits = (f.view(np.uint32) >> 16).astype(np.uint16)
    return np.where(np.isnan(y), np.uint16(0x7FC0), bits).astype(np.uint16)


# ---------------------------------------------------------------- glue
def add(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Residual connection: round(a + b)."""
    return round_bf16(bf16_to_f64(a) + bf16_to_f64(b))


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float = LLAMA_EPS, res: np.ndarray | None = None):
    """RMSNorm over each row: y = h / sqrt(mean_j h_j^2 + eps) * g, with h = x
    or, given the residual branch res, h = round(x + res).  Returns (h, y) as
    bf16 bit patterns."""
    h = x if res is None else add(x, res)
    hv = bf16_to_f64(h)
    ms = np.mean(hv * hv, axis=-1, keepdims=True)
    y = hv / np.sqrt(ms + eps) * bf16_to_f64(g)[None, :]
    return np.asarray(h, dtype=np.uint16), round_bf16(y)


def rope_f64(x: np.ndarray, seq_len: int, d_head: int, theta: float = ROPE_THETA) -> np.ndarray:
    """Rotary embedding of every head of x ([rows, heads * d_head] bf16 bits),
    unrounded: row r is at position r mod seq_len; element i < d_head/2 of a
    head pairs with element i + d_head/2, rotated by pos * theta^(-2i/d_head)."""
    rows, cols = x.shape
    half = d_head // 2
    v = bf16_to_f64(x).reshape(rows, cols // d_head, d_head)
    pos = (np.arange(rows) % seq_len).astype(np.float64)
    freq = theta ** (-2.0 * np.arange(half) / d_head)
    ang = pos[:, None] * freq[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = v[..., :half], v[..., half:]
    out = np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)
    return out.reshape(rows, cols)


def rope(x: np.ndarray, seq_len: int, d_head: int, theta: float = ROPE_THETA) -> np.ndarray:
    return round_bf16(rope_f64(x, seq_len, d_head, theta))


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, seq_len: int, n_heads: int,
              n_kv_heads: int, d_head: int) -> np.ndarray:
    """Causal softmax attention, per sequence of seq_len consecutive rows
    (the last may be shorter): o_i = sum_{j <= i} softmax_j(q_i . k_j /
    sqrt(d_head)) v_j for each query head; query head h uses key/value head
    h // (n_heads / n_kv_heads).  q [R, n_heads*d_head], k and v
    [R, n_kv_heads*d_head], bf16 bits.  Per sequence and head, the scores are
    one fp64 matrix product, masked above the diagonal; the softmax weights
    are exp(s - max_j s) and the weighted sum of values is divided by their
    sum.  Returns bf16 bits."""
    R = q.shape[0]
    group = n_heads // n_kv_heads
    qv, kv, vv = bf16_to_f64(q), bf16_to_f64(k), bf16_to_f64(v)
    out = np.zeros((R, n_heads * d_head))
    for s0 in range(0, R, seq_len):
        s1 = min(s0 + seq_len, R)
        causal = np.tril(np.ones((s1 - s0, s1 - s0), dtype=bool))
        for h in range(n_heads):
            hk = h // group
            Q = qv[s0:s1, h * d_head:(h + 1) * d_head]
            K = kv[s0:s1, hk * d_head:(hk + 1) * d_head]
            V = vv[s0:s1, hk * d_head:(hk + 1) * d_head]
            sc = np.where(causal, Q @ K.T / np.sqrt(d_head), -np.inf)
            p = np.exp(sc - sc.max(axis=1, keepdims=True))
            out[s0:s1, h * d_head:(h + 1) * d_head] = (p @ V) / p.sum(axis=1, keepdims=True)
    return round_bf16(out)


def swiglu(gu: np.ndarray, ffn: int) -> np.ndarray:
    """SwiGLU on the fused gate+up output [rows, 2 ffn]: a = g * sigmoid(g) * u
    with g = gu[:, :ffn], u = gu[:, ffn:2 ffn]."""
    v = bf16_to_f64(gu)
    g, u = v[:, :ffn], v[:, ffn:2 * ffn]
    return round_bf16(g / (1.0 + np.exp(-g)) * u)


# ---------------------------------------------------------------- FP8 linears
def gemm_e4(a8: np.ndarray, ba: int, b8t: np.ndarray, bb: int) -> np.ndarray:
    """Forward FP8 matmul of two E4M3 operands, both stored contiguous along
    the contraction ([M, K] and [N, K] codes): Y = 2^-(ba+bb) * A . B^T, one
    rounding to bf16 (Sec. 2.1 Eq. 2).  Every E4M3 value is an integer
    multiple of 2^-9 below 2^9, so every product is an integer multiple of
    2^-18 below 2^18 and, for K < 2^15, every partial sum is exact in fp64
    whatever the order: the library fp64 matmul gives the exact sum."""
    K = a8.shape[1]
    if K >= 1 << 15:
        raise ValueError("exactness of the fp64 sum needs K < 2^15")
    t = decode_table(E4M3)
    s = t[a8] @ t[b8t].T
    return round_bf16(np.ldexp(s, -(int(ba) + int(bb))))


def quantise(x: np.ndarray):
    """FP8-AMAX of one activation tensor (E4): returns (codes, bias)."""
    b, _, _ = scale_bias(np.ascontiguousarray(x), E4M3)
    return cast(np.ascontiguousarray(x), E4M3, b), b


def quantise_per_sequence(x: np.ndarray, seq_len: int):
    """FP8-AMAX of each sequence of seq_len consecutive rows as a tensor of its
    own (the per-data-sample activation biases of App. D): returns (codes,
    list of biases, bias of every row)."""
    rows = x.shape[0]
    q = np.empty(x.shape, dtype=np.uint8)
    row_bias = np.empty(rows, dtype=np.int64)
    biases = []
    for s0 in range(0, rows, seq_len):
        q[s0:s0 + seq_len], b = quantise(x[s0:s0 + seq_len])
        row_bias[s0:s0 + seq_len] = b
        biases.append(b)
    return q, biases, row_bias


def gemm_e4_rows(a8: np.ndarray, row_bias: np.ndarray, b8t: np.ndarray, bb: int) -> np.ndarray:
    """gemm_e4 with one bias per row of a8: row m unscaled by 2^-(row_bias[m] + bb)."""
    out = np.empty((a8.shape[0], b8t.shape[0]), dtype=np.uint16)
    for v in np.unique(row_bias):
        rows = np.nonzero(row_bias == v)[0]
        out[rows] = gemm_e4(a8[rows], int(v), b8t, bb)
    return out


def layer_forward(H: np.ndarray, p: dict, seq_len: int, n_heads: int, n_kv_heads: int,
                  d_head: int, ffn: int, eps: float = LLAMA_EPS, per_sequence: bool = False) -> dict:
    """One Llama 2 decoder layer, forward, with the four linears in FP8
    (App. E) and weights quantised beforehand (Sec. 3.1).  H is [rows, d]
    bf16 bits; p holds the RMSNorm gains g_attn, g_mlp (bf16 bits) and for
    each linear ("qkv", "o", "gate_up", "down") its transposed E4M3 codes
    p[name + "_w8t"] ([N, K]) and bias p[name + "_bw"].  Each activation that
    enters a linear gets one bias for the whole call, or with per_sequence one
    per sequence (then "b_*" are lists).  Returns every intermediate tensor and
    activation bias, ending with "out"."""
    r = {}
    dq, dkv = n_heads * d_head, n_kv_heads * d_head

    def quant(x):
        if per_sequence:
            q, biases, rb = quantise_per_sequence(x, seq_len)
            return q, biases, rb
        q, b = quantise(x)
        return q, b, None

    def lin(x8, b, rb, name):
        if per_sequence:
            return gemm_e4_rows(x8, rb, p[name + "_w8t"], p[name + "_bw"])
        return gemm_e4(x8, b, p[name + "_w8t"], p[name + "_bw"])

    _, r["xn"] = rmsnorm(H, p["g_attn"], eps)
    r["xn8"], r["b_xn"], rb = quant(r["xn"])
    r["qkv"] = lin(r["xn8"], r["b_xn"], rb, "qkv")
    r["q"] = rope(r["qkv"][:, :dq], seq_len, d_head)
    r["k"] = rope(r["qkv"][:, dq:dq + dkv], seq_len, d_head)
    r["v"] = r["qkv"][:, dq + dkv:dq + 2 * dkv]
    r["attn"] = attention(r["q"], r["k"], r["v"], seq_len, n_heads, n_kv_heads, d_head)
    r["attn8"], r["b_attn"], rb = quant(r["attn"])
    r["o"] = lin(r["attn8"], r["b_attn"], rb, "o")
    r["h1"], r["hn"] = rmsnorm(r["o"], p["g_mlp"], eps, res=H)
    r["hn8"], r["b_hn"], rb = quant(r["hn"])
    r["gu"] = lin(r["hn8"], r["b_hn"], rb, "gate_up")
    r["act"] = swiglu(r["gu"], ffn)
    r["act8"], r["b_act"], rb = quant(r["act"])
    r["down"] = lin(r["act8"], r["b_act"], rb, "down")
    r["out"] = add(r["h1"], r["down"])
    return r
