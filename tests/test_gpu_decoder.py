"""GPU parity of the Llama 2 decoder-layer glue (App. E: the layers kept in
higher precision around the four FP8 linears) and of the fused FP8-AMAX
quantise of their outputs, against oracle/decoder.py.

Bars (the tolerances follow from the arithmetic):
  * residual add: bit-exact (the fp32 sum of two bf16 values rounds to the
    correctly rounded bf16 sum);
  * RMSNorm, RoPE, SwiGLU: fp32 arithmetic (a few fp32 roundings, about 2e-7
    relative) rounded once to bf16, against the fp64 value rounded once:
    every element within one bf16 quantum of the oracle, and at most 1e-3 of
    the elements not identical (a difference needs the exact value within
    ~2e-7 relative of a bf16 rounding midpoint, which are 2^-8 apart);
  * attention: the probabilities are rounded to bf16 (relative 2^-9) before
    their product with V, and the output once more: relative Frobenius
    error per head <= 1e-2 (five bf16 unit roundoffs);
  * fused quantise: the bias equals the oracle's on the oracle's tensor, and
    the codes, bias, amax and flags are bit for bit those of fp8_quantise of
    the kernel's own bf16 output (whatever the prediction); the codes equal
    the oracle's cast wherever the bf16 outputs agree.
"""
import numpy as np
import pytest
import torch

import oracle as orc_mod
from oracle import decoder as D
from paper_2309_17224_amd import fp8lin as F
from paper_2309_17224_amd import workloads as wl
from parity_util import as_f64, i32, np_bits, rel_f, u32

pytestmark = pytest.mark.gpu

GLUE_MISMATCH_FRAC = 1e-3
ATTN_REL_F = 1e-2


def bf16_dev(bits: np.ndarray, dev) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)


def rand_bits(shape, seed, std=1.0):
    return wl.bf16_bits(wl.draw(shape[0], shape[1], "normal", std, (), seed))


def quantum(v: np.ndarray) -> np.ndarray:
    e = np.maximum(np.abs(v), 2.0 ** -126)
    return np.exp2(np.floor(np.log2(e)) - 7)


def ulp_check(got: np.ndarray, ref: np.ndarray, frac=GLUE_MISMATCH_FRAC, slack=0.0):
    """Every element within one bf16 quantum (plus an absolute slack where
    the fp32 arithmetic cancels), few not identical.  With got = round(v'),
    ref = round(v) and |v' - v| <= slack: |got - ref| <= q/2 + slack + q/2."""
    g, r = as_f64(got), as_f64(ref)
    bound = np.maximum(quantum(g), quantum(r)) * (1 + 1e-12) + slack
    assert np.all(np.abs(g - r) <= bound), "an element is more than one bf16 quantum off"
    assert np.mean(got != ref) <= frac, f"{np.mean(got != ref):.2e} of the elements differ"


def quant_args(dev, ws_bytes, rows, cols, pred=None):
    q = torch.full((rows, cols), 0xAB, dtype=torch.uint8, device=dev)
    scal = torch.zeros(3, dtype=torch.int32, device=dev)
    ws = torch.empty(max(ws_bytes, 4), dtype=torch.uint8, device=dev)
    bp = None if pred is None else torch.tensor([pred], dtype=torch.int32, device=dev)
    return F.FusedQuant(q, scal[0:1], ws, F.E4M3, 0, bias_pred=bp, amax_bits=scal[1:2], flags=scal[2:3]), scal


def check_fused(y_dev, fq, scal, ref_bits, orc):
    """Fused quantise vs fp8_quantise of the kernel's own output (bit for
    bit) and vs the oracle's bias on the oracle's tensor."""
    q2, _, b2, a2, f2 = F.fp8_quantise(y_dev, F.E4M3, 0)
    torch.cuda.synchronize()
    assert np.array_equal(fq.q.cpu().numpy(), q2.cpu().numpy())
    assert [i32(scal[0]), u32(scal[1]), u32(scal[2])] == [i32(b2), u32(a2), u32(f2)]
    ob, _, ofl = orc.scale_bias(ref_bits, orc.E4M3)
    assert (i32(scal[0]), u32(scal[2])) == (ob, ofl)
    oq = orc.cast(ref_bits, orc.E4M3, ob)
    same = np_bits(y_dev) == ref_bits
    assert np.array_equal(fq.q.cpu().numpy()[same], oq[same])


# ---------------------------------------------------------------- residual add
@pytest.mark.parametrize("n", [8, 2048 * 8 + 24, 3 * 1000 * 1000])
def test_residual_add_bit_exact(gpu, n):
    rng = np.random.default_rng(n)
    a = wl.bf16_bits(torch.from_numpy((rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)).to(torch.bfloat16).reshape(1, -1))
    b = wl.bf16_bits(torch.from_numpy((rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)).to(torch.bfloat16).reshape(1, -1))
    da, db = bf16_dev(a, gpu), bf16_dev(b, gpu)
    out = F.llama_residual_add(da, db)
    F.llama_residual_add(da, db, out=da)  # in place
    torch.cuda.synchronize()
    ref = D.add(a, b)
    assert np.array_equal(np_bits(out), ref)
    assert np.array_equal(np_bits(da), ref)


# ---------------------------------------------------------------- RMSNorm
@pytest.mark.parametrize("rows,cols,res", [(1, 8, False), (37, 512, False), (64, 8192, True), (300, 1048, True),
                                           (7, 8200, False), (3, 16384, True), (2, 16392, True), (5, 28672, False)])
def test_rmsnorm(gpu, orc, rows, cols, res):
    x = rand_bits((rows, cols), 10 + rows)
    r = rand_bits((rows, cols), 20 + rows, 3.0) if res else None
    g = rand_bits((1, cols), 30 + rows, 0.5)[0]
    h_ref, y_ref = D.rmsnorm(x, g, res=r)
    dx, dg = bf16_dev(x, gpu), bf16_dev(g, gpu)
    dr = bf16_dev(r, gpu) if res else None
    h = torch.empty((rows, cols), dtype=torch.bfloat16, device=gpu) if res else None
    fq, scal = quant_args(gpu, F.llama_rmsnorm_ws_bytes(rows), rows, cols, pred=3)
    y = F.llama_rmsnorm_quantise(dx, dg, 1e-5, res=dr, h=h, fq=fq)
    y_plain = F.llama_rmsnorm_quantise(dx, dg, 1e-5, res=dr)
    torch.cuda.synchronize()
    if res:
        assert np.array_equal(np_bits(h), h_ref)
    ulp_check(np_bits(y), y_ref)
    assert np.array_equal(np_bits(y), np_bits(y_plain))
    check_fused(y, fq, scal, y_ref, orc)


def test_rmsnorm_strided_and_predictions(gpu, orc):
    rows, cols = 100, 640
    big = rand_bits((rows, cols + 64), 41)
    g = rand_bits((1, cols), 42)[0]
    dbig = bf16_dev(big, gpu)
    dx = dbig[:, 32:32 + cols]
    _, y_ref = D.rmsnorm(np.ascontiguousarray(big[:, 32:32 + cols]), g)
    outs = []
    for pred in (None, 0, 2, -5, 100):
        fq, scal = quant_args(gpu, F.llama_rmsnorm_ws_bytes(rows), rows, cols, pred=pred)
        y = F.llama_rmsnorm_quantise(dx, bf16_dev(g, gpu), 1e-5, fq=fq)
        torch.cuda.synchronize()
        check_fused(y, fq, scal, y_ref, orc)
        outs.append((fq.q.cpu().numpy(), scal.cpu().numpy()))
    for q, s in outs[1:]:
        assert np.array_equal(q, outs[0][0]) and np.array_equal(s, outs[0][1])


# ---------------------------------------------------------------- RoPE
@pytest.mark.parametrize("rows,seq_len,heads", [(16, 16, 2), (300, 150, 12), (2048, 2048, 9)])
def test_rope(gpu, rows, seq_len, heads):
    dh = 128
    x = rand_bits((rows, heads * dh + 256), 50 + rows)   # extra columns stay untouched
    ref = x.copy()
    ref[:, :heads * dh] = D.rope(x[:, :heads * dh], seq_len, dh)
    dx = bf16_dev(x, gpu)
    table = F.llama_rope_table(seq_len, dh, 10000.0, device=gpu)
    F.llama_rope(dx[:, :heads * dh], heads, dh, seq_len, table)
    torch.cuda.synchronize()
    got = np_bits(dx)
    assert np.array_equal(got[:, heads * dh:], x[:, heads * dh:])
    # a cos - b sin in fp32 with a table rounded to fp32: a few roundings of
    # terms of size |a| + |b|, absolute error <= 2^-21 (|a| + |b|) where the
    # terms cancel
    v = as_f64(x[:, :heads * dh]).reshape(rows, heads, 2, dh // 2)
    pair = np.abs(v[:, :, 0]) + np.abs(v[:, :, 1])
    slack = np.zeros((rows, heads * dh + 256))
    slack[:, :heads * dh] = np.concatenate([pair, pair], axis=-1).reshape(rows, heads * dh) * 2.0 ** -21
    ulp_check(got, ref, slack=slack)


# ---------------------------------------------------------------- attention
ATTN_CASES = [
    # rows, seq_len, n_heads, n_kv_heads
    (1, 1, 1, 1),
    (40, 40, 2, 1),
    (200, 200, 4, 4),
    (300, 150, 8, 2),
    (256, 64, 2, 2),
    (520, 260, 4, 1),
    (2048, 2048, 8, 1),
]


def attn_inputs(rows, nh, nkv, seed):
    dh = 128
    return rand_bits((rows, (nh + 2 * nkv) * dh), seed)


@pytest.mark.parametrize("rows,seq_len,nh,nkv", ATTN_CASES)
def test_attention(gpu, orc, rows, seq_len, nh, nkv):
    dh = 128
    qkv = attn_inputs(rows, nh, nkv, 60 + rows + nh)
    q, k, v = qkv[:, :nh * dh], qkv[:, nh * dh:(nh + nkv) * dh], qkv[:, (nh + nkv) * dh:]
    ref = D.attention(q, k, v, seq_len, nh, nkv, dh)
    dq = bf16_dev(qkv, gpu)
    fq, scal = quant_args(gpu, F.llama_attention_ws_bytes(rows, seq_len, nh), rows, nh * dh, pred=6)
    o = F.llama_attention(dq, seq_len, nh, nkv, dh, fq=fq)
    o_plain = F.llama_attention(dq, seq_len, nh, nkv, dh)
    torch.cuda.synchronize()
    got = np_bits(o)
    assert np.array_equal(got, np_bits(o_plain))
    worst = max(rel_f(got[:, h * dh:(h + 1) * dh], ref[:, h * dh:(h + 1) * dh]) for h in range(nh))
    assert worst <= ATTN_REL_F, worst
    if seq_len == 1:
        assert np.array_equal(got, np.concatenate([v] * nh, axis=1))
    check_fused(o, fq, scal, ref, orc)


def test_attention_first_rows_exact_value(gpu):
    # the first query of every sequence sees only its own key: o = v exactly
    rows, seq_len, nh, nkv, dh = 390, 130, 4, 2, 128
    qkv = attn_inputs(rows, nh, nkv, 77)
    o = np_bits(F.llama_attention(bf16_dev(qkv, gpu), seq_len, nh, nkv, dh))
    v = qkv[:, (nh + nkv) * dh:]
    for s0 in range(0, rows, seq_len):
        for h in range(nh):
            hk = h // (nh // nkv)
            assert np.array_equal(o[s0, h * dh:(h + 1) * dh], v[s0, hk * dh:(hk + 1) * dh])


# ---------------------------------------------------------------- SwiGLU
@pytest.mark.parametrize("rows,ffn", [(1, 8), (16, 28672), (300, 1408), (2048, 2816)])
def test_swiglu(gpu, orc, rows, ffn):
    gu = rand_bits((rows, 2 * ffn), 90 + rows, 2.0)
    ref = D.swiglu(gu, ffn)
    fq, scal = quant_args(gpu, F.llama_swiglu_ws_bytes(), rows, ffn, pred=-2)
    a = F.llama_swiglu_quantise(bf16_dev(gu, gpu), ffn, fq=fq)
    torch.cuda.synchronize()
    ulp_check(np_bits(a), ref)
    check_fused(a, fq, scal, ref, orc)


# ---------------------------------------------------------------- argument checks
def test_glue_rejects_bad_arguments(gpu):
    x = torch.zeros((4, 12), dtype=torch.bfloat16, device=gpu)     # cols not a multiple of 8
    g = torch.zeros(12, dtype=torch.bfloat16, device=gpu)
    with pytest.raises(F.Fp8Error):
        F.llama_rmsnorm_quantise(x, g)
    qkv = torch.zeros((4, 3 * 64), dtype=torch.bfloat16, device=gpu)
    with pytest.raises(F.Fp8Error) as e:
        F.llama_attention(qkv, 4, 1, 1, 64)                          # head dim 64: not supported
    assert e.value.status == F.ENOTSUP
    qkv = torch.zeros((4, 5 * 128), dtype=torch.bfloat16, device=gpu)
    with pytest.raises(F.Fp8Error):
        F.llama_attention(qkv, 4, 3, 2, 128)                         # 2 does not divide 3
    with pytest.raises(F.Fp8Error):
        F.llama_swiglu_quantise(torch.zeros((2, 20), dtype=torch.bfloat16, device=gpu), 10)


# ---------------------------------------------------------------- edge cases
def test_glue_empty_outputs_give_zero_bias_and_flag(gpu):
    # an empty output with the quantise asked for: amax 0, bias 0, FLAG_ZERO (as fp8_quantise)
    for make in (
        lambda fq: F.llama_rmsnorm_quantise(torch.zeros((0, 64), dtype=torch.bfloat16, device=gpu),
                                            torch.ones(64, dtype=torch.bfloat16, device=gpu), fq=fq),
        lambda fq: F.llama_swiglu_quantise(torch.zeros((0, 64), dtype=torch.bfloat16, device=gpu), 32, fq=fq),
        lambda fq: F.llama_attention(torch.zeros((0, 3 * 128), dtype=torch.bfloat16, device=gpu), 16, 1, 1, 128,
                                     fq=fq),
    ):
        fq, scal = quant_args(gpu, 64, 1, 64, pred=5)
        scal.fill_(-7)
        make(fq)
        torch.cuda.synchronize()
        assert scal.cpu().tolist() == [0, 0, F.FLAG_ZERO]


def test_rmsnorm_zero_and_nonfinite_rows(gpu, orc):
    rows, cols = 6, 256
    x = rand_bits((rows, cols), 301)
    x[1] = 0                      # all-zero row: y = 0 (the eps keeps the scale finite)
    x[3, 17] = 0x7F80             # +inf: the mean square is inf, the row scales by 0, inf * 0 = NaN
    x[4, 5] = 0x7FC1              # NaN propagates through the row's mean square
    g = rand_bits((1, cols), 302)[0]
    _, y_ref = D.rmsnorm(x, g)
    fq, scal = quant_args(gpu, F.llama_rmsnorm_ws_bytes(rows), rows, cols, pred=2)
    y = np_bits(F.llama_rmsnorm_quantise(bf16_dev(x, gpu), bf16_dev(g, gpu), 1e-5, fq=fq))
    torch.cuda.synchronize()
    nan_g, nan_r = (y & 0x7FFF) > 0x7F80, (y_ref & 0x7FFF) > 0x7F80
    assert np.array_equal(nan_g, nan_r)
    assert np.all(y[1] & 0x7FFF == 0)
    ulp_check(np.where(nan_g, 0, y).astype(np.uint16), np.where(nan_r, 0, y_ref).astype(np.uint16))
    # the tensor holds NaN: the Eq. 3 bias is 0 with FLAG_NONFINITE, the amax the
    # canonical NaN, NaN codes are 0x7F with the sign
    assert (i32(scal[0]), u32(scal[1]), u32(scal[2])) == (0, 0x7FC00000, F.FLAG_NONFINITE)
    codes = fq.q.cpu().numpy()
    assert np.all(codes[nan_g] & 0x7F == 0x7F)
    q2, _, _, _, _ = F.fp8_quantise(bf16_dev(y, gpu), F.E4M3, 0)
    assert np.array_equal(codes, q2.cpu().numpy())


def test_swiglu_nonfinite(gpu, orc):
    rows, ffn = 4, 64
    gu = rand_bits((rows, 2 * ffn), 303)
    gu[0, 3] = 0x7F80             # gate +inf: inf * sigmoid(inf) * u = +-inf
    gu[1, 4] = 0xFF80             # gate -inf: -inf / (1 + inf) = NaN
    gu[2, ffn + 7] = 0x7FC0       # up NaN
    ref = D.swiglu(gu, ffn)
    fq, scal = quant_args(gpu, F.llama_swiglu_ws_bytes(), rows, ffn, pred=0)
    a = np_bits(F.llama_swiglu_quantise(bf16_dev(gu, gpu), ffn, fq=fq))
    torch.cuda.synchronize()
    nan_g, nan_r = (a & 0x7FFF) > 0x7F80, (ref & 0x7FFF) > 0x7F80
    assert np.array_equal(nan_g, nan_r)
    assert np.array_equal(a[~nan_g] & 0x7FFF == 0x7F80, ref[~nan_r] & 0x7FFF == 0x7F80)   # same infinities
    assert (i32(scal[0]), u32(scal[1]), u32(scal[2])) == (0, 0x7FC00000, F.FLAG_NONFINITE)
