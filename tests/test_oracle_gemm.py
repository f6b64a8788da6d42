"""Pins of the oracle's FP8 matmul with unscale (CPU only).

Sec. 2 / 2.2: FP8 inputs, higher-precision accumulation; Sec. 2.1 Eq. 2: the
output is unscaled by -(b_a + b_b).  The oracle sums in fp64 and rounds once.
* Brute force with exact rational arithmetic (fractions.Fraction) on tiny
  shapes, fp32 output compared bit for bit.  For E4M3 x E4M3 every product is
  a multiple of 2^-18 below 2^18, so with K <= 2^14 the fp64 sum is exact and
  the rounded result is unique.
* Library: numpy's fp64 matmul of the decoded operands (torch decode tables)
  on non-square shapes, which catches a transposed or swapped operand.
* Unscale invariant: raising b_a by one halves the output exactly.
* The single rounding to bf16 on hand-worked values where rounding through
  fp32 first would give a different answer.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

TORCH = {0: torch.float8_e4m3fn, 1: torch.float8_e5m2}


def torch_decode(codes: np.ndarray, f: int) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(codes)).view(TORCH[f]).to(torch.float64).numpy()


def finite_codes(f: int) -> np.ndarray:
    t = torch_decode(np.arange(256, dtype=np.uint8), f)
    return np.nonzero(np.isfinite(t))[0].astype(np.uint8)


@pytest.mark.parametrize("shape", [(1, 1, 1), (3, 5, 7), (4, 2, 33), (6, 9, 130)])
def test_exact_e4_products_bit_for_bit(orc, shape):
    M, N, K = shape
    rng = np.random.default_rng(sum(shape))
    codes = finite_codes(0)
    a = rng.choice(codes, size=(M, K))
    b = rng.choice(codes, size=(N, K))
    ba, bb = 3, -5
    got = orc.gemm_nt(a, 0, ba, b, 0, bb, out_dt=orc.F32)
    da = [[Fraction(float(v)) for v in row] for row in torch_decode(a, 0)]
    db = [[Fraction(float(v)) for v in row] for row in torch_decode(b, 0)]
    scale = Fraction(2) ** -(ba + bb)
    for i in range(M):
        for j in range(N):
            s = sum(da[i][k] * db[j][k] for k in range(K)) * scale
            exp = np.float32(float(s))  # float(Fraction) is exact here
            assert got[i, j] == exp, (i, j, got[i, j], exp)


def test_small_integer_values_mixed_formats(orc):
    # values {0, +-1, +-2, +-3, +-4, +-6, +-8} are exact in both formats
    vals = [0, 1, 2, 3, 4, 6, 8, -1, -2, -3, -4, -6, -8]
    rng = np.random.default_rng(0)
    for f_a, f_b in ((0, 1), (1, 0), (1, 1)):
        ca = np.array([orc.encode(f_a, v) for v in vals], dtype=np.uint8)
        cb = np.array([orc.encode(f_b, v) for v in vals], dtype=np.uint8)
        ia = rng.integers(0, len(vals), size=(13, 257))
        ib = rng.integers(0, len(vals), size=(11, 257))
        got = orc.gemm_nt(ca[ia], f_a, 0, cb[ib], f_b, 0, out_dt=orc.F32)
        va = np.array(vals, dtype=np.int64)
        exp = va[ia] @ va[ib].T
        assert np.array_equal(got, exp.astype(np.float32))


@pytest.mark.parametrize("fa,fb", [(0, 0), (1, 0), (0, 1)])
def test_matches_numpy_fp64_matmul(orc, fa, fb):
    rng = np.random.default_rng(fa * 2 + fb)
    M, N, K = 37, 19, 301
    a = rng.choice(finite_codes(fa), size=(M, K))
    b = rng.choice(finite_codes(fb), size=(N, K))
    ba, bb = 7, 11
    ref = (torch_decode(a, fa) @ torch_decode(b, fb).T) * 2.0 ** -(ba + bb)
    got = orc.gemm_nt(a, fa, ba, b, fb, bb, out_dt=orc.F32).astype(np.float64)
    err = np.abs(got - ref)
    assert (err <= 2.0 ** -23 * np.abs(ref) + 1e-30).all()
    # a transposed or swapped operand would not match
    assert got.shape == (M, N)


def test_unscale_halves_exactly(orc):
    rng = np.random.default_rng(2)
    a = rng.choice(finite_codes(0), size=(8, 64))
    b = rng.choice(finite_codes(1), size=(5, 64))
    y0 = orc.gemm_nt(a, 0, 4, b, 1, 20)
    y1 = orc.gemm_nt(a, 0, 5, b, 1, 20)
    assert np.array_equal(y1, y0 / 2)


def test_row_sampling_equals_full_rows(orc):
    rng = np.random.default_rng(4)
    a = rng.choice(finite_codes(0), size=(50, 96))
    b = rng.choice(finite_codes(0), size=(20, 96))
    full = orc.gemm_nt(a, 0, 2, b, 0, 1, out_dt=orc.BF16)
    rows = np.array([49, 0, 17, 17, 3])
    part = orc.gemm_nt(a, 0, 2, b, 0, 1, out_dt=orc.BF16, rows=rows)
    assert np.array_equal(part, full[rows])


def test_bf16_output_single_rounding(orc):
    # 1 + 2^-8 + 2^-40: above the halfway point between bf16 neighbours 1 and
    # 1 + 2^-7, so it rounds up; through fp32 it would become the tie 1 + 2^-8
    # and round to even (down).
    assert orc.round_bf16(1 + 2.0 ** -8 + 2.0 ** -40) == 0x3F81
    assert orc.round_bf16(1 + 2.0 ** -8) == 0x3F80           # tie -> even
    assert orc.round_bf16(1 + 3 * 2.0 ** -8) == 0x3F82       # tie -> even (up)
    assert orc.round_bf16(-(1 + 2.0 ** -8 + 2.0 ** -40)) == 0xBF81
    assert orc.round_bf16(2.0 ** 128) == 0x7F80               # overflow -> inf
    assert orc.round_bf16(2.0 ** -134) == 0x0000              # half the smallest subnormal: tie -> 0
    assert orc.round_bf16(1.5 * 2.0 ** -134) == 0x0001
    # agreement with torch's fp32 -> bf16 (round to nearest even) where the
    # value is an fp32
    rng = np.random.default_rng(8)
    x = (rng.standard_normal(20000) * np.exp2(rng.uniform(-130, 120, 20000))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([orc.round_bf16(float(v)) for v in x], dtype=np.uint16)
    assert np.array_equal(got, ref)


def test_empty_contraction_gives_zeros(orc):
    a = np.zeros((3, 0), dtype=np.uint8)
    b = np.zeros((4, 0), dtype=np.uint8)
    assert np.array_equal(orc.gemm_nt(a, 0, 0, b, 0, 0), np.zeros((3, 4), np.float32))


def test_ptq_is_bias_then_cast(orc):
    import paper_2309_17224_amd.workloads as wl
    w = wl.bf16_bits(wl.small(64, 96, std=0.01, seed=3))
    w8, w8t, bw, flags = orc.ptq_quantise_weights(w)
    b, _, fl = orc.scale_bias(w, orc.E4M3)
    assert (bw, flags) == (b, fl) and bw == 13  # 0.01 * N(0,1), amax ~ 0.03
    assert np.array_equal(w8, orc.cast(w, orc.E4M3, b))
    assert np.array_equal(w8t, w8.T)
