"""Pins of the oracle's scale-and-cast (CPU only).

Sec. 2.1 Eq. 1: the scaling bias is added to the exponent, i.e. the value is
multiplied by 2^b before the cast.  App. A: overflow clips to the largest
value.  Rounding is to nearest, ties to even (the paper does not name a
rounding mode for the cast; this is the reading taken).

* Library: torch's float8 casts round to nearest even but do not saturate, so
  they pin every value with |x * 2^b| <= max, exhaustively over all 65536 bf16
  patterns at several biases, and over random fp32 patterns.
* Clipping, NaN and signed-zero rules (App. A and App. B).
* Invariants: cast(2^k x, b - k) == cast(x, b); after the bias of Eq. 3 the
  largest code magnitude lies in (max/2, max].
"""
import numpy as np
import pytest
import torch

TORCH = {0: torch.float8_e4m3fn, 1: torch.float8_e5m2, 2: torch.float8_e4m3fnuz,
         3: torch.float8_e5m2fnuz}
ALL_BF16 = np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(256, 256)
BIASES = [-140, -126, -100, -30, -9, -3, -1, 0, 1, 2, 5, 8, 12, 15, 23, 40, 100, 126, 133, 148, 157]


def fits_fp32(v: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        return v.astype(np.float32).astype(np.float64) == v


def bf16_values(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def torch_codes(v: np.ndarray, f: int) -> np.ndarray:
    # v must be exactly representable in fp32 (checked by the caller)
    t = torch.from_numpy(v.astype(np.float32))
    return t.to(TORCH[f]).view(torch.uint8).numpy()


@pytest.mark.parametrize("f", [0, 1, 2, 3])
def test_cast_all_bf16_matches_torch_in_range(orc, f):
    mx = orc.max_num(f)
    x = bf16_values(ALL_BF16)
    for b in BIASES:
        q = orc.cast(ALL_BF16, f, b)
        v = np.ldexp(x, b)
        exact32 = fits_fp32(v)
        sel = ~np.isnan(v) & (np.abs(v) <= mx) & exact32
        ref = torch_codes(np.where(sel, v, 0.0), f)
        bad = sel & (q != ref)
        assert not bad.any(), (f, b, np.argwhere(bad)[:5], q[bad][:5], ref[bad][:5])
        # values below fp32's range are all far below half the smallest FP8
        # subnormal: they must become signed zeros
        tiny = ~np.isnan(v) & ~exact32 & (np.abs(v) < 1e-30)
        zero = 0x00 if f >= 2 else None
        if tiny.any():
            got = q[tiny]
            if zero is None:
                assert np.array_equal(got, np.where(np.signbit(v[tiny]), 0x80, 0x00))
            else:
                assert (got == 0).all()


@pytest.mark.parametrize("f", [0, 1])
def test_cast_random_fp32_matches_torch(orc, f):
    rng = np.random.default_rng(1234)
    bits = rng.integers(0, 2 ** 32, size=200_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = np.where(np.isfinite(x), x, np.float32(1.0)).astype(np.float32)
    mx = orc.max_num(f)
    for b in (-60, -5, 0, 7, 60):
        q = orc.cast(x, f, b)
        v = np.ldexp(x.astype(np.float64), b)
        exact32 = fits_fp32(v)
        sel = (np.abs(v) <= mx) & exact32
        ref = torch_codes(np.where(sel, v, 0.0), f)
        assert np.array_equal(q[sel], ref[sel])
    # values around the FP8 range, where rounding matters most
    x = (rng.standard_normal(200_000) * np.exp2(rng.uniform(-20, 12, 200_000))).astype(np.float32)
    q = orc.cast(x, f, 0)
    sel = np.abs(x) <= mx
    assert np.array_equal(q[sel], torch_codes(x[sel].astype(np.float64), f))


@pytest.mark.parametrize("f,maxcode", [(0, 0x7E), (1, 0x7B), (2, 0x7F), (3, 0x7F)])
def test_clip_nan_and_zero_rules(orc, f, maxcode):
    mx = orc.max_num(f)
    vals = np.array([mx * 1.01, mx * 4, 1e30, np.inf, -mx * 1.01, -np.inf, np.nan, -np.nan,
                     0.0, -0.0, -1e-30], dtype=np.float32)
    q = orc.cast(vals, f, 0)
    neg_zero = 0x80 if f < 2 else 0x00
    nan = [0x7F, 0xFF] if f < 2 else [0x80, 0x80]
    exp = [maxcode, maxcode, maxcode, maxcode, maxcode | 0x80, maxcode | 0x80,
           nan[0], nan[1], 0x00, neg_zero, neg_zero]
    assert q.tolist() == exp


def test_ties_round_to_even(orc):
    # E4M3: 1.0 = 0x38, next 1.125 = 0x39, next 1.25 = 0x3A.
    q = orc.cast(np.array([1.0625, 1.1875, -1.0625, 0.5 * 2 ** -9, 1.5 * 2 ** -9], np.float32), 0, 0)
    assert q.tolist() == [0x38, 0x3A, 0xB8, 0x00, 0x02]
    # E5M2: 1.0 = 0x3C, 1.25 = 0x3D; 1.125 ties to 1.0, 1.375 ties to 1.5
    q = orc.cast(np.array([1.125, 1.375], np.float32), 1, 0)
    assert q.tolist() == [0x3C, 0x3E]


@pytest.mark.parametrize("f", [0, 1])
def test_shift_invariance(orc, f):
    rng = np.random.default_rng(7)
    x = (rng.standard_normal(50_000) * np.exp2(rng.uniform(-30, 30, 50_000))).astype(np.float32)
    x = x[np.abs(x) > 2.0 ** -100]
    for b, k in ((0, 3), (5, -7), (-20, 11), (13, 40)):
        q1 = orc.cast(x, f, b)
        q2 = orc.cast((x.astype(np.float64) * 2.0 ** k).astype(np.float32), f, b - k)
        assert np.array_equal(q1, q2)


@pytest.mark.parametrize("f", [0, 1])
def test_amax_bias_fills_top_binade(orc, f):
    rng = np.random.default_rng(11)
    mx = orc.max_num(f)
    for s in (1e-6, 0.02, 1.0, 300.0, 1e5):
        x = (rng.standard_normal(4096) * s).astype(np.float32)
        b, _, _ = orc.scale_bias(x, f)
        q = orc.cast(x, f, b)
        top = np.abs(orc.decode_table(f)[q]).max()
        assert mx / 2 < top <= mx


def test_transposed_copy(orc):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((37, 53)).astype(np.float32)
    q, qT = orc.cast(x, 0, 4, transpose=True)
    assert np.array_equal(q.T, qT)
