"""The paper's FP8 formats (Table 7 rows "(a)": E4 bias 8, max 240; E5 bias 16,
max 57344; NaN = 0x80, no infinity, no -0) against the OCP formats the matrix
cores consume (rows "(b)"), through the oracle.

Pins, all derived from Table 7 rather than from either codec:
* Eq. 3 bias: E4 b_(b) - b_(a) = 1 - [f > 1.75] + [f > 1.875] for an amax
  f * 2^e (max 1.75 * 2^8 against 1.875 * 2^7); E5 biases are equal (both
  maxima are 1.75 * 2^15).
* Every code finite in both formats decodes to half in (a): so with
  b_(b) = b_(a) + 1 the two casts give the same code for every element except
  NaN (0x7F|s against 0x80) and values rounding to -0 (0x80 against 0x00).
* With equal biases (E5) the represented values x_hat = dec(q) 2^-b differ
  only for elements below the smallest normal of (b) after scaling.
The per-workload counts are written by tests/golden/formats_report.py.
"""
import numpy as np
import pytest
import torch

from parity_util import np_bits

E4B, E5B, E4A, E5A = 0, 1, 2, 3


def _frac_exp(amax_bits: int):
    f = np.uint32(amax_bits).view(np.float32).item()
    m, e = np.frexp(f)  # f = m 2^e, m in [0.5, 1)
    return 2 * m, e - 1


def _tensors():
    g = torch.Generator().manual_seed(123)
    out = []
    for scale in (1.0, 0.02, 1e-4, 37.0, 3e-6):
        out.append((torch.randn(300, 200, generator=g) * scale).to(torch.bfloat16))
    # amax mantissas on both sides of 1.75 and 1.875
    for m in (1.5, 1.74, 1.76, 1.8, 1.875, 1.9, 1.99):
        x = (torch.rand(50, 40, generator=g) * 2 - 1).to(torch.bfloat16)
        x[7, 3] = m * 2.0 ** 5
        out.append(x)
    return out


@pytest.mark.parametrize("i", range(12))
def test_bias_relation_between_format_families(orc, i):
    x = np_bits(_tensors()[i])
    for fb, fa in ((E4B, E4A), (E5B, E5A)):
        bb, ab, _ = orc.scale_bias(x, fb)
        ba, aa, _ = orc.scale_bias(x, fa)
        assert ab == aa  # the amax does not depend on the format
        f, _ = _frac_exp(ab)
        if fb == E4B:
            assert bb - ba == 1 - int(f > 1.75) + int(f > 1.875)
        else:
            assert bb == ba


@pytest.mark.parametrize("i", range(12))
def test_e4_codes_agree_when_biases_differ_by_one(orc, i):
    x = np_bits(_tensors()[i])
    bb, _, _ = orc.scale_bias(x, E4B)
    ba, _, _ = orc.scale_bias(x, E4A)
    if bb != ba + 1:
        pytest.skip("amax mantissa in (1.75, 1.875]: the biases are equal")
    qb, qa = orc.cast(x, E4B, bb), orc.cast(x, E4A, ba)
    neg_zero = qb == 0x80
    assert np.array_equal(qa[~neg_zero], qb[~neg_zero])
    assert np.all(qa[neg_zero] == 0x00)  # (a) has no -0


def test_special_codes_differ_as_table7_says(orc):
    x = np.array([0x7FC0, 0xFFC0, 0x8001, 0x8000, 0x3F80], dtype=np.uint16)  # NaN, -NaN, tiny<0, -0, 1
    for fb, fa in ((E4B, E4A), (E5B, E5A)):
        qb, qa = orc.cast(x, fb, 0), orc.cast(x, fa, -1)
        assert list(qa[:2]) == [0x80, 0x80]          # (a): the single NaN code
        assert list(qb[:2]) == [0x7F, 0xFF]          # (b): 0x7F with the sign
        assert qa[2] == 0x00 and qb[2] == 0x80       # underflow to -0 in (b) only
        assert qa[3] == 0x00 and qb[3] == 0x80
        assert qa[4] == qb[4]                         # 1.0: same code


@pytest.mark.parametrize("i", range(12))
def test_e5_represented_values_differ_only_below_normal_range(orc, i):
    x = np_bits(_tensors()[i])
    b, _, _ = orc.scale_bias(x, E5B)
    qb, qa = orc.cast(x, E5B, b), orc.cast(x, E5A, b)
    tb, ta = orc.decode_table(E5B), orc.decode_table(E5A)
    vb = tb[qb].astype(np.float64) * 2.0 ** -b
    va = ta[qa].astype(np.float64) * 2.0 ** -b
    xv = (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    differ = vb != va
    # the smallest (b) normal is 2^-14 after scaling by 2^b
    assert np.all(np.abs(xv[differ]) * 2.0 ** b < 2.0 ** -14)
