"""Pins of the oracle's amax and scaling bias (CPU only).

Sec. 2.3 Eq. 3: amax = max |tensor|, bias = floor(log2(max_num / amax)), with
floor(a) the largest integer not above a; Sec. 3.2: a margin lowers the bias.
* Hand-worked values of Eq. 3 (tests/golden/eq3_bias_cases.txt).
* Brute force: the bias is the largest integer b with amax * 2^b <= max_num
  (exact in fp64 for every fp32 amax), for many random amax values.
* Shift invariance bias(2^k T) = bias(T) - k; flags for zero and non-finite.
* amax against numpy's max(abs) on finite tensors, and the NaN / inf / -0 rules.
"""
import math
import os

import numpy as np
import pytest

GOLD = os.path.join(os.path.dirname(__file__), "golden", "eq3_bias_cases.txt")
FMT_IDS = {"E4M3": 0, "E5M2": 1, "E4_A": 2, "E5_A": 3}


def f32_bits(v: float) -> int:
    return int(np.array([v], dtype=np.float32).view(np.uint32)[0])


def golden_cases():
    out = []
    for line in open(GOLD):
        line = line.split("#")[0].strip()
        if line:
            a, f, margin, b = line.split()
            out.append((float.fromhex(a), FMT_IDS[f], int(margin), int(b)))
    return out


@pytest.mark.parametrize("case", golden_cases(), ids=lambda c: "%s-%d-%d" % (c[0].hex(), c[1], c[2]))
def test_eq3_hand_worked(orc, case):
    amax, f, margin, expected = case
    assert np.float32(amax) == amax  # every case is an exact fp32 value
    b, flags = orc.bias_from_amax(f32_bits(amax), f, margin)
    assert (b, flags) == (expected, 0)


def brute_force_bias(amax: float, mx: float) -> int:
    b = -400
    while math.ldexp(amax, b + 1) <= mx:
        b += 1
    return b


@pytest.mark.parametrize("f", [0, 1, 2, 3])
def test_bias_is_largest_b_that_fits(orc, f):
    rng = np.random.default_rng(100 + f)
    mx = orc.max_num(f)
    bits = rng.integers(1, 0x7F800000, size=3000, dtype=np.uint64).astype(np.uint32)
    # plus values on and next to the power-of-two and max_num boundaries
    extra = []
    for k in range(-140, 128, 7):
        for v in (2.0 ** k, mx * 2.0 ** k):
            if 2.0 ** -149 <= v < 3.4e38:
                for d in (-1, 0, 1):
                    u = f32_bits(v) + d
                    if 0 < u < 0x7F800000:
                        extra.append(u)
    for u in list(bits) + extra:
        amax = float(np.array([u], dtype=np.uint32).view(np.float32)[0])
        b, flags = orc.bias_from_amax(int(u), f)
        assert flags == 0
        assert b == brute_force_bias(amax, mx), (f, amax)
        assert math.ldexp(amax, b) <= mx < math.ldexp(amax, b + 1)


def test_bias_flags(orc):
    for f in range(4):
        assert orc.bias_from_amax(0, f) == (0, 2)
        assert orc.bias_from_amax(0x7F800000, f) == (0, 1)        # +inf
        assert orc.bias_from_amax(0x7FC00000, f) == (0, 1)        # NaN
        assert orc.bias_from_amax(0x00000001, f, 0)[1] == 0      # smallest fp32 subnormal


def test_bias_shift_invariance(orc):
    rng = np.random.default_rng(5)
    x = (rng.standard_normal(1000)).astype(np.float32)
    for f in (0, 1):
        b0, _, _ = orc.scale_bias(x, f)
        for k in (-50, -3, 1, 17, 60):
            bk, _, _ = orc.scale_bias((x * np.float32(2.0 ** k)).astype(np.float32), f)
            assert bk == b0 - k


def test_margin_is_subtracted(orc):
    x = np.array([0.75, -3.0, 1e-3], dtype=np.float32)
    b0, _, _ = orc.scale_bias(x, 1)
    for m in (0, 1, 3, 5):
        assert orc.scale_bias(x, 1, margin=m)[0] == b0 - m


def test_amax_matches_numpy(orc):
    import torch
    g = torch.Generator().manual_seed(9)
    for n in (1, 7, 4096, 100_003):
        x = torch.randn(n, generator=g) * 3
        xb = x.to(torch.bfloat16)
        bits = xb.view(torch.int16).numpy().view(np.uint16)
        ref = np.abs(xb.float().numpy()).max()
        assert orc.amax_bits(bits) == f32_bits(float(ref))
        xf = x.numpy().astype(np.float32)
        assert orc.amax_bits(xf) == f32_bits(float(np.abs(xf).max()))


def test_amax_special_values(orc):
    z = np.array([0.0, -0.0], dtype=np.float32)
    assert orc.amax_bits(z) == 0
    assert orc.amax_bits(np.array([-0.0], dtype=np.float32)) == 0
    assert orc.amax_bits(np.array([1.0, -np.inf, 3.0], dtype=np.float32)) == 0x7F800000
    a = orc.amax_bits(np.array([1.0, np.nan, np.inf], dtype=np.float32))
    assert (a & 0x7F800000) == 0x7F800000 and (a & 0x7FFFFF) != 0
    # bf16 subnormals are kept, not flushed
    sub = np.array([0x0001, 0x8003, 0x0002], dtype=np.uint16)
    assert orc.amax_bits(sub) == 0x00030000
    b, amax, flags = orc.scale_bias(np.array([], dtype=np.uint16), 0)
    assert (b, amax, flags) == (0, 0, 2)
