"""Pins of the oracle's FP8 codecs (CPU only).

* Table 7 of the paper (App. A): exponent/mantissa widths, exponent range,
  largest normal, smallest subnormal and bias of every FP8 format.
* App. B special values: E4 (b) has a single NaN pattern per sign and no
  infinity, E5 (b) follows IEEE, the (a) formats use the negative-zero code.
* Library decoders: torch's float8_e4m3fn / float8_e5m2 (OCP = rows (b)) and
  float8_e4m3fnuz / float8_e5m2fnuz (bias 8 / 16 = rows (a)), all 256 codes.
"""
import math
import os

import numpy as np
import pytest
import torch

GOLD = os.path.join(os.path.dirname(__file__), "golden", "table7_fp8_formats.txt")
FMT_IDS = {"E4M3": 0, "E5M2": 1, "E4_A": 2, "E5_A": 3}
TORCH = {0: torch.float8_e4m3fn, 1: torch.float8_e5m2, 2: torch.float8_e4m3fnuz,
         3: torch.float8_e5m2fnuz}


def table7():
    rows = []
    for line in open(GOLD):
        line = line.split("#")[0].strip()
        if line:
            f, E, M, mx, mn, maxn, minsub, bias = line.split()
            rows.append((f, int(E), int(M), int(mx), int(mn), float(maxn), float(minsub), int(bias)))
    return rows


@pytest.mark.parametrize("row", table7(), ids=lambda r: r[0])
def test_table7_constants(orc, row):
    name, E, M, max_exp, min_exp, max_normal, min_sub, bias = row
    f = FMT_IDS[name]
    tab = orc.decode_table(f)
    fin = tab[np.isfinite(tab)]
    pos = fin[fin > 0]
    # largest finite value: printed exactly in Table 7
    assert orc.max_num(f) == max_normal == pos.max()
    # smallest subnormal: printed to two significant digits
    assert abs(pos.min() - min_sub) / min_sub < 0.03
    assert pos.min() == 2.0 ** (min_exp - M)
    # exponent range: smallest normal is 2^min_exp, largest binade is 2^max_exp
    normals = pos[pos >= 2.0 ** min_exp]
    assert normals.min() == 2.0 ** min_exp
    assert math.floor(math.log2(pos.max())) == max_exp
    # bias: the code with exponent field == bias and zero mantissa is 1.0
    assert orc.decode(f, bias << M) == 1.0
    # E and M: 2^M codes per binade
    binade = pos[(pos >= 1.0) & (pos < 2.0)]
    assert len(binade) == 2 ** M


@pytest.mark.parametrize("f", [0, 1, 2, 3])
def test_decode_matches_torch(orc, f):
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(TORCH[f]).to(torch.float64).numpy()
    ours = orc.decode_table(f)
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(ours[ok], ref[ok])
    # signed zeros agree too (-0 exists only in the OCP formats)
    assert np.array_equal(np.signbit(ours[ok]), np.signbit(ref[ok]))


def test_special_values(orc):
    t = orc.decode_table(0)  # E4 (b): NaN only at S.1111.111, no infinity
    assert [c for c in range(256) if np.isnan(t[c])] == [0x7F, 0xFF]
    assert not np.isinf(t).any()
    t = orc.decode_table(1)  # E5 (b): IEEE-like
    assert [c for c in range(256) if np.isinf(t[c])] == [0x7C, 0xFC]
    assert [c for c in range(256) if np.isnan(t[c])] == [0x7D, 0x7E, 0x7F, 0xFD, 0xFE, 0xFF]
    for f in (2, 3):  # (a): negative-zero code is the single NaN/inf
        t = orc.decode_table(f)
        assert [c for c in range(256) if np.isnan(t[c])] == [0x80]


@pytest.mark.parametrize("f", [0, 1, 2, 3])
def test_round_trip_every_code(orc, f):
    mx = orc.max_num(f)
    for c in range(256):
        v = orc.decode(f, c)
        if math.isnan(v):
            assert orc.encode(f, v) == (0x80 if f >= 2 else 0x7F)
        elif math.isinf(v):  # saturating cast clips infinity to the maximum
            assert orc.encode(f, v) == orc.encode(f, math.copysign(mx, v))
        else:
            assert orc.encode(f, v) == c, (f, c, v)


def test_a_formats_are_half_of_ocp_on_common_codes(orc):
    # The (a) formats have bias one higher than (b): every code finite in both
    # decodes to half the value (App. B, Table 7 bias column).
    for fa, fb in ((2, 0), (3, 1)):
        ta, tb = orc.decode_table(fa), orc.decode_table(fb)
        both = np.isfinite(ta) & np.isfinite(tb) & (np.arange(256) != 0x80)
        assert np.array_equal(ta[both], tb[both] / 2)
