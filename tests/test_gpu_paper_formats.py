"""GPU parity for the paper's own FP8 formats (Table 7 rows "(a)": E4 bias 8,
max 240; E5 bias 16, max 57344; NaN = 0x80; no infinity, no -0) against the
oracle's (a) codec, which is pinned to torch's float8_*fnuz dtypes and to the
closed-form relations with the OCP formats (tests/test_oracle_formats*.py).

Bar: bit-exact (integer work): codes, transposed codes, biases, amax, flags.
"""
import numpy as np
import pytest
import torch

from paper_2309_17224_amd import fp8lin as F
from parity_util import i32, np_bits, u32

pytestmark = pytest.mark.gpu

PAPER = [F.E4_A, F.E5_A]


def bf16_all_patterns() -> torch.Tensor:
    return torch.arange(65536, dtype=torch.int32).to(torch.int16).view(torch.bfloat16).reshape(256, 256)


@pytest.mark.parametrize("fmt", PAPER)
def test_cast_every_bf16_pattern(orc, gpu, fmt):
    """All 65536 bf16 patterns (NaNs, infinities, -0, subnormals) at biases that
    put them below the smallest code, across the whole range, and beyond the
    largest code (the (a) values above the OCP maximum included)."""
    x = bf16_all_patterns()
    xd = x.to(gpu)
    bits = np_bits(x)
    for b in (-600, -140, -60, -20, -3, -1, 0, 1, 2, 5, 8, 9, 15, 16, 17, 40, 130, 600):
        bias = torch.tensor([b], dtype=torch.int32, device=gpu)
        q, qT = F.fp8_cast(xd, fmt, bias, want_qT=True)
        torch.cuda.synchronize()
        ref, refT = orc.cast(bits, fmt, b, transpose=True)
        assert np.array_equal(q.cpu().numpy(), ref), f"bias {b}"
        assert np.array_equal(qT.cpu().numpy(), refT), f"bias {b} (transposed)"


@pytest.mark.parametrize("fmt", PAPER)
def test_cast_top_of_range_dense(orc, gpu, fmt):
    """Dense sweep of magnitudes around the OCP maximum, where the (a) codes
    come from the fix-up rather than the converter (ties to even included)."""
    top = 480.0 if fmt == F.E4_A else 114688.0
    v = torch.linspace(0.85 * top / 2, 1.3 * top / 2, 40000, dtype=torch.float64)
    x = torch.cat([v, -v]).to(torch.bfloat16).reshape(200, 400)
    for b in (-1, 0):
        bias = torch.tensor([b], dtype=torch.int32, device=gpu)
        q, _ = F.fp8_cast(x.to(gpu), fmt, bias)
        torch.cuda.synchronize()
        assert np.array_equal(q.cpu().numpy(), orc.cast(np_bits(x), fmt, b))


@pytest.mark.parametrize("fmt", PAPER)
def test_cast_fp32_patterns(orc, gpu, fmt):
    g = torch.Generator().manual_seed(17 + fmt)
    u = torch.randint(-(2 ** 31), 2 ** 31 - 1, (300, 301), generator=g, dtype=torch.int64)
    x = u.to(torch.int32).view(torch.float32)
    for b in (-130, -7, 0, 3, 60):
        bias = torch.tensor([b], dtype=torch.int32, device=gpu)
        q, qT = F.fp8_cast(x.to(gpu), fmt, bias, want_qT=True)
        torch.cuda.synchronize()
        ref, refT = orc.cast(x.numpy(), fmt, b, transpose=True)
        assert np.array_equal(q.cpu().numpy(), ref) and np.array_equal(qT.cpu().numpy(), refT)


SPECIAL = {
    "zeros": [0] * 1000,
    "neg_zero": [0x8000] * 37,
    "one_nan": [0x3F80] * 500 + [0x7FC1] + [0x3F80] * 10,
    "neg_inf": [0xFF80] + [0x4000] * 3000,
    "subnormals": [0x0001, 0x8003, 0x0042, 0x807F] * 333,
    "amax_is_240": [0x4370, 0x3F80],      # 240
    "amax_above_1_75": [0x3FF0, 0x3F80],  # 1.875
    "amax_1_8": [0x3FE6],                 # 1.796875
    "amax_is_57344": [0x4760, 0x3F80],
    "bf16_max": [0x7F7F, 0x0001],
}


@pytest.mark.parametrize("name", sorted(SPECIAL))
@pytest.mark.parametrize("fmt", PAPER)
def test_bias_special_tensors(orc, gpu, name, fmt):
    bits = np.asarray(SPECIAL[name], dtype=np.uint16)
    x = torch.tensor(bits.view(np.int16)).view(torch.bfloat16)
    ob, oa, ofl = orc.scale_bias(bits, fmt)
    b, a, fl = F.fp8_scale_bias(x.to(gpu), fmt)
    torch.cuda.synchronize()
    assert (i32(b), u32(fl)) == (ob, ofl)
    if (oa & 0x7F800000) == 0x7F800000 and (oa & 0x7FFFFF):
        assert (u32(a) & 0x7F800000) == 0x7F800000 and (u32(a) & 0x7FFFFF)
    else:
        assert u32(a) == oa


@pytest.mark.parametrize("fmt", PAPER)
@pytest.mark.parametrize("pred", [None, 0, 1])
@pytest.mark.parametrize("shape", [(1, 1), (300, 517), (1000, 64)])
def test_quantise_paper_formats(orc, gpu, fmt, pred, shape):
    g = torch.Generator().manual_seed(shape[0] + 7 * shape[1])
    x = (torch.randn(*shape, generator=g) * 3.0).to(torch.bfloat16)
    bits = np_bits(x)
    ob, oa, ofl = orc.scale_bias(bits, fmt)
    oq, oqT = orc.cast(bits, fmt, ob, transpose=True)
    bias_pred = None if pred is None else torch.tensor([ob + pred], dtype=torch.int32, device=gpu)
    q, qT, b, a, fl = F.fp8_quantise(x.to(gpu), fmt, bias_pred=bias_pred, want_qT=True)
    torch.cuda.synchronize()
    assert (i32(b), u32(a), u32(fl)) == (ob, oa, ofl)
    assert np.array_equal(q.cpu().numpy(), oq) and np.array_equal(qT.cpu().numpy(), oqT)


def test_bias_from_amax_paper_formats(orc, gpu):
    for a_bits in (0x3F800000, 0x3FF00000, 0x3FE80000, 0x43700000, 0x00000001, 0x7F7FFFFF):
        amax = torch.tensor([a_bits], dtype=torch.int64).to(torch.int32).to(gpu)
        for fmt in PAPER:
            b, fl = F.fp8_bias_from_amax(amax, fmt)
            torch.cuda.synchronize()
            assert (i32(b), u32(fl)) == orc.bias_from_amax(a_bits, fmt)
