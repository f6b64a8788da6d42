"""Pins of the oracle's per-segment quantise, per-row-bias matmul and bias
mode (one bias per micro batch / data sample, Sec. 4 and App. D; the mode of
App. D and F), against things the definition fixes rather than against a
retyped formula:
* one segment covering every row is the whole-tensor quantise;
* scaling one segment by 2^k moves only that segment's bias, by -k (Eq. 3),
  and leaves every code unchanged (Eq. 1 is exact under power-of-two scaling
  away from the format's ends);
* an empty segment has amax 0, bias 0 and the zero flag;
* the per-row matmul with a constant bias is the plain matmul, and adding d
  to one row's bias scales that row by exactly 2^-d (exact products);
* the mode on hand-made cases (ties go to the smallest value, clamping).
"""
import numpy as np
import pytest
import torch

from parity_util import np_bits


def _x(rows, cols, seed, scales=None):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(rows, cols, generator=g)
    if scales is not None:
        x = x * torch.tensor(scales, dtype=torch.float32)[:, None]
    return np_bits(x.to(torch.bfloat16))


@pytest.mark.parametrize("fmt", [0, 1, 2, 3])
def test_one_segment_is_the_whole_tensor(orc, fmt):
    x = _x(70, 33, 1)
    q, qT, b, a, fl, rb = orc.quantise_segments(x, [0, 70], fmt, 1)
    b0, a0, f0 = orc.scale_bias(x, fmt, 1)
    q0, qT0 = orc.cast(x, fmt, b0, transpose=True)
    assert (b, a, fl) == ([b0], [a0], [f0])
    assert np.array_equal(q, q0) and np.array_equal(qT, qT0) and np.all(rb == b0)


@pytest.mark.parametrize("fmt", [0, 1])
def test_scaling_a_segment_moves_only_its_bias(orc, fmt):
    off = [0, 13, 40, 41, 64]
    x = _x(64, 50, 2)
    q, qT, b, a, fl, rb = orc.quantise_segments(x, off, fmt)
    k = 3
    xs = x.copy()
    seg = ((xs[13:40].astype(np.uint32) << 16).view(np.float32) * 2.0 ** k).astype(np.float32)
    xs[13:40] = (seg.view(np.uint32) >> 16).astype(np.uint16)  # exact: a power-of-two scale of bf16 values
    q2, qT2, b2, a2, fl2, rb2 = orc.quantise_segments(xs, off, fmt)
    assert b2 == [b[0], b[1] - k, b[2], b[3]]
    assert np.array_equal(q2, q) and np.array_equal(qT2, qT)
    assert np.all(rb2[13:40] == b[1] - k) and np.all(rb2[:13] == b[0])


def test_empty_segment(orc):
    x = _x(20, 8, 3)
    q, qT, b, a, fl, rb = orc.quantise_segments(x, [0, 0, 12, 12, 20], 0)
    assert (b[0], a[0], fl[0]) == (0, 0, orc.FLAG_ZERO) and (b[2], a[2], fl[2]) == (0, 0, orc.FLAG_ZERO)
    b1, _, _ = orc.scale_bias(x[:12], 0)
    b3, _, _ = orc.scale_bias(x[12:], 0)
    assert (b[1], b[3]) == (b1, b3)


def test_row_bias_matmul(orc):
    vals = np.array([0x00, 0x38, 0x40, 0x44, 0x48], dtype=np.uint8)  # E4M3 0, 1, 2, 3, 4
    rng = np.random.default_rng(4)
    a8 = vals[rng.integers(0, len(vals), size=(24, 64))]
    b8 = vals[rng.integers(0, len(vals), size=(40, 64))]
    y = orc.gemm_nt(a8, 0, 2, b8, 0, 1, out_dt=orc.F32)
    assert np.array_equal(orc.gemm_nt_rows(a8, 0, [2] * 24, b8, 0, 1, out_dt=orc.F32), y)
    d = np.arange(24) % 5 - 2
    yr = orc.gemm_nt_rows(a8, 0, 2 + d, b8, 0, 1, out_dt=orc.F32)
    assert np.array_equal(yr, (y.astype(np.float64) * 2.0 ** -d[:, None]).astype(np.float32))


def test_bias_mode_cases(orc):
    assert orc.bias_mode([3, 3, 5]) == 3
    assert orc.bias_mode([5, 3]) == 3
    assert orc.bias_mode([7]) == 7
    assert orc.bias_mode([-1, 4, 4, -1, 9]) == -1
    assert orc.bias_mode([-2000]) == -1024
    assert orc.bias_mode([2000, 2000, -5]) == 1023
