"""Pins of the oracle's delayed scaling (oracle.quantise_delayed): the bias of
a call is Eq. 3 (Sec. 2.3) of the largest amax recorded by the previous calls
(the amax-history remedy Sec. 3 cites for the second pass over a tensor),
used as it is, with App. A clipping when the tensor outgrows it."""
import os

import numpy as np
import pytest

import oracle as orc

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "delayed_bias_cases.txt")


def tensor_with_amax(amax: float, n: int = 64, seed: int = 0) -> np.ndarray:
    """fp32 values of magnitude at most amax / 2, and amax itself once."""
    rng = np.random.default_rng(seed)
    x = (rng.uniform(-0.5, 0.5, n) * amax).astype(np.float32)
    x[seed % n] = -amax if seed % 2 else amax
    return x


def test_hand_worked_sequence():
    rows = [list(map(float, l.split())) for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    xs = [tensor_with_amax(r[1], seed=i) for i, r in enumerate(rows)]
    out, hist = orc.quantise_delayed(xs, orc.E4M3, history_len=2)
    for r, o in zip(rows, out):
        assert o["bias"] == int(r[2]) and o["next_bias"] == int(r[3])
        assert bool(o["flags"] & orc.FLAG_SATURATED) == bool(r[4])
    assert [orc._f32(h) for h in hist] == [0.5, 0.5]


def test_codes_are_the_cast_with_the_bias_used_and_clip():
    xs = [tensor_with_amax(a, seed=i) for i, a in enumerate([1.0, 8.0, 2.0])]
    out, _ = orc.quantise_delayed(xs, orc.E4M3, history_len=2)
    for x, o in zip(xs, out):
        assert np.array_equal(o["q"], orc.cast(x, orc.E4M3, o["bias"]))
    # call 1 saturates: its largest magnitude clips to 448 (code 0x7E with the sign)
    q1 = out[1]["q"]
    assert (q1 & 0x7F).max() == 0x7E and orc.decode(orc.E4M3, int(q1[1 % 64])) in (448.0, -448.0)


def test_history_of_one_is_the_previous_calls_exact_bias():
    rng = np.random.default_rng(5)
    xs = [(rng.standard_normal(200) * 2.0 ** rng.integers(-12, 12)).astype(np.float32) for _ in range(12)]
    for fmt in (orc.E4M3, orc.E5M2):
        out, _ = orc.quantise_delayed(xs, fmt, history_len=1, bias0=3)
        assert out[0]["bias"] == 3
        for t in range(1, len(xs)):
            assert out[t]["bias"] == orc.scale_bias(xs[t - 1], fmt)[0]


def test_unchanged_tensor_gives_the_just_in_time_codes_after_one_call():
    x = tensor_with_amax(37.0, n=500, seed=9)
    exact, _, _ = orc.scale_bias(x, orc.E4M3)
    out, _ = orc.quantise_delayed([x] * 4, orc.E4M3, history_len=3)
    assert out[0]["bias"] == 0
    for o in out[1:]:
        assert o["bias"] == exact and o["flags"] == 0
        assert np.array_equal(o["q"], orc.cast(x, orc.E4M3, exact))


def test_largest_of_the_window_and_forgetting():
    # amax 64 then six tensors of amax 1, history of 4: the bias stays Eq. 3 of
    # 64 while 64 is among the last four calls, then returns to Eq. 3 of 1
    xs = [tensor_with_amax(64.0, seed=1)] + [tensor_with_amax(1.0, seed=i) for i in range(2, 8)]
    out, _ = orc.quantise_delayed(xs, orc.E4M3, history_len=4)
    b64, b1 = orc.bias_from_amax(0x42800000, orc.E4M3)[0], orc.bias_from_amax(0x3F800000, orc.E4M3)[0]
    assert (b64, b1) == (2, 8)
    assert [o["next_bias"] for o in out] == [b64, b64, b64, b64, b1, b1, b1]


def test_margin_and_flags():
    xs = [np.zeros(10, np.float32), tensor_with_amax(4.0), np.array([1.0, np.nan], np.float32),
          tensor_with_amax(4.0)]
    out, _ = orc.quantise_delayed(xs, orc.E5M2, margin=3, history_len=2)
    assert out[0]["flags"] == orc.FLAG_ZERO and out[0]["next_bias"] == 0      # zero history: bias 0
    assert out[1]["next_bias"] == orc.bias_from_amax(0x40800000, orc.E5M2)[0] - 3
    assert out[2]["flags"] == orc.FLAG_NONFINITE and out[2]["amax"] == 0x7FC00000
    assert out[2]["next_bias"] == 0                                           # NaN in the history
    assert out[3]["next_bias"] == 0                                           # still in the window


def test_history_max_orders_values_and_nan():
    assert orc.history_max([0x3F800000, 0x40000000, 0]) == 0x40000000
    assert orc.history_max([0x00000001, 0]) == 1
    assert orc.history_max([0x7F800000, 0x3F800000]) == 0x7F800000
    assert orc.history_max([0x3F800000, 0x7FC00000, 0x7F800000]) == 0x7FC00000
    assert orc.history_max([]) == 0
    with pytest.raises(ValueError):
        orc.quantise_delayed([], orc.E4M3, history_len=0)
