"""GPU parity of fp8_quantise (amax + Eq. 3 bias + scale-and-cast in one call)
against the oracle, with and without a predicted bias.

Bar: bit-exact (integer work) for the codes, their transpose, the bias, the
amax pattern and the flags, whatever the prediction: right, wrong by one or
many binades, out of range, absent, or the bias word itself (the steady
state of a training step).  Sec. 2.3 Eq. 3, Sec. 2.1 Eq. 1, App. A.
"""
import numpy as np
import pytest
import torch

from paper_2309_17224_amd import fp8lin as F
from parity_util import i32, np_bits, u32

pytestmark = pytest.mark.gpu

PRED_DELTAS = [None, 0, 1, -1, 7, -40, "huge", "alias"]


def oracle_expect(orc, x_cpu, fmt, margin=0):
    bits = np_bits(x_cpu)
    b, a, fl = orc.scale_bias(bits, fmt, margin)
    q, qT = orc.cast(bits, fmt, b, transpose=True)
    return b, a, fl, q, qT


def run_quantise(x_dev, fmt, pred, exact_bias, margin=0, want_q=True, want_qT=True, x_view=None):
    dev = x_dev.device
    bias = torch.zeros(1, dtype=torch.int32, device=dev)
    if pred is None:
        bias_pred = None
    elif pred == "alias":
        bias.fill_(exact_bias - 3)  # a stale value in the output word itself
        bias_pred = bias
    elif pred == "huge":
        bias_pred = torch.tensor([-(2**31) + 5], dtype=torch.int32, device=dev)
    else:
        bias_pred = torch.tensor([exact_bias + pred], dtype=torch.int32, device=dev)
    xv = x_dev if x_view is None else x_view
    rows, cols = xv.shape
    q = torch.full((rows, cols), 0xAB, dtype=torch.uint8, device=dev) if want_q else None
    qT = torch.full((cols, rows), 0xCD, dtype=torch.uint8, device=dev) if want_qT else None
    q, qT, b, a, fl = F.fp8_quantise(xv, fmt, margin, bias_pred=bias_pred, bias=bias, q=q, qT=qT,
                                     want_q=want_q, want_qT=want_qT)
    torch.cuda.synchronize()
    return (None if q is None else q.cpu().numpy(), None if qT is None else qT.cpu().numpy(),
            i32(b), u32(a), u32(fl))


def check(orc, x_cpu, fmt, dev, pred, margin=0):
    ob, oa, ofl, oq, oqT = oracle_expect(orc, x_cpu, fmt, margin)
    q, qT, b, a, fl = run_quantise(x_cpu.to(dev), fmt, pred, ob, margin)
    assert (b, fl, a) == (ob, ofl, oa)  # a NaN amax is 0x7FC00000 on both sides
    assert np.array_equal(q, oq), "codes differ"
    assert np.array_equal(qT, oqT), "transposed codes differ"


def bf16_from_bits(bits, shape) -> torch.Tensor:
    return torch.tensor(np.asarray(bits, dtype=np.uint16).view(np.int16)).view(torch.bfloat16).reshape(shape)


@pytest.mark.parametrize("pred", PRED_DELTAS)
@pytest.mark.parametrize("fmt", [0, 1])
@pytest.mark.parametrize("shape", [(1, 1), (128, 128), (300, 517), (1000, 64), (64, 1000), (7, 3)])
def test_quantise_predictions(orc, gpu, pred, fmt, shape):
    g = torch.Generator().manual_seed(shape[0] * 1000 + shape[1])
    x = (torch.randn(*shape, generator=g) * 2.0 ** (shape[1] % 9 - 4)).to(torch.bfloat16)
    check(orc, x, fmt, gpu, pred)


@pytest.mark.parametrize("pred", [None, 0, 2])
@pytest.mark.parametrize("fmt", [0, 1])
def test_quantise_fp32_input(orc, gpu, pred, fmt):
    g = torch.Generator().manual_seed(11)
    x = torch.randn(257, 390, generator=g) * 1e-30  # tiny values: large positive biases
    x[5, 7] = 3e-38
    check(orc, x, fmt, gpu, pred)


SPECIAL = {
    "zeros": [0] * 1000,
    "one_nan": [0x3F80] * 500 + [0x7FC1] + [0x3F80] * 499,
    "neg_inf": [0xFF80] + [0x4000] * 999,
    "subnormals": [0x0001, 0x8003, 0x0042, 0x807F] * 250,
    "amax_is_448": [0x43E0, 0x3F80] * 500,
}


@pytest.mark.parametrize("name", sorted(SPECIAL))
@pytest.mark.parametrize("pred", [None, 0, 5])
@pytest.mark.parametrize("fmt", [0, 1])
def test_quantise_special_tensors(orc, gpu, name, pred, fmt):
    check(orc, bf16_from_bits(SPECIAL[name], (40, 25)), fmt, gpu, pred)


@pytest.mark.parametrize("margin", [-3, 0, 3])
def test_quantise_margin(orc, gpu, margin):
    g = torch.Generator().manual_seed(3)
    x = (torch.randn(200, 300, generator=g) * 1e-3).to(torch.bfloat16)
    for pred in (None, 0, 1):
        check(orc, x, 1, gpu, pred, margin)


def test_quantise_strided_and_single_outputs(orc, gpu):
    g = torch.Generator().manual_seed(9)
    big = (torch.randn(300, 700, generator=g) * 5).to(torch.bfloat16)
    view_cpu = big[:, 37:37 + 500]
    ob, oa, ofl, oq, oqT = oracle_expect(orc, view_cpu.contiguous(), 0)
    dev_big = big.to(gpu)
    view = dev_big[:, 37:37 + 500]
    for pred in (None, 0, -2):
        q, qT, b, a, fl = run_quantise(dev_big, 0, pred, ob, x_view=view)
        assert (b, a, fl) == (ob, oa, ofl)
        assert np.array_equal(q, oq) and np.array_equal(qT, oqT)
        q, qT, b, _, _ = run_quantise(dev_big, 0, pred, ob, x_view=view, want_q=False)
        assert q is None and np.array_equal(qT, oqT) and b == ob
        q, qT, b, _, _ = run_quantise(dev_big, 0, pred, ob, x_view=view, want_qT=False)
        assert qT is None and np.array_equal(q, oq) and b == ob


def test_quantise_matches_two_pass_entry_points(gpu):
    """Same bytes as fp8_scale_bias followed by fp8_cast_e5 (the two-pass path)."""
    g = torch.Generator().manual_seed(21)
    x = (torch.randn(1024, 3000, generator=g) * 1e-4).to(torch.bfloat16).to(gpu)
    b2, a2, f2 = F.fp8_scale_bias(x, F.E5M2)
    q2, qT2 = F.fp8_cast_e5(x, b2, want_q=True, want_qT=True)
    bias = torch.zeros(1, dtype=torch.int32, device=gpu)
    for _ in range(3):  # steady state: the bias word predicts itself
        q, qT, b, a, fl = F.fp8_quantise(x, F.E5M2, bias_pred=bias, bias=bias, want_qT=True)
    torch.cuda.synchronize()
    assert torch.equal(q, q2) and torch.equal(qT, qT2)
    assert torch.equal(b, b2) and torch.equal(a, a2) and torch.equal(fl, f2)


def test_quantise_empty(gpu):
    x = torch.empty(0, 16, dtype=torch.bfloat16, device=gpu)
    bias = torch.full((1,), 77, dtype=torch.int32, device=gpu)
    _, _, b, a, fl = F.fp8_quantise(x, F.E4M3, bias_pred=bias, bias=bias, want_q=True, ws=None)
    torch.cuda.synchronize()
    assert (i32(b), u32(a), u32(fl)) == (0, 0, F.FLAG_ZERO)


def test_quantise_rejects_small_workspace(gpu):
    x = torch.ones(256, 256, dtype=torch.bfloat16, device=gpu)
    ws = torch.empty(8, dtype=torch.uint8, device=gpu)
    with pytest.raises(F.Fp8Error):
        F.fp8_quantise(x, F.E4M3, ws=ws)


def test_quantise_workspace_reused(orc, gpu):
    """One workspace across calls of different tensors and shapes (the steady
    state of a step reuses one per tensor): every call matches the oracle,
    whether its prediction is wrong (the first call, a new tensor) or right."""
    from paper_2309_17224_amd import workloads as wl
    ws = F.quantise_workspace(300, 1000, gpu)   # tiles of the largest shape
    bias = torch.zeros(1, dtype=torch.int32, device=gpu)
    for rows, cols, seed, std, fmt in ((300, 520, 1, 1.0, F.E4M3), (300, 520, 1, 1.0, F.E4M3),
                                       (64, 64, 2, 3e-3, F.E5M2), (129, 1000, 3, 40.0, F.E4M3),
                                       (129, 1000, 3, 40.0, F.E4M3)):
        x = wl.small(rows, cols, std, seed)
        ob, oa, ofl, oq, oqT = oracle_expect(orc, x, fmt)
        q, qT, b, a, fl = F.fp8_quantise(x.to(gpu), fmt, 0, bias_pred=bias, bias=bias, want_qT=True, ws=ws)
        torch.cuda.synchronize()
        assert (i32(b), u32(a), u32(fl)) == (ob, oa, ofl)
        assert np.array_equal(q.cpu().numpy(), oq) and np.array_equal(qT.cpu().numpy(), oqT)


@pytest.mark.parametrize("fmt", [F.E4M3, F.E5M2], ids=["e4", "e5"])
@pytest.mark.parametrize("preds", [None, (0, 0, 0, 0), (0, 2, -1, "alias")], ids=["none", "right", "mixed"])
def test_quantise_batch_equals_separate_calls(orc, gpu, fmt, preds):
    """fp8_quantise_batch over ragged, strided, codes-only and transposed-only
    tensors (and an empty one) gives, for each tensor, the oracle's bits and
    the bits of a separate fp8_quantise call, whatever its prediction."""
    from paper_2309_17224_amd import workloads as wl
    shapes = [(300, 520, 1.0, True, True), (129, 1000, 40.0, True, False), (64, 64, 3e-3, False, True),
              (200, 300, 0.5, True, True)]
    items, expect = [], []
    for k, (rows, cols, std, want_q, want_qT) in enumerate(shapes):
        x = wl.small(rows, cols, std, 10 + k)
        if k == 3:  # strided: the first 300 columns of a wider tensor
            wide = wl.small(rows, 320, std, 20).to(gpu)
            wide[:, :cols] = x.to(gpu)
            xd = wide[:, :cols]
        else:
            xd = x.to(gpu)
        ob, oa, ofl, oq, oqT = oracle_expect(orc, x, fmt)
        bias = torch.zeros(1, dtype=torch.int32, device=gpu)
        pred = None
        if preds is not None:
            p = preds[k]
            if p == "alias":
                bias.fill_(ob - 3)
                pred = bias
            else:
                pred = torch.tensor([ob + p], dtype=torch.int32, device=gpu)
        it = dict(x=xd, bias=bias, bias_pred=pred, amax_bits=torch.zeros(1, dtype=torch.int32, device=gpu),
                  flags=torch.zeros(1, dtype=torch.int32, device=gpu),
                  q=torch.empty((rows, cols), dtype=torch.uint8, device=gpu) if want_q else None,
                  qT=torch.empty((cols, rows), dtype=torch.uint8, device=gpu) if want_qT else None,
                  ws=F.quantise_workspace(rows, cols, gpu))
        items.append(it)
        expect.append((ob, oa, ofl, oq if want_q else None, oqT if want_qT else None))
    empty = dict(x=torch.empty((0, 8), dtype=torch.bfloat16, device=gpu),
                 bias=torch.full((1,), 9, dtype=torch.int32, device=gpu),
                 flags=torch.zeros(1, dtype=torch.int32, device=gpu),
                 q=torch.empty((0, 8), dtype=torch.uint8, device=gpu), ws=torch.empty(4, dtype=torch.uint8, device=gpu))
    F.fp8_quantise_batch(items[:2] + [empty], fmt)
    F.fp8_quantise_batch(items[2:], fmt)
    torch.cuda.synchronize()
    assert i32(empty["bias"]) == 0 and u32(empty["flags"]) == F.FLAG_ZERO
    for it, (ob, oa, ofl, oq, oqT) in zip(items, expect):
        assert (i32(it["bias"]), u32(it["amax_bits"]), u32(it["flags"])) == (ob, oa, ofl)
        if oq is not None:
            assert np.array_equal(it["q"].cpu().numpy(), oq)
        if oqT is not None:
            assert np.array_equal(it["qT"].cpu().numpy(), oqT)
        # the same call alone
        q, qT, b, a, fl = F.fp8_quantise(it["x"], fmt, 0, want_q=oq is not None, want_qT=oqT is not None)
        torch.cuda.synchronize()
        assert (i32(b), u32(a), u32(fl)) == (ob, oa, ofl)
        if oq is not None:
            assert torch.equal(q, it["q"])
        if oqT is not None:
            assert torch.equal(qT, it["qT"])


def test_quantise_batch_four_large_tensors(orc, gpu):
    """Four tensors whose tiles exceed the pass-2 workgroup cap each (a
    misprediction makes every tensor's finishing workgroups recast it)."""
    from paper_2309_17224_amd import workloads as wl
    items, ref = [], []
    for k, (rows, cols) in enumerate([(2048, 1024), (1024, 2304), (640, 3000), (4096, 512)]):
        x = wl.small(rows, cols, 1.0 + k, 30 + k)
        ob, oa, ofl, oq, oqT = oracle_expect(orc, x, F.E4M3)
        items.append(dict(x=x.to(gpu), bias=torch.zeros(1, dtype=torch.int32, device=gpu),
                          bias_pred=torch.tensor([ob + (k % 2)], dtype=torch.int32, device=gpu),
                          q=torch.empty((rows, cols), dtype=torch.uint8, device=gpu),
                          qT=torch.empty((cols, rows), dtype=torch.uint8, device=gpu),
                          ws=F.quantise_workspace(rows, cols, gpu)))
        ref.append((ob, oq, oqT))
    F.fp8_quantise_batch(items, F.E4M3)
    torch.cuda.synchronize()
    for it, (ob, oq, oqT) in zip(items, ref):
        assert i32(it["bias"]) == ob
        assert np.array_equal(it["q"].cpu().numpy(), oq) and np.array_equal(it["qT"].cpu().numpy(), oqT)
