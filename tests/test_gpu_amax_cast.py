"""GPU parity of amax, scaling bias and scale-and-cast against the oracle.

Bar: bit-exact (integer work).  Calls go through the C ABI (ctypes binding);
the oracle receives the same bytes.  Sec. 2.3 Eq. 3 (amax, bias), Sec. 2.1
Eq. 1 (scale), App. A (clip), App. B (special values).
"""
import numpy as np
import pytest
import torch

from paper_2309_17224_amd import fp8lin as F
from paper_2309_17224_amd import workloads as wl
from parity_util import i32, np_bits, u32

pytestmark = pytest.mark.gpu


def gpu_bias(x_dev, fmt, margin=0):
    b, a, fl = F.fp8_scale_bias(x_dev, fmt, margin)
    torch.cuda.synchronize()
    return i32(b), u32(a), u32(fl)


def check_bias(orc, x_cpu, fmt, dev, margin=0):
    ob, oa, ofl = orc.scale_bias(np_bits(x_cpu), fmt, margin)
    gb, ga, gfl = gpu_bias(x_cpu.to(dev), fmt, margin)
    assert (gb, gfl, ga) == (ob, ofl, oa)  # a NaN amax is 0x7FC00000 on both sides
    return gb


def bf16_from_bits(bits) -> torch.Tensor:
    return torch.tensor(np.asarray(bits, dtype=np.uint16).view(np.int16)).view(torch.bfloat16)


# ------------------------------------------------------------------ amax / bias
SPECIAL = {
    "zeros": bf16_from_bits([0] * 1000),
    "neg_zero": bf16_from_bits([0x8000] * 37),
    "one_nan": bf16_from_bits([0x3F80] * 500 + [0x7FC1] + [0x3F80] * 10),
    "pos_inf": bf16_from_bits([0x3F80] * 100 + [0x7F80]),
    "neg_inf": bf16_from_bits([0xFF80] + [0x4000] * 3000),
    "subnormals": bf16_from_bits([0x0001, 0x8003, 0x0042, 0x807F] * 333),
    "pow2_amax": bf16_from_bits([0x4100, 0xC100, 0x3F00]),          # 8, -8, 0.5
    "amax_is_448": bf16_from_bits([0x43E0, 0x3F80]),                # 448
    "amax_is_57344": bf16_from_bits([0x4760, 0x3F80]),              # 57344
    "single": bf16_from_bits([0xBC00]),
    "bf16_max": bf16_from_bits([0x7F7F, 0x0001]),
}


@pytest.mark.parametrize("name", sorted(SPECIAL))
@pytest.mark.parametrize("fmt", [0, 1])
def test_bias_special_tensors(orc, gpu, name, fmt):
    check_bias(orc, SPECIAL[name], fmt, gpu)


@pytest.mark.parametrize("n", [1, 2, 7, 8, 9, 15, 16, 17, 255, 1000, 8191, 8192, 8193, 100_003,
                               3_000_017])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_bias_lengths_and_dtypes(orc, gpu, n, dtype):
    g = torch.Generator().manual_seed(n)
    x = (torch.randn(n, generator=g) * 3.7).to(dtype)
    # put the maximum at a position that exercises the tail
    x[-1] = 1000.0
    for fmt in (0, 1):
        check_bias(orc, x, fmt, gpu)


def test_bias_unaligned_pointer(orc, gpu):
    g = torch.Generator().manual_seed(5)
    base = torch.randn(4097, generator=g).to(torch.bfloat16)
    dev = base.to(gpu)
    for off in (1, 3, 5):
        x = dev[off:]
        assert x.data_ptr() % 16 != 0
        ob, oa, ofl = orc.scale_bias(np_bits(base[off:]), 0)
        assert gpu_bias(x, 0) == (ob, oa, ofl)


@pytest.mark.parametrize("margin", [-2, 0, 3, 5])
def test_bias_margin(orc, gpu, margin):
    x = wl.small(64, 96, std=1e-3, seed=1)
    check_bias(orc, x, 1, gpu, margin)


def test_bias_from_amax_entry(orc, gpu):
    vals = [0x3F800000, 0x43E00000, 0x43E08000, 0x00000001, 0x7F7FFFFF, 0, 0x7F800000, 0x7FC00000,
            0x3DCCCCCD, 0x00800000, 0x007FFFFF]
    for fmt in (0, 1):
        for margin in (0, 3):
            for v in vals:
                a = torch.tensor([v], dtype=torch.int64).to(torch.int32).to(gpu)
                b, fl = F.fp8_bias_from_amax(a, fmt, margin)
                torch.cuda.synchronize()
                assert (i32(b), u32(fl)) == orc.bias_from_amax(v, fmt, margin)


def test_empty_tensor_bias(orc, gpu):
    x = torch.empty(0, dtype=torch.bfloat16, device=gpu)
    b, a, fl = F.fp8_scale_bias(x, 0)
    torch.cuda.synchronize()
    assert (i32(b), u32(a), u32(fl)) == (0, 0, F.FLAG_ZERO)


# ------------------------------------------------------------------ cast
def gpu_cast(x_dev, fmt, bias_val, want_qT=True):
    b = torch.tensor([bias_val], dtype=torch.int32, device=x_dev.device)
    fn = F.fp8_cast_e4 if fmt == 0 else F.fp8_cast_e5
    q, qT = fn(x_dev, b, want_qT=want_qT)
    torch.cuda.synchronize()
    return q.cpu().numpy(), (qT.cpu().numpy() if qT is not None else None)


@pytest.mark.parametrize("fmt", [0, 1])
def test_cast_every_bf16_pattern(orc, gpu, fmt):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(256, 256)
    x = bf16_from_bits(bits.ravel()).reshape(256, 256)
    xd = x.to(gpu)
    for bias in (-140, -30, -9, 0, 1, 7, 15, 23, 40, 133, 157, 600, -600):
        q, qT = gpu_cast(xd, fmt, bias)
        ref = orc.cast(bits, fmt, bias)
        assert np.array_equal(q, ref), (fmt, bias, np.argwhere(q != ref)[:4])
        assert np.array_equal(qT, ref.T)


@pytest.mark.parametrize("fmt", [0, 1])
def test_cast_fp32_patterns(orc, gpu, fmt):
    rng = np.random.default_rng(fmt)
    u = rng.integers(0, 2 ** 32, size=(300, 257), dtype=np.uint64).astype(np.uint32)
    u[0, :8] = [0x7F800000, 0xFF800000, 0x7FC00000, 0xFFC00001, 0, 0x80000000, 1, 0x80000001]
    x = u.view(np.float32)
    xd = torch.from_numpy(x.copy()).to(gpu)
    for bias in (-150, -20, 0, 9, 30, 150):
        q, qT = gpu_cast(xd, fmt, bias)
        ref = orc.cast(x, fmt, bias)
        assert np.array_equal(q, ref)
        assert np.array_equal(qT, ref.T)
    # around the FP8 range
    y = (rng.standard_normal((129, 1000)) * np.exp2(rng.uniform(-25, 12, (129, 1000)))).astype(np.float32)
    q, qT = gpu_cast(torch.from_numpy(y).to(gpu), fmt, 0)
    assert np.array_equal(q, orc.cast(y, fmt, 0))


SHAPES = [(1, 1), (1, 7), (3, 5), (4, 8), (17, 129), (64, 128), (65, 127), (100, 300), (129, 255),
          (255, 1000), (1000, 17)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "%dx%d" % s)
@pytest.mark.parametrize("fmt", [0, 1])
def test_cast_ragged_shapes(orc, gpu, shape, fmt):
    x = wl.small(*shape, std=2.0, seed=shape[0] * 1000 + shape[1])
    bias = check_bias(orc, x, fmt, gpu)
    q, qT = gpu_cast(x.to(gpu), fmt, bias)
    ref, refT = orc.cast(np_bits(x), fmt, bias, transpose=True)
    assert np.array_equal(q, ref)
    assert np.array_equal(qT, refT)


def test_cast_strided_input_and_outputs(orc, gpu):
    base = wl.small(70, 300, seed=9)
    x = base[3:67, 5:250]                       # row stride 300, unaligned start
    bits = np_bits(x.contiguous())
    bias = torch.tensor([4], dtype=torch.int32, device=gpu)
    xd = base.to(gpu)[3:67, 5:250]
    qbuf = torch.zeros((64, 260), dtype=torch.uint8, device=gpu)
    qTbuf = torch.zeros((245, 80), dtype=torch.uint8, device=gpu)
    q, qT = F.fp8_cast_e4(xd, bias, q=qbuf[:, :245], qT=qTbuf[:, :64])
    torch.cuda.synchronize()
    ref, refT = orc.cast(bits, 0, 4, transpose=True)
    assert np.array_equal(qbuf[:, :245].cpu().numpy(), ref)
    assert np.array_equal(qTbuf[:, :64].cpu().numpy(), refT)
    assert int(qbuf[:, 245:].abs().sum()) == 0 and int(qTbuf[:, 64:].abs().sum()) == 0


def test_cast_only_transposed_output(orc, gpu):
    x = wl.small(96, 160, seed=2)
    b = torch.tensor([3], dtype=torch.int32, device=gpu)
    q, qT = F.fp8_cast_e5(x.to(gpu), b, want_q=False, want_qT=True)
    torch.cuda.synchronize()
    assert q is None
    assert np.array_equal(qT.cpu().numpy(), orc.cast(np_bits(x), 1, 3).T)


def test_cast_is_deterministic(gpu):
    x = wl.small(333, 777, seed=4).to(gpu)
    b = torch.tensor([6], dtype=torch.int32, device=gpu)
    q1, t1 = F.fp8_cast_e4(x, b, want_qT=True)
    q2, t2 = F.fp8_cast_e4(x, b, want_qT=True)
    torch.cuda.synchronize()
    assert torch.equal(q1, q2) and torch.equal(t1, t2)
