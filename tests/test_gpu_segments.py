"""Per-segment FP8-AMAX (fp8_quantise_segments), the matmul with one
activation bias per row (fp8_linear_fwd_rows) and the bias-mode ring buffer
(fp8_bias_mode), against the oracle.

Bar: bit-exact (integer work: codes, transposed codes, biases, amax, flags,
row biases, modes); the per-row matmul bit-exact against the per-segment
fp8_linear_fwd calls and, on exact products, against the oracle.
"""
import numpy as np
import pytest
import torch

from paper_2309_17224_amd import fp8lin as F
from parity_util import i32, np_bits, u32

pytestmark = pytest.mark.gpu

LAYOUTS = {
    "one": lambda r: [0, r],
    "ragged": lambda r: sorted({0, r, *np.random.default_rng(r).integers(0, r, size=7).tolist()}),
    "with_empty": lambda r: [0, 0, r // 3, r // 3, r // 3 + 1, r, r],
    "many_small": lambda r: list(range(0, r, 5)) + [r],
}


def data(rows, cols, seed, dt):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(rows, cols, generator=g)
    # rows of very different magnitudes, so segments get different biases
    x = x * torch.pow(2.0, torch.randint(-8, 9, (rows, 1), generator=g).float())
    return x.to(torch.bfloat16) if dt == F.DT_BF16 else x


def host(x):
    return np_bits(x) if x.dtype == torch.bfloat16 else x.numpy()


@pytest.mark.parametrize("shape", [(300, 520), (1000, 64), (257, 1000), (64, 4096), (33, 7)], ids=str)
@pytest.mark.parametrize("layout", sorted(LAYOUTS))
@pytest.mark.parametrize("fmt", [F.E4M3, F.E5M2, F.E4_A, F.E5_A])
def test_segments_match_oracle(orc, gpu, shape, layout, fmt):
    rows, cols = shape
    off = LAYOUTS[layout](rows)
    for dt, margin in ((F.DT_BF16, 0), (F.DT_F32, 2)):
        x = data(rows, cols, rows + cols + fmt, dt)
        offsets = torch.tensor(off, dtype=torch.int32, device=gpu)
        q, qT, b, a, fl, rb = F.fp8_quantise_segments(x.to(gpu), offsets, fmt, margin, want_qT=True)
        torch.cuda.synchronize()
        oq, oqT, ob, oa, ofl, orb = orc.quantise_segments(host(x), off, fmt, margin)
        assert b.cpu().tolist() == ob and (a.cpu().numpy().view(np.uint32) == np.array(oa, dtype=np.uint32)).all()
        assert (fl.cpu().numpy().view(np.uint32) == np.array(ofl, dtype=np.uint32)).all()
        assert np.array_equal(rb.cpu().numpy(), orb)
        assert np.array_equal(q.cpu().numpy(), oq) and np.array_equal(qT.cpu().numpy(), oqT)


def test_one_segment_equals_whole_tensor_quantise(gpu):
    x = data(2048, 1536, 5, F.DT_BF16).to(gpu)
    offsets = torch.tensor([0, 2048], dtype=torch.int32, device=gpu)
    q, qT, b, a, fl, rb = F.fp8_quantise_segments(x, offsets, F.E4M3, want_qT=True)
    q0, qT0, b0, a0, f0 = F.fp8_quantise(x, F.E4M3, want_qT=True)
    torch.cuda.synchronize()
    assert (i32(b[0]), u32(a[0]), u32(fl[0])) == (i32(b0), u32(a0), u32(f0))
    assert torch.equal(q, q0) and torch.equal(qT, qT0) and bool((rb == b0).all())


def test_special_values_per_segment(orc, gpu):
    """A NaN in one segment, an all-zero segment, an infinity in another."""
    x = data(96, 40, 7, F.DT_BF16)
    x[5, 3] = float("nan")
    x.view(torch.int16)[6, 8] = 0x7FC5      # a NaN with a payload: the amax is still 0x7FC00000
    x[40:64] = 0
    x[70, 1] = float("-inf")
    x.view(torch.int16)[90, 2] = -93        # 0xFFA3: a negative NaN with a payload
    off = [0, 32, 40, 64, 96]
    q, qT, b, a, fl, rb = F.fp8_quantise_segments(x.to(gpu), torch.tensor(off, dtype=torch.int32, device=gpu),
                                                  F.E4M3, want_qT=True)
    torch.cuda.synchronize()
    oq, oqT, ob, oa, ofl, orb = orc.quantise_segments(np_bits(x), off, F.E4M3)
    assert b.cpu().tolist() == ob and (fl.cpu().numpy().view(np.uint32) == np.array(ofl, np.uint32)).all()
    assert ofl[0] == F.FLAG_NONFINITE and ofl[2] == F.FLAG_ZERO and ofl[3] == F.FLAG_NONFINITE
    assert oa[0] == 0x7FC00000 and oa[3] == 0x7FC00000
    assert (a.cpu().numpy().view(np.uint32) == np.array(oa, np.uint32)).all()
    assert np.array_equal(q.cpu().numpy(), oq) and np.array_equal(qT.cpu().numpy(), oqT)


@pytest.mark.parametrize("shape", [(300, 520, 384), (16, 1024, 256), (20, 512, 256), (100, 64, 100),
                                   (2048, 1024, 512), (12, 1000, 1024), (9, 96, 10240)], ids=str)
def test_fwd_rows_is_the_product_unscaled_per_row(gpu, shape):
    """Y of the per-row matmul is the same kernel's fp32 product S (taken with
    zero biases), unscaled row by row: Y[m] = round(S[m] * 2^-(rb[m] + bw)),
    on the 256 x 256, decode (both staged row counts and the fragment-loading
    kernel) and fallback kernels; and its epilogue amax."""
    M, N, K = shape
    x = data(M, K, M + K, F.DT_BF16).to(gpu)
    g = torch.Generator().manual_seed(N)
    w = (torch.randn(N, K, generator=g) * 0.02).to(torch.bfloat16).to(gpu)
    w8t, _, bw, _, _ = F.fp8_quantise(w, F.E4M3)
    off = sorted({0, M, M // 3, M // 2, M // 2 + 1, 7 % M})
    offsets = torch.tensor(off, dtype=torch.int32, device=gpu)
    x8, _, b, a, fl, rb = F.fp8_quantise_segments(x, offsets, F.E4M3)
    zero = torch.zeros(1, dtype=torch.int32, device=gpu)
    S = F.fp8_linear_fwd(x8, zero, w8t, zero, out_dt=F.DT_F32)
    torch.cuda.synchronize()
    sh = -(rb.cpu().to(torch.int32) + int(bw.cpu()))
    expect = torch.ldexp(S.cpu(), sh[:, None].float())
    for out_dt in (F.DT_BF16, F.DT_F32):
        amax = torch.zeros(1, dtype=torch.int32, device=gpu)
        y = F.fp8_linear_fwd_rows(x8, rb, w8t, bw, out_dt=out_dt, y_amax_bits=amax)
        torch.cuda.synchronize()
        if out_dt == F.DT_BF16:
            assert torch.equal(y.cpu().view(torch.int16), expect.to(torch.bfloat16).view(torch.int16))
        else:
            assert torch.equal(y.cpu().view(torch.int32), expect.view(torch.int32))
        got = torch.tensor([u32(amax)], dtype=torch.int64).to(torch.int32).view(torch.float32)
        assert float(got) == float(y.float().abs().max())


def test_fwd_rows_against_oracle_on_exact_products(orc, gpu):
    vals = np.array([0x00, 0x38, 0x40, 0x44, 0x48, 0x4C, 0x50], dtype=np.uint8)
    rng = np.random.default_rng(12)

    def codes(r, c):
        v = vals[rng.integers(0, len(vals), size=(r, c))]
        return (v | (rng.integers(0, 2, size=(r, c)).astype(np.uint8) << 7) * (v != 0)).astype(np.uint8)

    for M, K in ((300, 256), (20, 256), (12, 512)):
        N = 512
        x8, w8t = codes(M, K), codes(N, K)
        rows_b = (np.arange(M) % 9 - 4).astype(np.int32)
        yref = orc.gemm_nt_rows(x8, 0, rows_b, w8t, 0, 1, out_dt=orc.BF16)
        y = F.fp8_linear_fwd_rows(torch.from_numpy(x8).to(gpu), torch.from_numpy(rows_b).to(gpu),
                                  torch.from_numpy(w8t).to(gpu), torch.tensor([1], dtype=torch.int32, device=gpu))
        torch.cuda.synchronize()
        assert np.array_equal(np_bits(y), yref)


def test_bias_mode_ring(orc, gpu):
    rng = np.random.default_rng(3)
    cases = [rng.integers(-5, 30, size=1000), np.array([4, 4, 9, 9, 2]), np.array([7]),
             np.array([-3000, -3000, 12]), rng.integers(-200, 200, size=70000)]
    ring = torch.full((3,), -777, dtype=torch.int32, device=gpu)
    count = torch.zeros(1, dtype=torch.int32, device=gpu)
    expect = []
    for c in cases:
        F.fp8_bias_mode(torch.from_numpy(c.astype(np.int32)).to(gpu), ring, count)
        expect.append(orc.bias_mode(c.tolist()))
    torch.cuda.synchronize()
    assert i32(count) == len(cases)
    got = ring.cpu().tolist()
    for i, e in enumerate(expect[-3:], start=len(cases) - 3):
        assert got[i % 3] == e, (i, got, expect)
