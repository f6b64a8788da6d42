"""The matmul epilogue's fused quantise (fp8_linear_fwd_quantise,
fp8_linear_bwd_dx_quantise): bias, amax, flags and the codes (and transposed
codes) of the bf16 output, for the next layer.

Bar: bit-exact against the unfused calls (the matmul, then fp8_quantise on
its output, itself bit-exact against the oracle), for predictions that hold,
miss, are absent or alias the bias word, in every FP8 format, on shapes that
take the fused 256x256 kernel and on shapes that fall back (M <= 32, K not a
multiple of 128).  Where the product is exact (small integer codes), the
oracle's own product, quantised by the oracle, is the reference.
"""
import numpy as np
import pytest
import torch

from paper_2309_17224_amd import fp8lin as F
from parity_util import i32, np_bits, u32

pytestmark = pytest.mark.gpu

SHAPES = [(256, 256, 128), (300, 520, 384), (1024, 768, 768), (2048, 4096, 1024),  # fused
          (16, 1024, 256), (130, 200, 100)]                                          # fallback
PREDS = [None, 0, 1, -3, "alias"]


def operands(gpu, M, N, K, seed):
    g = torch.Generator().manual_seed(seed)
    x = (torch.randn(M, K, generator=g)).to(torch.bfloat16).to(gpu)
    w = (torch.randn(N, K, generator=g) * 0.02).to(torch.bfloat16).to(gpu)
    x8, _, bx, _, _ = F.fp8_quantise(x, F.E4M3)
    w8t, _, bw, _, _ = F.fp8_quantise(w, F.E4M3)
    return x8, bx, w8t, bw


def reference(x8, bx, w8t, bw, fmt, margin):
    y = F.fp8_linear_fwd(x8, bx, w8t, bw)
    q, qT, b, a, fl = F.fp8_quantise(y, fmt, margin, want_qT=True)
    return y, q, qT, b, a, fl


def pred_tensors(gpu, pred, exact):
    bias = torch.zeros(1, dtype=torch.int32, device=gpu)
    if pred is None:
        return None, bias
    if pred == "alias":
        bias.fill_(exact - 2)
        return bias, bias
    return torch.tensor([exact + pred], dtype=torch.int32, device=gpu), bias


@pytest.mark.parametrize("shape", SHAPES, ids=str)
@pytest.mark.parametrize("pred", PREDS, ids=str)
@pytest.mark.parametrize("fmt", [F.E4M3, F.E5M2, F.E4_A, F.E5_A])
def test_fwd_fused_quantise_matches_unfused(gpu, shape, pred, fmt):
    M, N, K = shape
    x8, bx, w8t, bw = operands(gpu, M, N, K, M + N + K)
    y0, q0, qT0, b0, a0, f0 = reference(x8, bx, w8t, bw, fmt, 0)
    torch.cuda.synchronize()
    bp, bias = pred_tensors(gpu, pred, i32(b0))
    y, q, qT, b, a, fl = F.fp8_linear_fwd_quantise(x8, bx, w8t, bw, fmt, 0, bias_pred=bp, bias=bias,
                                                   want_y8t=True)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y0.view(torch.int16))
    assert (i32(b), u32(a), u32(fl)) == (i32(b0), u32(a0), u32(f0))
    assert torch.equal(q, q0), "codes differ"
    assert torch.equal(qT, qT0), "transposed codes differ"


@pytest.mark.parametrize("shape", [(512, 384, 640), (40, 256, 128), (1000, 300, 260)], ids=str)
@pytest.mark.parametrize("pred", [None, 0, 2], ids=str)
def test_dx_fused_quantise_matches_unfused(gpu, shape, pred):
    M, N, K = shape  # dX [M, K] = dY8 [M, N] . W8 [K, N]^T
    g = torch.Generator().manual_seed(M * N)
    dy = (torch.randn(M, N, generator=g) * 1e-4).to(torch.bfloat16).to(gpu)
    w = (torch.randn(K, N, generator=g) * 0.02).to(torch.bfloat16).to(gpu)
    dy8, _, bg, _, _ = F.fp8_quantise(dy, F.E5M2)
    w8, _, bw, _, _ = F.fp8_quantise(w, F.E4M3)
    dx0 = F.fp8_linear_bwd_dx(dy8, bg, w8, bw)
    q0, qT0, b0, a0, f0 = F.fp8_quantise(dx0, F.E5M2, 1, want_qT=True)
    torch.cuda.synchronize()
    bp, bias = pred_tensors(gpu, pred, i32(b0))
    dx, q, qT, b, a, fl = F.fp8_linear_bwd_dx_quantise(dy8, bg, w8, bw, F.E5M2, 1, bias_pred=bp, bias=bias,
                                                       want_dx8t=True)
    torch.cuda.synchronize()
    assert torch.equal(dx.view(torch.int16), dx0.view(torch.int16))
    assert (i32(b), u32(a), u32(fl)) == (i32(b0), u32(a0), u32(f0))
    assert torch.equal(q, q0) and torch.equal(qT, qT0)


def test_fused_quantise_against_oracle_on_exact_products(orc, gpu):
    """Codes from {0, +-1, +-2, +-3, +-4, +-6, +-8} with K < 2^14 give exact
    fp32 sums, so the oracle's product is the GPU's, and the oracle's bias and
    cast of it are the reference for the fused epilogue."""
    M, N, K = 384, 512, 256
    vals = np.array([0x00, 0x38, 0x40, 0x44, 0x48, 0x4C, 0x50], dtype=np.uint8)  # E4M3 0,1,2,3,4,6,8
    rng = np.random.default_rng(5)
    def codes(r, c):
        v = vals[rng.integers(0, len(vals), size=(r, c))]
        return (v | (rng.integers(0, 2, size=(r, c)).astype(np.uint8) << 7) * (v != 0)).astype(np.uint8)
    x8, w8t = codes(M, K), codes(N, K)
    bx = bw = 2
    yref = orc.gemm_nt(x8, 0, bx, w8t, 0, bw, out_dt=orc.BF16)
    for fmt in (F.E4M3, F.E5M2, F.E4_A):
        ob, oa, ofl = orc.scale_bias(yref, fmt)
        oq, oqT = orc.cast(yref, fmt, ob, transpose=True)
        dx8 = torch.from_numpy(x8).to(gpu)
        dw8t = torch.from_numpy(w8t).to(gpu)
        b2 = torch.tensor([bx], dtype=torch.int32, device=gpu)
        pred = torch.tensor([ob + 1], dtype=torch.int32, device=gpu)
        y, q, qT, b, a, fl = F.fp8_linear_fwd_quantise(dx8, b2, dw8t, b2, fmt, bias_pred=pred, want_y8t=True)
        torch.cuda.synchronize()
        assert np.array_equal(np_bits(y), yref)
        assert (i32(b), u32(a), u32(fl)) == (ob, oa, ofl)
        assert np.array_equal(q.cpu().numpy(), oq) and np.array_equal(qT.cpu().numpy(), oqT)


def test_fused_quantise_empty_and_rejects(gpu):
    x8 = torch.zeros(0, 128, dtype=torch.uint8, device=gpu)
    w8t = torch.zeros(64, 128, dtype=torch.uint8, device=gpu)
    z = torch.zeros(1, dtype=torch.int32, device=gpu)
    y, q, qT, b, a, fl = F.fp8_linear_fwd_quantise(x8, z, w8t, z, F.E4M3)
    torch.cuda.synchronize()
    assert (i32(b), u32(a), u32(fl)) == (0, 0, F.FLAG_ZERO)
    x8 = torch.zeros(256, 128, dtype=torch.uint8, device=gpu)
    with pytest.raises(F.Fp8Error):
        F.fp8_linear_fwd_quantise(x8, z, w8t, z, F.E4M3, ws=torch.empty(4, dtype=torch.uint8, device=gpu))
