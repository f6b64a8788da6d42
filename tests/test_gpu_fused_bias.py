"""fp8_linear_fwd_bias / fp8_linear_bwd_dx_bias: the matmul with the Eq. 3
bias of its output taken in the same launch (the last workgroup folds the
running maximum into amax, bias and flags).

Bar: bit-exact against the unfused calls (the matmul with its epilogue amax,
then fp8_bias_from_amax), for every format and margin, bf16 and fp32 outputs,
shapes that take the 256 x 256 kernel and shapes that fall back (M <= 32, K
not a multiple of 128); the workspace must be zero after every call.  Where
the product is exact (small integer codes), the oracle's product and bias are
the reference.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2309_17224_amd import fp8lin as F
from parity_util import i32, np_bits, u32

pytestmark = pytest.mark.gpu

SHAPES = [(256, 256, 128), (300, 520, 384), (1024, 768, 768), (2048, 4096, 1024),  # 256 x 256 kernel
          (16, 1024, 256), (130, 200, 100)]                                          # fallbacks
FMTS = [F.E4M3, F.E5M2, F.E4_A, F.E5_A]


def operands(gpu, M, N, K, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    x = (torch.randn(M, K, generator=g) * scale).to(torch.bfloat16).to(gpu)
    w = (torch.randn(N, K, generator=g) * 0.02).to(torch.bfloat16).to(gpu)
    x8, _, bx, _, _ = F.fp8_quantise(x, F.E4M3)
    w8t, _, bw, _, _ = F.fp8_quantise(w, F.E4M3)
    return x8, bx, w8t, bw


def unfused_fwd(x8, bx, w8t, bw, fmt, margin, out_dt):
    amax = torch.zeros(1, dtype=torch.int32, device=x8.device)
    y = F.fp8_linear_fwd(x8, bx, w8t, bw, out_dt=out_dt, y_amax_bits=amax)
    b, fl = F.fp8_bias_from_amax(amax, fmt, margin)
    return y, b, amax, fl


def bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


@pytest.mark.parametrize("shape", SHAPES, ids=str)
@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("out_dt", [F.DT_BF16, F.DT_F32])
def test_fwd_bias_matches_unfused(gpu, shape, fmt, out_dt):
    M, N, K = shape
    x8, bx, w8t, bw = operands(gpu, M, N, K, M * 7 + N + K)
    ws = F.bias_workspace(gpu)
    for margin in (0, 2):
        y0, b0, a0, f0 = unfused_fwd(x8, bx, w8t, bw, fmt, margin, out_dt)
        y, b, a, fl = F.fp8_linear_fwd_bias(x8, bx, w8t, bw, fmt, margin, out_dt=out_dt, ws=ws)
        torch.cuda.synchronize()
        assert torch.equal(bits(y), bits(y0))
        assert (i32(b), u32(a), u32(fl)) == (i32(b0), u32(a0), u32(f0)), f"margin {margin}"
        assert not ws.any(), "workspace not left zero"


@pytest.mark.parametrize("shape", [(512, 384, 640), (40, 256, 128), (1000, 300, 260), (4096, 1024, 2048)], ids=str)
@pytest.mark.parametrize("fmt", [F.E5M2, F.E5_A])
def test_dx_bias_matches_unfused(gpu, shape, fmt):
    M, N, K = shape  # dX [M, K] = dY8 [M, N] . W8 [K, N]^T
    g = torch.Generator().manual_seed(M + N)
    dy = (torch.randn(M, N, generator=g) * 1e-4).to(torch.bfloat16).to(gpu)
    w = (torch.randn(K, N, generator=g) * 0.02).to(torch.bfloat16).to(gpu)
    dy8, _, bg, _, _ = F.fp8_quantise(dy, F.E5M2)
    w8, _, bw, _, _ = F.fp8_quantise(w, F.E4M3)
    ws = F.bias_workspace(gpu)
    for margin in (0, 1, 3):
        amax = torch.zeros(1, dtype=torch.int32, device=gpu)
        dx0 = F.fp8_linear_bwd_dx(dy8, bg, w8, bw, dx_amax_bits=amax)
        b0, f0 = F.fp8_bias_from_amax(amax, fmt, margin)
        dx, b, a, fl = F.fp8_linear_bwd_dx_bias(dy8, bg, w8, bw, fmt, margin, ws=ws)
        torch.cuda.synchronize()
        assert torch.equal(dx.view(torch.int16), dx0.view(torch.int16))
        assert (i32(b), u32(a), u32(fl)) == (i32(b0), u32(amax), u32(f0))
        assert not ws.any()


def test_workspace_reuse_across_calls_and_shapes(gpu):
    """One workspace, calls of different sizes and magnitudes back to back on
    the stream: each call's bias is its own (nothing carried over)."""
    ws = F.bias_workspace(gpu)
    outs, refs = [], []
    for i, (M, N, K, scale) in enumerate([(2048, 2048, 512, 100.0), (512, 768, 256, 1e-3),
                                          (16, 512, 256, 5.0), (1024, 1024, 1024, 0.25)]):
        x8, bx, w8t, bw = operands(gpu, M, N, K, 100 + i, scale)
        refs.append(unfused_fwd(x8, bx, w8t, bw, F.E4M3, 0, F.DT_BF16))
        outs.append(F.fp8_linear_fwd_bias(x8, bx, w8t, bw, F.E4M3, 0, ws=ws))
    torch.cuda.synchronize()
    for (y0, b0, a0, f0), (y, b, a, fl) in zip(refs, outs):
        assert torch.equal(y.view(torch.int16), y0.view(torch.int16))
        assert (i32(b), u32(a), u32(fl)) == (i32(b0), u32(a0), u32(f0))
    assert not ws.any()


@pytest.mark.parametrize("shape", [(512, 512, 256), (16, 256, 128), (100, 64, 100)], ids=str)
def test_null_amax_and_flags(gpu, shape):
    """The C entry point with no amax or flags output (the fallback kernels
    then use the workspace as their atomic target and clear it again)."""
    M, N, K = shape
    x8, bx, w8t, bw = operands(gpu, M, N, K, 9)
    y0, b0, _, _ = unfused_fwd(x8, bx, w8t, bw, F.E5M2, 1, F.DT_BF16)
    y = torch.empty(M, N, dtype=torch.bfloat16, device=gpu)
    b = torch.zeros(1, dtype=torch.int32, device=gpu)
    ws = F.bias_workspace(gpu)
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    st = F.lib().fp8_linear_fwd_bias(p(x8), p(bx), p(w8t), p(bw), p(y), F.DT_BF16, M, N, K, F.E5M2, 1, p(b),
                                     None, None, p(ws), 8, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == F.OK
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y0.view(torch.int16)) and i32(b) == i32(b0)
    assert not ws.any()


def test_special_outputs(gpu):
    """All-zero product (bias 0, FLAG_ZERO) and a NaN code in X (NaN row of Y,
    FLAG_NONFINITE), on the 256 x 256 kernel and on a fallback."""
    ws = F.bias_workspace(gpu)
    for M, N, K in ((512, 512, 256), (20, 256, 128)):
        x8 = torch.zeros(M, K, dtype=torch.uint8, device=gpu)
        w8t = torch.full((N, K), 0x38, dtype=torch.uint8, device=gpu)
        z = torch.zeros(1, dtype=torch.int32, device=gpu)
        y, b, a, fl = F.fp8_linear_fwd_bias(x8, z, w8t, z, F.E4M3, ws=ws)
        torch.cuda.synchronize()
        assert (i32(b), u32(a), u32(fl)) == (0, 0, F.FLAG_ZERO)
        x8[3, 5] = 0x7F  # E4M3 NaN
        y0, b0, a0, f0 = unfused_fwd(x8, z, w8t, z, F.E4M3, 0, F.DT_BF16)
        y, b, a, fl = F.fp8_linear_fwd_bias(x8, z, w8t, z, F.E4M3, ws=ws)
        torch.cuda.synchronize()
        assert u32(fl) == F.FLAG_NONFINITE and (i32(b), u32(a), u32(fl)) == (i32(b0), u32(a0), u32(f0))
        assert torch.equal(y.view(torch.int16), y0.view(torch.int16))
        assert not ws.any()


def test_empty_output(gpu):
    ws = F.bias_workspace(gpu)
    x8 = torch.zeros(0, 128, dtype=torch.uint8, device=gpu)
    w8t = torch.zeros(64, 128, dtype=torch.uint8, device=gpu)
    z = torch.zeros(1, dtype=torch.int32, device=gpu)
    y, b, a, fl = F.fp8_linear_fwd_bias(x8, z, w8t, z, F.E4M3, ws=ws)
    torch.cuda.synchronize()
    assert (i32(b), u32(a), u32(fl)) == (0, 0, F.FLAG_ZERO)
    with pytest.raises(F.Fp8Error):
        F.fp8_linear_fwd_bias(x8, z, w8t, z, F.E4M3, ws=torch.zeros(1, dtype=torch.int32, device=gpu))


def test_against_oracle_on_exact_products(orc, gpu):
    """Codes from {0, +-1, +-2, +-3, +-4, +-6, +-8} with K < 2^14 give exact
    fp32 sums, so the oracle's product, amax and bias are the reference."""
    M, N, K = 768, 512, 384
    vals = np.array([0x00, 0x38, 0x40, 0x44, 0x48, 0x4C, 0x50], dtype=np.uint8)
    rng = np.random.default_rng(11)

    def codes(r, c):
        v = vals[rng.integers(0, len(vals), size=(r, c))]
        return (v | (rng.integers(0, 2, size=(r, c)).astype(np.uint8) << 7) * (v != 0)).astype(np.uint8)

    x8, w8t = codes(M, K), codes(N, K)
    bx, bw = 3, -1
    yref = orc.gemm_nt(x8, 0, bx, w8t, 0, bw, out_dt=orc.BF16)
    ws = F.bias_workspace(gpu)
    for fmt in FMTS:
        for margin in (0, 2):
            ob, oa, ofl = orc.scale_bias(yref, fmt, margin)
            y, b, a, fl = F.fp8_linear_fwd_bias(torch.from_numpy(x8).to(gpu),
                                                torch.tensor([bx], dtype=torch.int32, device=gpu),
                                                torch.from_numpy(w8t).to(gpu),
                                                torch.tensor([bw], dtype=torch.int32, device=gpu),
                                                fmt, margin, ws=ws)
            torch.cuda.synchronize()
            assert np.array_equal(np_bits(y), yref)
            assert (i32(b), u32(a), u32(fl)) == (ob, oa, ofl), (fmt, margin)
