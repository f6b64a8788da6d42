"""GPU parity of the three FP8 matmuls (forward, grad-input, grad-weight)
against the oracle's fp64-accumulated result (Sec. 2, 2.2; Eq. 2).

Bar: rel_F = ||Y - Y_ref||_F / ||Y_ref||_F <= 1e-3 with Y_ref rounded to the
same output type; bit-for-bit where every partial sum is exact in fp32.
"""
import numpy as np
import pytest
import torch

from paper_2309_17224_amd import fp8lin as F
from parity_util import REL_F_TOL, i32, np_bits, rel_f, u32

pytestmark = pytest.mark.gpu

ODT = {F.DT_BF16: torch.bfloat16, F.DT_F32: torch.float32}


def rand_codes(shape, fmt, rng, orc):
    """Random finite FP8 codes (uniform over codes, so all binades appear)."""
    tab = orc.decode_table(fmt)
    ok = np.nonzero(np.isfinite(tab))[0].astype(np.uint8)
    return rng.choice(ok, size=shape)


def run_nt(entry, A, fa, ba, B, fb, bb, out_dt, gpu, M, N, K, amax=False):
    """Call one entry point on operands A [M,K], B [N,K] given in NT form."""
    dev = gpu
    ta = torch.from_numpy(np.ascontiguousarray(A)).to(dev)
    tb = torch.from_numpy(np.ascontiguousarray(B)).to(dev)
    pa = torch.tensor([ba], dtype=torch.int32, device=dev)
    pb = torch.tensor([bb], dtype=torch.int32, device=dev)
    am = torch.zeros(1, dtype=torch.int32, device=dev) if amax else None
    if entry == "fwd":      # Y[M,N] = X8[M,K] . W8T[N,K]^T
        out = F.fp8_linear_fwd(ta, pa, tb, pb, out_dt=out_dt, y_amax_bits=am)
    elif entry == "dx":     # dX[M,K'] = dY8[M,N'] . W8[K',N']^T: here N' = K, K' = N
        out = F.fp8_linear_bwd_dx(ta, pa, tb, pb, out_dt=out_dt, dx_amax_bits=am)
    else:                   # dW[K',N'] = X8T[K',M'] . dY8T[N',M']^T: K' = M, M' = K
        out = F.fp8_linear_bwd_dw(ta, pa, tb, pb, out_dt=out_dt)
    torch.cuda.synchronize()
    return np_bits(out), (u32(am) if amax else None)


ENTRY_FMTS = {"fwd": (0, 0), "dx": (1, 0), "dw": (0, 1)}
SHAPES = [(1, 1, 128), (16, 16, 128), (256, 256, 256), (300, 200, 384), (17, 129, 1000),
          (255, 1, 17), (1, 255, 640), (129, 257, 128), (513, 300, 512), (64, 64, 0), (5, 70, 1024),
          (300, 200, 400), (65, 257, 144), (40, 33, 16)]


def scaled_normal_codes(shape, fmt, rng, orc):
    """Codes as the method produces them: N(0,1) data, AMAX bias, cast."""
    x = (rng.standard_normal(shape) * np.exp2(rng.uniform(-8, 8))).astype(np.float32)
    b, _, _ = orc.scale_bias(x, fmt)
    return orc.cast(x, fmt, b), b


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "%dx%dx%d" % s)
@pytest.mark.parametrize("entry", ["fwd", "dx", "dw"])
@pytest.mark.parametrize("out_dt", [F.DT_BF16, F.DT_F32], ids=["bf16", "f32"])
def test_gemm_scaled_normal_codes(orc, gpu, shape, entry, out_dt):
    """The parity bar, rel_F <= 1e-3, on operands distributed as the method
    produces them (AMAX-scaled normal tensors cast to FP8)."""
    M, N, K = shape
    fa, fb = ENTRY_FMTS[entry]
    rng = np.random.default_rng(M * 7 + N * 11 + K)
    A, ba = scaled_normal_codes((M, K), fa, rng, orc)
    B, bb = scaled_normal_codes((N, K), fb, rng, orc)
    got, _ = run_nt(entry, A, fa, ba, B, fb, bb, out_dt, gpu, M, N, K)
    ref = orc.gemm_nt(A, fa, ba, B, fb, bb, out_dt=out_dt)
    assert got.shape == (M, N)
    assert rel_f(got, ref) <= REL_F_TOL


# Elementwise bound for arbitrary codes.  The matrix core sums each group of
# 16 products of a 16x16x128 instruction keeping about 13 significant bits
# relative to the group's largest product (measured on gfx950: 65536 + 4 -> 65536
# inside a group, exact across groups and across instructions, which add in
# fp32).  Summed over groups this gives |err| of about 2^-13 sum_k |a_k b_k| per
# output before the unscale; the largest ratio measured over these cases is
# 2^-11.88 (forward, 255 x 1 x 17), and the test allows 2^-11.
ELEM_BOUND = 2.0 ** -11


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "%dx%dx%d" % s)
@pytest.mark.parametrize("entry", ["fwd", "dx", "dw"])
def test_gemm_uniform_codes_elementwise_bound(orc, gpu, shape, entry):
    """Codes drawn uniformly over every finite value (36 binades of product
    magnitudes, heavy cancellation): elementwise bound relative to the sum of
    absolute products, fp32 output."""
    M, N, K = shape
    fa, fb = ENTRY_FMTS[entry]
    rng = np.random.default_rng(M * 7 + N * 11 + K + 1)
    A = rand_codes((M, K), fa, rng, orc)
    B = rand_codes((N, K), fb, rng, orc)
    ba, bb = 9, 14 if fb == 1 else 6
    got, _ = run_nt(entry, A, fa, ba, B, fb, bb, F.DT_F32, gpu, M, N, K)
    ref = orc.gemm_nt(A, fa, ba, B, fb, bb, out_dt=orc.F32).astype(np.float64)
    da, db = np.abs(orc.decode_table(fa)[A]), np.abs(orc.decode_table(fb)[B])
    absum = (da @ db.T) * 2.0 ** -(ba + bb)
    err = np.abs(got.astype(np.float64) - ref)
    ratio = float((err / np.maximum(absum, 1e-300)).max()) if err.size else 0.0
    print(f"\n[uniform codes] {entry} {shape}: max err/sum|ab| = 2^{np.log2(max(ratio, 1e-300)):.2f}, "
          f"rel_F = {rel_f(got, ref.astype(np.float32)):.3e}", flush=True)
    assert (err <= ELEM_BOUND * absum + 1e-38).all()


@pytest.mark.parametrize("shape", [(16, 16, 128), (256, 512, 1024), (77, 300, 2048), (300, 77, 333)],
                         ids=lambda s: "%dx%dx%d" % s)
@pytest.mark.parametrize("entry", ["fwd", "dx", "dw"])
def test_gemm_exact_small_integers_bit_for_bit(orc, gpu, shape, entry):
    # Values in {0, +-1, ..., +-8} are exact in E4M3 and E5M2 and every
    # partial sum stays an integer below 2^24: the fp32 result is unique.
    M, N, K = shape
    fa, fb = ENTRY_FMTS[entry]
    vals = [0, 1, 2, 3, 4, 6, 8, -1, -2, -3, -4, -6, -8]
    ca = np.array([orc.encode(fa, v) for v in vals], dtype=np.uint8)
    cb = np.array([orc.encode(fb, v) for v in vals], dtype=np.uint8)
    rng = np.random.default_rng(K)
    ia = rng.integers(0, len(vals), (M, K))
    ib = rng.integers(0, len(vals), (N, K))
    got, _ = run_nt(entry, ca[ia], fa, 0, cb[ib], fb, 0, F.DT_F32, gpu, M, N, K)
    v = np.array(vals, dtype=np.int64)
    exact = (v[ia] @ v[ib].T).astype(np.float32)
    assert np.array_equal(got, exact)
    # the unscale is an exact power of two
    got2, _ = run_nt(entry, ca[ia], fa, 3, cb[ib], fb, -1, F.DT_F32, gpu, M, N, K)
    assert np.array_equal(got2, exact / 4)


@pytest.mark.parametrize("out_dt", [F.DT_BF16, F.DT_F32], ids=["bf16", "f32"])
def test_epilogue_amax(orc, gpu, out_dt):
    M, N, K = 300, 520, 256
    rng = np.random.default_rng(3)
    A = rand_codes((M, K), 0, rng, orc)
    B = rand_codes((N, K), 0, rng, orc)
    got, amax = run_nt("fwd", A, 0, 10, B, 0, 10, out_dt, gpu, M, N, K, amax=True)
    mag = np.abs(got.astype(np.uint16) & 0x7FFF).astype(np.uint32) << 16 if out_dt == F.DT_BF16 \
        else got.view(np.uint32) & 0x7FFFFFFF
    assert amax == int(mag.max())
    # its bias equals the oracle's bias of the output tensor
    ob, oa, ofl = orc.scale_bias(got, 0)
    assert oa == amax
    a = torch.tensor([amax], dtype=torch.int64).to(torch.int32).to(gpu)
    b, fl = F.fp8_bias_from_amax(a, 0)
    torch.cuda.synchronize()
    assert (i32(b), u32(fl)) == (ob, ofl)
    gotdx, amax_dx = run_nt("dx", rand_codes((M, K), 1, rng, orc), 1, 20, B, 0, 10, out_dt, gpu,
                            M, N, K, amax=True)
    _, oa2, _ = orc.scale_bias(gotdx, 1)
    assert amax_dx == oa2


# Shapes of the 256 x 256 kernel (with and without a narrow last round), the
# decode kernels and the byte-load kernel (K not a multiple of 128).
NAN_SHAPES = [(300, 520, 256), (512, 700, 384), (16, 640, 512), (24, 100, 256), (40, 90, 200)]


@pytest.mark.parametrize("shape", NAN_SHAPES, ids=lambda s: "%dx%dx%d" % s)
@pytest.mark.parametrize("out_dt", [F.DT_BF16, F.DT_F32], ids=["bf16", "f32"])
def test_epilogue_amax_of_nan_output_is_canonical(orc, gpu, shape, out_dt):
    """A NaN code in an operand makes outputs NaN; their amax, through the
    epilogue atomics and through the in-launch bias, is 0x7FC00000 with
    FP8_FLAG_NONFINITE and bias 0, the oracle's amax of a tensor holding NaN."""
    M, N, K = shape
    rng = np.random.default_rng(M + N + K)
    A = rand_codes((M, K), 0, rng, orc)
    B = rand_codes((N, K), 0, rng, orc)
    A[M // 2, K // 3] = 0xFF            # E4M3 NaN (negative sign)
    got, amax = run_nt("fwd", A, 0, 3, B, 0, 2, out_dt, gpu, M, N, K, amax=True)
    assert amax == 0x7FC00000
    ref_nan = orc.gemm_nt(A, 0, 3, B, 0, 2, out_dt=out_dt, rows=np.array([M // 2]))
    assert orc.scale_bias(ref_nan, 0)[1] == 0x7FC00000
    ta, tb = (torch.from_numpy(np.ascontiguousarray(v)).to(gpu) for v in (A, B))
    pa = torch.tensor([3], dtype=torch.int32, device=gpu)
    pb = torch.tensor([2], dtype=torch.int32, device=gpu)
    _, b, a, fl = F.fp8_linear_fwd_bias(ta, pa, tb, pb, F.E4M3, 0, out_dt=out_dt)
    torch.cuda.synchronize()
    assert (i32(b), u32(a), u32(fl)) == (0, 0x7FC00000, F.FLAG_NONFINITE)


def test_gemm_zero_sizes(gpu):
    e = torch.empty((0, 128), dtype=torch.uint8, device=gpu)
    w = torch.zeros((64, 128), dtype=torch.uint8, device=gpu)
    b = torch.zeros(1, dtype=torch.int32, device=gpu)
    y = F.fp8_linear_fwd(e, b, w, b)
    assert y.shape == (0, 64)
    # an empty output has amax 0: the amax word is written, not left stale
    am = torch.full((1,), 0x12345, dtype=torch.int32, device=gpu)
    F.fp8_linear_fwd(e, b, w, b, y_amax_bits=am)
    dxam = torch.full((1,), 0x12345, dtype=torch.int32, device=gpu)
    F.fp8_linear_bwd_dx(e, b, torch.zeros((0, 128), dtype=torch.uint8, device=gpu), b, dx_amax_bits=dxam)
    torch.cuda.synchronize()
    assert u32(am) == 0 and u32(dxam) == 0
    # K == 0: zeros
    x0 = torch.empty((5, 0), dtype=torch.uint8, device=gpu)
    w0 = torch.empty((7, 0), dtype=torch.uint8, device=gpu)
    y = F.fp8_linear_fwd(x0, b, w0, b, out_dt=F.DT_F32)
    torch.cuda.synchronize()
    assert y.shape == (5, 7) and float(y.abs().sum()) == 0.0


def test_gemm_deterministic(orc, gpu):
    rng = np.random.default_rng(12)
    A = torch.from_numpy(rand_codes((512, 1024), 0, rng, orc)).to(gpu)
    B = torch.from_numpy(rand_codes((768, 1024), 0, rng, orc)).to(gpu)
    b = torch.tensor([5], dtype=torch.int32, device=gpu)
    y1 = F.fp8_linear_fwd(A, b, B, b, out_dt=F.DT_F32)
    y2 = F.fp8_linear_fwd(A, b, B, b, out_dt=F.DT_F32)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


# Decode shapes (M <= 32 routes to the weight-streaming kernels; 33 does not).
# M <= 16 with K a multiple of 512 takes the LDS-staged kernel: 64 weight rows
# per workgroup (K <= 8192 or N >= 16384) or 32; one stage (K = 512), exactly
# as many stages as buffers (1536), long K with few workgroups, ragged N.
DECODE = [(1, 64, 128), (2, 1000, 1024), (15, 65, 896), (16, 4096, 8192), (17, 130, 384),
          (31, 192, 2048), (32, 1, 128), (33, 100, 256), (16, 63, 28672), (1, 130, 512),
          (7, 33, 1536), (16, 200, 9216), (12, 16390, 512)]


@pytest.mark.parametrize("shape", DECODE, ids=lambda s: "%dx%dx%d" % s)
@pytest.mark.parametrize("out_dt", [F.DT_BF16, F.DT_F32], ids=["bf16", "f32"])
def test_gemm_decode_shapes(orc, gpu, shape, out_dt):
    M, N, K = shape
    rng = np.random.default_rng(M * 131 + N + K)
    A, ba = scaled_normal_codes((M, K), 0, rng, orc)
    B, bb = scaled_normal_codes((N, K), 0, rng, orc)
    got, amax = run_nt("fwd", A, 0, ba, B, 0, bb, out_dt, gpu, M, N, K, amax=True)
    ref = orc.gemm_nt(A, 0, ba, B, 0, bb, out_dt=out_dt)
    assert rel_f(got, ref) <= REL_F_TOL
    mag = (got.astype(np.uint32) & 0x7FFF) << 16 if out_dt == F.DT_BF16 else got.view(np.uint32) & 0x7FFFFFFF
    assert amax == int(mag.max())
    # exact small integers: bit for bit
    vals = [0, 1, 2, 3, -1, -2, -4]
    c = np.array([orc.encode(0, v) for v in vals], dtype=np.uint8)
    ia, ib = rng.integers(0, len(vals), (M, K)), rng.integers(0, len(vals), (N, K))
    got, _ = run_nt("fwd", c[ia], 0, 0, c[ib], 0, 0, F.DT_F32, gpu, M, N, K)
    v = np.array(vals, dtype=np.int64)
    assert np.array_equal(got, (v[ia] @ v[ib].T).astype(np.float32))
