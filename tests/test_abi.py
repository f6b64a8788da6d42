"""The C ABI on the host (no GPU needed): the library loads, exports every
function include/fp8lin.h declares, and rejects bad arguments before it would
launch anything (status FP8_EINVAL, see the header's conventions)."""
import ctypes
import os
import re

import pytest

from paper_2309_17224_amd import fp8lin as F

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fp8lin.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(F.LIB_PATH):
        from paper_2309_17224_amd import build
        build.build()
    return F.lib()


def test_header_and_binding_agree():
    assert declared_functions() == sorted(F.EXPORTS)


def test_every_declared_symbol_is_exported(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_status_strings(L):
    assert L.fp8_status_string(0) == b"ok"
    assert L.fp8_status_string(1) == b"invalid argument"
    assert L.fp8_status_string(99) == b"unknown status"
    assert L.fp8_abi_version() == 1


def test_workspace_size(L):
    assert L.fp8_scale_bias_ws_bytes(0) == 0
    assert L.fp8_scale_bias_ws_bytes(1) == 4
    assert L.fp8_scale_bias_ws_bytes(10 ** 9) == 4 * 2048


FAKE = ctypes.c_void_p(0x100000)       # aligned, never dereferenced: rejected before launch
ODD = ctypes.c_void_p(0x100001)
A8 = ctypes.c_void_p(0x100008)         # 8-byte but not 16-byte aligned
NULL = None


def test_scale_bias_rejects(L):
    f = L.fp8_scale_bias
    assert f(FAKE, 2, 10, 0, 0, FAKE, NULL, NULL, FAKE, 64, NULL) == F.EINVAL      # dtype
    assert f(FAKE, 0, 10, 7, 0, FAKE, NULL, NULL, FAKE, 64, NULL) == F.EINVAL      # format
    assert f(FAKE, 0, -1, 0, 0, FAKE, NULL, NULL, FAKE, 64, NULL) == F.EINVAL      # n < 0
    assert f(NULL, 0, 10, 0, 0, FAKE, NULL, NULL, FAKE, 64, NULL) == F.EINVAL      # x
    assert f(FAKE, 0, 10, 0, 0, NULL, NULL, NULL, FAKE, 64, NULL) == F.EINVAL      # bias
    assert f(ODD, 0, 10, 0, 0, FAKE, NULL, NULL, FAKE, 64, NULL) == F.EINVAL       # alignment
    assert f(FAKE, 0, 10, 0, 0, FAKE, NULL, NULL, NULL, 64, NULL) == F.EINVAL      # workspace
    assert f(FAKE, 0, 10 ** 8, 0, 0, FAKE, NULL, NULL, FAKE, 4, NULL) == F.EINVAL  # too small
    assert f(FAKE, 0, 10, 0, 1 << 20, FAKE, NULL, NULL, FAKE, 64, NULL) == F.EINVAL  # margin


def test_cast_rejects(L):
    for f in (L.fp8_cast_e4, L.fp8_cast_e5):
        assert f(FAKE, 0, 4, 8, 8, FAKE, NULL, 8, NULL, 4, NULL) == F.EINVAL   # no output
        assert f(FAKE, 0, 4, 8, 7, FAKE, FAKE, 8, NULL, 4, NULL) == F.EINVAL   # ldx < cols
        assert f(FAKE, 0, 4, 8, 8, FAKE, FAKE, 7, NULL, 4, NULL) == F.EINVAL   # ldq < cols
        assert f(FAKE, 0, 4, 8, 8, FAKE, NULL, 0, FAKE, 3, NULL) == F.EINVAL   # ldqT < rows
        assert f(NULL, 0, 4, 8, 8, FAKE, FAKE, 8, NULL, 4, NULL) == F.EINVAL   # x
        assert f(FAKE, 0, 4, 8, 8, NULL, FAKE, 8, NULL, 4, NULL) == F.EINVAL   # bias
        assert f(FAKE, 5, 4, 8, 8, FAKE, FAKE, 8, NULL, 4, NULL) == F.EINVAL   # dtype
        assert f(ODD, 0, 4, 8, 8, FAKE, FAKE, 8, NULL, 4, NULL) == F.EINVAL    # alignment
        assert f(FAKE, 0, -4, 8, 8, FAKE, FAKE, 8, NULL, 4, NULL) == F.EINVAL  # rows < 0
        assert f(NULL, 0, 0, 8, 8, NULL, NULL, 8, NULL, 4, NULL) == F.OK       # empty: no-op
        big = 1 << 39  # 2^32 x 2^32 tiles of 128 x 128: more workgroups than one launch holds
        assert f(FAKE, 0, big, big, big, FAKE, FAKE, big, NULL, big, NULL) == F.ENOTSUP


def test_quantise_workspace_size(L):
    assert L.fp8_quantise_ws_bytes(0, 5) == 0
    assert L.fp8_quantise_ws_bytes(128, 128) == 4 * (1 + 1)
    assert L.fp8_quantise_ws_bytes(129, 300) == 4 * (1 + 2 * 3)


def test_quantise_rejects(L):
    f = L.fp8_quantise
    WS = 4 * 64
    #        x     dt rows cols ldx fmt marg pred  bias  amax  flags q     ldq qT    ldqT ws    wsb  stream
    assert f(FAKE, 0, 4, 8, 8, 0, 0, NULL, FAKE, NULL, NULL, NULL, 8, NULL, 4, FAKE, WS, NULL) == F.EINVAL  # no output
    assert f(FAKE, 0, 4, 8, 7, 0, 0, NULL, FAKE, NULL, NULL, FAKE, 8, NULL, 4, FAKE, WS, NULL) == F.EINVAL  # ldx
    assert f(FAKE, 0, 4, 8, 8, 0, 0, NULL, FAKE, NULL, NULL, FAKE, 7, NULL, 4, FAKE, WS, NULL) == F.EINVAL  # ldq
    assert f(FAKE, 0, 4, 8, 8, 0, 0, NULL, FAKE, NULL, NULL, NULL, 0, FAKE, 3, FAKE, WS, NULL) == F.EINVAL  # ldqT
    assert f(NULL, 0, 4, 8, 8, 0, 0, NULL, FAKE, NULL, NULL, FAKE, 8, NULL, 4, FAKE, WS, NULL) == F.EINVAL  # x
    assert f(FAKE, 0, 4, 8, 8, 0, 0, NULL, NULL, NULL, NULL, FAKE, 8, NULL, 4, FAKE, WS, NULL) == F.EINVAL  # bias
    assert f(FAKE, 0, 4, 8, 8, 0, 0, ODD, FAKE, NULL, NULL, FAKE, 8, NULL, 4, FAKE, WS, NULL) == F.EINVAL   # pred align
    assert f(FAKE, 0, 4, 8, 8, 0, 0, NULL, FAKE, NULL, NULL, FAKE, 8, NULL, 4, NULL, WS, NULL) == F.EINVAL  # ws
    assert f(FAKE, 0, 4, 8, 8, 0, 0, NULL, FAKE, NULL, NULL, FAKE, 8, NULL, 4, FAKE, 4, NULL) == F.EINVAL   # ws small
    assert f(FAKE, 3, 4, 8, 8, 0, 0, NULL, FAKE, NULL, NULL, FAKE, 8, NULL, 4, FAKE, WS, NULL) == F.EINVAL  # dtype
    assert f(FAKE, 0, 4, 8, 8, 4, 0, NULL, FAKE, NULL, NULL, FAKE, 8, NULL, 4, FAKE, WS, NULL) == F.EINVAL  # format
    assert f(FAKE, 0, 4, 8, 8, 0, 1 << 20, NULL, FAKE, NULL, NULL, FAKE, 8, NULL, 4, FAKE, WS, NULL) == F.EINVAL  # margin
    assert f(FAKE, 0, -1, 8, 8, 0, 0, NULL, FAKE, NULL, NULL, FAKE, 8, NULL, 4, FAKE, WS, NULL) == F.EINVAL  # rows < 0


def test_generic_cast_rejects(L):
    f = L.fp8_cast
    assert f(FAKE, 0, 4, 8, 8, 4, FAKE, FAKE, 8, NULL, 4, NULL) == F.EINVAL    # format
    assert f(FAKE, 0, 4, 8, 8, -1, FAKE, FAKE, 8, NULL, 4, NULL) == F.EINVAL   # format
    assert f(FAKE, 0, 4, 8, 8, 2, NULL, FAKE, 8, NULL, 4, NULL) == F.EINVAL    # bias
    assert f(FAKE, 0, 4, 8, 8, 3, FAKE, NULL, 8, NULL, 4, NULL) == F.EINVAL    # no output


def test_gemm_rejects(L):
    for f in (L.fp8_linear_fwd, L.fp8_linear_bwd_dx):
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 3, 4, 4, 4, NULL, NULL) == F.EINVAL    # out dtype
        assert f(NULL, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, NULL, NULL) == F.EINVAL    # operand
        assert f(FAKE, NULL, FAKE, FAKE, FAKE, 0, 4, 4, 4, NULL, NULL) == F.EINVAL    # bias
        assert f(FAKE, FAKE, FAKE, FAKE, NULL, 0, 4, 4, 4, NULL, NULL) == F.EINVAL    # output
        assert f(FAKE, FAKE, FAKE, FAKE, ODD, 0, 4, 4, 4, NULL, NULL) == F.EINVAL     # alignment
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 0, -1, 4, 4, NULL, NULL) == F.EINVAL   # M < 0
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, ODD, NULL) == F.EINVAL     # amax
        assert f(NULL, NULL, NULL, NULL, NULL, 0, 0, 4, 4, NULL, NULL) == F.OK        # empty
        # FP8 operands must start on 16-byte boundaries (also where K is not a
        # multiple of 128): rejected, not routed to another kernel
        assert f(ODD, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, NULL, NULL) == F.EINVAL     # operand A
        assert f(FAKE, FAKE, A8, FAKE, FAKE, 0, 4, 4, 4, NULL, NULL) == F.EINVAL      # operand B
        assert f(FAKE, FAKE, A8, FAKE, FAKE, 0, 4, 4, 20, NULL, NULL) == F.EINVAL     # any K
    f = L.fp8_linear_bwd_dw
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 2, 4, 4, 4, NULL) == F.EINVAL
    assert f(FAKE, FAKE, NULL, FAKE, FAKE, 0, 4, 4, 4, NULL) == F.EINVAL
    assert f(A8, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, NULL) == F.EINVAL
    assert f(FAKE, FAKE, ODD, FAKE, FAKE, 0, 4, 4, 4, NULL) == F.EINVAL
    assert f(NULL, NULL, NULL, NULL, NULL, 0, 4, 0, 4, NULL) == F.OK
    f = L.fp8_linear_fwd_rows
    assert f(ODD, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, NULL, NULL) == F.EINVAL
    assert f(FAKE, FAKE, A8, FAKE, FAKE, 0, 4, 4, 4, NULL, NULL) == F.EINVAL


def test_ptq_and_bias_from_amax_reject(L):
    assert L.ptq_quantise_weights(FAKE, 0, 4, 4, NULL, NULL, FAKE, NULL, FAKE, 64, NULL) == F.EINVAL
    assert L.ptq_quantise_weights(FAKE, 0, 4, 4, FAKE, NULL, NULL, NULL, FAKE, 64, NULL) == F.EINVAL
    assert L.ptq_quantise_weights(FAKE, 9, 4, 4, FAKE, NULL, FAKE, NULL, FAKE, 64, NULL) == F.EINVAL
    # K * N past the element count an amax call accepts (2^46), including products past 2^63
    assert L.ptq_quantise_weights(FAKE, 0, 1 << 24, 1 << 23, FAKE, NULL, FAKE, NULL, FAKE, 64, NULL) == F.EINVAL
    assert L.ptq_quantise_weights(FAKE, 0, 1 << 33, 1 << 33, FAKE, NULL, FAKE, NULL, FAKE, 64, NULL) == F.EINVAL
    assert L.fp8_bias_from_amax(NULL, 0, 0, FAKE, NULL, NULL) == F.EINVAL
    assert L.fp8_bias_from_amax(FAKE, 5, 0, FAKE, NULL, NULL) == F.EINVAL
    assert L.fp8_bias_from_amax(FAKE, 0, 0, ODD, NULL, NULL) == F.EINVAL


def test_gemm_bias_rejects(L):
    assert L.fp8_linear_bias_ws_bytes() == 8
    for f in (L.fp8_linear_fwd_bias, L.fp8_linear_bwd_dx_bias):
        # (a, ba, b, bb, c, c_dt, M, N, K, fmt, margin, bias, amax, flags, ws, ws_bytes, stream)
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 3, 4, 4, 4, 0, 0, FAKE, NULL, NULL, FAKE, 8, NULL) == F.EINVAL   # dtype
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, 4, 0, FAKE, NULL, NULL, FAKE, 8, NULL) == F.EINVAL   # format
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, 0, 1 << 20, FAKE, NULL, NULL, FAKE, 8, NULL) == F.EINVAL  # margin
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, 0, 0, NULL, NULL, NULL, FAKE, 8, NULL) == F.EINVAL   # bias
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, 0, 0, FAKE, NULL, NULL, NULL, 8, NULL) == F.EINVAL   # ws
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, 0, 0, FAKE, NULL, NULL, FAKE, 4, NULL) == F.EINVAL   # ws small
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, 0, 0, FAKE, NULL, NULL, ODD, 8, NULL) == F.EINVAL    # ws align
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, 0, 0, FAKE, ODD, NULL, FAKE, 8, NULL) == F.EINVAL    # amax align
        assert f(NULL, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, 0, 0, FAKE, NULL, NULL, FAKE, 8, NULL) == F.EINVAL   # operand
        assert f(FAKE, FAKE, FAKE, FAKE, NULL, 0, 4, 4, 4, 0, 0, FAKE, NULL, NULL, FAKE, 8, NULL) == F.EINVAL   # output
        assert f(FAKE, FAKE, FAKE, FAKE, ODD, 0, 4, 4, 4, 0, 0, FAKE, NULL, NULL, FAKE, 8, NULL) == F.EINVAL    # out align
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 0, -1, 4, 4, 0, 0, FAKE, NULL, NULL, FAKE, 8, NULL) == F.EINVAL  # M < 0
        assert f(A8, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 4, 0, 0, FAKE, NULL, NULL, FAKE, 8, NULL) == F.EINVAL    # A align
        assert f(FAKE, FAKE, ODD, FAKE, FAKE, 0, 4, 4, 4, 0, 0, FAKE, NULL, NULL, FAKE, 8, NULL) == F.EINVAL   # B align


def test_segments_mode_rows_reject(L):
    f = L.fp8_quantise_segments
    # (x, dt, rows, cols, ldx, fmt, margin, offsets, nseg, bias, amax, flags, row_bias, q, ldq, qT, ldqT, stream)
    ok = [FAKE, 0, 4, 8, 8, 0, 0, FAKE, 2, FAKE, FAKE, NULL, FAKE, FAKE, 8, NULL, 0, NULL]
    for i, bad in ((1, 3), (5, 9), (6, 1 << 20), (8, 0), (7, NULL), (9, NULL), (10, NULL), (12, NULL), (0, NULL),
                   (0, ODD), (4, 7), (14, 7), (2, -1)):
        args = list(ok)
        args[i] = bad
        assert f(*args) == F.EINVAL, (i, bad)
    g = L.fp8_linear_fwd_rows
    assert g(FAKE, NULL, FAKE, FAKE, FAKE, 0, 4, 4, 4, NULL, NULL) == F.EINVAL   # row biases
    assert g(FAKE, ODD, FAKE, FAKE, FAKE, 0, 4, 4, 4, NULL, NULL) == F.EINVAL    # alignment
    assert g(FAKE, FAKE, FAKE, FAKE, FAKE, 3, 4, 4, 4, NULL, NULL) == F.EINVAL   # dtype
    assert g(NULL, NULL, NULL, NULL, NULL, 0, 0, 4, 4, NULL, NULL) == F.OK       # empty
    h = L.fp8_bias_mode
    assert h(FAKE, 4, FAKE, 0, FAKE, NULL) == F.EINVAL     # capacity
    assert h(FAKE, 4, NULL, 3, FAKE, NULL) == F.EINVAL     # ring
    assert h(FAKE, 4, FAKE, 3, NULL, NULL) == F.EINVAL     # count
    assert h(NULL, 4, FAKE, 3, FAKE, NULL) == F.EINVAL     # biases
    assert h(NULL, 0, FAKE, 3, FAKE, NULL) == F.OK         # nothing to count


def test_decoder_glue_workspace_sizes(L):
    assert L.llama_rmsnorm_ws_bytes(0) == 0
    assert L.llama_rmsnorm_ws_bytes(2048) == 4 * (1 + 2048)
    assert L.llama_swiglu_ws_bytes() == 4 * (1 + 2048)
    # one maximum per (query head, sequence, block of 128 queries)
    assert L.llama_attention_ws_bytes(2048, 2048, 64) == 4 * (1 + 64 * 16)
    assert L.llama_attention_ws_bytes(300, 150, 8) == 4 * (1 + 8 * 2 * 2)
    assert L.llama_attention_ws_bytes(0, 16, 8) == 0


def test_decoder_glue_rejects(L):
    A = ctypes.c_void_p(0x100000)
    ws = 4 * 4097
    # llama_rmsnorm_quantise(x, ldx, res, ldr, g, rows, cols, eps, h, ldh, y, ldy, fmt, margin, pred, bias,
    #                        amax, flags, q, ldq, ws, ws_bytes, stream)
    ok = [A, 64, NULL, 0, A, 4, 64, 1e-5, NULL, 0, A, 64, 0, 0, NULL, A, NULL, NULL, A, 64, A, ws, NULL]
    for i, bad in ((0, NULL), (0, ctypes.c_void_p(0x100008)), (1, 60), (1, 68), (4, NULL), (6, 12), (7, -1.0),
                   (7, float("nan")), (10, NULL), (11, 32), (12, 9), (15, NULL), (18, ODD), (19, 60),
                   (20, NULL), (21, 8), (5, -1)):
        args = list(ok)
        args[i] = bad
        assert L.llama_rmsnorm_quantise(*args) == F.EINVAL, (i, bad)
    # llama_attention(qkv, rows, ld, seq_len, nh, nkv, dh, o, ldo, fmt, margin, pred, bias, amax, flags, q, ldq,
    #                 ws, ws_bytes, stream)
    ok = [A, 256, 12 * 128, 256, 8, 2, 128, A, 8 * 128, 0, 0, NULL, A, NULL, NULL, NULL, 0, NULL, 0, NULL]
    for i, bad, st in ((6, 64, F.ENOTSUP), (5, 3, F.EINVAL), (4, 0, F.EINVAL), (3, 0, F.EINVAL),
                       (2, 11 * 128, F.EINVAL), (8, 7 * 128, F.EINVAL), (0, NULL, F.EINVAL), (7, ODD, F.EINVAL)):
        args = list(ok)
        args[i] = bad
        assert L.llama_attention(*args) == st, (i, bad)
    # with codes requested, the quantise arguments are checked too
    args = list(ok)
    args[15], args[16], args[17], args[18] = A, 8 * 128, A, 8   # workspace too small
    assert L.llama_attention(*args) == F.EINVAL
    # llama_swiglu_quantise(gu, ldgu, rows, ffn, a, lda, fmt, margin, pred, bias, amax, flags, q, ldq, ws, ws_bytes, s)
    ok = [A, 2816, 16, 1408, A, 1408, 0, 0, NULL, NULL, NULL, NULL, NULL, 0, NULL, 0, NULL]
    for i, bad in ((3, 1404), (1, 2808), (5, 1400), (0, NULL), (4, ODD)):
        args = list(ok)
        args[i] = bad
        assert L.llama_swiglu_quantise(*args) == F.EINVAL, (i, bad)
    # llama_rope(x, rows, ld, n_heads, d_head, seq_len, table, stream); llama_rope_table(seq, dh, theta, table, s)
    assert L.llama_rope(A, 4, 1024, 8, 120, 4, A, NULL) == F.EINVAL     # d_head not a multiple of 16
    assert L.llama_rope(A, 4, 1000, 8, 128, 4, A, NULL) == F.EINVAL     # row stride
    assert L.llama_rope(A, 4, 1024, 8, 128, 0, A, NULL) == F.EINVAL     # seq_len
    assert L.llama_rope(A, 4, 1024, 8, 128, 4, NULL, NULL) == F.EINVAL  # table
    assert L.llama_rope(NULL, 0, 1024, 8, 128, 4, NULL, NULL) == F.OK   # nothing to rotate
    assert L.llama_rope_table(16, 128, -1.0, A, NULL) == F.EINVAL
    assert L.llama_rope_table(0, 128, 1e4, A, NULL) == F.EINVAL
    # llama_residual_add(a, b, out, n, stream)
    assert L.llama_residual_add(A, A, A, 12, NULL) == F.EINVAL
    assert L.llama_residual_add(A, ODD, A, 16, NULL) == F.EINVAL
    assert L.llama_residual_add(NULL, NULL, NULL, 0, NULL) == F.OK


def test_quantise_noalloc_rejects(L):
    f = L.fp8_quantise_noalloc
    # (x, dt, rows, cols, ldx, fmt, margin, pred, bias, amax, flags, q, ldq, qT, ldqT, stream)
    assert f(FAKE, 0, 4, 8, 8, 9, 0, NULL, FAKE, NULL, NULL, FAKE, 8, NULL, 0, NULL) == F.EINVAL     # format
    assert f(FAKE, 0, 4, 8, 8, 0, 0, NULL, NULL, NULL, NULL, FAKE, 8, NULL, 0, NULL) == F.EINVAL     # bias
    assert f(FAKE, 0, 4, 8, 8, 0, 0, NULL, FAKE, NULL, NULL, NULL, 8, NULL, 0, NULL) == F.EINVAL     # no output
    assert f(FAKE, 0, 4, 8, 4, 0, 0, NULL, FAKE, NULL, NULL, FAKE, 8, NULL, 0, NULL) == F.EINVAL     # ldx
    # more 128 x 128 tiles than the static scratch holds (512 x 513 > 262143)
    r, c = 512 * 128, 513 * 128
    assert f(FAKE, 0, r, c, c, 0, 0, NULL, FAKE, NULL, NULL, FAKE, c, NULL, 0, NULL) == F.EINVAL
    assert F.NOALLOC_SCRATCH_BYTES == 4 * (F.NOALLOC_MAX_TILES + 1)


def test_quantise_delayed_rejects(L):
    f = L.fp8_quantise_delayed
    # (x, dt, rows, cols, ldx, fmt, margin, bias, history, hlen, count, amax, flags, q, ldq, qT, ldqT, ws, ws_bytes, stream)
    ok = (FAKE, 0, 4, 8, 8, 0, 0, FAKE, FAKE, 16, FAKE, NULL, NULL, FAKE, 8, NULL, 0, FAKE, 64, NULL)
    def call(i, v):
        a = list(ok)
        a[i] = v
        return f(*a)
    assert call(5, 9) == F.EINVAL                 # format
    assert call(7, NULL) == F.EINVAL              # bias
    assert call(8, NULL) == F.EINVAL              # history
    assert call(8, ODD) == F.EINVAL               # history alignment
    assert call(9, 0) == F.EINVAL                 # history length
    assert call(9, 65537) == F.EINVAL
    assert call(10, NULL) == F.EINVAL             # count
    assert call(17, NULL) == F.EINVAL             # workspace
    assert call(18, 4) == F.EINVAL                # workspace too small
    assert call(13, NULL) == F.EINVAL             # no output


def test_quantise_batch_rejects(L):
    """fp8_quantise_batch checks every tensor as fp8_quantise does, plus the
    batch size and that predictions are given for all tensors or none."""
    def args(**kw):
        a = F.QuantiseArgs(x=FAKE, rows=4, cols=8, ldx=8, bias_pred=None, bias=FAKE, amax_bits=None,
                           flags=None, q=FAKE, ldq=8, qT=None, ldqT=0, ws=FAKE, ws_bytes=4 * 64)
        for k, v in kw.items():
            setattr(a, k, v)
        return a

    def call(items, n=None, dt=0, fmt=0, margin=0):
        arr = (F.QuantiseArgs * max(len(items), 1))(*items)
        return L.fp8_quantise_batch(len(items) if n is None else n, ctypes.cast(arr, ctypes.c_void_p), dt, fmt,
                                    margin, NULL)

    assert L.fp8_quantise_batch(0, NULL, 0, 0, 0, NULL) == F.OK            # nothing to do
    assert L.fp8_quantise_batch(1, NULL, 0, 0, 0, NULL) == F.EINVAL        # no array
    assert call([args()] * 5) == F.EINVAL                                  # more than the maximum
    assert call([args()], n=-1) == F.EINVAL
    assert call([args(), args(ldx=7)]) == F.EINVAL                         # second tensor's stride
    assert call([args(), args(ws_bytes=4)]) == F.EINVAL                    # second tensor's workspace
    assert call([args(), args(q=None)]) == F.EINVAL                        # no output
    assert call([args(bias=None)]) == F.EINVAL
    assert call([args(bias_pred=FAKE), args()]) == F.EINVAL                # mixed predictions
    assert call([args()], dt=3) == F.EINVAL
    assert call([args()], fmt=4) == F.EINVAL
    assert call([args()], margin=1 << 20) == F.EINVAL
    assert F.QUANTISE_BATCH_MAX == 4 and "FP8_QUANTISE_BATCH_MAX 4" in open(HEADER).read()


PROBE_HEADER = os.path.join(ROOT, "include", "fp8probe.h")


def test_probe_library_exports_and_rejects():
    """The measurement aid libfp8probe.so (include/fp8probe.h): every declared
    function is exported, and bad arguments are rejected before any launch."""
    from paper_2309_17224_amd import build
    if not os.path.exists(build.PROBE_LIB):
        build.build()
    P = ctypes.CDLL(build.PROBE_LIB)
    text = re.sub(r"/\*.*?\*/", "", open(PROBE_HEADER).read(), flags=re.S)
    names = set(re.findall(r"^\s*[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", text, re.M))
    assert names == {"fp8probe_mfma_loop_flops", "fp8probe_mfma_loop", "fp8probe_stream",
                     "fp8probe_lds_src_bytes", "fp8probe_lds"}
    for n in names:
        assert hasattr(P, n), n
    P.fp8probe_lds_src_bytes.restype = ctypes.c_int64
    assert P.fp8probe_lds_src_bytes() == 64 << 20
    P.fp8probe_lds.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    assert P.fp8probe_lds(4, 10, FAKE, FAKE, NULL) == 1      # unknown mode
    assert P.fp8probe_lds(0, 0, FAKE, FAKE, NULL) == 1       # no iterations
    assert P.fp8probe_lds(0, 10, NULL, FAKE, NULL) == 1      # no source
    assert P.fp8probe_lds(0, 10, A8, FAKE, NULL) == 1        # source not 16-byte aligned
    P.fp8probe_stream.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    assert P.fp8probe_stream(FAKE, 24, FAKE, NULL, NULL) == 1  # n not a multiple of 16
    P.fp8probe_mfma_loop.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    assert P.fp8probe_mfma_loop(0, 10, 1, FAKE, NULL) == 1   # no workgroups
