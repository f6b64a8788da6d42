"""GPU parity at the full sizes of the benchmark workloads, in the launch
configuration the benchmark times (paper_2309_17224_amd.linear).

* Biases and amax: bit-exact against the oracle on every tensor.
* Casts: the GPU casts whole tensors; rows sampled at random (plus the first
  and last row) are compared bit for bit with the oracle, for the codes and
  for the transposed copy.
* Matmuls: rel_F <= 1e-3 on sampled output rows, recomputed by the oracle
  from the same FP8 codes and biases.
* PTQ inference (Sec. 3.1): weight quantised once, activations per call.
"""
import functools

import numpy as np
import pytest
import torch

from paper_2309_17224_amd import fp8lin as F
from paper_2309_17224_amd import linear as L
from paper_2309_17224_amd import workloads as wl
from parity_util import REL_F_TOL, i32, np_bits, rel_f, sample_rows, u32

pytestmark = pytest.mark.gpu

TRAIN = ["gpt111m-linear", "llama2-7b-up", "llama2-13b-qkv", "llama2-70b-mlp"]


@functools.lru_cache(maxsize=4)
def tensor(workload: str, name: str) -> torch.Tensor:
    return wl.make_tensor(wl.WORKLOADS[workload], name)


def n_sample(M: int, K: int) -> int:
    # oracle cost per sampled row is N*K multiply-adds
    return 256 if M * K <= 8192 * 5120 else 64


def linears(name):
    return [(name, lin.name) for lin in wl.WORKLOADS[name].linears]


@pytest.mark.parametrize("wname,lname", [p for w in TRAIN for p in linears(w)],
                         ids=lambda v: str(v))
def test_train_step_parity(orc, gpu, wname, lname):
    w = wl.WORKLOADS[wname]
    lin = [l for l in w.linears if l.name == lname][0]
    print(f"\n[case] {wname}/{lname} M={lin.M} K={lin.K} N={lin.N}", flush=True)
    X, W, dY = tensor(wname, lin.x), tensor(wname, lin.w), tensor(wname, lin.dy)
    b = L.alloc(lin.M, lin.K, lin.N, gpu)
    L.train_step(X.to(gpu), W.to(gpu), dY.to(gpu), b)
    torch.cuda.synchronize()
    x_bits, w_bits, dy_bits = np_bits(X), np_bits(W), np_bits(dY)

    # biases and amax: bit-exact
    bx, ax, fx = orc.scale_bias(x_bits, orc.E4M3)
    bw, aw, fw = orc.scale_bias(w_bits, orc.E4M3)
    bg, ag, fg = orc.scale_bias(dy_bits, orc.E5M2)
    assert (i32(b.bx), u32(b.amax_x), u32(b.flags_x)) == (bx, ax, fx)
    assert (i32(b.bw), u32(b.amax_w), u32(b.flags_w)) == (bw, aw, fw)
    assert (i32(b.bg), u32(b.amax_g), u32(b.flags_g)) == (bg, ag, fg)

    # casts on sampled rows (codes and the transposed copies)
    rx = sample_rows(lin.M, 64, 1)
    rw = sample_rows(lin.K, 64, 2)
    x8, x8t = b.x8.cpu().numpy(), b.x8t.cpu().numpy()
    w8, w8t = b.w8.cpu().numpy(), b.w8t.cpu().numpy()
    dy8, dy8t = b.dy8.cpu().numpy(), b.dy8t.cpu().numpy()
    assert np.array_equal(x8[rx], orc.cast(x_bits[rx], orc.E4M3, bx))
    assert np.array_equal(x8t[:, rx], x8[rx].T)
    assert np.array_equal(w8[rw], orc.cast(w_bits[rw], orc.E4M3, bw))
    assert np.array_equal(w8t[:, rw], w8[rw].T)
    assert np.array_equal(dy8[rx], orc.cast(dy_bits[rx], orc.E5M2, bg))
    assert np.array_equal(dy8t[:, rx], dy8[rx].T)
    # transposes checked in full (cheap, exact)
    assert np.array_equal(x8t, x8.T) and np.array_equal(w8t, w8.T) and np.array_equal(dy8t, dy8.T)

    # matmuls on sampled output rows, from the GPU's codes (checked above)
    ry = sample_rows(lin.M, n_sample(lin.M, lin.K), 3)
    y = np_bits(b.y)
    yref = orc.gemm_nt(x8, 0, bx, w8t, 0, bw, out_dt=orc.BF16, rows=ry)
    assert rel_f(y[ry], yref) <= REL_F_TOL
    dx = np_bits(b.dx)
    dxref = orc.gemm_nt(dy8, 1, bg, w8, 0, bw, out_dt=orc.BF16, rows=ry)
    assert rel_f(dx[ry], dxref) <= REL_F_TOL
    rdw = sample_rows(lin.K, n_sample(lin.K, lin.M), 4)
    dw = np_bits(b.dw)
    dwref = orc.gemm_nt(x8t, 0, bx, dy8t, 1, bg, out_dt=orc.F32, rows=rdw)
    assert rel_f(dw[rdw], dwref) <= REL_F_TOL

    # epilogue amax of Y and dX and the next consumers' biases
    ymag = (y.astype(np.uint32) & 0x7FFF) << 16
    assert u32(b.amax_y) == int(ymag.max())
    assert i32(b.by) == orc.bias_from_amax(u32(b.amax_y), orc.E4M3)[0]
    dxmag = (dx.astype(np.uint32) & 0x7FFF) << 16
    assert u32(b.amax_dx) == int(dxmag.max())
    assert i32(b.bdx) == orc.bias_from_amax(u32(b.amax_dx), orc.E5M2)[0]


@pytest.mark.parametrize("wname", ["gpt111m-linear", "llama2-7b-up"])
def test_train_step_matches_oracle_chain(orc, gpu, wname):
    """Whole-tensor check of Y against the oracle computing every step itself
    (its own biases and casts, not the GPU's codes)."""
    w = wl.WORKLOADS[wname]
    lin = w.linears[0]
    X, W, dY = tensor(wname, lin.x), tensor(wname, lin.w), tensor(wname, lin.dy)
    b = L.alloc(lin.M, lin.K, lin.N, gpu)
    L.train_step(X.to(gpu), W.to(gpu), dY.to(gpu), b)
    torch.cuda.synchronize()
    xb, wb = np_bits(X), np_bits(W)
    bx, _, _ = orc.scale_bias(xb, 0)
    bw, _, _ = orc.scale_bias(wb, 0)
    rows = sample_rows(lin.M, 128, 7)
    x8 = orc.cast(xb[rows], 0, bx)
    w8t = orc.cast(wb, 0, bw, transpose=True)[1]
    yref = orc.gemm_nt(x8, 0, bx, w8t, 0, bw, out_dt=orc.BF16)
    assert rel_f(np_bits(b.y)[rows], yref) <= REL_F_TOL


PTQ = wl.WORKLOADS["llama2-70b-ptq"]


@pytest.mark.parametrize("lname", [l.name for l in PTQ.linears])
def test_ptq_inference_parity(orc, gpu, lname):
    lin = [l for l in PTQ.linears if l.name == lname][0]
    print(f"\n[case] ptq/{lname} M={lin.M} K={lin.K} N={lin.N}", flush=True)
    W, X = tensor(PTQ.name, lin.w), tensor(PTQ.name, lin.x)
    b = L.alloc(lin.M, lin.K, lin.N, gpu, train=False)
    F.ptq_quantise_weights(W.to(gpu), want_w8=False, w8t=b.w8t, bw=b.bw, flags=b.flags_w, ws=b.ws)
    L.infer_step(X.to(gpu), b)
    torch.cuda.synchronize()
    wb, xb = np_bits(W), np_bits(X)
    bw, _, fw = orc.scale_bias(wb, 0)
    assert (i32(b.bw), u32(b.flags_w)) == (bw, fw)
    bx, ax, fx = orc.scale_bias(xb, 0)
    assert (i32(b.bx), u32(b.amax_x)) == (bx, ax)
    w8t = b.w8t.cpu().numpy()
    rn = sample_rows(lin.N, 64, 5)
    assert np.array_equal(w8t[rn], orc.cast(wb[:, rn].copy(), 0, bw).T)
    x8 = b.x8.cpu().numpy()
    ry = sample_rows(lin.M, 64, 6)
    assert np.array_equal(x8[ry], orc.cast(xb[ry], 0, bx))
    yref = orc.gemm_nt(x8, 0, bx, w8t, 0, bw, out_dt=orc.BF16, rows=ry)
    assert rel_f(np_bits(b.y)[ry], yref) <= REL_F_TOL


def test_ptq_entry_matches_oracle(orc, gpu):
    W = wl.small(1000, 777, std=0.01, seed=21)
    w8, w8t, bw, fl = F.ptq_quantise_weights(W.to(gpu))
    torch.cuda.synchronize()
    ow8, ow8t, obw, ofl = orc.ptq_quantise_weights(np_bits(W))
    assert (i32(bw), u32(fl)) == (obw, ofl)
    assert np.array_equal(w8.cpu().numpy(), ow8)
    assert np.array_equal(w8t.cpu().numpy(), ow8t)


@pytest.mark.parametrize("cbias", [0, 3, -2])
def test_cscale_step_parity(orc, gpu, cbias):
    """FP8-CSCALE (Sec. 3): every tensor cast with one constant bias, no amax.
    Codes bit-exact against the oracle's cast with that bias (App. A clipping
    included: a constant bias can push values past the largest code); the
    matmuls rel_F <= 1e-3 against the oracle on the same codes."""
    w = wl.WORKLOADS["gpt111m-linear"]
    lin = w.linears[0]
    tens = {t.name: tensor(w.name, t.name).to(gpu) for t in w.tensors}
    step = L.WorkloadStep(w, tens, gpu, quant="cscale", cscale_bias=cbias)
    step.run()
    torch.cuda.synchronize()
    assert not any(k == "amax" or k == "quantise" or k == "bias" for _, k, _, _ in step.calls)
    xq, wq, gq = step.q[lin.x], step.q[lin.w], step.q[lin.dy]
    for qt in (xq, wq, gq):
        assert i32(qt.bias) == cbias
    X, W, dY = (np_bits(tensor(w.name, n)) for n in (lin.x, lin.w, lin.dy))
    x8, x8t = orc.cast(X, orc.E4M3, cbias, transpose=True)
    w8, w8t = orc.cast(W, orc.E4M3, cbias, transpose=True)
    g8, g8t = orc.cast(dY, orc.E5M2, cbias, transpose=True)
    assert np.array_equal(xq.q.cpu().numpy(), x8) and np.array_equal(xq.qT.cpu().numpy(), x8t)
    assert np.array_equal(wq.q.cpu().numpy(), w8) and np.array_equal(wq.qT.cpu().numpy(), w8t)
    assert np.array_equal(gq.q.cpu().numpy(), g8) and np.array_equal(gq.qT.cpu().numpy(), g8t)
    o = step.out[lin.name]
    rows = sample_rows(lin.M, 128, 7)
    yref = orc.gemm_nt(x8, 0, cbias, w8t, 0, cbias, out_dt=orc.BF16, rows=rows)
    assert rel_f(np_bits(o["y"])[rows], yref) <= REL_F_TOL
    dxref = orc.gemm_nt(g8, 1, cbias, w8, 0, cbias, out_dt=orc.BF16, rows=rows)
    assert rel_f(np_bits(o["dx"])[rows], dxref) <= REL_F_TOL
    rdw = sample_rows(lin.K, 128, 8)
    dwref = orc.gemm_nt(x8t, 0, cbias, g8t, 1, cbias, out_dt=orc.F32, rows=rdw)
    assert rel_f(np_bits(o["dw"])[rdw], dwref) <= REL_F_TOL
