"""GPU parity at the full sizes of the benchmark workloads.

test_bench_step_parity builds the step exactly as bench.py builds the step it
times (bench.step_kwargs of the default arguments: fp8_quantise_batch with
the previous step's bias as the prediction, forward and grad-input matmuls
that take their output's Eq. 3 bias in the same launch, one HIP graph per
step), runs it eagerly once (the bias words start at zero, so the predictions
fail), captures it and replays it twice (the predictions hold), then compares
with the oracle:

* every quantised tensor (Sec. 2.3 Eq. 3, Sec. 2.1 Eq. 1): bias, amax and
  flags, and the whole code tensor and its transposed copy, bit for bit;
* the bias, amax and flags the matmuls give their outputs, bit for bit against
  the oracle's Eq. 3 of those outputs;
* every matmul (Sec. 2, 2.2, Eq. 2): rel_F <= 1e-3 on 256 sampled output rows
  (all rows below 256), recomputed by the oracle in fp64 from its own codes.

Then it doubles every per-step input in place (exact in bf16), so every Eq. 3
bias moves by one and every prediction fails, replays the graph once more and
checks again (biases and whole code tensors against the oracle; matmuls on 64
rows against the oracle, and exactly 4x (training) or 2x (inference) the
previous outputs, the unscale being an exact power of two).

The separate-call path (fp8_scale_bias, fp8_cast, fp8_linear_*,
fp8_bias_from_amax) and the PTQ entry point are checked at full size below.
"""
import functools
import importlib.util
import os

import numpy as np
import pytest
import torch

from paper_2309_17224_amd import fp8lin as F
from paper_2309_17224_amd import linear as L
from paper_2309_17224_amd import workloads as wl
from parity_util import REL_F_TOL, i32, np_bits, rel_f, sample_rows, u32

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCHED = ["gpt111m-linear", "llama2-7b-up", "llama2-13b-qkv", "llama2-70b-mlp", "llama2-70b-ptq"]
ROWS = 256


@functools.lru_cache(maxsize=1)
def bench_module():
    spec = importlib.util.spec_from_file_location("bench_for_parity", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def bench_step_kwargs() -> dict:
    b = bench_module()
    return b.step_kwargs(b.parse([]))


def check_against_oracle(orc, step, cpu, scale, nrows):
    """Compare every output of the last step with the oracle, whose inputs
    are `scale` times the generated tensors (for the per-step inputs)."""
    w = step.w
    per_step = set(step.step_inputs())
    ptq_weights = {l.w for l in w.linears} if not w.train else set()
    expect = {}
    for name, fmt, margin in step.quantised():
        x = cpu[name] * scale if name in per_step else cpu[name]
        xb = np_bits(x)
        ob, oa, ofl = orc.scale_bias(xb, fmt, margin)
        qt = step.q[name]
        if name in ptq_weights:  # ptq_quantise_weights writes bias and flags
            assert (i32(qt.bias), u32(qt.flags)) == (ob, ofl), name
        else:
            assert (i32(qt.bias), u32(qt.amax), u32(qt.flags)) == (ob, oa, ofl), name
        oq, oqT = orc.cast(xb, fmt, ob, transpose=True)
        if qt.q is not None:
            assert np.array_equal(qt.q.cpu().numpy(), oq), f"codes of {name}"
        if qt.qT is not None:
            assert np.array_equal(qt.qT.cpu().numpy(), oqT), f"transposed codes of {name}"
        expect[name] = (oq, oqT, ob, fmt, margin)
        del xb
    for k, l in enumerate(w.linears):
        xq, wq = expect[l.x], expect[l.w]
        o = step.out[l.name]
        ry = sample_rows(l.M, nrows, 3 + k)
        y = np_bits(o["y"])
        yref = orc.gemm_nt(xq[0], xq[3], xq[2], wq[1], wq[3], wq[2], out_dt=orc.BF16, rows=ry)
        err = rel_f(y[ry], yref)
        print(f"[parity] {w.name}/{l.name} fwd rel_F {err:.2e} on {len(ry)} rows", flush=True)
        assert err <= REL_F_TOL
        if not w.train:
            continue
        # the bias each matmul gave its output: Eq. 3 of that output, exactly
        ob, oa, ofl = orc.scale_bias(y, orc.E4M3, 0)
        assert [i32(o["y_scal"][0]), u32(o["y_scal"][1]), u32(o["y_scal"][2])] == [ob, oa, ofl]
        gq = expect[l.dy]
        dx = np_bits(o["dx"])
        dxref = orc.gemm_nt(gq[0], gq[3], gq[2], wq[0], wq[3], wq[2], out_dt=orc.BF16, rows=ry)
        err = rel_f(dx[ry], dxref)
        print(f"[parity] {w.name}/{l.name} dx rel_F {err:.2e}", flush=True)
        assert err <= REL_F_TOL
        ob, oa, ofl = orc.scale_bias(dx, orc.E5M2, gq[4])
        assert [i32(o["dx_scal"][0]), u32(o["dx_scal"][1]), u32(o["dx_scal"][2])] == [ob, oa, ofl]
        rdw = sample_rows(l.K, nrows, 40 + k)
        dw = np_bits(o["dw"])
        dwref = orc.gemm_nt(xq[1], xq[3], xq[2], gq[1], gq[3], gq[2], out_dt=orc.F32, rows=rdw)
        err = rel_f(dw[rdw], dwref)
        print(f"[parity] {w.name}/{l.name} dw rel_F {err:.2e}", flush=True)
        assert err <= REL_F_TOL


@pytest.mark.timeout(900)
@pytest.mark.parametrize("wname", BENCHED)
def test_bench_step_parity(orc, gpu, wname):
    w = wl.WORKLOADS[wname]
    print(f"\n[case] bench step {wname}: {[(l.name, l.M, l.K, l.N) for l in w.linears]}", flush=True)
    cpu = {t.name: wl.make_tensor(w, t.name) for t in w.tensors}
    tens = {k: v.to(gpu) for k, v in cpu.items()}
    kw = bench_step_kwargs()
    assert kw["quant"] == "predicted" and kw["batch_quant"] and kw["fused_bias"] and not kw["concurrent"]
    step = L.WorkloadStep(w, tens, gpu, **kw)
    if not w.train:
        step.prepare_inference()
    step.run()                       # predictions from zeroed bias words: they fail
    torch.cuda.synchronize()
    first = step.prediction_hits()
    step.capture()
    step.replay()
    step.replay()
    torch.cuda.synchronize()
    hits, n = step.prediction_hits()
    print(f"[case] predictions held: first step {first[0]}/{first[1]}, replays {hits}/{n}", flush=True)
    assert first[0] < first[1] and hits == n
    check_against_oracle(orc, step, cpu, 1, ROWS)

    # every per-step input doubled: every bias moves by one, no prediction holds
    keep = {name: {k: v.clone() for k, v in o.items() if k in ("y", "dx", "dw")} for name, o in step.out.items()}
    for name in step.step_inputs():
        tens[name].mul_(2)
    step.replay()
    torch.cuda.synchronize()
    hits, n = step.prediction_hits()
    assert hits == 0, f"{hits} of {n} predictions held after the inputs doubled"
    factor = 4 if w.train else 2
    for name, outs in keep.items():
        for k, v in outs.items():
            assert torch.equal(step.out[name][k], v * factor), f"{name} {k} not {factor}x"
    check_against_oracle(orc, step, cpu, 2, 64)


# ------------------------------------------------ separate calls, full size
SEPARATE = ["gpt111m-linear", "llama2-7b-up", "llama2-13b-qkv"]


@functools.lru_cache(maxsize=4)
def tensor(workload: str, name: str) -> torch.Tensor:
    return wl.make_tensor(wl.WORKLOADS[workload], name)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("wname", SEPARATE)
def test_separate_calls_parity(orc, gpu, wname):
    """The linear layer as separate library calls (linear.train_step:
    fp8_scale_bias, fp8_cast_e4/e5, fp8_linear_fwd/bwd_dx with the epilogue
    amax, fp8_bias_from_amax, fp8_linear_bwd_dw) on the full workload."""
    w = wl.WORKLOADS[wname]
    lin = w.linears[0]
    print(f"\n[case] separate calls {wname} M={lin.M} K={lin.K} N={lin.N}", flush=True)
    X, W, dY = tensor(wname, lin.x), tensor(wname, lin.w), tensor(wname, lin.dy)
    b = L.alloc(lin.M, lin.K, lin.N, gpu)
    L.train_step(X.to(gpu), W.to(gpu), dY.to(gpu), b)
    torch.cuda.synchronize()
    x_bits, w_bits, dy_bits = np_bits(X), np_bits(W), np_bits(dY)
    bx, ax, fx = orc.scale_bias(x_bits, orc.E4M3)
    bw, aw, fw = orc.scale_bias(w_bits, orc.E4M3)
    bg, ag, fg = orc.scale_bias(dy_bits, orc.E5M2)
    assert (i32(b.bx), u32(b.amax_x), u32(b.flags_x)) == (bx, ax, fx)
    assert (i32(b.bw), u32(b.amax_w), u32(b.flags_w)) == (bw, aw, fw)
    assert (i32(b.bg), u32(b.amax_g), u32(b.flags_g)) == (bg, ag, fg)
    x8, x8t = orc.cast(x_bits, orc.E4M3, bx, transpose=True)
    w8, w8t = orc.cast(w_bits, orc.E4M3, bw, transpose=True)
    g8, g8t = orc.cast(dy_bits, orc.E5M2, bg, transpose=True)
    for got, ref in ((b.x8, x8), (b.x8t, x8t), (b.w8, w8), (b.w8t, w8t), (b.dy8, g8), (b.dy8t, g8t)):
        assert np.array_equal(got.cpu().numpy(), ref)
    ry = sample_rows(lin.M, ROWS, 3)
    y = np_bits(b.y)
    assert rel_f(y[ry], orc.gemm_nt(x8, 0, bx, w8t, 0, bw, out_dt=orc.BF16, rows=ry)) <= REL_F_TOL
    dx = np_bits(b.dx)
    assert rel_f(dx[ry], orc.gemm_nt(g8, 1, bg, w8, 0, bw, out_dt=orc.BF16, rows=ry)) <= REL_F_TOL
    rdw = sample_rows(lin.K, ROWS, 4)
    dw = np_bits(b.dw)
    assert rel_f(dw[rdw], orc.gemm_nt(x8t, 0, bx, g8t, 1, bg, out_dt=orc.F32, rows=rdw)) <= REL_F_TOL
    # epilogue amax of Y and dX and the next consumers' biases
    assert u32(b.amax_y) == orc.scale_bias(y, orc.E4M3)[1]
    assert i32(b.by) == orc.bias_from_amax(u32(b.amax_y), orc.E4M3)[0]
    assert u32(b.amax_dx) == orc.scale_bias(dx, orc.E5M2)[1]
    assert i32(b.bdx) == orc.bias_from_amax(u32(b.amax_dx), orc.E5M2)[0]


PTQ = wl.WORKLOADS["llama2-70b-ptq"]


@functools.lru_cache(maxsize=4)
def oracle_ptq(wname: str):
    """The oracle's PTQ of one Llama-2-70B weight (shared by its prefill and
    decode cases)."""
    import oracle
    return oracle.ptq_quantise_weights(np_bits(tensor(PTQ.name, wname)))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("lname", [l.name for l in PTQ.linears])
def test_ptq_inference_parity(orc, gpu, lname):
    """ptq_quantise_weights then linear.infer_step (separate calls), every
    Llama-2-70B prefill (2048 tokens) and decode (16) shape: whole code
    tensors bit for bit, 256 output rows (all 16 at decode)."""
    lin = [l for l in PTQ.linears if l.name == lname][0]
    print(f"\n[case] ptq/{lname} M={lin.M} K={lin.K} N={lin.N}", flush=True)
    W, X = tensor(PTQ.name, lin.w), tensor(PTQ.name, lin.x)
    b = L.alloc(lin.M, lin.K, lin.N, gpu, train=False)
    F.ptq_quantise_weights(W.to(gpu), want_w8=False, w8t=b.w8t, bw=b.bw, flags=b.flags_w, ws=b.ws)
    L.infer_step(X.to(gpu), b)
    torch.cuda.synchronize()
    xb = np_bits(X)
    _, ow8t, obw, ofw = oracle_ptq(lin.w)
    assert (i32(b.bw), u32(b.flags_w)) == (obw, ofw)
    w8t = b.w8t.cpu().numpy()
    assert np.array_equal(w8t, ow8t)
    bx, ax, fx = orc.scale_bias(xb, 0)
    assert (i32(b.bx), u32(b.amax_x), u32(b.flags_x)) == (bx, ax, fx)
    x8 = orc.cast(xb, 0, bx)
    assert np.array_equal(b.x8.cpu().numpy(), x8)
    ry = sample_rows(lin.M, ROWS, 6)
    yref = orc.gemm_nt(x8, 0, bx, ow8t, 0, obw, out_dt=orc.BF16, rows=ry)
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
