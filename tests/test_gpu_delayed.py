"""GPU parity of delayed scaling (fp8_quantise_delayed; the amax-history
remedy Sec. 3 cites for the second pass over a tensor) against the oracle's
quantise_delayed, call by call: the bias each call casts with, the codes and
transposed codes, the tensor's amax and flags (FP8_FLAG_SATURATED where the
codes clip, App. A), the next call's bias (Eq. 3 of the history maximum) and
the history ring itself.  Bar: bit for bit (integer work)."""
import numpy as np
import pytest
import torch

from paper_2309_17224_amd import fp8lin as F
from paper_2309_17224_amd import linear as L
from paper_2309_17224_amd import workloads as wl
from parity_util import REL_F_TOL, i32, np_bits, rel_f, sample_rows, u32

pytestmark = pytest.mark.gpu


def with_amax(rows, cols, amax, seed, dtype=torch.bfloat16):
    """Values of magnitude at most amax / 2 and amax itself once (exact in
    bf16 for the powers of two and small integers used here)."""
    g = torch.Generator().manual_seed(seed)
    x = (torch.rand(rows, cols, generator=g) - 0.5) * amax
    x[seed % rows, (3 * seed) % cols] = amax if seed % 2 else -amax
    return x.to(dtype)


def run_sequence(orc, gpu, xs, fmt, hlen, margin=0, bias0=0):
    bias = torch.tensor([bias0], dtype=torch.int32, device=gpu)
    hist = torch.zeros(hlen, dtype=torch.int32, device=gpu)
    count = torch.zeros(1, dtype=torch.int32, device=gpu)
    cpu_xs = [x if x.dtype == torch.float32 else x for x in xs]
    ref, ref_hist = orc.quantise_delayed([np_bits(x) for x in cpu_xs], fmt, margin, hlen, bias0)
    for t, (x, r) in enumerate(zip(xs, ref)):
        used = i32(bias)
        q, qT, _, a, fl = F.fp8_quantise_delayed(x.to(gpu), fmt, bias, hist, count, margin, want_qT=True)
        torch.cuda.synchronize()
        print(f"[case] call {t} {tuple(x.shape)} used {used} -> next {i32(bias)} flags {u32(fl)}", flush=True)
        assert used == r["bias"]
        assert (i32(bias), u32(a), u32(fl)) == (r["next_bias"], r["amax"], r["flags"])
        rq = r["q"].reshape(x.shape) if x.numel() else r["q"]
        assert np.array_equal(q.cpu().numpy(), rq)
        assert np.array_equal(qT.cpu().numpy(), rq.T)
    assert (hist.cpu().numpy().view(np.uint32) == np.array(ref_hist, np.uint32)).all()
    assert u32(count) == len(xs)
    return ref


def test_hand_worked_sequence(orc, gpu):
    # amaxes 1, 8, 2, 0.5, 0.5 with a history of 2 (tests/golden/delayed_bias_cases.txt)
    xs = [with_amax(130, 257, a, seed=i + 1) for i, a in enumerate([1.0, 8.0, 2.0, 0.5, 0.5])]
    ref = run_sequence(orc, gpu, xs, F.E4M3, 2)
    assert [r["bias"] for r in ref] == [0, 8, 5, 5, 7]
    assert [bool(r["flags"] & F.FLAG_SATURATED) for r in ref] == [False, True, False, False, False]


@pytest.mark.parametrize("fmt", [F.E4M3, F.E5M2])
@pytest.mark.parametrize("hlen", [1, 3, 300])
def test_random_sequences(orc, gpu, fmt, hlen):
    g = torch.Generator().manual_seed(hlen * 10 + fmt)
    xs = []
    for t in range(7):
        scale = 2.0 ** float(torch.randint(-20, 8, (1,), generator=g))
        shape = [(300, 517), (128, 128), (1, 1000), (257, 3), (1000, 129), (64, 64), (17, 900)][t]
        xs.append((torch.randn(*shape, generator=g) * scale).to(torch.bfloat16))
    run_sequence(orc, gpu, xs, fmt, hlen, margin=1 if fmt == F.E5M2 else 0, bias0=-3)


def test_special_tensors_and_fp32(orc, gpu):
    z = torch.zeros(50, 70)
    nan = torch.randn(50, 70)
    nan[3, 4] = float("nan")
    inf = torch.randn(50, 70)
    inf[7, 1] = float("-inf")
    big = torch.randn(50, 70) * 1e30
    xs = [torch.randn(50, 70), z, nan, torch.randn(50, 70), inf, big, torch.randn(50, 70) * 1e-30]
    run_sequence(orc, gpu, xs, F.E5M2, 2)                           # fp32 inputs
    run_sequence(orc, gpu, [x.to(torch.bfloat16) for x in xs], F.E4M3, 3, margin=2)


def test_empty_tensor_records_zero(orc, gpu):
    xs = [torch.randn(40, 40).to(torch.bfloat16), torch.empty(0, 40, dtype=torch.bfloat16),
          torch.randn(40, 40).to(torch.bfloat16)]
    bias = torch.zeros(1, dtype=torch.int32, device=gpu)
    hist = torch.zeros(2, dtype=torch.int32, device=gpu)
    count = torch.zeros(1, dtype=torch.int32, device=gpu)
    ref, _ = orc.quantise_delayed([np_bits(x) for x in xs], F.E4M3, 0, 2, 0)
    for x, r in zip(xs, ref):
        used = i32(bias)
        q, _, _, a, fl = F.fp8_quantise_delayed(x.to(gpu), F.E4M3, bias, hist, count)
        torch.cuda.synchronize()
        assert (used, i32(bias), u32(a), u32(fl)) == (r["bias"], r["next_bias"], r["amax"], r["flags"])


def test_step_in_delayed_mode(orc, gpu):
    """WorkloadStep(quant="delayed") on the GPT-111M workload: the first step
    casts every tensor with bias 0 (clipping and flushing), later steps with
    the history's Eq. 3 bias, which for unchanged tensors is the exact one:
    the codes of step 3 are FP8-AMAX's, the matmuls rel_F <= 1e-3."""
    w = wl.WORKLOADS["gpt111m-linear"]
    cpu = {t.name: wl.make_tensor(w, t.name) for t in w.tensors}
    tens = {k: v.to(gpu) for k, v in cpu.items()}
    step = L.WorkloadStep(w, tens, gpu, quant="delayed", history_len=4)
    lin = w.linears[0]
    fmts = {lin.x: F.E4M3, lin.w: F.E4M3, lin.dy: F.E5M2}
    step.run()
    torch.cuda.synchronize()
    for name, fmt in fmts.items():
        oq = orc.cast(np_bits(cpu[name]), fmt, 0)
        assert np.array_equal(step.q[name].q.cpu().numpy(), oq)
    step.run()
    step.run()
    torch.cuda.synchronize()
    codes = {}
    for name, fmt in fmts.items():
        ob, oa, _ = orc.scale_bias(np_bits(cpu[name]), fmt)
        qt = step.q[name]
        assert (i32(qt.bias), u32(qt.amax), u32(qt.flags)) == (ob, oa, 0)
        oq, oqT = orc.cast(np_bits(cpu[name]), fmt, ob, transpose=True)
        assert np.array_equal(qt.q.cpu().numpy(), oq) and np.array_equal(qt.qT.cpu().numpy(), oqT)
        codes[name] = (oq, oqT, ob)
    o = step.out[lin.name]
    rows = sample_rows(lin.M, 256, 1)
    x8, x8t, bx = codes[lin.x]
    w8, w8t, bw = codes[lin.w]
    g8, g8t, bg = codes[lin.dy]
    assert rel_f(np_bits(o["y"])[rows], orc.gemm_nt(x8, 0, bx, w8t, 0, bw, out_dt=orc.BF16, rows=rows)) <= REL_F_TOL
    assert rel_f(np_bits(o["dx"])[rows], orc.gemm_nt(g8, 1, bg, w8, 0, bw, out_dt=orc.BF16, rows=rows)) <= REL_F_TOL
    rdw = sample_rows(lin.K, 256, 2)
    assert rel_f(np_bits(o["dw"])[rdw], orc.gemm_nt(x8t, 0, bx, g8t, 1, bg, out_dt=orc.F32, rows=rdw)) <= REL_F_TOL
