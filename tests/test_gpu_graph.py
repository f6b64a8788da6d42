"""A whole training step recorded into a HIP graph and replayed.

Every replay must reproduce the eager step bit for bit: the library launches
only kernels (no memset or copy nodes) and every kernel of the step is
deterministic (the only atomics are integer maxima).  Outputs are clobbered
before each replay and unrelated eager work runs between replays, so a replay
that skipped or reordered work would show.
"""
import pytest
import torch

from paper_2309_17224_amd import linear as L
from paper_2309_17224_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _outputs(step):
    out = {}
    for name, qt in step.q.items():
        if qt.q is not None:
            out[f"{name}.q"] = qt.q
        if qt.qT is not None:
            out[f"{name}.qT"] = qt.qT
        out[f"{name}.scal"] = qt.scal
    for lname, o in step.out.items():
        for k, v in o.items():
            out[f"{lname}.{k}"] = v
    return out


def _bits(t):
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.view(torch.int16)
    if t.dtype == torch.float32:
        return t.view(torch.int32)
    return t


def _make_step(dev, name="gpt111m-linear"):
    w = wl.WORKLOADS[name]
    tens = {t.name: wl.make_tensor(w, t.name).to(dev) for t in w.tensors}
    return w, tens, L.WorkloadStep(w, tens, dev)


def test_graph_replay_matches_eager(gpu):
    w, tens, step = _make_step(gpu)
    step.run()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in _outputs(step).items()}
    step.capture()
    junk = torch.randn(1 << 20, device=gpu)
    for rep in range(4):
        for v in _outputs(step).values():
            if v.is_floating_point():
                v.fill_(float("nan"))
            else:
                v.fill_(0x5A)
        junk.mul_(1.0001).add_(0.5)  # unrelated eager work between replays
        float(junk.sum())
        step.replay()
        torch.cuda.synchronize()
        for k, v in _outputs(step).items():
            assert torch.equal(_bits(v), _bits(ref[k])), f"replay {rep}: {k} differs from the eager step"


def test_graph_replay_reads_current_inputs(gpu):
    """Doubling X after capture: its bias drops by one, its codes stay, and
    Y and dW (which carry one factor of X) double exactly."""
    w, tens, step = _make_step(gpu)
    step.capture()
    step.replay()
    torch.cuda.synchronize()
    lin = w.linears[0]
    ref = {k: v.clone() for k, v in _outputs(step).items()}
    tens[lin.x].mul_(2)
    step.replay()
    torch.cuda.synchronize()
    out = _outputs(step)
    assert int(out[f"{lin.x}.scal"][0]) == int(ref[f"{lin.x}.scal"][0]) - 1
    assert torch.equal(out[f"{lin.x}.q"], ref[f"{lin.x}.q"])
    assert torch.equal(_bits(out[f"{lin.name}.y"]), _bits(ref[f"{lin.name}.y"] * 2))
    assert torch.equal(_bits(out[f"{lin.name}.dw"]), _bits(ref[f"{lin.name}.dw"] * 2))
    assert torch.equal(_bits(out[f"{lin.name}.dx"]), _bits(ref[f"{lin.name}.dx"]))


def test_step_quant_modes_identical(gpu):
    """Predicted-bias quantise, two-pass quantise and the separate amax + cast
    calls give the same bits for every output of the step, eager and replayed
    (the predicted mode is right after the first step and wrong in the first)."""
    w = wl.WORKLOADS["gpt111m-linear"]
    tens = {t.name: wl.make_tensor(w, t.name).to(gpu) for t in w.tensors}
    outs = {}
    for mode in ("predicted", "twopass", "separate"):
        step = L.WorkloadStep(w, tens, gpu, quant=mode)
        step.run()
        step.capture()
        step.replay()
        step.replay()
        torch.cuda.synchronize()
        outs[mode] = {k: v.clone() for k, v in _outputs(step).items()}
    ref = outs["separate"]
    for mode in ("predicted", "twopass"):
        for k, v in outs[mode].items():
            assert torch.equal(_bits(v), _bits(ref[k])), f"{mode}: {k} differs"


@pytest.mark.parametrize("workload", ["gpt111m-linear", "llama2-70b-mlp"])
@pytest.mark.parametrize("fused_bias", [True, False])
def test_concurrent_graph_matches_sequential(gpu, workload, fused_bias):
    """The two-stream graph (independent quantises and each linear's
    grad-input / grad-weight matmuls forked onto a side stream) gives the bits
    of the one-stream eager step, replay after replay."""
    w = wl.WORKLOADS[workload]
    tens = {t.name: wl.make_tensor(w, t.name).to(gpu) for t in w.tensors}
    seq = L.WorkloadStep(w, tens, gpu, fused_bias=fused_bias, concurrent=False)
    seq.run()
    seq.run()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in _outputs(seq).items()}
    del seq
    step = L.WorkloadStep(w, tens, gpu, fused_bias=fused_bias, concurrent=True)
    assert any(b == 1 for _, b in step.sched)
    step.run()
    step.capture()
    for rep in range(3):
        for v in _outputs(step).values():
            if v.is_floating_point():
                v.fill_(float("nan"))
            else:
                v.fill_(0x5A)
        step.replay()
        torch.cuda.synchronize()
        for k, v in _outputs(step).items():
            assert torch.equal(_bits(v), _bits(ref[k])), f"replay {rep}: {k}"
