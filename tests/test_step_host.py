"""Host-side properties of WorkloadStep (no GPU needed): the schedule of
independent calls, and that a step is freed as soon as it is dropped (no
reference cycle), so a step that owns a HIP graph is never destroyed by the
cyclic garbage collector in the middle of another step's graph capture."""
import gc
import weakref

import pytest
import torch

from paper_2309_17224_amd import linear as L
from paper_2309_17224_amd import workloads as wl


def cpu_step(name, **kw):
    w = wl.WORKLOADS[name]
    tens = {t.name: torch.zeros(t.rows, t.cols, dtype=torch.bfloat16) for t in w.tensors}
    return w, L.WorkloadStep(w, tens, "cpu", **kw)


@pytest.mark.parametrize("fused_bias", [True, False])
@pytest.mark.parametrize("quant", ["predicted", "separate", "cscale"])
def test_step_is_not_a_reference_cycle(fused_bias, quant):
    was = gc.isenabled()
    gc.disable()
    try:
        _, step = cpu_step("llama2-70b-mlp", fused_bias=fused_bias, quant=quant)
        ref = weakref.ref(step)
        del step
        assert ref() is None, "WorkloadStep is kept alive by a reference cycle"
    finally:
        if was:
            gc.enable()


def test_schedule_pairs_independent_calls():
    w, step = cpu_step("llama2-70b-mlp")
    labels = [c[0] for c in step.calls]
    assert len(step.sched) == len(step.calls)
    for l in w.linears:
        i, j = labels.index(f"dx {l.name}"), labels.index(f"dw {l.name}")
        assert step.sched[i][0] == step.sched[j][0] and step.sched[i][1] != step.sched[j][1]
    # forwards run on their own; quantise phases hold only quantise calls
    for (label, kind, _, _), (phase, _) in zip(step.calls, step.sched):
        if label.startswith("fwd"):
            assert phase is None
        if phase is not None and phase.startswith("quantise"):
            assert kind == "quantise"
    assert not step.concurrent  # CPU device: no side stream


def test_separate_bias_stays_after_its_matmul_on_one_branch():
    _, step = cpu_step("gpt111m-linear", fused_bias=False)
    labels = [c[0] for c in step.calls]
    for name in ("linear",):
        i, j = labels.index(f"dx {name}"), labels.index(f"bias dx {name}")
        assert j == i + 1 and step.sched[i] == step.sched[j]
