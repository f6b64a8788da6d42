#!/usr/bin/env python3
"""Benchmark of the FP8 linear layer (amax + bias + cast + FP8 matmuls) on one GPU.

A step is one pass of the whole path over one batch of a workload (see
paper_2309_17224_amd.workloads): weight bias and cast, activation bias and
cast, forward matmul with epilogue amax, gradient bias and cast (E5), grad-input
matmul with epilogue amax, grad-weight matmul.  Inputs are synthetic, seeded,
already resident in HBM when timing starts.

Timed steps replay one HIP graph that holds the whole step (--launch eager
issues one host call per library call instead); a separate eager pass brackets
every call with HIP events for the per-kernel table.

Prints one JSON line:
  value      = 6*M*N*K per linear (fwd + bwd matmul FLOPs) / step time, TFLOP/s,
               on the Llama-2-70B MLP step (gate, up, down; 4096 tokens) by default
  roofline   = the dominant kernel against its roofline, timed with HIP events
  cpu_baseline = the CPU oracle on a bounded sample, extrapolated to one step
  configs    = the other workloads (GPT-111M, Llama-2-7B up, Llama-2-13B QKV,
               Llama-2-70B PTQ prefill + decode) timed in the same run
  mispredicted = the headline step over two input sets whose Eq. 3 biases
               differ, so that no bias prediction holds (every quantise casts
               twice)
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FP8_PEAK_TFLOPS = 5000.0     # MI355X dense FP8 MFMA, published
BF16_PEAK_TFLOPS = 2500.0    # MI355X dense bf16 MFMA, published
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, published
METRIC = "FP8 linear fwd+bwd TFLOP/s incl. amax+cast, % of FP8 MFMA peak"
DEFAULT_WORKLOAD = "llama2-70b-mlp"
# Workloads timed next to the headline in one default run (fewer steps each).
SIDE_WORKLOADS = ("gpt111m-linear", "llama2-7b-up", "llama2-13b-qkv", "llama2-70b-ptq")


def parse(argv=None):
    p = argparse.ArgumentParser(description=__doc__)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default=DEFAULT_WORKLOAD)
    p.add_argument("--margin", type=int, default=0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-budget", type=float, default=12.0,
                   help="seconds of oracle GEMM work in the CPU baseline sample")
    p.add_argument("--flush-mb", type=int, default=0,
                   help="write this many MB before every step (evicts the 256 MB MALL), and in the "
                        "per-call pass also before every decode matmul (weights from HBM, as in "
                        "token-by-token decode)")
    p.add_argument("--quant", choices=("predicted", "twopass", "separate", "delayed", "cscale"), default="predicted",
                   help="bias + cast of X, W, dY: one fp8_quantise call predicting each bias from "
                        "the previous step (identical bits; one read of an unchanged tensor), "
                        "fp8_quantise without prediction, fp8_scale_bias + fp8_cast, delayed scaling "
                        "(fp8_quantise_delayed: Eq. 3 of the largest amax of the last --history-len steps, "
                        "never re-cast: other bits than the just-in-time modes), or FP8-CSCALE "
                        "(constant bias --cscale-bias, no amax); the last two are not the headline metric")
    p.add_argument("--history-len", type=int, default=16, help="amax history length of --quant delayed")
    p.add_argument("--cscale-bias", type=int, default=0)
    p.add_argument("--streams", type=int, choices=(1, 2), default=1,
                   help="graph of the timed steps: independent calls (input quantises, gradient "
                        "quantises, each linear's grad-input and grad-weight matmuls) on two "
                        "streams, or everything on one")
    p.add_argument("--bias", choices=("fused", "separate"), default="fused",
                   help="bias of Y and dX: taken by the matmul launch itself (last workgroup), "
                        "or epilogue amax + fp8_bias_from_amax (identical bits)")
    p.add_argument("--launch", choices=("graph", "eager"), default="graph",
                   help="timed steps: replays of one HIP graph holding the whole step, or "
                        "one host call per library call")
    p.add_argument("--bias-per", choices=("tensor", "sequence"), default="tensor",
                   help="decoder-layer workloads: one activation bias per tensor and call (quantise fused "
                        "into the producing kernels), or one per sequence (segmented quantise, per-row-bias "
                        "matmuls)")
    p.add_argument("--no-quant-batch", action="store_true",
                   help="one fp8_quantise call per tensor instead of fp8_quantise_batch over the "
                        "tensors of each quantise phase (identical bits)")
    p.add_argument("--amax-mb", type=int, default=0,
                   help="only time fp8_scale_bias on a bf16 tensor of this many MB, --steps calls "
                        "(read-bandwidth reference for the amax kernel), then exit")
    p.add_argument("--copy-mb", type=int, default=0,
                   help="only run a plain device-to-device copy of this many MB, --steps times "
                        "(reference kernel for scaling hardware traffic counters), then exit")
    p.add_argument("--mfma-ceiling", type=int, default=0, metavar="ITERS",
                   help="only run the register-operand FP8 MFMA loop of libfp8probe.so (ITERS x 8 "
                        "instructions per wave, 8 waves on each of 256 workgroups), --steps launches: the "
                        "sustained matrix-core rate with no memory traffic, then exit")
    p.add_argument("--lds-probe", type=int, default=0, metavar="ITERS",
                   help="time the LDS read / LDS-copy probe of libfp8probe.so (ITERS loop trips) and exit")
    p.add_argument("--stream-ceiling", type=int, default=0, metavar="MB",
                   help="only run the cast-shaped stream of libfp8probe.so on a bf16 tensor of MB megabytes "
                        "(2 bytes read, 1 or 2 written per element; a read + write reference rate), --steps "
                        "launches each, then exit")
    p.add_argument("--no-configs", action="store_true",
                   help="time the chosen workload only (no table of the other workloads)")
    p.add_argument("--no-mispredicted", action="store_true",
                   help="skip the step over two input sets whose bias predictions never hold")
    p.add_argument("--side-steps", type=int, default=20,
                   help="timed steps of each workload in the configs table")
    return p.parse_args(argv)


def step_kwargs(args) -> dict:
    """WorkloadStep options of a bench run (the tests build the timed step
    with these, so that the benchmark times the configuration they check)."""
    return dict(margin=args.margin, quant=args.quant, cscale_bias=args.cscale_bias,
                fused_bias=args.bias == "fused", concurrent=args.streams == 2,
                batch_quant=not args.no_quant_batch, history_len=args.history_len)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def make_inputs(w):
    from paper_2309_17224_amd import workloads as wl
    t0 = time.time()
    cpu = {t.name: wl.make_tensor(w, t.name) for t in w.tensors}
    log(f"[bench] generated {len(cpu)} tensors in {time.time() - t0:.1f}s")
    return cpu


# Kernel kinds that, with --flush-mb, the per-call pass also times right after
# a flush: token-by-token decode reads each layer's weights once per token,
# with every other layer's weights read in between, so they come from HBM.
COLD_KINDS = ("gemm_decode",)


def time_steps(step, steps, warmup, flush=None):
    import torch
    for _ in range(warmup):
        if flush is not None:
            flush.add_(1)
        step.run()
    torch.cuda.synchronize()
    ncalls = len(step.calls)
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(ncalls)] for _ in range(steps)]
    fl_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        if flush is not None:
            fl_ev[s][0].record()
            flush.add_(1)
            fl_ev[s][1].record()
        for i, (_, kind, _, fn) in enumerate(step.calls):
            if flush is not None and kind in COLD_KINDS:
                fl_ev.append((torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)))
                fl_ev[-1][0].record()
                flush.add_(1)
                fl_ev[-1][1].record()
            ev[s][i][0].record()
            fn()
            ev[s][i][1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_call = [[ev[s][i][0].elapsed_time(ev[s][i][1]) * 1e-3 for i in range(ncalls)]
                for s in range(steps)]
    flush_s = sum(a.elapsed_time(b) * 1e-3 for a, b in fl_ev) if flush is not None else 0.0
    return wall, per_call, flush_s


def time_graph(step, steps, warmup, flush=None, capture=True):
    """Wall time of `steps` replays of the captured step (HIP graph).  With
    capture=False the step was captured beforehand (so that no idle gap for
    the capture lets the clocks fall right before the timed replays)."""
    import torch
    if capture:
        step.capture()
    for _ in range(warmup):
        if flush is not None:
            flush.add_(1)
        step.replay()
    torch.cuda.synchronize()
    fl_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(steps)]
    t0 = time.perf_counter()
    for s in range(steps):
        if flush is not None:
            fl_ev[s][0].record()
            flush.add_(1)
            fl_ev[s][1].record()
        step.replay()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    flush_s = sum(a.elapsed_time(b) * 1e-3 for a, b in fl_ev) if flush is not None else 0.0
    return wall, flush_s


def roofline(step, per_call):
    """Group per-call HIP-event durations by kernel kind; the dominant kind
    (largest total time) is reported against its roofline."""
    steps = len(per_call)
    kinds = {}
    for i, (label, kind, work, _) in enumerate(step.calls):
        t = sum(per_call[s][i] for s in range(steps))
        k = kinds.setdefault(kind, {"time": 0.0, "work": 0, "launches": 0})
        k["time"] += t
        k["work"] += work * steps
        k["launches"] += steps
    table = {}
    for kind, k in kinds.items():
        avg = k["time"] / k["launches"]
        per_launch = k["work"] / k["launches"]
        if kind == "gemm_decode":
            ach = per_launch / avg / 1e9 if avg > 0 else 0.0
            table[kind] = dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s",
                               frac=ach / HBM_PEAK_GBS, avg_us=avg * 1e6, per_launch=per_launch,
                               total_ms=k["time"] / steps * 1e3)
        elif kind.startswith("gemm"):
            ach = per_launch / avg / 1e12 if avg > 0 else 0.0
            table[kind] = dict(bound="mfma", achieved=ach, peak=FP8_PEAK_TFLOPS, unit="TFLOP/s",
                               frac=ach / FP8_PEAK_TFLOPS, avg_us=avg * 1e6, per_launch=per_launch,
                               total_ms=k["time"] / steps * 1e3)
        elif kind == "attention":
            ach = per_launch / avg / 1e12 if avg > 0 else 0.0
            table[kind] = dict(bound="mfma", achieved=ach, peak=BF16_PEAK_TFLOPS, unit="TFLOP/s",
                               frac=ach / BF16_PEAK_TFLOPS, avg_us=avg * 1e6, per_launch=per_launch,
                               total_ms=k["time"] / steps * 1e3)
        elif kind in ("amax", "cast", "quantise", "glue"):
            ach = per_launch / avg / 1e9 if avg > 0 else 0.0
            table[kind] = dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s",
                               frac=ach / HBM_PEAK_GBS, avg_us=avg * 1e6, per_launch=per_launch,
                               total_ms=k["time"] / steps * 1e3)
        else:
            table[kind] = dict(avg_us=avg * 1e6, total_ms=k["time"] / steps * 1e3)
    dom = max((k for k in table if "bound" in table[k]), key=lambda k: table[k]["total_ms"])
    d = table[dom]
    roof = {"bound": d["bound"], "achieved": round(d["achieved"], 2), "peak": d["peak"],
            "unit": d["unit"], "frac": round(d["frac"], 4), "traffic": None,
            "kernel": dom, "avg_launch_us": round(d["avg_us"], 2)}
    return roof, table


def measured_traffic(workload: str, kind: str):
    """HBM bytes per launch of `kind` from the hardware-counter runs stored in
    profiles/ (FETCH_SIZE and WRITE_SIZE scaled by a plain copy kernel), or
    None when there is no measurement for this workload or the kernel sources
    changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    h = hashlib.sha256()
    for src in ("fp8lin_gemm.hip", "fp8lin_amax_cast.hip", "fp8lin_fp8.h"):
        with open(os.path.join(ROOT, "paper_2309_17224_amd", "csrc", src), "rb") as f:
            h.update(f.read())
    if rec.get("kernel_sources_sha256") != h.hexdigest():
        return None
    return rec.get("bytes_per_launch", {}).get(kind)


def cpu_baseline(w, cpu_tensors, budget_s):
    """The oracle, as it is, on a bounded sample of one step: amax, bias and
    cast on the full tensors, the matmuls on sampled rows, extrapolated
    linearly in rows (every output row costs the same)."""
    import numpy as np
    import oracle as orc
    from paper_2309_17224_amd import workloads as wl
    bits = {k: wl.bf16_bits(v) for k, v in cpu_tensors.items()}
    t_quant = 0.0
    codes = {}
    fmt_of = {}
    for l in w.linears:
        fmt_of.setdefault(l.w, orc.E4M3)
        fmt_of.setdefault(l.x, orc.E4M3)
        if w.train:
            fmt_of.setdefault(l.dy, orc.E5M2)
    for name, fmt in fmt_of.items():
        t0 = time.perf_counter()
        b, _, _ = orc.scale_bias(bits[name], fmt)
        q, qT = orc.cast(bits[name], fmt, b, transpose=True)
        t_quant += time.perf_counter() - t0
        codes[name] = (q, qT, b, fmt)
    gemms = []
    for l in w.linears:
        x, wq = codes[l.x], codes[l.w]
        gemms.append(("fwd", x[0], x[3], x[2], wq[1], wq[3], wq[2], l.M))
        if w.train:
            g = codes[l.dy]
            gemms.append(("dx", g[0], g[3], g[2], wq[0], wq[3], wq[2], l.M))
            gemms.append(("dw", x[1], x[3], x[2], g[1], g[3], g[2], l.K))
    # calibrate rows per matmul so that the sample costs about budget_s
    per_row = []
    for name, A, fa, ba, B, fb, bb, rows in gemms:
        r = np.arange(min(4, rows))
        t0 = time.perf_counter()
        orc.gemm_nt(A, fa, ba, B, fb, bb, rows=r)
        per_row.append((time.perf_counter() - t0) / len(r))
    share = budget_s / max(1, len(gemms))
    t_gemm = 0.0
    sampled = []
    for (name, A, fa, ba, B, fb, bb, rows), pr in zip(gemms, per_row):
        nr = int(max(4, min(rows, share / max(pr, 1e-9))))
        r = np.linspace(0, rows - 1, nr).astype(np.int64)
        t0 = time.perf_counter()
        orc.gemm_nt(A, fa, ba, B, fb, bb, rows=r)
        dt = time.perf_counter() - t0
        t_gemm += dt * rows / nr
        sampled.append(f"{name}:{nr}/{rows} rows")
    flops = sum(2 * l.M * l.N * l.K * (3 if w.train else 1) for l in w.linears)
    total = t_quant + t_gemm
    cores = orc.num_threads()
    quant_elems = sum(bits[k].size for k in fmt_of)
    # amax + bias + cast at one thread on the first 2^24 elements of the
    # largest tensor (the oracle's two passes: amax, then the cast)
    big = max(fmt_of, key=lambda k: bits[k].size)
    sample = np.ascontiguousarray(bits[big].reshape(-1)[: 1 << 24])
    orc.set_num_threads(1)
    try:
        t0 = time.perf_counter()
        b1, _, _ = orc.scale_bias(sample, fmt_of[big])
        orc.cast(sample, fmt_of[big], b1)
        t1 = time.perf_counter() - t0
    finally:
        orc.set_num_threads(cores)
    return {"value": round(flops / total / 1e12, 6), "unit": "TFLOP/s", "cores": cores,
            "kind": "oracle",
            "sample": "amax+bias+cast of every tensor in full (%.1fs); matmuls on %s, fp64 "
                      "accumulation, extrapolated by rows to %.1fs" % (t_quant, ", ".join(sampled),
                                                                     t_gemm),
            "quantise": {"threads": cores, "elements": int(quant_elems), "seconds": round(t_quant, 3),
                         "GB_per_s": round(3 * quant_elems / t_quant / 1e9, 3),
                         "note": "amax + bias + cast (codes and transposed codes) of every tensor; "
                                 "GB/s counts 3 bytes per element"},
            "quantise_1_thread": {"threads": 1, "elements": int(sample.size), "tensor": big,
                                  "seconds": round(t1, 3), "GB_per_s": round(3 * sample.size / t1 / 1e9, 3),
                                  "note": "amax + bias + cast (codes only) of the first 2^24 elements"}}


def cpu_baseline_layer(cfg, cpu_tensors, sample_rows=256):
    """The oracle layer on the first `sample_rows` tokens of the call, with the
    weights quantised by the oracle beforehand (PTQ, not timed, as on the
    GPU); extrapolated linearly in tokens (the four linears, >99% of the
    work, cost the same per token; attention grows faster, so the estimate
    is optimistic for the oracle)."""
    import oracle as orc
    from oracle import decoder as D
    from paper_2309_17224_amd import workloads as wl
    bits = {k: wl.bf16_bits(v) for k, v in cpu_tensors.items()}
    p = {"g_attn": bits["g_attn"][0], "g_mlp": bits["g_mlp"][0]}
    for name, key in (("qkv", "Wqkv"), ("o", "Wo"), ("gate_up", "Wgu"), ("down", "Wd")):
        _, w8t, bw, _ = orc.ptq_quantise_weights(bits[key])
        p[name + "_w8t"], p[name + "_bw"] = w8t, bw
    n = min(sample_rows, cfg.rows)
    t0 = time.perf_counter()
    D.layer_forward(bits["H"][:n], p, min(cfg.seq_len, n), cfg.n_heads, cfg.n_kv_heads, cfg.d_head, cfg.ffn)
    dt = time.perf_counter() - t0
    flops = sum(2 * cfg.rows * K * N for _, K, N in cfg.linears())
    est = dt * cfg.rows / n
    return {"value": round(flops / est / 1e12, 6), "unit": "TFLOP/s", "cores": orc.num_threads(),
            "kind": "oracle",
            "sample": "oracle decoder layer (fp64; numpy matmuls of exactly decoded E4M3 codes) on the first "
                      "%d of %d tokens, %.1fs, extrapolated linearly in tokens to %.1fs" % (n, cfg.rows, dt, est)}


def bench_layer(args, cfg):
    """One forward call of a Llama 2 decoder layer with its four linears in
    FP8 (PTQ weights, per-call activation biases fused into the producing
    kernels).  value = FLOPs of the four linears / layer time."""
    import torch
    from paper_2309_17224_amd import decoder as DL
    from paper_2309_17224_amd import workloads as wl
    dev = torch.device("cuda:0")
    t0 = time.time()
    cpu = {t.name: wl.make_layer_tensor(cfg, t.name) for t in cfg.tensors()}
    log(f"[bench] generated {len(cpu)} tensors in {time.time() - t0:.1f}s")
    W = {k: v.to(dev) for k, v in cpu.items() if k != "H"}
    layer = DL.DecoderLayer(cfg, W, dev, bias_per=args.bias_per)
    layer.H.copy_(cpu["H"].to(dev))
    del W
    torch.cuda.synchronize()
    log(f"[bench] {cfg.name}: {len(layer.calls)} calls per layer; warmup {args.warmup}, steps {args.steps}")
    wall, per_call, _ = time_steps(layer, args.steps, args.warmup)
    eager_s = wall / args.steps
    step_s = eager_s
    if args.launch == "graph":
        gwall, _ = time_graph(layer, args.steps, args.warmup)
        step_s = gwall / args.steps
    flops = layer.linear_flops()
    value = flops / step_s / 1e12
    roof, table = roofline(layer, per_call)
    for kind, d in sorted(table.items()):
        log(f"[bench] {kind:9s} " + " ".join(f"{k}={v:.4g}" if isinstance(v, float) else f"{k}={v}"
                                             for k, v in d.items()))
    for i, (label, kind, work, _) in enumerate(layer.calls):
        avg = sum(pc[i] for pc in per_call) / len(per_call)
        log(f"[bench]   {label:32s} {avg * 1e6:8.1f} us")
    out = {
        "metric": METRIC, "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_s * 1e3, 4),
        "eager_ms_per_step": round(eager_s * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "fp8",
        "data": "synthetic",
        "config": {"workload": cfg.name, "description": cfg.description,
                   "linears": [dict(name=n, M=cfg.rows, K=K, N=N) for n, K, N in cfg.linears()],
                   "mode": "PTQ inference, one decoder layer fwd (four FP8 linears; RMSNorm, RoPE, "
                           "attention, SwiGLU in bf16 with fused FP8-AMAX quantise)",
                   "accumulate": "fp32", "outputs": "bf16", "activation_bias": f"per {args.bias_per}",
                   "launch": ("one HIP graph replay per layer call" if args.launch == "graph"
                              else "one host call per library call")},
        "frac_of_fp8_peak": round(value / FP8_PEAK_TFLOPS, 4),
        "roofline": roof,
        "kernels": {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv) for kk, vv in d.items()}
                    for k, d in table.items()},
    }
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline_layer(cfg, cpu)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


def time_alternating(step_a, step_b, steps, warmup):
    """Wall time per step of replays alternating between two captured steps
    that share their FP8 buffers (each predicts its biases from the other's
    last step), and the prediction hits of the last one."""
    import torch
    step_a.capture()
    step_b.capture()
    for _ in range(max(warmup, 5)):
        step_a.replay()
        step_b.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        (step_a if s % 2 == 0 else step_b).replay()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    last = step_a if (steps - 1) % 2 == 0 else step_b
    return wall / steps, last.prediction_hits()


def quantise_table(step, per_call):
    """Per quantise call: algorithmic bytes (2 read + 1 written per element),
    average time and rates against HBM peak, with and without the transposed
    copy of the codes (layout overhead)."""
    out = []
    steps = len(per_call)
    for i, (label, kind, work, _) in enumerate(step.calls):
        if kind not in ("quantise", "cast", "amax"):
            continue
        avg = sum(per_call[s][i] for s in range(steps)) / steps
        lay = getattr(step, "layout_bytes", {}).get(label, 0)
        gbs = work / avg / 1e9 if avg > 0 else 0.0
        out.append({"call": label, "avg_us": round(avg * 1e6, 2), "bytes": int(work), "GB_per_s": round(gbs, 1),
                    "frac_hbm": round(gbs / HBM_PEAK_GBS, 4), "transpose_bytes": int(lay),
                    "GB_per_s_incl_transpose": round((work + lay) / avg / 1e9, 1) if avg > 0 else 0.0,
                    "input_mb": round(2 * work / 3 / 1e6, 1)})
    return out


def stream_ceilings(mb=1024, launches=5):
    """Read + write rates of a cast-shaped stream (libfp8probe.so): GB/s for
    2 bytes read + 1 written and 2 read + 2 written per element.  A reference
    measured in the same run, not a bound: the tiled quantise passes exceed it
    on some tensors."""
    import ctypes
    import torch
    P = probe_lib()
    n = (mb << 20) // 2 // 16 * 16
    src = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    d1 = torch.empty(n, dtype=torch.uint8, device="cuda")
    d2 = torch.empty(n, dtype=torch.uint8, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    out = {}
    for label, second, nbytes in (("read2_write1", None, 3 * n), ("read2_write2", d2, 4 * n)):
        ts = []
        for i in range(launches + 2):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            if P.fp8probe_stream(ctypes.c_void_p(src.data_ptr()), n, ctypes.c_void_p(d1.data_ptr()),
                                 None if second is None else ctypes.c_void_p(second.data_ptr()), stream) != 0:
                raise SystemExit("fp8probe_stream failed")
            b.record()
            torch.cuda.synchronize()
            if i >= 2:
                ts.append(a.elapsed_time(b) * 1e-3)
        out[label] = round(nbytes / sorted(ts)[len(ts) // 2] / 1e9, 1)
    del src, d1, d2
    torch.cuda.empty_cache()
    return out


def input_hashes(cpu):
    from paper_2309_17224_amd import workloads as wl
    h = {k: wl.sha256(v) for k, v in cpu.items()}
    for k, v in h.items():
        log(f"[bench] input {k} {tuple(cpu[k].shape)} sha256 {v}")
    return h


def bench_workload(args, w, steps, warmup, cpu_baseline_budget=None, mispredicted=False):
    """Time one linear workload: eager per-call pass (HIP events), then
    graph replays (or eager steps).  Returns the result fields."""
    import torch
    from paper_2309_17224_amd import linear as L
    dev = torch.device("cuda:0")
    cpu = make_inputs(w)
    hashes = input_hashes(cpu)
    tens = {k: v.to(dev) for k, v in cpu.items()}
    torch.cuda.synchronize()
    step = L.WorkloadStep(w, tens, dev, **step_kwargs(args))
    if not w.train:
        step.prepare_inference()
    flush = None
    if args.flush_mb:
        flush = torch.zeros(args.flush_mb * (1 << 20) // 4, dtype=torch.float32, device=dev)
    log(f"[bench] {w.name}: {len(step.calls)} calls per step; warmup {warmup}, steps {steps}")
    if args.launch == "graph":
        # one untimed eager step, then the capture, both before any timing: the
        # GPU then stays busy from the eager pass into the replays (an idle gap
        # lets the clocks drop and the first timed replays run slow)
        step.run()
        step.capture()
    # eager pass: every call bracketed by HIP events on its stream (roofline table)
    wall, per_call, flush_s = time_steps(step, steps, warmup, flush)
    eager_step_s = (wall - flush_s) / steps
    step_s = eager_step_s
    if args.launch == "graph":
        gwall, gflush = time_graph(step, steps, warmup, flush, capture=False)
        step_s = (gwall - gflush) / steps
    hits = step.prediction_hits()
    flops = step.gemm_flops()
    roof, table = roofline(step, per_call)
    roof["traffic"] = measured_traffic(w.name, roof["kernel"])
    # The whole step at the rooflines (each call's work at the MFMA or HBM
    # peak): a step that takes far longer than that is bound by launch and
    # ramp latency, and no roofline fraction is claimed for it.
    floor_s = sum(work / (FP8_PEAK_TFLOPS * 1e12) if kind.startswith("gemm") and kind != "gemm_decode"
                  else work / (HBM_PEAK_GBS * 1e9) for _, kind, work, _ in step.calls)
    if floor_s < 0.1 * step_s:
        roof = {"bound": "latency", "achieved": None, "peak": None, "unit": None, "frac": None, "traffic": None,
                "kernel": roof["kernel"], "avg_launch_us": roof["avg_launch_us"],
                "note": "step at the rooflines %.1f us against %.1f us measured: launch-latency bound, "
                        "no roofline fraction claimed" % (floor_s * 1e6, step_s * 1e6)}
    for kind, d in sorted(table.items()):
        log(f"[bench] {kind:11s} " + " ".join(f"{k}={v:.4g}" if isinstance(v, float) else f"{k}={v}"
                                               for k, v in d.items()))
    res = {
        "value": round(flops / step_s / 1e12, 3), "ms_per_step": round(step_s * 1e3, 4),
        "eager_ms_per_step": round(eager_step_s * 1e3, 4),
        "frac_of_fp8_peak": round(flops / step_s / 1e12 / FP8_PEAK_TFLOPS, 4),
        "config": {"workload": w.name, "description": w.description,
                   "linears": [dict(name=l.name, M=l.M, K=l.K, N=l.N) for l in w.linears],
                   "mode": "train fwd+bwd" if w.train else "PTQ inference fwd",
                   "accumulate": "fp32", "outputs": "Y,dX bf16; dW fp32" if w.train else "Y bf16",
                   "margin": args.margin, "mall_flush_mb": args.flush_mb, "quant": args.quant,
                   "history_len": args.history_len if args.quant == "delayed" else None,
                   "quant_batch": not args.no_quant_batch, "output_bias": args.bias,
                   "launch": (f"one HIP graph replay per step, {args.streams} stream(s)" if args.launch == "graph"
                              else "one host call per library call"),
                   "inputs_sha256": hashes},
        "prediction_hits": {"hits": hits[0], "tensors": hits[1],
                            "note": "last timed step; inputs unchanged between steps"},
        "roofline": roof,
        "kernels": {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv) for kk, vv in d.items()}
                    for k, d in table.items()},
        "quantise_calls": quantise_table(step, per_call),
    }
    if mispredicted and args.quant == "predicted" and args.launch == "graph":
        # the same step over 2x the inputs (exact in bf16): every Eq. 3 bias
        # moves by one, so each replay's predictions (the other set's biases)
        # fail and every quantise re-casts its tensor
        tens2 = {k: v * 2 for k, v in tens.items()}
        step2 = L.WorkloadStep(w, tens2, dev, share=step, **step_kwargs(args))
        ms, mh = time_alternating(step, step2, steps, warmup)
        res["mispredicted"] = {"value": round(flops / ms / 1e12, 3), "ms_per_step": round(ms * 1e3, 4),
                               "prediction_hits": {"hits": mh[0], "tensors": mh[1]},
                               "inputs": "alternating steps over X, W, dY and over 2 X, 2 W, 2 dY"}
        del step2, tens2
    if cpu_baseline_budget is not None:
        log("[bench] timing the CPU oracle on a bounded sample")
        res["cpu_baseline"] = cpu_baseline(w, cpu, cpu_baseline_budget)
    del step, tens
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def probe_lib():
    import ctypes
    path = os.path.join(ROOT, "paper_2309_17224_amd", "libfp8probe.so")
    if not os.path.exists(path):
        raise SystemExit(f"{path} is missing: build it with `python -m paper_2309_17224_amd.build`")
    P = ctypes.CDLL(path)
    P.fp8probe_mfma_loop.restype = ctypes.c_int32
    P.fp8probe_mfma_loop.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_void_p]
    P.fp8probe_mfma_loop_flops.restype = ctypes.c_int64
    P.fp8probe_mfma_loop_flops.argtypes = [ctypes.c_int32, ctypes.c_int32]
    P.fp8probe_stream.restype = ctypes.c_int32
    P.fp8probe_stream.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                  ctypes.c_void_p]
    P.fp8probe_lds_src_bytes.restype = ctypes.c_int64
    P.fp8probe_lds_src_bytes.argtypes = []
    P.fp8probe_lds.restype = ctypes.c_int32
    P.fp8probe_lds.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    return P


def lds_probe(args):
    """LDS read and LDS-copy rates per compute unit of the matmul's main-loop
    traffic in isolation (measurement aid libfp8probe.so): 256 workgroups of
    8 waves, HIP events around each launch; bytes per compute unit = waves x
    iters x 8 KiB for each role."""
    import ctypes
    import torch
    P = probe_lib()
    src = torch.ones(int(P.fp8probe_lds_src_bytes()), dtype=torch.uint8, device="cuda")
    out = torch.zeros(256, dtype=torch.int32, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    iters = args.lds_probe
    roles = {0: (8, 0), 1: (0, 8), 2: (4, 4), 3: (4, 0)}  # (reading waves, copying waves)
    names = {0: "read_8_waves", 1: "copy_8_waves", 2: "copy_4_read_4", 3: "read_4_waves"}
    res = {}
    for mode in (0, 1, 2, 3):
        ts = []
        for i in range(max(args.warmup, 1) + args.steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            if P.fp8probe_lds(mode, iters, ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                              stream) != 0:
                raise SystemExit("fp8probe_lds failed")
            b.record()
            torch.cuda.synchronize()
            if i >= max(args.warmup, 1):
                ts.append(a.elapsed_time(b) * 1e-3)
        med = sorted(ts)[len(ts) // 2]
        rd, cp = roles[mode]
        per = iters * 8 * 1024
        res[names[mode]] = {"median_us": round(med * 1e6, 1),
                            "read_GB_per_s_per_cu": round(rd * per / med / 1e9, 1),
                            "copy_GB_per_s_per_cu": round(cp * per / med / 1e9, 1), "launches": len(ts)}
    print(json.dumps({"lds_probe": {"workgroups": 256, "iters": iters, **res}}), flush=True)


def stream_ceiling(args):
    """Read + write rate of a cast-shaped stream (measurement aid
    libfp8probe.so): 2 bytes read and 1 (codes) or 2 (codes and a second
    copy) written per element, HIP events around each launch."""
    import ctypes
    import torch
    P = probe_lib()
    n = (args.stream_ceiling << 20) // 2 // 16 * 16
    src = torch.randn(n, dtype=torch.float32, device="cuda").to(torch.bfloat16)
    d1 = torch.empty(n, dtype=torch.uint8, device="cuda")
    d2 = torch.empty(n, dtype=torch.uint8, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    res = {}
    for label, second, nbytes in (("read2_write1", None, 3 * n), ("read2_write2", d2, 4 * n)):
        ts = []
        for i in range(max(args.warmup, 1) + args.steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            st = P.fp8probe_stream(ctypes.c_void_p(src.data_ptr()), n, ctypes.c_void_p(d1.data_ptr()),
                                   None if second is None else ctypes.c_void_p(second.data_ptr()), stream)
            if st != 0:
                raise SystemExit("fp8probe_stream failed")
            b.record()
            torch.cuda.synchronize()
            if i >= max(args.warmup, 1):
                ts.append(a.elapsed_time(b) * 1e-3)
        med = sorted(ts)[len(ts) // 2]
        res[label] = {"bytes_per_launch": nbytes, "median_us": med * 1e6, "GB_per_s": nbytes / med / 1e9,
                      "frac_of_8TBps": nbytes / med / 8e12, "launches": len(ts)}
    print(json.dumps({"stream": {"elements": n, "input_mb": 2 * n / 1e6, **res}}), flush=True)


def mfma_ceiling(args):
    """Sustained FP8 matrix-core rate with no memory traffic (measurement aid
    libfp8probe.so): HIP events around each launch on the current stream."""
    import ctypes
    import torch
    P = probe_lib()
    blocks, iters = torch.cuda.get_device_properties(0).multi_processor_count, args.mfma_ceiling
    out = torch.zeros(blocks * 8, dtype=torch.float32, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    flops = P.fp8probe_mfma_loop_flops(blocks, iters)
    res = {}
    for vary in (1, 0):
        ts = []
        for i in range(max(args.warmup, 1) + args.steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            if P.fp8probe_mfma_loop(blocks, iters, vary, ctypes.c_void_p(out.data_ptr()), stream) != 0:
                raise SystemExit("fp8probe_mfma_loop failed")
            b.record()
            torch.cuda.synchronize()
            if i >= max(args.warmup, 1):
                ts.append(a.elapsed_time(b) * 1e-3)
        med = sorted(ts)[len(ts) // 2]
        res["random_operands" if vary else "fixed_operands"] = {
            "median_s": med, "TFLOP_per_s": flops / med / 1e12,
            "frac_of_fp8_peak": flops / med / 1e12 / FP8_PEAK_TFLOPS, "launches": len(ts)}
    print(json.dumps({"mfma_loop": {"workgroups": blocks, "waves_per_workgroup": 8, "iters": iters,
                                    "flop_per_launch": flops, **res}}), flush=True)


def main(argv=None):
    args = parse(argv)
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py measures one GPU only; --gpus %d is not supported: the "
                                   "path shards with no FP8-specific exchange (see the design notes), "
                                   "and this build measures the one-GPU share" % args.gpus}))
        sys.exit(2)
    import torch
    from paper_2309_17224_amd import fp8lin
    from paper_2309_17224_amd import workloads as wl
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    if args.copy_mb:
        nbytes = args.copy_mb << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_launch": nbytes, "launches": args.steps}))
        return
    if args.mfma_ceiling:
        mfma_ceiling(args)
        return
    if args.stream_ceiling:
        stream_ceiling(args)
        return
    if args.lds_probe:
        lds_probe(args)
        return
    fp8lin.lib()  # fails loudly when the HIP library is missing
    if args.amax_mb:
        # fp8_scale_bias (amax + Eq. 3 bias) of one bf16 tensor larger than the
        # 256 MB MALL, so every launch reads it from HBM
        n = (args.amax_mb << 20) // 2
        x = torch.randn(n, dtype=torch.float32, device="cuda").to(torch.bfloat16)
        ws = fp8lin.workspace(n, x.device)
        for _ in range(max(args.warmup, 1)):
            fp8lin.fp8_scale_bias(x, fp8lin.E4M3, ws=ws)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
        for a, b in ev:
            a.record()
            fp8lin.fp8_scale_bias(x, fp8lin.E4M3, ws=ws)
            b.record()
        torch.cuda.synchronize()
        ts = sorted(a.elapsed_time(b) * 1e-3 for a, b in ev)
        med = ts[len(ts) // 2]
        print(json.dumps({"amax_bytes_per_call": 2 * n, "calls": args.steps, "median_us": med * 1e6,
                          "GB_per_s": 2 * n / med / 1e9, "frac_of_8TBps": 2 * n / med / 8e12}))
        return
    if args.workload in wl.LAYERS:
        bench_layer(args, wl.LAYERS[args.workload])
        return
    w = wl.WORKLOADS[args.workload]
    ceil = stream_ceilings()
    log(f"[bench] cast-shaped stream reference (GB/s): {ceil}")
    res = bench_workload(args, w, args.steps, args.warmup,
                         cpu_baseline_budget=None if args.no_cpu_baseline else args.cpu_budget,
                         mispredicted=not args.no_mispredicted)
    out = {"metric": METRIC, "value": res.pop("value"), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": res.pop("ms_per_step"),
           "eager_ms_per_step": res.pop("eager_ms_per_step"), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "fp8", "data": "synthetic", "config": res.pop("config")}
    out.update(res)
    out.setdefault("cpu_baseline", None)
    # every quantise call against HBM peak (3 bytes per element) and against a
    # stream with the same bytes read and written, measured in the same run
    out["stream_reference_GBps"] = {
        **ceil, "source": "libfp8probe.so cast-shaped stream (contiguous range per workgroup, no arithmetic), "
                          "1 GiB bf16, HIP events; a reference, not a bound: tiled quantise passes exceed it "
                          "on some tensors"}
    for q in out.get("quantise_calls", []):
        wr2 = q["transpose_bytes"] > 0
        c = ceil["read2_write2"] if wr2 else ceil["read2_write1"]
        q["vs_stream_reference"] = round(q["GB_per_s_incl_transpose" if wr2 else "GB_per_s"] / c, 4)
    if not args.no_configs and args.workload == DEFAULT_WORKLOAD:
        side = {}
        for name in SIDE_WORKLOADS:
            r = bench_workload(args, wl.WORKLOADS[name], args.side_steps, min(args.warmup, 5))
            side[name] = {"value": r["value"], "unit": "TFLOP/s", "ms_per_step": r["ms_per_step"],
                          "frac_of_fp8_peak": r["frac_of_fp8_peak"], "steps": args.side_steps,
                          "description": r["config"]["description"],
                          "inputs_sha256": r["config"]["inputs_sha256"],
                          "roofline": r["roofline"],
                          "kernels": {k: {kk: v[kk] for kk in ("achieved", "unit", "frac", "avg_us")
                                          if kk in v} for k, v in r["kernels"].items()}}
        out["configs"] = side
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
