"""The FP8 linear layer of the paper as a sequence of library calls.

Training (Sec. 2, 2.2, 2.3, 3): three scaling biases per layer and call,
  b_w = bias(W, E4)   W8, W8T = cast_E4(W * 2^b_w)     (after each weight update)
  b_x = bias(X, E4)   X8, X8T = cast_E4(X * 2^b_x)
  Y   = 2^-(b_x + b_w) X8 . W8                          (fp32 accumulate)
  b_g = bias(dY, E5) - margin   dY8, dY8T = cast_E5(dY * 2^b_g)
  dX  = 2^-(b_g + b_w) dY8 . W8^T
  dW  = 2^-(b_x + b_g) X8^T . dY8
The forward and grad-input matmuls also return the amax of their outputs
(epilogue reduction), from which the next consumer's bias is taken without a
second read of Y or dX (fp8_bias_from_amax).

Inference (Sec. 3.1): W8T and b_w come once from ptq_quantise_weights; each
call computes b_x and X8, then the forward matmul.

Every buffer is allocated once, up front; a step launches kernels only.
"""
from __future__ import annotations

import gc
from dataclasses import dataclass

import torch

from . import fp8lin as F


@dataclass
class LinearBuffers:
    M: int
    K: int
    N: int
    device: torch.device
    w8: torch.Tensor
    w8t: torch.Tensor
    x8: torch.Tensor
    x8t: torch.Tensor
    dy8: torch.Tensor
    dy8t: torch.Tensor
    y: torch.Tensor
    dx: torch.Tensor
    dw: torch.Tensor
    scal: torch.Tensor      # int32 [16]: biases, amax bits, flags
    ws: torch.Tensor

    # views into scal
    @property
    def bw(self): return self.scal[0:1]
    @property
    def bx(self): return self.scal[1:2]
    @property
    def bg(self): return self.scal[2:3]
    @property
    def by(self): return self.scal[3:4]       # bias of Y for the next layer (E4)
    @property
    def bdx(self): return self.scal[4:5]      # bias of dX for the previous layer (E5)
    @property
    def amax_w(self): return self.scal[5:6]
    @property
    def amax_x(self): return self.scal[6:7]
    @property
    def amax_g(self): return self.scal[7:8]
    @property
    def amax_y(self): return self.scal[8:9]
    @property
    def amax_dx(self): return self.scal[9:10]
    @property
    def flags_w(self): return self.scal[10:11]
    @property
    def flags_x(self): return self.scal[11:12]
    @property
    def flags_g(self): return self.scal[12:13]
    @property
    def flags_y(self): return self.scal[13:14]
    @property
    def flags_dx(self): return self.scal[14:15]


def alloc(M: int, K: int, N: int, device, y_dtype=torch.bfloat16, dx_dtype=torch.bfloat16,
          dw_dtype=torch.float32, train: bool = True) -> LinearBuffers:
    u8 = dict(dtype=torch.uint8, device=device)
    e = torch.empty
    nmax = max(M * K, K * N, M * N)
    return LinearBuffers(
        M, K, N, torch.device(device),
        w8=e((K, N), **u8) if train else e((0, 0), **u8), w8t=e((N, K), **u8),
        x8=e((M, K), **u8), x8t=e((K, M), **u8) if train else e((0, 0), **u8),
        dy8=e((M, N), **u8) if train else e((0, 0), **u8),
        dy8t=e((N, M), **u8) if train else e((0, 0), **u8),
        y=e((M, N), dtype=y_dtype, device=device),
        dx=e((M, K), dtype=dx_dtype, device=device) if train else e((0, 0), dtype=dx_dtype, device=device),
        dw=e((K, N), dtype=dw_dtype, device=device) if train else e((0, 0), dtype=dw_dtype, device=device),
        scal=torch.zeros(16, dtype=torch.int32, device=device),
        ws=F.workspace(nmax, device),
    )


def quantise_weight(w: torch.Tensor, b: LinearBuffers) -> None:
    """bias + cast of the weight: after every weight update (Sec. 3.2), or
    once at checkpoint load (Sec. 3.1)."""
    F.fp8_scale_bias(w, F.E4M3, 0, bias=b.bw, amax_bits=b.amax_w, flags=b.flags_w, ws=b.ws)
    F.fp8_cast_e4(w, b.bw, q=b.w8, qT=b.w8t)


def forward(x: torch.Tensor, b: LinearBuffers, keep_xt: bool = True) -> torch.Tensor:
    F.fp8_scale_bias(x, F.E4M3, 0, bias=b.bx, amax_bits=b.amax_x, flags=b.flags_x, ws=b.ws)
    F.fp8_cast_e4(x, b.bx, q=b.x8, qT=b.x8t if keep_xt else None, want_qT=keep_xt)
    F.fp8_linear_fwd(b.x8, b.bx, b.w8t, b.bw, y=b.y, y_amax_bits=b.amax_y)
    F.fp8_bias_from_amax(b.amax_y, F.E4M3, 0, bias=b.by, flags=b.flags_y)
    return b.y


def backward(dy: torch.Tensor, b: LinearBuffers, margin: int = 0):
    F.fp8_scale_bias(dy, F.E5M2, margin, bias=b.bg, amax_bits=b.amax_g, flags=b.flags_g, ws=b.ws)
    F.fp8_cast_e5(dy, b.bg, q=b.dy8, qT=b.dy8t)
    F.fp8_linear_bwd_dx(b.dy8, b.bg, b.w8, b.bw, dx=b.dx, dx_amax_bits=b.amax_dx)
    F.fp8_bias_from_amax(b.amax_dx, F.E5M2, margin, bias=b.bdx, flags=b.flags_dx)
    F.fp8_linear_bwd_dw(b.x8t, b.bx, b.dy8t, b.bg, dw=b.dw)
    return b.dx, b.dw


def train_step(x: torch.Tensor, w: torch.Tensor, dy: torch.Tensor, b: LinearBuffers,
               margin: int = 0):
    """One fwd + bwd pass of one FP8 linear layer, weight cast included."""
    quantise_weight(w, b)
    y = forward(x, b)
    dx, dw = backward(dy, b, margin)
    return y, dx, dw


def infer_step(x: torch.Tensor, b: LinearBuffers) -> torch.Tensor:
    """PTQ inference call: activation bias + cast, then the forward matmul
    with the weight quantised beforehand (quantise_weight / ptq)."""
    F.fp8_scale_bias(x, F.E4M3, 0, bias=b.bx, amax_bits=b.amax_x, flags=b.flags_x, ws=b.ws)
    F.fp8_cast_e4(x, b.bx, q=b.x8)
    F.fp8_linear_fwd(b.x8, b.bx, b.w8t, b.bw, y=b.y)
    return b.y


# ---------------------------------------------------------------- workloads
class Fp8Tensor:
    """Device buffers of one high-precision tensor's FP8 form: codes, the
    transposed codes, and [bias, amax bits, flags] as int32."""

    def __init__(self, rows: int, cols: int, device, want_q=True, want_qT=True):
        u8 = dict(dtype=torch.uint8, device=device)
        self.q = torch.empty((rows, cols), **u8) if want_q else None
        self.qT = torch.empty((cols, rows), **u8) if want_qT else None
        self.scal = torch.zeros(3, dtype=torch.int32, device=device)
        self.qws = self.sws = None  # quantise / scale-bias workspaces (set by the step)

    @property
    def bias(self): return self.scal[0:1]
    @property
    def amax(self): return self.scal[1:2]
    @property
    def flags(self): return self.scal[2:3]


class WorkloadStep:
    """One pass of the FP8 path over all linear layers of a workload.

    Training: every weight and every distinct activation / gradient tensor is
    amax-scaled and cast once (an activation shared by several linears, such
    as the input of gate and up projections, is cast once), then the forward,
    grad-input and grad-weight matmuls of each linear run, the first two with
    the epilogue amax and the bias of their outputs.  Inference: activations
    are scaled and cast per call, weights once beforehand (PTQ).
    ``calls`` lists (label, kind, flops_or_bytes, fn); running them in order
    is one step.

    quant: how each tensor gets its bias and codes.
      "predicted": fp8_quantise with the tensor's previous bias as the
                   prediction (one read of the tensor when it is unchanged);
      "twopass":   fp8_quantise without a prediction (amax pass, then cast);
      "separate":  fp8_scale_bias followed by fp8_cast_e4/e5.
    All three give identical bits (FP8-AMAX, Sec. 2.3).
      "delayed":   delayed scaling (the amax-history remedy of Sec. 3):
                   fp8_quantise_delayed casts each tensor once with Eq. 3 of
                   the largest amax of its last `history_len` steps (0 before
                   the first), records its own amax, never recasts; a tensor
                   that outgrows its history clips (App. A).
      "cscale":    FP8-CSCALE (Sec. 3): one constant bias `cscale_bias` for every
                   weight, activation and gradient; no amax, only the casts and
                   the matmuls (no epilogue amax either).
    fused_bias: the forward and grad-input matmuls take the bias of their
      outputs in the same launch (fp8_linear_fwd_bias / fp8_linear_bwd_dx_bias);
      False: epilogue amax, then fp8_bias_from_amax (identical bits).
    batch_quant: with "predicted" or "twopass" and one stream, the weight and
      the input of each linear, which are ready together before its forward
      matmul, go through one fp8_quantise_batch call: two launches instead of
      four, same bits.  Tensors of different linears are never batched (in a
      network one linear's input is produced by the linear before it).
    concurrent: capture() records independent calls on two streams (the
      quantise calls of the weights and activations, those of the gradients,
      and each linear's grad-input and grad-weight matmuls), so that the last
      partial round of workgroups of one kernel can overlap the other; run()
      always issues the calls one after another.  Same bits either way.  Off
      by default: on the measured workloads it gained nothing (the paired
      matmuls still need the same number of rounds of workgroups) and cost 3 %
      on the Llama-2-70B MLP step (operand panels of two kernels share L2).
    """

    QUANT_MODES = ("predicted", "twopass", "separate", "delayed", "cscale")

    def __init__(self, workload, tensors: dict, device, margin: int = 0, quant: str = "predicted",
                 cscale_bias: int = 0, fused_bias: bool = True, concurrent: bool = False,
                 batch_quant: bool = True, share: "WorkloadStep | None" = None, history_len: int = 16):
        """share: another step of the same workload whose FP8 buffers, biases
        and outputs this one uses (its own input tensors only): steps over two
        input sets that write one set of codes, each taking its bias
        predictions from the other's last step."""
        if quant not in self.QUANT_MODES:
            raise ValueError(f"quant must be one of {self.QUANT_MODES}")
        self.fused_bias = bool(fused_bias)
        self.w = workload
        self.t = tensors
        self.dev = torch.device(device)
        self.margin = margin
        self.quant = quant
        self.cscale_bias = int(cscale_bias)
        lin = workload.linears
        train = workload.train
        if share is not None:
            if share.w is not workload:
                raise ValueError("a shared step must run the same workload")
            self.ws, self.q, self.out, self.bws = share.ws, share.q, share.out, share.bws
        else:
            nmax = max(x.numel() for x in tensors.values())
            self.ws = F.workspace(nmax, device)
            self.q = {}
            for l in lin:
                K, N, M = l.K, l.N, l.M
                if l.w not in self.q:
                    self.q[l.w] = Fp8Tensor(K, N, device, want_q=train, want_qT=True)
                if l.x not in self.q:
                    self.q[l.x] = Fp8Tensor(M, K, device, want_q=True, want_qT=train)
                if train and l.dy not in self.q:
                    self.q[l.dy] = Fp8Tensor(M, N, device, want_q=True, want_qT=True)
            self.out = {}
            for l in lin:
                o = dict(y=torch.empty((l.M, l.N), dtype=torch.bfloat16, device=device),
                         y_scal=torch.zeros(3, dtype=torch.int32, device=device))
                if train:
                    o.update(dx=torch.empty((l.M, l.K), dtype=torch.bfloat16, device=device),
                             dw=torch.empty((l.K, l.N), dtype=torch.float32, device=device),
                             dx_scal=torch.zeros(3, dtype=torch.int32, device=device))
                self.out[l.name] = o
            # bias workspaces of the forward and grad-input matmuls (zero between calls)
            self.bws = {l.name: F.bias_workspace(device) for l in lin}
            # a workspace per tensor: calls on different streams never share one
            for name, qt in self.q.items():
                x = tensors[name]
                qt.qws = torch.empty(max(F.fp8_quantise_ws_bytes(*x.shape), 4), dtype=torch.uint8, device=device)
                qt.sws = F.workspace(x.numel(), device)
        # transposed-code bytes each quantise / cast call writes beyond its
        # algorithmic 3 bytes per element (layout overhead, reported apart)
        self.layout_bytes = {}
        # delayed scaling: per tensor an amax history (zeros) and a call count
        self.history_len = int(history_len)
        self.hist = {}
        if quant == "delayed":
            for name in self.q:
                self.hist[name] = (torch.zeros(self.history_len, dtype=torch.int32, device=device),
                                   torch.zeros(1, dtype=torch.int32, device=device))
                self.q[name].bias.zero_()
        self.concurrent = bool(concurrent) and self.dev.type == "cuda"
        self.batch_quant = bool(batch_quant) and not self.concurrent and quant in ("predicted", "twopass")
        self.side = torch.cuda.Stream(self.dev) if self.concurrent else None  # default priority
        self.sched = []
        self.calls = self._build()

    def _layout(self, name) -> int:
        """Bytes of the second (transposed) copy of a tensor's codes."""
        qt = self.q[name]
        return self.t[name].numel() if qt.qT is not None and qt.q is not None else 0

    def _quant(self, name, fmt, margin):
        """Work of a quantise or cast call: its algorithmic bytes, 2 read + 1
        written per element; a transposed copy is layout overhead, recorded in
        layout_bytes under the call's label."""
        x = self.t[name]
        qt = self.q[name]
        cast = F.fp8_cast_e4 if fmt == F.E4M3 else F.fp8_cast_e5
        n = x.numel()
        if self.quant == "cscale":
            qt.bias.fill_(self.cscale_bias)
            self.layout_bytes[f"cast {name}"] = self._layout(name)
            return [(f"cast {name}", "cast", 3 * n,
                     lambda: cast(x, qt.bias, q=qt.q, qT=qt.qT, want_q=qt.q is not None,
                                  want_qT=qt.qT is not None))]
        if self.quant == "delayed":
            hist, count = self.hist[name]
            self.layout_bytes[f"quantise {name}"] = self._layout(name)
            return [(f"quantise {name}", "quantise", 3 * n,
                     lambda: F.fp8_quantise_delayed(x, fmt, qt.bias, hist, count, margin, amax_bits=qt.amax,
                                                    flags=qt.flags, q=qt.q, qT=qt.qT, want_q=qt.q is not None,
                                                    want_qT=qt.qT is not None, ws=qt.qws))]
        if self.quant != "separate":
            pred = qt.bias if self.quant == "predicted" else None
            # one read of the tensor and its codes when the prediction holds
            self.layout_bytes[f"quantise {name}"] = self._layout(name)
            return [(f"quantise {name}", "quantise", 3 * n,
                     lambda: F.fp8_quantise(x, fmt, margin, bias_pred=pred, bias=qt.bias,
                                            amax_bits=qt.amax, flags=qt.flags, q=qt.q, qT=qt.qT,
                                            want_q=qt.q is not None, want_qT=qt.qT is not None,
                                            ws=qt.qws))]
        self.layout_bytes[f"cast {name}"] = self._layout(name)
        return [
            (f"amax+bias {name}", "amax", 2 * n,
             lambda: F.fp8_scale_bias(x, fmt, margin, bias=qt.bias, amax_bits=qt.amax,
                                      flags=qt.flags, ws=qt.sws)),
            (f"cast {name}", "cast", 3 * n,
             lambda: cast(x, qt.bias, q=qt.q, qT=qt.qT, want_q=qt.q is not None,
                          want_qT=qt.qT is not None)),
        ]

    def _quant_batch(self, names, fmt, margin):
        """The quantise calls of `names`, up to QUANTISE_BATCH_MAX tensors per
        fp8_quantise_batch call (work counted as in _quant)."""
        calls = []
        for g in range(0, len(names), F.QUANTISE_BATCH_MAX):
            grp = names[g:g + F.QUANTISE_BATCH_MAX]
            items, work, layout = [], 0, 0
            for name in grp:
                x, qt = self.t[name], self.q[name]
                work += 3 * x.numel()
                layout += self._layout(name)
                items.append(dict(x=x, bias=qt.bias, bias_pred=qt.bias if self.quant == "predicted" else None,
                                  amax_bits=qt.amax, flags=qt.flags, q=qt.q, qT=qt.qT, ws=qt.qws))
            label = f"quantise {'+'.join(grp)}"
            self.layout_bytes[label] = layout
            calls.append((label, "quantise", work,
                          lambda items=items: F.fp8_quantise_batch(items, fmt, margin)))
        return calls

    def quantised(self):
        """(name, format, margin) of every tensor the step quantises."""
        out = {}
        for l in self.w.linears:
            out.setdefault(l.w, (F.E4M3, 0))
            out.setdefault(l.x, (F.E4M3, 0))
            if self.w.train:
                out.setdefault(l.dy, (F.E5M2, self.margin))
        return [(k, f, m) for k, (f, m) in out.items()]

    def step_inputs(self):
        """Names of the tensors every step quantises (inference weights are
        quantised once beforehand, by prepare_inference)."""
        names = [n for n, _, _ in self.quantised()]
        if not self.w.train:
            weights = {l.w for l in self.w.linears}
            names = [n for n in names if n not in weights]
        return names

    def prediction_hits(self):
        """(hits, tensors) of the last step's bias predictions ("predicted"
        mode): a tensor's prediction held when the bias its codes were first
        cast with (word 0 of its quantise workspace) is its exact bias."""
        if self.quant != "predicted":
            return 0, 0
        names = self.step_inputs()
        used = torch.stack([self.q[n].qws[:4].view(torch.int32)[0] for n in names]).cpu()
        exact = torch.stack([self.q[n].bias[0] for n in names]).cpu()
        return int((used == exact).sum()), len(names)

    def _build(self):
        """The step's calls in issue order; self.sched[i] = (phase, branch) of
        call i: consecutive calls of one phase are independent across branches
        (phase None: on its own)."""
        calls, sched = [], []

        def add(cs, phase=None, branch=0):
            calls.extend(cs)
            sched.extend([(phase, branch)] * len(cs))

        lin = self.w.linears
        done = set()
        weights = [l.w for l in lin]
        names = list(dict.fromkeys(weights)) if self.w.train else []
        names += [x for x in dict.fromkeys(l.x for l in lin) if x not in names]
        if self.batch_quant:
            for l in lin:  # one call per linear: its weight and input
                grp = [n for n in ((l.w,) if self.w.train else ()) + (l.x,) if n not in done]
                done.update(grp)
                if grp:
                    add(self._quant_batch(grp, F.E4M3, 0), "quantise inputs")
        else:
            done.update(names)
            for nq, name in enumerate(names):
                add(self._quant(name, F.E4M3, 0), "quantise inputs", nq % 2)
        for l in lin:
            xq, wq, o = self.q[l.x], self.q[l.w], self.out[l.name]
            flop = 2 * l.M * l.N * l.K
            # M <= 32 runs the weight-streaming kernel: its work is counted in
            # bytes (weight + activations + bf16 output), it is HBM-bound
            kind, work = "gemm_fwd", flop
            if l.M <= 32:
                kind, work = "gemm_decode", l.N * l.K + l.M * l.K + 2 * l.M * l.N
            amax_y = self.w.train and self.quant != "cscale"
            if amax_y and self.fused_bias:
                add([(f"fwd {l.name}", kind, work,
                      lambda xq=xq, wq=wq, o=o, bws=self.bws[l.name]: F.fp8_linear_fwd_bias(
                          xq.q, xq.bias, wq.qT, wq.bias, F.E4M3, 0, y=o["y"],
                          bias=o["y_scal"][0:1], amax_bits=o["y_scal"][1:2],
                          flags=o["y_scal"][2:3], ws=bws))])
                continue
            add([(f"fwd {l.name}", kind, work,
                  lambda xq=xq, wq=wq, o=o, amax_y=amax_y: F.fp8_linear_fwd(
                      xq.q, xq.bias, wq.qT, wq.bias, y=o["y"],
                      y_amax_bits=o["y_scal"][1:2] if amax_y else None))])
            if amax_y:
                add([(f"bias y {l.name}", "bias", 0,
                      lambda o=o: F.fp8_bias_from_amax(o["y_scal"][1:2], F.E4M3, 0,
                                                       bias=o["y_scal"][0:1],
                                                       flags=o["y_scal"][2:3]))])
        if self.w.train:
            grads = [g for g in dict.fromkeys(l.dy for l in lin) if g not in done]
            done.update(grads)
            for nq, name in enumerate(grads):  # each gradient on its own
                add(self._quant_batch([name], F.E5M2, self.margin) if self.batch_quant
                    else self._quant(name, F.E5M2, self.margin), "quantise gradients", nq % 2)
            for l in lin:
                xq, wq, gq, o = self.q[l.x], self.q[l.w], self.q[l.dy], self.out[l.name]
                flop = 2 * l.M * l.N * l.K
                amax_dx = self.quant != "cscale"
                ph = f"backward {l.name}"
                if amax_dx and self.fused_bias:
                    add([(f"dx {l.name}", "gemm_dx", flop,
                          lambda wq=wq, gq=gq, o=o, bws=self.bws[l.name], mg=self.margin: F.fp8_linear_bwd_dx_bias(
                              gq.q, gq.bias, wq.q, wq.bias, F.E5M2, mg, dx=o["dx"],
                              bias=o["dx_scal"][0:1], amax_bits=o["dx_scal"][1:2],
                              flags=o["dx_scal"][2:3], ws=bws))], ph, 0)
                else:
                    add([(f"dx {l.name}", "gemm_dx", flop,
                          lambda wq=wq, gq=gq, o=o, amax_dx=amax_dx: F.fp8_linear_bwd_dx(
                              gq.q, gq.bias, wq.q, wq.bias, dx=o["dx"],
                              dx_amax_bits=o["dx_scal"][1:2] if amax_dx else None))], ph, 0)
                if amax_dx and not self.fused_bias:
                    add([(f"bias dx {l.name}", "bias", 0,
                          lambda o=o, mg=self.margin: F.fp8_bias_from_amax(o["dx_scal"][1:2], F.E5M2,
                                                                           mg, bias=o["dx_scal"][0:1],
                                                           flags=o["dx_scal"][2:3]))], ph, 0)
                add([(f"dw {l.name}", "gemm_dw", flop,
                      lambda xq=xq, gq=gq, o=o: F.fp8_linear_bwd_dw(
                          xq.qT, xq.bias, gq.qT, gq.bias, dw=o["dw"]))], ph, 1)
        self.sched = sched
        return calls

    def prepare_inference(self):
        """PTQ: quantise every weight once (not part of the per-call step)."""
        for name in dict.fromkeys(l.w for l in self.w.linears):
            qt = self.q[name]
            F.ptq_quantise_weights(self.t[name], want_w8=False, w8t=qt.qT, bw=qt.bias,
                                   flags=qt.flags, ws=self.ws)

    def run(self):
        for _, _, _, fn in self.calls:
            fn()

    def run_concurrent(self):
        """The step with independent calls forked onto the side stream: for
        each phase, branch-1 calls run on the side stream after an event of
        the current stream, and the current stream waits for them before the
        next phase."""
        main = torch.cuda.current_stream(self.dev)
        i, n = 0, len(self.calls)
        while i < n:
            phase = self.sched[i][0]
            j = i + 1
            while phase is not None and j < n and self.sched[j][0] == phase:
                j += 1
            group = range(i, j)
            if all(self.sched[k][1] == 0 for k in group):
                for k in group:
                    self.calls[k][3]()
            else:
                fork = torch.cuda.Event()
                fork.record(main)
                self.side.wait_event(fork)
                for k in group:
                    if self.sched[k][1] == 0:
                        self.calls[k][3]()
                with torch.cuda.stream(self.side):
                    for k in group:
                        if self.sched[k][1] != 0:
                            self.calls[k][3]()
                join = torch.cuda.Event()
                join.record(self.side)
                main.wait_event(join)
            i = j

    def capture(self):
        """Record one step into a HIP graph, so that replay() launches the
        whole step with one host call (independent calls on two streams when
        concurrent).  The library launches only kernels (no memset or copy
        nodes) on the current stream, and every buffer is allocated
        beforehand, so replays recompute the step from the current contents of
        the input tensors."""
        torch.cuda.synchronize(self.dev)
        g = torch.cuda.CUDAGraph()
        # Dead objects that own HIP resources (an earlier step's graph) must
        # not be destroyed while the stream is capturing: collect them now and
        # keep the cyclic collector off until the capture ends.
        gc.collect()
        was_enabled = gc.isenabled()
        gc.disable()
        try:
            with torch.cuda.graph(g):
                if self.concurrent:
                    self.run_concurrent()
                else:
                    self.run()
        finally:
            if was_enabled:
                gc.enable()
        torch.cuda.synchronize(self.dev)
        self.graph = g
        return g

    def replay(self):
        self.graph.replay()

    def gemm_flops(self) -> int:
        return sum(2 * l.M * l.N * l.K * (3 if self.w.train else 1) for l in self.w.linears)
