"""One Llama 2 decoder layer with its four linears in FP8, as library calls.

The paper quantises the QKV projection, the attention output projection and
the two feed-forward layers of every decoder layer to FP8 and keeps the rest
in higher precision (App. E); weights are quantised once (post-training
quantisation, Sec. 3.1) and every activation that enters an FP8 linear gets
its own FP8-AMAX bias per call (Sec. 2.3 Eq. 3, Sec. 3).  The layer:

  xn  = RMSNorm(H) g_attn          -> E4 codes, bias   (fused quantise)
  qkv = xn8 . Wqkv8                 (FP8 matmul, bf16 out)
  RoPE on the Q and K heads of qkv (in place)
  att = causal GQA attention(qkv)  -> E4 codes, bias   (fused quantise)
  o   = att8 . Wo8
  h1  = H + o;  hn = RMSNorm(h1) g_mlp -> E4 codes, bias (one kernel)
  gu  = hn8 . Wgu8                  (gate | up)
  a   = silu(gate) * up            -> E4 codes, bias   (fused quantise)
  out = h1 + a8 . Wd8

Each fused quantise casts with the previous call's bias as a prediction and
re-casts only if the exact bias differs, so the codes are always those of the
exact FP8-AMAX bias.  Buffers are allocated once; a call launches kernels only
and can be captured in a HIP graph.

Bias granularity: one bias per activation tensor and call ("tensor"), or one
per sequence of the call ("sequence": the per-data-sample activation biases of
the paper's inference, App. D): then each glue kernel writes its bf16 output
only, fp8_quantise_segments gives every sequence its own Eq. 3 bias and codes,
and fp8_linear_fwd_rows unscales each output row by its sequence's bias.
"""
from __future__ import annotations

import gc

import torch

from . import fp8lin as F
from .workloads import LayerConfig

LLAMA_EPS = 1e-5
ROPE_THETA = 10000.0


class _Act:
    """An activation that enters an FP8 linear: bf16 tensor, its E4 codes,
    [bias, amax bits, flags] and the fused-quantise workspace."""

    def __init__(self, rows, cols, ws_bytes, device):
        self.x = torch.empty((rows, cols), dtype=torch.bfloat16, device=device)
        self.q = torch.empty((rows, cols), dtype=torch.uint8, device=device)
        self.scal = torch.zeros(3, dtype=torch.int32, device=device)
        self.ws = torch.empty(max(ws_bytes, 4), dtype=torch.uint8, device=device)

    @property
    def bias(self): return self.scal[0:1]

    def fq(self):
        return F.FusedQuant(self.q, self.bias, self.ws, F.E4M3, 0, bias_pred=self.bias,
                            amax_bits=self.scal[1:2], flags=self.scal[2:3])

    def segments(self, nseg, device):
        """Per-sequence bias buffers: [nseg] biases, amax bits and flags, and
        the bias of every row."""
        i32 = dict(dtype=torch.int32, device=device)
        self.seg_bias = torch.zeros(nseg, **i32)
        self.seg_amax = torch.zeros(nseg, **i32)
        self.seg_flags = torch.zeros(nseg, **i32)
        self.row_bias = torch.zeros(self.x.shape[0], **i32)

    def quantise_segments(self, offsets):
        F.fp8_quantise_segments(self.x, offsets, F.E4M3, 0, bias=self.seg_bias, amax_bits=self.seg_amax,
                                flags=self.seg_flags, row_bias=self.row_bias, q=self.q)


class DecoderLayer:
    """Buffers and calls of one decoder layer for a fixed number of tokens.

    weights: dict of bf16 device tensors Wqkv [d, (nh + 2 nkv) dh], Wo
    [nh dh, d], Wgu [d, 2 ffn] (gate columns first), Wd [ffn, d], g_attn and
    g_mlp [d] (or [1, d]); they are quantised once here (PTQ).
    ``calls`` lists (label, kind, work, fn) in issue order; running them is
    one forward call of the layer on ``self.H``."""

    BIAS_PER = ("tensor", "sequence")

    def __init__(self, cfg: LayerConfig, weights: dict, device, bias_per: str = "tensor"):
        if bias_per not in self.BIAS_PER:
            raise ValueError(f"bias_per must be one of {self.BIAS_PER}")
        self.bias_per = bias_per
        self.cfg = c = cfg
        dev = self.dev = torch.device(device)
        R, d, nh, nkv, dh, ffn = c.rows, c.d_model, c.n_heads, c.n_kv_heads, c.d_head, c.ffn
        self.dq, self.dkv = nh * dh, nkv * dh
        bf = dict(dtype=torch.bfloat16, device=dev)
        self.g_attn = weights["g_attn"].reshape(-1).contiguous()
        self.g_mlp = weights["g_mlp"].reshape(-1).contiguous()
        # PTQ: transposed E4 codes [N, K] and one bias per weight
        self.w8t, self.wscal = {}, {}
        ws = F.workspace(max(w.numel() for k, w in weights.items() if k.startswith("W")), dev)
        for name, key in (("qkv", "Wqkv"), ("o", "Wo"), ("gate_up", "Wgu"), ("down", "Wd")):
            w = weights[key]
            K, N = w.shape
            self.w8t[name] = torch.empty((N, K), dtype=torch.uint8, device=dev)
            self.wscal[name] = torch.zeros(2, dtype=torch.int32, device=dev)
            F.ptq_quantise_weights(w, want_w8=False, w8t=self.w8t[name], bw=self.wscal[name][0:1],
                                   flags=self.wscal[name][1:2], ws=ws)
        self.table = F.llama_rope_table(c.seq_len, dh, ROPE_THETA, device=dev)
        # activations
        self.H = torch.empty((R, d), **bf)
        self.xn = _Act(R, d, F.llama_rmsnorm_ws_bytes(R), dev)
        self.qkv = torch.empty((R, (nh + 2 * nkv) * dh), **bf)
        self.att = _Act(R, self.dq, F.llama_attention_ws_bytes(R, c.seq_len, nh), dev)
        self.o = torch.empty((R, d), **bf)
        self.h1 = torch.empty((R, d), **bf)
        self.hn = _Act(R, d, F.llama_rmsnorm_ws_bytes(R), dev)
        self.gu = torch.empty((R, 2 * ffn), **bf)
        self.act = _Act(R, ffn, F.llama_swiglu_ws_bytes(), dev)
        self.down = torch.empty((R, d), **bf)
        self.out = torch.empty((R, d), **bf)
        self.nseg = (R + c.seq_len - 1) // c.seq_len
        self.offsets = torch.tensor([min(s * c.seq_len, R) for s in range(self.nseg + 1)], dtype=torch.int32,
                                    device=dev)
        if bias_per == "sequence":
            for a in (self.xn, self.att, self.hn, self.act):
                a.segments(self.nseg, dev)
        self.graph = None
        self.calls = self._build_sequence() if bias_per == "sequence" else self._build()

    def bw(self, name):
        return self.wscal[name][0:1]

    def _build(self):
        c = self.cfg
        R, d, ffn = c.rows, c.d_model, c.ffn
        att_flop = 4 * c.n_heads * c.d_head * sum(
            (min(c.seq_len, R - s) * (min(c.seq_len, R - s) + 1)) // 2 for s in range(0, R, c.seq_len))

        def lin(name, a: _Act, y):
            K, N = a.x.shape[1], y.shape[1]
            return (f"{name}", "gemm_fwd", 2 * R * N * K,
                    lambda: F.fp8_linear_fwd(a.q, a.bias, self.w8t[name], self.bw(name), y=y))

        return [
            ("rmsnorm+quantise attn", "glue", 2 * R * d + 3 * R * d,
             lambda: F.llama_rmsnorm_quantise(self.H, self.g_attn, LLAMA_EPS, y=self.xn.x, fq=self.xn.fq())),
            lin("qkv", self.xn, self.qkv),
            ("rope", "glue", 4 * R * (self.dq + self.dkv),
             lambda: F.llama_rope(self.qkv[:, :self.dq + self.dkv], c.n_heads + c.n_kv_heads, c.d_head,
                                  c.seq_len, self.table)),
            ("attention+quantise", "attention", att_flop,
             lambda: F.llama_attention(self.qkv, c.seq_len, c.n_heads, c.n_kv_heads, c.d_head, o=self.att.x,
                                       fq=self.att.fq())),
            lin("o", self.att, self.o),
            ("residual+rmsnorm+quantise mlp", "glue", 4 * R * d + 5 * R * d,
             lambda: F.llama_rmsnorm_quantise(self.o, self.g_mlp, LLAMA_EPS, res=self.H, h=self.h1,
                                              y=self.hn.x, fq=self.hn.fq())),
            lin("gate_up", self.hn, self.gu),
            ("swiglu+quantise", "glue", 4 * R * ffn + 3 * R * ffn,
             lambda: F.llama_swiglu_quantise(self.gu, ffn, a=self.act.x, fq=self.act.fq())),
            lin("down", self.act, self.down),
            ("residual", "glue", 6 * R * d, lambda: F.llama_residual_add(self.h1, self.down, out=self.out)),
        ]

    def _build_sequence(self):
        """The layer with one activation bias per sequence: glue kernels
        without the fused quantise, then a segmented quantise and the matmul
        with per-row biases."""
        c = self.cfg
        R, d, ffn = c.rows, c.d_model, c.ffn
        att_flop = 4 * c.n_heads * c.d_head * sum(
            (min(c.seq_len, R - s) * (min(c.seq_len, R - s) + 1)) // 2 for s in range(0, R, c.seq_len))

        def quant(a: _Act, label):
            n = a.x.numel()
            return (f"quantise/seq {label}", "quantise", 2 * 2 * n + n, lambda: a.quantise_segments(self.offsets))

        def lin(name, a: _Act, y):
            K, N = a.x.shape[1], y.shape[1]
            return (f"{name}", "gemm_fwd", 2 * R * N * K,
                    lambda: F.fp8_linear_fwd_rows(a.q, a.row_bias, self.w8t[name], self.bw(name), y=y))

        return [
            ("rmsnorm attn", "glue", 2 * R * d + 2 * R * d,
             lambda: F.llama_rmsnorm_quantise(self.H, self.g_attn, LLAMA_EPS, y=self.xn.x)),
            quant(self.xn, "attn input"),
            lin("qkv", self.xn, self.qkv),
            ("rope", "glue", 4 * R * (self.dq + self.dkv),
             lambda: F.llama_rope(self.qkv[:, :self.dq + self.dkv], c.n_heads + c.n_kv_heads, c.d_head,
                                  c.seq_len, self.table)),
            ("attention", "attention", att_flop,
             lambda: F.llama_attention(self.qkv, c.seq_len, c.n_heads, c.n_kv_heads, c.d_head, o=self.att.x)),
            quant(self.att, "attention"),
            lin("o", self.att, self.o),
            ("residual+rmsnorm mlp", "glue", 4 * R * d + 4 * R * d,
             lambda: F.llama_rmsnorm_quantise(self.o, self.g_mlp, LLAMA_EPS, res=self.H, h=self.h1, y=self.hn.x)),
            quant(self.hn, "mlp input"),
            lin("gate_up", self.hn, self.gu),
            ("swiglu", "glue", 4 * R * ffn + 2 * R * ffn,
             lambda: F.llama_swiglu_quantise(self.gu, ffn, a=self.act.x)),
            quant(self.act, "down input"),
            lin("down", self.act, self.down),
            ("residual", "glue", 6 * R * d, lambda: F.llama_residual_add(self.h1, self.down, out=self.out)),
        ]

    def run(self):
        for _, _, _, fn in self.calls:
            fn()
        return self.out

    def capture(self):
        """Record one call into a HIP graph (kernels only; see WorkloadStep)."""
        torch.cuda.synchronize(self.dev)
        g = torch.cuda.CUDAGraph()
        gc.collect()
        was_enabled = gc.isenabled()
        gc.disable()
        try:
            with torch.cuda.graph(g):
                self.run()
        finally:
            if was_enabled:
                gc.enable()
        torch.cuda.synchronize(self.dev)
        self.graph = g
        return g

    def replay(self):
        self.graph.replay()

    def linear_flops(self) -> int:
        return sum(w for _, k, w, _ in self.calls if k == "gemm_fwd")

    def biases(self) -> dict:
        """Activation and weight biases (host ints; synchronises); with one
        bias per sequence, the activation entries are lists."""
        b = {n: int(self.bw(n).item()) for n in self.w8t}
        for n, a in (("xn", self.xn), ("att", self.att), ("hn", self.hn), ("act", self.act)):
            b[n] = a.seg_bias.cpu().tolist() if self.bias_per == "sequence" else int(a.bias.item())
        return b
