"""Seeded synthetic inputs shaped like the paper's linear layers.

This module only draws random numbers: it contains none of the FP8 method's
arithmetic (no amax, bias, cast or matmul), and it imports neither the HIP
library binding nor the oracle.  Both sides of every parity check receive the
same bytes from here.

Shapes follow the model table of the paper (Table 1: d_model and d_ffn of GPT
111M and Llama 2 7B / 13B / 70B) and the linear layers it quantises (App. E:
QKV, attention output, FF up, FF down).  The paper's datasets and checkpoints
are not available, so normally distributed tensors stand in for activations,
weights and gradients.

Conventions: X is [M, K] (tokens x d_in), W is [K, N] (d_in x d_out), dY is
[M, N]; all bf16, row-major.  N(0, s) means standard deviation s.  Each tensor
is drawn in fp32 from a CPU ``torch.Generator`` seeded with
``base_seed(config) + t`` (t = position of the tensor in the list below) and
rounded to bf16 (round to nearest even).
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import torch


@dataclass(frozen=True)
class Tensor:
    name: str
    rows: int
    cols: int
    kind: str            # "normal", "outlier_cols", "row_log2_uniform", "gain"
    std: float = 1.0
    extra: tuple = ()


@dataclass(frozen=True)
class Linear:
    """One FP8 linear layer: X [M,K] @ W [K,N] with gradient dY [M,N]."""
    name: str
    x: str
    w: str
    dy: str | None
    M: int
    K: int
    N: int


@dataclass(frozen=True)
class Workload:
    name: str
    index: int           # position in the list of workloads (seed base)
    description: str
    tensors: tuple
    linears: tuple
    train: bool = True   # fwd + bwd; False = PTQ inference (fwd only)
    extra: dict = field(default_factory=dict)

    def tensor(self, name: str) -> Tensor:
        for t in self.tensors:
            if t.name == name:
                return t
        raise KeyError(name)


def _w(name, K, N, std):
    return Tensor(name, K, N, "normal", std)


WORKLOADS = {
    # GPT 111M (d_model 768): one linear 1024 tokens x 768 -> 768.
    "gpt111m-linear": Workload(
        "gpt111m-linear", 0,
        "GPT-111M-shaped FP8 linear fwd+bwd: X 1024x768 N(0,1), W 768x768 N(0,0.02), "
        "dY 1024x768 N(0,1e-3)",
        (Tensor("X", 1024, 768, "normal", 1.0), _w("W", 768, 768, 0.02),
         Tensor("dY", 1024, 768, "normal", 1e-3)),
        (Linear("linear", "X", "W", "dY", 1024, 768, 768),),
    ),
    # Llama 2 7B MLP up-projection (d_model 4096 -> d_ffn 11008), 4096 tokens.
    "llama2-7b-up": Workload(
        "llama2-7b-up", 1,
        "Llama-2-7B MLP up-proj fwd+bwd: X 4096x4096 N(0,1) with 0.1% of columns x50, "
        "W 4096x11008 N(0,0.02), dY 4096x11008 N(0,1e-4)",
        (Tensor("X", 4096, 4096, "outlier_cols", 1.0, (0.001, 50.0)),
         _w("W", 4096, 11008, 0.02), Tensor("dY", 4096, 11008, "normal", 1e-4)),
        (Linear("up", "X", "W", "dY", 4096, 4096, 11008),),
    ),
    # Llama 2 13B fused QKV (d_model 5120 -> 3 x 5120), 8192 tokens; gradient
    # rows spread over ten binades to stress the E5 range.
    "llama2-13b-qkv": Workload(
        "llama2-13b-qkv", 2,
        "Llama-2-13B fused QKV fwd+bwd: X 8192x5120 N(0,1), W 5120x15360 N(0,0.015), "
        "dY 8192x15360 rows 2^u * N(0,1), u ~ U[-20,-10]",
        (Tensor("X", 8192, 5120, "normal", 1.0), _w("W", 5120, 15360, 0.015),
         Tensor("dY", 8192, 15360, "row_log2_uniform", 1.0, (-20.0, -10.0))),
        (Linear("qkv", "X", "W", "dY", 8192, 5120, 15360),),
    ),
    # Llama 2 70B MLP (d_model 8192, d_ffn 28672), 4096 tokens, unsharded.
    # X is shared by gate and up; the input of down is a synthetic tensor
    # (the SwiGLU between them is not part of the FP8 path).
    "llama2-70b-mlp": Workload(
        "llama2-70b-mlp", 3,
        "Llama-2-70B MLP fwd+bwd on one GPU: X 4096x8192 N(0,1), gate/up W 8192x28672, "
        "down W 28672x8192 N(0,0.01), dY N(0,1e-4)",
        (Tensor("X", 4096, 8192, "normal", 1.0), Tensor("Xd", 4096, 28672, "normal", 1.0),
         _w("Wg", 8192, 28672, 0.01), _w("Wu", 8192, 28672, 0.01), _w("Wd", 28672, 8192, 0.01),
         Tensor("dYg", 4096, 28672, "normal", 1e-4), Tensor("dYu", 4096, 28672, "normal", 1e-4),
         Tensor("dYd", 4096, 8192, "normal", 1e-4)),
        (Linear("gate", "X", "Wg", "dYg", 4096, 8192, 28672),
         Linear("up", "X", "Wu", "dYu", 4096, 8192, 28672),
         Linear("down", "Xd", "Wd", "dYd", 4096, 28672, 8192)),
    ),
    # Llama 2 70B decoder layer, PTQ inference: weights quantised once, then
    # per-call activation scaling at prefill (2048 tokens) and decode (16).
    "llama2-70b-ptq": Workload(
        "llama2-70b-ptq", 4,
        "Llama-2-70B decoder-layer PTQ inference: W QKV 8192x10240, O 8192x8192, "
        "gate+up 8192x57344, down 28672x8192 N(0,0.01); X N(0,1) at M=2048 and M=16",
        (_w("Wqkv", 8192, 10240, 0.01), _w("Wo", 8192, 8192, 0.01),
         _w("Wgu", 8192, 57344, 0.01), _w("Wd", 28672, 8192, 0.01),
         Tensor("Xp", 2048, 8192, "normal", 1.0), Tensor("Xpd", 2048, 28672, "normal", 1.0),
         Tensor("Xs", 16, 8192, "normal", 1.0), Tensor("Xsd", 16, 28672, "normal", 1.0)),
        (Linear("qkv", "Xp", "Wqkv", None, 2048, 8192, 10240),
         Linear("o", "Xp", "Wo", None, 2048, 8192, 8192),
         Linear("gateup", "Xp", "Wgu", None, 2048, 8192, 57344),
         Linear("down", "Xpd", "Wd", None, 2048, 28672, 8192),
         Linear("qkv_dec", "Xs", "Wqkv", None, 16, 8192, 10240),
         Linear("o_dec", "Xs", "Wo", None, 16, 8192, 8192),
         Linear("gateup_dec", "Xs", "Wgu", None, 16, 8192, 57344),
         Linear("down_dec", "Xsd", "Wd", None, 16, 28672, 8192)),
        train=False,
    ),
}


@dataclass(frozen=True)
class LayerConfig:
    """One Llama 2 decoder layer: the dimensions of Table 1, its four FP8
    linears (App. E: QKV [d, (n_heads + 2 n_kv_heads) d_head], O
    [n_heads d_head, d], gate+up [d, 2 ffn], down [ffn, d]) and a call of
    `rows` tokens in sequences of `seq_len`."""
    name: str
    index: int           # seed base, after the linear workloads
    description: str
    d_model: int
    n_heads: int
    n_kv_heads: int
    d_head: int
    ffn: int
    rows: int
    seq_len: int
    w_std: float = 0.01

    def tensors(self) -> tuple:
        d, q = self.d_model, self.n_heads * self.d_head
        return (Tensor("H", self.rows, d, "normal", 1.0),
                Tensor("g_attn", 1, d, "gain", 0.1), Tensor("g_mlp", 1, d, "gain", 0.1),
                _w("Wqkv", d, (self.n_heads + 2 * self.n_kv_heads) * self.d_head, self.w_std),
                _w("Wo", q, d, self.w_std), _w("Wgu", d, 2 * self.ffn, self.w_std),
                _w("Wd", self.ffn, d, self.w_std))

    def linears(self) -> tuple:
        """(name, K, N) of the four linears, in call order."""
        d = self.d_model
        return (("qkv", d, (self.n_heads + 2 * self.n_kv_heads) * self.d_head),
                ("o", self.n_heads * self.d_head, d), ("gate_up", d, 2 * self.ffn), ("down", self.ffn, d))


LAYERS = {
    # Llama 2 70B decoder layer (d 8192, 64 query / 8 key-value heads of 128,
    # ffn 28672), post-training-quantised weights, prefill of one 2048-token
    # sequence: input hidden state N(0,1), RMSNorm gains 1 + N(0, 0.1).
    "llama2-70b-layer": LayerConfig(
        "llama2-70b-layer", 5,
        "Llama-2-70B decoder layer, PTQ inference, prefill 2048 tokens: H 2048x8192 N(0,1), "
        "W QKV 8192x10240, O 8192x8192, gate+up 8192x57344, down 28672x8192 N(0,0.01), "
        "RMSNorm gains 1+N(0,0.1); GQA 64/8 heads of 128, causal",
        8192, 64, 8, 128, 28672, 2048, 2048),
    # Llama 2 7B decoder layer (32 heads, no grouping), two 2048-token sequences.
    "llama2-7b-layer": LayerConfig(
        "llama2-7b-layer", 6,
        "Llama-2-7B decoder layer, PTQ inference, prefill 2x2048 tokens: H 4096x4096 N(0,1), "
        "W QKV 4096x12288, O 4096x4096, gate+up 4096x22016, down 11008x4096 N(0,0.02); 32 heads of 128",
        4096, 32, 32, 128, 11008, 4096, 2048, 0.02),
    # Small layer for parity against the oracle: grouped heads (8 / 2), two
    # sequences of 150 tokens (ragged query and key blocks).
    "tiny-layer": LayerConfig(
        "tiny-layer", 7, "small decoder layer for parity: d 512, 8/2 heads of 128, ffn 1408, 2x150 tokens",
        512, 8, 2, 128, 1408, 300, 150, 0.05),
}


def make_layer_tensor(cfg: LayerConfig, name: str) -> torch.Tensor:
    ts = cfg.tensors()
    idx = [t.name for t in ts].index(name)
    t = ts[idx]
    return draw(t.rows, t.cols, t.kind, t.std, t.extra, 1000 * cfg.index + idx)


def base_seed(w: Workload) -> int:
    return 1000 * w.index


def make_tensor(w: Workload, name: str) -> torch.Tensor:
    """Draw one tensor of a workload (bf16, CPU, contiguous)."""
    idx = [t.name for t in w.tensors].index(name)
    t = w.tensors[idx]
    return draw(t.rows, t.cols, t.kind, t.std, t.extra, base_seed(w) + idx)


def draw(rows: int, cols: int, kind: str = "normal", std: float = 1.0, extra: tuple = (),
         seed: int = 0) -> torch.Tensor:
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    x = torch.randn((rows, cols), generator=g, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    if kind == "outlier_cols":
        frac, factor = extra
        ncol = max(1, int(round(frac * cols)))
        cols_idx = torch.randperm(cols, generator=g)[:ncol]
        x[:, cols_idx] *= factor
    elif kind == "row_log2_uniform":
        lo, hi = extra
        u = torch.rand((rows, 1), generator=g, dtype=torch.float64) * (hi - lo) + lo
        x.mul_(torch.exp2(u).to(torch.float32))
    elif kind == "gain":            # RMSNorm gain: 1 + N(0, std)
        x.add_(1.0)
    elif kind != "normal":
        raise ValueError(kind)
    return x.to(torch.bfloat16)


def small(rows: int, cols: int, std: float = 1.0, seed: int = 0) -> torch.Tensor:
    """A plain N(0, std) bf16 tensor for small parity cases."""
    return draw(rows, cols, "normal", std, (), seed)


def sha256(t: torch.Tensor) -> str:
    return hashlib.sha256(t.contiguous().view(torch.uint8).numpy().tobytes()).hexdigest()


def bf16_bits(t: torch.Tensor):
    """bf16 CPU tensor -> numpy uint16 bit patterns (no arithmetic)."""
    return t.contiguous().view(torch.int16).numpy().view("uint16")
