"""GPU parity of one Llama 2 decoder layer with its four linears in FP8
(App. E; weights quantised once, Sec. 3.1; FP8-AMAX activation biases per
call, Sec. 2.3 Eq. 3) against the oracle chain in oracle/decoder.py.

Both sides start from the same seeded bf16 tensors and each computes every
intermediate itself.  Bars:
  * the weight biases and the four activation biases equal the oracle's
    (integers: exact), and each activation's codes equal the oracle's
    wherever the bf16 tensors agree;
  * up to the attention, the two chains differ only by bf16 roundings:
    RMSNorm output and the QKV projection within rel_F 1e-3 (the FP8 matmul
    bar), the attention within its own bar, rel_F 1e-2;
  * from the cast of the attention output on, the chains quantise slightly
    different tensors: where a bf16 value differs, its E4M3 code can move by
    one step (2^-3 relative), and every later stage carries these flips.  The
    bar there is half an E4M3 step, rel_F <= 2^-4: the agreement an FP8 chain
    can promise; a wiring mistake (a wrong residual, gate and up swapped, a
    wrong bias or head mapping) gives errors of order one.  Measured: 0.5e-2
    to 3.6e-2 on both layers below.
Graph replays match the eager call bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle as orc_mod
from oracle import decoder as D
from paper_2309_17224_amd import decoder as DL
from paper_2309_17224_amd import workloads as wl
from parity_util import np_bits, rel_f

pytestmark = pytest.mark.gpu

FP8_CHAIN = 2.0 ** -4
TOL = {"xn": 1e-3, "qkv": 1e-3, "attn": 1e-2, "o": FP8_CHAIN, "h1": FP8_CHAIN, "hn": FP8_CHAIN, "gu": FP8_CHAIN,
       "act": FP8_CHAIN, "down": FP8_CHAIN, "out": FP8_CHAIN}


def layer_inputs(cfg):
    return {t.name: wl.make_layer_tensor(cfg, t.name) for t in cfg.tensors()}


def oracle_layer(cfg, T):
    bits = {k: wl.bf16_bits(v) for k, v in T.items()}
    p = {"g_attn": bits["g_attn"][0], "g_mlp": bits["g_mlp"][0]}
    for name, key in (("qkv", "Wqkv"), ("o", "Wo"), ("gate_up", "Wgu"), ("down", "Wd")):
        _, w8t, bw, _ = orc_mod.ptq_quantise_weights(bits[key])
        p[name + "_w8t"], p[name + "_bw"] = w8t, bw
    r = D.layer_forward(bits["H"], p, cfg.seq_len, cfg.n_heads, cfg.n_kv_heads, cfg.d_head, cfg.ffn)
    return p, r


def gpu_layer(cfg, T, dev):
    W = {k: v.to(dev) for k, v in T.items() if k != "H"}
    layer = DL.DecoderLayer(cfg, W, dev)
    layer.H.copy_(T["H"].to(dev))
    return layer


def compare(cfg, layer, p, r):
    dq = cfg.n_heads * cfg.d_head
    b = layer.biases()
    assert [b["qkv"], b["o"], b["gate_up"], b["down"]] == [p["qkv_bw"], p["o_bw"], p["gate_up_bw"], p["down_bw"]]
    assert [b["xn"], b["att"], b["hn"], b["act"]] == [r["b_xn"], r["b_attn"], r["b_hn"], r["b_act"]]
    got = {"xn": layer.xn.x, "qkv": layer.qkv, "attn": layer.att.x, "o": layer.o, "h1": layer.h1,
           "hn": layer.hn.x, "gu": layer.gu, "act": layer.act.x, "down": layer.down, "out": layer.out}
    errs = {}
    for k, t in got.items():
        g = np_bits(t)
        ref = r[k]
        if k == "qkv":   # after RoPE on the GPU (in place): compare the V columns and the rotated Q, K
            ref = np.concatenate([r["q"], r["k"], r["v"]], axis=1)
        errs[k] = rel_f(g, ref)
    print(cfg.name, "rel_F:", {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    for k, e in errs.items():
        assert e <= TOL[k], (k, e)
    # codes of each FP8 activation equal the oracle's wherever its bf16 input agrees
    for a, ref_x, ref_q in ((layer.xn, r["xn"], r["xn8"]), (layer.att, r["attn"], r["attn8"]),
                            (layer.hn, r["hn"], r["hn8"]), (layer.act, r["act"], r["act8"])):
        same = np_bits(a.x) == ref_x
        assert np.array_equal(a.q.cpu().numpy()[same], ref_q[same])
    return errs


def test_tiny_layer_matches_oracle_and_graph_replays(gpu):
    cfg = wl.LAYERS["tiny-layer"]
    T = layer_inputs(cfg)
    p, r = oracle_layer(cfg, T)
    layer = gpu_layer(cfg, T, gpu)
    layer.run()            # first call: predictions still zero, every quantise re-casts
    layer.run()            # second call: predicted biases hold
    torch.cuda.synchronize()
    compare(cfg, layer, p, r)
    eager = {k: np_bits(t).copy() for k, t in (("out", layer.out), ("attn", layer.att.x), ("act", layer.act.x))}
    codes = layer.act.q.cpu().numpy().copy()
    layer.capture()
    for _ in range(3):
        layer.out.zero_()
        layer.act.q.zero_()
        layer.replay()
        torch.cuda.synchronize()
        assert np.array_equal(np_bits(layer.out), eager["out"])
        assert np.array_equal(layer.act.q.cpu().numpy(), codes)


def test_layer_7b_shape_matches_oracle(gpu):
    # Llama 2 7B head layout (32 heads, no grouping), fewer tokens: one
    # 256-token and one 128-token sequence (a short last sequence).
    full = wl.LAYERS["llama2-7b-layer"]
    cfg = wl.LayerConfig("7b-layer-384", 8, "Llama-2-7B layer dims, 384 tokens", full.d_model, full.n_heads,
                         full.n_kv_heads, full.d_head, full.ffn, 384, 256, full.w_std)
    T = layer_inputs(cfg)
    p, r = oracle_layer(cfg, T)
    layer = gpu_layer(cfg, T, gpu)
    layer.run()
    torch.cuda.synchronize()
    compare(cfg, layer, p, r)


@pytest.mark.timeout(900)
def test_70b_layer_full_size_matches_oracle(gpu):
    """The Llama 2 70B layer at 2048 tokens, the configuration the benchmark
    times, against the oracle chain computing every stage itself in fp64
    (each activation's Eq. 3 bias needs the whole tensor, so the oracle runs
    the whole chain: about two minutes of host time).  Same bars as the
    smaller layers."""
    cfg = wl.LAYERS["llama2-70b-layer"]
    T = layer_inputs(cfg)
    layer = gpu_layer(cfg, T, gpu)
    layer.run()
    layer.run()
    torch.cuda.synchronize()
    p, r = oracle_layer(cfg, T)
    errs = compare(cfg, layer, p, r)
    print("70B layer rel_F per stage:", {k: f"{v:.3e}" for k, v in errs.items()}, flush=True)


def test_70b_layer_full_size_properties(gpu):
    """Llama 2 70B layer at 2048 tokens, the configuration the benchmark
    times: properties that hold at any size, on inputs drawn on the GPU (the
    comparison with the oracle chain at this size is the test above)."""
    from paper_2309_17224_amd import fp8lin as F
    cfg = wl.LAYERS["llama2-70b-layer"]
    g = torch.Generator(device=gpu)
    g.manual_seed(1000 * cfg.index)
    W = {}
    for t in cfg.tensors():
        x = torch.randn((t.rows, t.cols), generator=g, device=gpu) * t.std
        W[t.name] = (x + 1.0 if t.kind == "gain" else x).to(torch.bfloat16)
    H = W.pop("H")
    layer = DL.DecoderLayer(cfg, W, gpu)
    layer.H.copy_(H)
    layer.run()
    layer.run()
    torch.cuda.synchronize()
    # each fused quantise = fp8_quantise of the layer's own bf16 tensor
    for a in (layer.xn, layer.att, layer.hn, layer.act):
        q2, _, b2, a2, f2 = F.fp8_quantise(a.x, F.E4M3, 0)
        torch.cuda.synchronize()
        assert torch.equal(a.q, q2)
        assert a.scal.cpu().tolist() == [int(b2.item()), int(a2.item()), int(f2.item())]
        assert int(f2.item()) == 0
    # the first query sees only its own key: its output is its value row
    dq, dkv, dh = layer.dq, layer.dkv, cfg.d_head
    v0 = layer.qkv[0, dq + dkv:dq + 2 * dkv].reshape(cfg.n_kv_heads, dh)
    o0 = layer.att.x[0].reshape(cfg.n_heads, dh)
    assert torch.equal(o0, v0.repeat_interleave(cfg.n_heads // cfg.n_kv_heads, dim=0))
    assert torch.isfinite(layer.out.float()).all()
    eager = layer.out.clone()
    layer.capture()
    for _ in range(2):
        layer.out.zero_()
        layer.replay()
        torch.cuda.synchronize()
        assert torch.equal(layer.out, eager)


@pytest.mark.parametrize("name", ["tiny-layer", "7b-layer-384"])
def test_layer_per_sequence_biases_match_oracle(gpu, name):
    """One activation bias per sequence (the per-data-sample biases of
    App. D): segmented quantise + per-row-bias matmuls on the GPU against
    the oracle chain with per-sequence quantisation; same bars."""
    if name == "tiny-layer":
        cfg = wl.LAYERS["tiny-layer"]
    else:
        full = wl.LAYERS["llama2-7b-layer"]
        cfg = wl.LayerConfig("7b-layer-384", 8, "Llama-2-7B layer dims, 384 tokens", full.d_model, full.n_heads,
                             full.n_kv_heads, full.d_head, full.ffn, 384, 256, full.w_std)
    T = layer_inputs(cfg)
    bits = {k: wl.bf16_bits(v) for k, v in T.items()}
    p, _ = oracle_layer(cfg, T)
    r = D.layer_forward(bits["H"], p, cfg.seq_len, cfg.n_heads, cfg.n_kv_heads, cfg.d_head, cfg.ffn,
                        per_sequence=True)
    W = {k: v.to(gpu) for k, v in T.items() if k != "H"}
    layer = DL.DecoderLayer(cfg, W, gpu, bias_per="sequence")
    layer.H.copy_(T["H"].to(gpu))
    layer.run()
    torch.cuda.synchronize()
    compare(cfg, layer, p, r)
    # graph replays match the eager call
    eager = np_bits(layer.out).copy()
    layer.capture()
    for _ in range(2):
        layer.out.zero_()
        layer.replay()
        torch.cuda.synchronize()
        assert np.array_equal(np_bits(layer.out), eager)
