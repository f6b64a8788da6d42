"""Pins of the decoder-layer oracle (oracle/decoder.py) to closed forms,
invariants, hand-worked values and library routines other than the ones it
calls.  CPU only."""
import math

import numpy as np
import pytest
import torch

import oracle as orc
from oracle import decoder as D


def bits(x) -> np.ndarray:
    """fp32-representable values -> bf16 patterns, via torch's RNE conversion."""
    t = torch.tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def vals(h) -> np.ndarray:
    return D.bf16_to_f64(h)


# ---------------------------------------------------------------- bf16 rounding
def test_round_bf16_matches_c_oracle_and_torch():
    rng = np.random.default_rng(0)
    y = np.concatenate([
        rng.standard_normal(4000) * np.exp2(rng.integers(-140, 128, 4000)),
        # exact midpoints between neighbouring bf16 values: ties to even
        (np.arange(256, 512) + 0.5) * 2.0 ** -8,
        np.array([0.0, -0.0, 2.0 ** -133, 2.0 ** -134, 3 * 2.0 ** -135, 2.0 ** -150,
                  (2 - 2 ** -8) * 2.0 ** 127, 2.0 ** 128, -2.0 ** 130, np.inf, -np.inf]),
    ])
    got = D.round_bf16(y)
    ref = np.array([orc.round_bf16(v) for v in y], dtype=np.uint16)
    assert np.array_equal(got, ref)
    # fp32-representable values: torch's fp32 -> bf16 conversion (RNE)
    f = y[np.abs(y) < 3.0e38].astype(np.float32)
    assert np.array_equal(D.round_bf16(f.astype(np.float64)), bits(f))
    assert D.round_bf16(np.array([np.nan]))[0] == 0x7FC0


# ---------------------------------------------------------------- residual add
def test_add_equals_torch_bf16_add():
    rng = np.random.default_rng(1)
    a = bits(rng.standard_normal(5000) * np.exp2(rng.integers(-20, 20, 5000)))
    b = bits(rng.standard_normal(5000) * np.exp2(rng.integers(-20, 20, 5000)))
    ta = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    tb = torch.from_numpy(b.view(np.int16)).view(torch.bfloat16)
    ref = (ta + tb).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(D.add(a, b), ref)


# ---------------------------------------------------------------- RMSNorm
def test_rmsnorm_hand_worked():
    # x = (3, 4): mean square 12.5, y = (3, 4) / sqrt(12.5) = (0.848528..., 1.131371...)
    # bf16: 0.848528 = 1.697056 * 2^-1 -> mantissa 89/128 -> 0x3F59;
    #       1.131371 = 1.131371 * 2^0 -> mantissa round(16.82) = 17 -> 0x3F91
    _, y = D.rmsnorm(bits([[3.0, 4.0]]), bits([1.0, 1.0]), eps=0.0)
    assert y.tolist() == [[0x3F59, 0x3F91]]
    # the gain multiplies elementwise: g = (2, -1) -> 2*0.848528 = 1.697056 (0x3FD9), -1.131371 (0xBF91)
    _, y = D.rmsnorm(bits([[3.0, 4.0]]), bits([2.0, -1.0]), eps=0.0)
    assert y.tolist() == [[0x3FD9, 0xBF91]]


def test_rmsnorm_constant_row_and_eps():
    # constant row c: y = c / sqrt(c^2 + eps)
    for c, eps in ((0.5, 1e-5), (-3.0, 1e-5), (1e-3, 1e-5), (2.0, 0.0)):
        _, y = D.rmsnorm(bits(np.full((1, 64), c)), bits(np.ones(64)), eps=eps)
        ref = D.round_bf16(np.array([c / math.sqrt(c * c + eps)]))[0]
        assert np.all(y == ref), (c, eps)


def test_rmsnorm_scale_invariance_and_unit_rms():
    rng = np.random.default_rng(2)
    x = bits(rng.standard_normal((8, 256)))
    g = bits(np.ones(256))
    _, y = D.rmsnorm(x, g, eps=0.0)
    for k in (-7, 3, 20):
        xs = bits(vals(x) * 2.0 ** k)           # exact power-of-two scaling
        _, ys = D.rmsnorm(xs, g, eps=0.0)
        assert np.array_equal(ys, y)
    ms = np.mean(vals(y) ** 2, axis=1)
    assert np.all(np.abs(ms - 1.0) < 4e-3)     # bf16 rounding of each element


def test_rmsnorm_residual_is_rounded_sum():
    rng = np.random.default_rng(3)
    x = bits(rng.standard_normal((4, 128)))
    r = bits(rng.standard_normal((4, 128)) * 10)
    h, y = D.rmsnorm(x, bits(np.ones(128)), res=r)
    assert np.array_equal(h, D.add(x, r))
    _, y2 = D.rmsnorm(h, bits(np.ones(128)))
    assert np.array_equal(y, y2)


# ---------------------------------------------------------------- RoPE
def test_rope_hand_worked_pairs_half_apart():
    # d_head 4, theta 10000: frequencies (1, 10000^-1/2 = 0.01); pairs (0, 2) and (1, 3).
    x = np.zeros((2, 4))
    x[:, 0] = 1.0   # first element of pair (0, 2)
    x[:, 3] = 1.0   # second element of pair (1, 3)
    out = D.rope_f64(bits(x), seq_len=2, d_head=4)
    assert np.allclose(out[0], [1, 0, 0, 1])                     # position 0: identity
    assert np.allclose(out[1], [math.cos(1), -math.sin(0.01), math.sin(1), math.cos(0.01)])


def test_rope_position_zero_is_identity_and_norm_kept():
    rng = np.random.default_rng(4)
    x = bits(rng.standard_normal((6, 2 * 128)))
    out = D.rope(x, seq_len=3, d_head=128)
    assert np.array_equal(out[0], x[0]) and np.array_equal(out[3], x[3])   # each sequence starts at 0
    f = D.rope_f64(x, seq_len=3, d_head=128).reshape(6, 2, 128)
    v = vals(x).reshape(6, 2, 128)
    n_in = v[..., :64] ** 2 + v[..., 64:] ** 2
    n_out = f[..., :64] ** 2 + f[..., 64:] ** 2
    assert np.allclose(n_in, n_out, rtol=1e-12, atol=1e-12)


def test_rope_scores_depend_on_relative_position_only():
    rng = np.random.default_rng(5)
    q = bits(rng.standard_normal((1, 128)))
    k = bits(rng.standard_normal((1, 128)))
    L = 64

    def at(x, p):   # x placed at position p of a sequence of length L
        rows = np.zeros((L, 128), dtype=np.uint16)
        rows[p] = x[0]
        return D.rope_f64(rows, L, 128)[p]

    s1 = at(q, 10) @ at(k, 3)
    s2 = at(q, 57) @ at(k, 50)
    assert abs(s1 - s2) < 1e-9 * max(1.0, abs(s1))
    assert abs(s1 - at(q, 10) @ at(k, 4)) > 1e-6


# ---------------------------------------------------------------- attention
def _heads(rows, nh, dh, rng, scale=1.0):
    return bits(rng.standard_normal((rows, nh * dh)) * scale)


def test_attention_single_token_returns_value():
    rng = np.random.default_rng(6)
    q, k, v = _heads(3, 2, 8, rng), _heads(3, 1, 8, rng), _heads(3, 1, 8, rng)
    o = D.attention(q, k, v, seq_len=1, n_heads=2, n_kv_heads=1, d_head=8)
    assert np.array_equal(o[:, :8], v) and np.array_equal(o[:, 8:], v)


def test_attention_zero_keys_give_causal_mean():
    rng = np.random.default_rng(7)
    R, dh = 12, 16
    q = _heads(R, 1, dh, rng)
    k = np.zeros((R, dh), dtype=np.uint16)
    v = _heads(R, 1, dh, rng)
    o = D.attention(q, k, v, seq_len=6, n_heads=1, n_kv_heads=1, d_head=dh)
    vv = vals(v)
    ref = np.stack([vv[(i // 6) * 6:i + 1].mean(axis=0) for i in range(R)])
    assert np.array_equal(o, D.round_bf16(ref))


def test_attention_scale_is_inverse_sqrt_dhead():
    # two keys whose scores differ by sqrt(dh) * ln 3: weights 3 : 1
    dh = 16
    q = np.zeros((2, dh))
    q[1, 0] = 1.0
    k = np.zeros((2, dh))
    k[1, 0] = math.sqrt(dh) * math.log(3.0)   # rounded to bf16 below: use the rounded value
    kb = bits(k)
    v = np.zeros((2, dh))
    v[0, :] = 1.0
    v[1, :] = 2.0
    o = D.attention(bits(q), kb, bits(v), seq_len=2, n_heads=1, n_kv_heads=1, d_head=dh)
    w = math.exp(vals(kb)[1, 0] / math.sqrt(dh))   # = 3 up to the rounding of k
    ref = (1.0 + 2.0 * w) / (1.0 + w)
    assert np.all(o[1] == D.round_bf16(np.array([ref]))[0])
    assert abs(ref - 1.75) < 2e-3


def test_attention_is_causal_and_sequences_are_separate():
    rng = np.random.default_rng(8)
    R, dh = 10, 8
    q, k, v = _heads(R, 2, dh, rng), _heads(R, 1, dh, rng), _heads(R, 1, dh, rng)
    o = D.attention(q, k, v, seq_len=5, n_heads=2, n_kv_heads=1, d_head=dh)
    k2, v2 = k.copy(), v.copy()
    k2[3:5] = _heads(2, 1, dh, rng)
    v2[3:5] = _heads(2, 1, dh, rng)
    o2 = D.attention(q, k2, v2, seq_len=5, n_heads=2, n_kv_heads=1, d_head=dh)
    assert np.array_equal(o[:3], o2[:3]) and np.array_equal(o[5:], o2[5:])
    assert not np.array_equal(o[3:5], o2[3:5])
    assert np.array_equal(o[5, :dh], v[5]) and np.array_equal(o[5, dh:], v[5])


def test_attention_grouped_query_mapping():
    # 4 query heads, 2 key/value heads: heads 0, 1 read kv head 0, heads 2, 3 kv head 1
    rng = np.random.default_rng(9)
    R, dh = 6, 8
    q = _heads(R, 4, dh, rng)
    k = _heads(R, 2, dh, rng)
    v = np.concatenate([np.zeros((R, dh)), np.ones((R, dh))], axis=1)
    o = vals(D.attention(q, k, bits(v), seq_len=R, n_heads=4, n_kv_heads=2, d_head=dh))
    assert np.all(o[:, :2 * dh] == 0.0) and np.all(o[:, 2 * dh:] == 1.0)


def test_attention_dominant_key():
    dh = 8
    q = np.zeros((4, dh))
    q[3, 0] = 64.0
    k = np.zeros((4, dh))
    k[1, 0] = 64.0          # score 64*64/sqrt(8) ~ 1448 for key 1 at query 3
    v = np.arange(4 * dh, dtype=np.float64).reshape(4, dh)
    o = D.attention(bits(q), bits(k), bits(v), seq_len=4, n_heads=1, n_kv_heads=1, d_head=dh)
    assert np.array_equal(o[3], bits(v[1]))


# ---------------------------------------------------------------- SwiGLU
def test_swiglu_closed_forms_and_torch_silu():
    # gate 0 -> 0; gate ln 3 -> sigmoid = 3/4; gate/up order matters
    gu = bits([[0.0, 1.0, 5.0, 2.0], [1.0, 1.0, 2.0, 1.0]])   # ffn 2: gate (g0, g1), up (u0, u1)
    a = vals(D.swiglu(gu, 2))
    assert a[0, 0] == 0.0
    assert a[1, 0] == vals(D.round_bf16(np.array([2.0 / (1 + math.exp(-1.0))])))[0]   # g=1, u=2
    g3 = vals(bits([math.log(3.0)]))[0]
    a3 = vals(D.swiglu(bits([[g3, 4.0]]), 1))[0, 0]
    assert a3 == vals(D.round_bf16(np.array([g3 * (1 / (1 + math.exp(-g3))) * 4.0])))[0]
    assert abs(a3 - 0.75 * math.log(3.0) * 4.0) < 0.02
    rng = np.random.default_rng(10)
    gu = bits(rng.standard_normal((16, 64)) * 4)
    v = vals(gu)
    ref = torch.nn.functional.silu(torch.from_numpy(v[:, :32])).numpy() * v[:, 32:]
    assert np.array_equal(D.swiglu(gu, 32), D.round_bf16(ref))


# ---------------------------------------------------------------- FP8 linears
def test_gemm_e4_equals_c_oracle_bit_for_bit():
    rng = np.random.default_rng(11)
    a8 = rng.integers(0, 256, (37, 300), dtype=np.uint8)
    b8 = rng.integers(0, 256, (53, 300), dtype=np.uint8)
    a8[(a8 & 0x7F) == 0x7F] = 0x3C   # no NaN codes
    b8[(b8 & 0x7F) == 0x7F] = 0x41
    got = D.gemm_e4(a8, 3, b8, -2)
    ref = orc.gemm_nt(a8, orc.E4M3, 3, b8, orc.E4M3, -2, out_dt=orc.BF16)
    assert np.array_equal(got, ref)
    with pytest.raises(ValueError):
        D.gemm_e4(np.zeros((1, 1 << 15), np.uint8), 0, np.zeros((1, 1 << 15), np.uint8), 0)


# ---------------------------------------------------------------- the chain
def _layer_params(rng, d, nh, nkv, dh, ffn, zero_o=False, zero_down=False):
    p = {"g_attn": bits(1 + 0.1 * rng.standard_normal(d)), "g_mlp": bits(1 + 0.1 * rng.standard_normal(d))}
    shapes = {"qkv": (d, (nh + 2 * nkv) * dh), "o": (nh * dh, d), "gate_up": (d, 2 * ffn), "down": (ffn, d)}
    for name, (K, N) in shapes.items():
        w = bits(rng.standard_normal((K, N)) * 0.05)
        if (name == "o" and zero_o) or (name == "down" and zero_down):
            w = np.zeros((K, N), dtype=np.uint16)
        _, w8t, bw, _ = orc.ptq_quantise_weights(w)
        p[name + "_w8t"], p[name + "_bw"] = w8t, bw
    return p


def test_layer_forward_zero_projections_pass_the_residual():
    rng = np.random.default_rng(12)
    d, nh, nkv, dh, ffn = 64, 4, 2, 16, 96
    H = bits(rng.standard_normal((12, d)))
    p = _layer_params(rng, d, nh, nkv, dh, ffn, zero_o=True, zero_down=True)
    r = D.layer_forward(H, p, seq_len=6, n_heads=nh, n_kv_heads=nkv, d_head=dh, ffn=ffn)
    assert np.array_equal(r["out"], H)          # out = H + 0 + 0
    assert np.all(vals(r["o"]) == 0) and np.all(vals(r["down"]) == 0)


def test_layer_forward_shapes_and_biases():
    rng = np.random.default_rng(13)
    d, nh, nkv, dh, ffn = 64, 4, 2, 16, 96
    H = bits(rng.standard_normal((12, d)))
    p = _layer_params(rng, d, nh, nkv, dh, ffn)
    r = D.layer_forward(H, p, seq_len=6, n_heads=nh, n_kv_heads=nkv, d_head=dh, ffn=ffn)
    assert r["qkv"].shape == (12, (nh + 2 * nkv) * dh)
    assert r["attn"].shape == (12, nh * dh) and r["act"].shape == (12, ffn)
    assert r["out"].shape == H.shape
    for t, b in (("xn", "b_xn"), ("attn", "b_attn"), ("hn", "b_hn"), ("act", "b_act")):
        m = np.max(np.abs(vals(r[t])))
        assert m * 2.0 ** r[b] <= 448 < m * 2.0 ** (r[b] + 1)     # Eq. 3
    # the attention input at position 0 of each sequence is the unrotated projection
    assert np.array_equal(r["q"][0], r["qkv"][0, :nh * dh])


def test_layer_forward_per_sequence_biases():
    rng = np.random.default_rng(14)
    d, nh, nkv, dh, ffn = 64, 4, 2, 16, 96
    H = bits(rng.standard_normal((12, d)) * np.repeat([1.0, 40.0], 6)[:, None])   # two sequences, scales apart
    p = _layer_params(rng, d, nh, nkv, dh, ffn)
    # one sequence: the per-sequence mode is the per-tensor mode
    a = D.layer_forward(H, p, seq_len=12, n_heads=nh, n_kv_heads=nkv, d_head=dh, ffn=ffn)
    b = D.layer_forward(H, p, seq_len=12, n_heads=nh, n_kv_heads=nkv, d_head=dh, ffn=ffn, per_sequence=True)
    assert np.array_equal(a["out"], b["out"])
    assert [b["b_xn"], b["b_attn"], b["b_hn"], b["b_act"]] == [[a["b_xn"]], [a["b_attn"]], [a["b_hn"]], [a["b_act"]]]
    # two sequences: Eq. 3 on each sequence's rows; the tensor's bias is the smallest of them
    t = D.layer_forward(H, p, seq_len=6, n_heads=nh, n_kv_heads=nkv, d_head=dh, ffn=ffn)
    s = D.layer_forward(H, p, seq_len=6, n_heads=nh, n_kv_heads=nkv, d_head=dh, ffn=ffn, per_sequence=True)
    for x, bk in (("xn", "b_xn"), ("attn", "b_attn"), ("hn", "b_hn"), ("act", "b_act")):
        assert len(s[bk]) == 2
        for seg, bseg in zip((s[x][:6], s[x][6:]), s[bk]):
            m = np.max(np.abs(vals(seg)))
            assert m * 2.0 ** bseg <= 448 < m * 2.0 ** (bseg + 1)
    assert min(s["b_xn"]) == t["b_xn"]          # same RMSNorm output in both modes
