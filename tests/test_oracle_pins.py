"""Pins of the CPU oracle against closed forms, invariants, library routines and brute force.

None of these compares the oracle with itself: each check would fail for a
plausible mistake (dropped term, wrong sign or pairing, transposed operand,
wrong GQA group, missing causal key, wrong tie-break).
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import (OracleKV, OracleStage, argmax_lowest, attention_rows, bf16_to_f64, decoder_layer,
                    head_logits, mlp_swiglu, rms_norm, rope, silu, softmax)
from tests import brute

TINY = synth.ModelShape(n_layers=3, hidden=16, n_q_heads=4, n_kv_heads=2, head_dim=4, ffn=24, vocab=50,
                        rms_eps=1e-5, rope_theta=10000.0)


def rng(seed=0):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- bf16 widening
def test_bf16_widening_exact():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x4049, 0x3C23, 0x7F7F], dtype=np.uint16)
    want = [1.0, -1.0, 0.0, 3.140625, 0.0099487304688, 3.3895313892515355e38]
    got = bf16_to_f64(bits)
    for g, w in zip(got, want):
        assert g == pytest.approx(w, rel=1e-12)


# ---------------------------------------------------------------- RMSNorm
def test_rmsnorm_rms_equals_gain_without_eps():
    x = rng(1).standard_normal((5, 64)) * 3.0
    for c in (1.0, 0.5, 2.75):
        y = rms_norm(x, np.full(64, c), 0.0)
        np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), c, rtol=1e-12)


def test_rmsnorm_closed_form_with_eps():
    x = rng(2).standard_normal((3, 32)) * 0.01  # small rows make eps visible
    eps, c = 1e-5, 1.5
    y = rms_norm(x, np.full(32, c), eps)
    m = np.mean(x * x, axis=-1)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), c * np.sqrt(m / (m + eps)), rtol=1e-12)


def test_rmsnorm_matches_torch():
    x = rng(3).standard_normal((4, 48))
    g = 1 + 0.1 * rng(4).standard_normal(48)
    want = F.rms_norm(torch.from_numpy(x), (48,), weight=torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(rms_norm(x, g, 1e-5), want, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- RoPE
def test_rope_head_dim_2_is_plane_rotation():
    # hd = 2: one pair at frequency theta^0 = 1, so the angle is the position itself.
    u = np.array([[0.3, -1.7]])
    for p in (0, 1, 5, 37):
        got = rope(u, np.array(p), 500.0)[0]
        c, s = math.cos(p), math.sin(p)
        np.testing.assert_allclose(got, [0.3 * c + 1.7 * s, -1.7 * c + 0.3 * s], rtol=1e-13)


def test_rope_head_dim_4_pairs_i_and_i_plus_half():
    theta, p = 10000.0, 7
    u = np.array([[1.0, 2.0, 3.0, 4.0]])
    got = rope(u, np.array(p), theta)[0]
    w1 = theta ** -0.5
    # pair (0, 2) at angle p, pair (1, 3) at angle p * theta^(-2/4)
    want = [1 * math.cos(p) - 3 * math.sin(p), 2 * math.cos(p * w1) - 4 * math.sin(p * w1),
            3 * math.cos(p) + 1 * math.sin(p), 4 * math.cos(p * w1) + 2 * math.sin(p * w1)]
    np.testing.assert_allclose(got, want, rtol=1e-13)


def test_rope_equals_complex_multiplication():
    hd, theta = 64, 5e5
    u = rng(5).standard_normal((3, 2, hd))
    pos = np.array([0, 11, 4095])
    got = rope(u, pos, theta)
    half = hd // 2
    z = u[..., :half] + 1j * u[..., half:]
    freq = theta ** (-np.arange(half) * 2.0 / hd)
    z = z * np.exp(1j * pos[:, None, None] * freq)
    np.testing.assert_allclose(got, np.concatenate([z.real, z.imag], axis=-1), rtol=1e-10, atol=1e-12)


def test_rope_norm_identity_and_relative_position():
    hd, theta = 128, 1e4
    q = rng(6).standard_normal((1, 1, hd))
    k = rng(7).standard_normal((1, 1, hd))
    assert np.array_equal(rope(q, np.array([0]), theta), q)
    for p in (1, 100, 4159):
        np.testing.assert_allclose(np.linalg.norm(rope(q, np.array([p]), theta)), np.linalg.norm(q), rtol=1e-12)
    d0 = np.sum(rope(q, np.array([9]), theta) * rope(k, np.array([3]), theta))
    d1 = np.sum(rope(q, np.array([9 + 50]), theta) * rope(k, np.array([3 + 50]), theta))
    assert d0 == pytest.approx(d1, rel=1e-9)


# ---------------------------------------------------------------- softmax and attention
def test_softmax_sums_to_one_and_is_shift_invariant():
    s = rng(8).standard_normal((6, 17)) * 20
    p = softmax(s)
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=1e-12)
    np.testing.assert_allclose(softmax(s + 123.0), p, rtol=1e-12)
    assert np.all(p > 0)


def test_single_key_attention_returns_value():
    q = rng(9).standard_normal((1, 4, 8))
    K = rng(10).standard_normal((1, 2, 8))
    V = rng(11).standard_normal((1, 2, 8))
    out = attention_rows(q, [K], [V], 2).reshape(4, 8)
    for h in range(4):
        assert np.array_equal(out[h], V[0, h // 2])


def test_equal_keys_give_mean_value():
    q = rng(12).standard_normal((1, 4, 8))
    K = np.repeat(rng(13).standard_normal((1, 2, 8)), 9, axis=0)
    V = rng(14).standard_normal((9, 2, 8))
    out = attention_rows(q, [K], [V], 2).reshape(4, 8)
    for h in range(4):
        np.testing.assert_allclose(out[h], V[:, h // 2].mean(0), rtol=1e-12)


def test_gqa_attention_matches_torch_sdpa():
    nq, nkv, hd, n = 8, 2, 16, 13
    q = rng(15).standard_normal((1, nq, hd))
    K = rng(16).standard_normal((n, nkv, hd))
    V = rng(17).standard_normal((n, nkv, hd))
    got = attention_rows(q, [K], [V], nkv).reshape(nq, hd)
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]  # [1, nq, 1, hd]
    tk = torch.from_numpy(K).permute(1, 0, 2)[None]
    tv = torch.from_numpy(V).permute(1, 0, 2)[None]
    want = F.scaled_dot_product_attention(tq, tk, tv, enable_gqa=True)[0, :, 0].numpy()
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------- SwiGLU
def test_silu_and_swiglu_match_torch():
    u = np.linspace(-30, 30, 101)
    np.testing.assert_allclose(silu(u), F.silu(torch.from_numpy(u)).numpy(), rtol=1e-12, atol=1e-300)
    assert silu(np.array(0.0)) == 0.0
    z = rng(18).standard_normal((2, 8))
    wg, wu, wd = (rng(19 + i).standard_normal(s) for i, s in enumerate([(12, 8), (12, 8), (8, 12)]))
    tz = torch.from_numpy(z)
    want = (F.silu(tz @ torch.from_numpy(wg).T) * (tz @ torch.from_numpy(wu).T)) @ torch.from_numpy(wd).T
    np.testing.assert_allclose(mlp_swiglu(z, wg, wu, wd), want.numpy(), rtol=1e-12)


# ---------------------------------------------------------------- layer wiring
def _tiny_weights(shape, lo, hi, seed=0, cfg=99):
    return {l: synth.layer_weights(shape, cfg, l, seed) for l in range(lo, hi)}


def test_zero_output_projections_give_identity():
    shape = TINY
    W = _tiny_weights(shape, 0, 1)[0]
    w = {k: bf16_to_f64(v) for k, v in W.items()}
    w["wo"][:] = 0.0
    w["wd"][:] = 0.0
    kv = OracleKV([0], 1, 8, shape.n_kv_heads, shape.head_dim)
    x = rng(20).standard_normal((3, shape.hidden))
    out = decoder_layer(x, w, shape, kv, 0, [0, 0, 0], [0, 1, 2])
    assert np.array_equal(out, x)


def _brute_weights(Wbits):
    return {l: {k: brute.widen(v) for k, v in w.items()} for l, w in Wbits.items()}


def test_layers_match_scalar_brute_force_prefill_then_ragged_decode():
    shape = TINY
    Wbits = _tiny_weights(shape, 0, 3)
    hb = synth.head_weights(shape, 99)
    orc = OracleStage(shape, 0, 3, lambda l: Wbits[l], hb, max_users=3, max_ctx=8)
    br = brute.BruteStage(shape, 0, 3, _brute_weights(Wbits), {k: brute.widen(v) for k, v in hb.items()})
    # prefill user 0 (4 tokens by id) and user 2 (2 hidden rows)
    toks = [3, 41, 7, 3]
    got = orc.prefill(0, 0, tokens=np.array(toks))
    want = br.forward(br.embed(toks), [0] * 4, [0, 1, 2, 3])
    np.testing.assert_allclose(got, np.array(want), rtol=1e-10, atol=1e-12)
    h2 = rng(21).standard_normal((2, shape.hidden))
    got = orc.prefill(2, 0, hidden=h2)
    want = br.forward(h2.tolist(), [2, 2], [0, 1])
    np.testing.assert_allclose(got, np.array(want), rtol=1e-10, atol=1e-12)
    # ragged batch decode: users 2, 0, 1 at positions 2, 4, 0
    hd = rng(22).standard_normal((3, shape.hidden))
    got = orc.decode([2, 0, 1], [2, 4, 0], hidden=hd)
    want = br.forward(hd.tolist(), [2, 0, 1], [2, 4, 0])
    np.testing.assert_allclose(got, np.array(want), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(orc.logits(got), np.array(br.logits(want)), rtol=1e-10, atol=1e-12)


# ---------------------------------------------------------------- whole model vs transformers' Llama
def test_stage_matches_transformers_llama_in_float64():
    transformers = pytest.importorskip("transformers")
    shape = synth.ModelShape(n_layers=3, hidden=32, n_q_heads=4, n_kv_heads=2, head_dim=8, ffn=40, vocab=64,
                             rms_eps=1e-5, rope_theta=500.0)
    Wbits = _tiny_weights(shape, 0, 3, cfg=98)
    hb = synth.head_weights(shape, 98)
    cfg = transformers.LlamaConfig(hidden_size=32, intermediate_size=40, num_attention_heads=4,
                                   num_key_value_heads=2, head_dim=8, num_hidden_layers=3, vocab_size=64,
                                   rms_norm_eps=1e-5, tie_word_embeddings=False,
                                   rope_parameters={"rope_type": "default", "rope_theta": 500.0},
                                   max_position_embeddings=64, attention_bias=False, mlp_bias=False)
    torch.manual_seed(0)
    m = transformers.LlamaForCausalLM(cfg).to(torch.float64).eval()
    names = {"attn_norm": "input_layernorm", "mlp_norm": "post_attention_layernorm", "wq": "self_attn.q_proj",
             "wk": "self_attn.k_proj", "wv": "self_attn.v_proj", "wo": "self_attn.o_proj", "wg": "mlp.gate_proj",
             "wu": "mlp.up_proj", "wd": "mlp.down_proj"}
    sd = {}
    for l, w in Wbits.items():
        for k, v in w.items():
            sd[f"model.layers.{l}.{names[k]}.weight"] = torch.from_numpy(bf16_to_f64(v))
    sd["model.embed_tokens.weight"] = torch.from_numpy(bf16_to_f64(hb["embed"]))
    sd["model.norm.weight"] = torch.from_numpy(bf16_to_f64(hb["final_norm"]))
    sd["lm_head.weight"] = torch.from_numpy(bf16_to_f64(hb["lm_head"]))
    m.load_state_dict(sd, strict=True)
    toks = [5, 17, 63, 0, 9, 33]
    orc = OracleStage(shape, 0, 3, lambda l: Wbits[l], hb, max_users=1, max_ctx=16)
    with torch.no_grad():
        out = m(torch.tensor([toks]), use_cache=True, output_hidden_states=True)
    x = orc.prefill(0, 0, tokens=np.array(toks))
    # HF applies the final norm to its last hidden state; compare logits instead
    np.testing.assert_allclose(orc.logits(x), out.logits[0].numpy(), rtol=2e-5, atol=2e-6)
    # middle stage: HF's per-layer hidden states are the stage boundaries
    mid = OracleStage(shape, 1, 3, lambda l: Wbits[l], None, max_users=1, max_ctx=16)
    h1 = out.hidden_states[1][0].numpy()
    y = mid.prefill(0, 0, hidden=h1)
    np.testing.assert_allclose(orc.logits(y), out.logits[0].numpy(), rtol=2e-5, atol=2e-6)
    # greedy decode steps with the cache
    past = out.past_key_values
    nxt = int(np.argmax(out.logits[0, -1].numpy()))
    for step in range(4):
        with torch.no_grad():
            o2 = m(torch.tensor([[nxt]]), past_key_values=past, use_cache=True)
        past = o2.past_key_values
        y = orc.decode([0], [len(toks) + step], tokens=np.array([nxt]))
        lo = orc.logits(y)
        np.testing.assert_allclose(lo, o2.logits[0].numpy(), rtol=2e-5, atol=2e-6)
        assert int(orc.argmax(y)[0]) == int(np.argmax(o2.logits[0, -1].numpy()))
        nxt = int(orc.argmax(y)[0])


# ---------------------------------------------------------------- Qwen3-style block vs transformers' Qwen3
def test_qk_norm_stage_matches_transformers_qwen3_in_float64():
    """Per-head q/k RMSNorm before RoPE, query width nq*hd != hidden, against Qwen3ForCausalLM."""
    transformers = pytest.importorskip("transformers")
    if not hasattr(transformers, "Qwen3ForCausalLM"):
        pytest.skip("transformers without Qwen3")
    shape = synth.ModelShape(n_layers=3, hidden=24, n_q_heads=4, n_kv_heads=2, head_dim=8, ffn=40, vocab=64,
                             rms_eps=1e-6, rope_theta=1000.0, qk_norm=True)
    assert shape.n_q_heads * shape.head_dim != shape.hidden
    Wbits = _tiny_weights(shape, 0, 3, cfg=97)
    assert set(Wbits[0]) == set(synth.LAYER_KINDS) | {"q_norm", "k_norm"}
    hb = synth.head_weights(shape, 97)
    cfg = transformers.Qwen3Config(hidden_size=24, intermediate_size=40, num_attention_heads=4,
                                   num_key_value_heads=2, head_dim=8, num_hidden_layers=3, vocab_size=64,
                                   rms_norm_eps=1e-6, tie_word_embeddings=False,
                                   rope_parameters={"rope_type": "default", "rope_theta": 1000.0},
                                   max_position_embeddings=64, attention_bias=False, use_sliding_window=False)
    torch.manual_seed(0)
    m = transformers.Qwen3ForCausalLM(cfg).to(torch.float64).eval()
    names = {"attn_norm": "input_layernorm", "mlp_norm": "post_attention_layernorm", "wq": "self_attn.q_proj",
             "wk": "self_attn.k_proj", "wv": "self_attn.v_proj", "wo": "self_attn.o_proj", "wg": "mlp.gate_proj",
             "wu": "mlp.up_proj", "wd": "mlp.down_proj", "q_norm": "self_attn.q_norm", "k_norm": "self_attn.k_norm"}
    sd = {}
    for l, w in Wbits.items():
        for k, v in w.items():
            sd[f"model.layers.{l}.{names[k]}.weight"] = torch.from_numpy(bf16_to_f64(v))
    sd["model.embed_tokens.weight"] = torch.from_numpy(bf16_to_f64(hb["embed"]))
    sd["model.norm.weight"] = torch.from_numpy(bf16_to_f64(hb["final_norm"]))
    sd["lm_head.weight"] = torch.from_numpy(bf16_to_f64(hb["lm_head"]))
    m.load_state_dict(sd, strict=True)
    toks = [3, 40, 63, 1, 22, 7]
    orc = OracleStage(shape, 0, 3, lambda l: Wbits[l], hb, max_users=1, max_ctx=16)
    with torch.no_grad():
        out = m(torch.tensor([toks]), use_cache=True)
    x = orc.prefill(0, 0, tokens=np.array(toks))
    np.testing.assert_allclose(orc.logits(x), out.logits[0].numpy(), rtol=2e-5, atol=2e-6)
    past = out.past_key_values
    nxt = int(np.argmax(out.logits[0, -1].numpy()))
    for step in range(3):
        with torch.no_grad():
            o2 = m(torch.tensor([[nxt]]), past_key_values=past, use_cache=True)
        past = o2.past_key_values
        y = orc.decode([0], [len(toks) + step], tokens=np.array([nxt]))
        np.testing.assert_allclose(orc.logits(y), o2.logits[0].numpy(), rtol=2e-5, atol=2e-6)
        nxt = int(orc.argmax(y)[0])


# ---------------------------------------------------------------- structural invariants
def test_prefill_equals_sequential_decode_and_chunking():
    shape = TINY
    Wbits = _tiny_weights(shape, 0, 2)
    h = rng(23).standard_normal((6, shape.hidden))
    a = OracleStage(shape, 0, 2, lambda l: Wbits[l], max_users=1, max_ctx=8)
    full = a.prefill(0, 0, hidden=h)
    b = OracleStage(shape, 0, 2, lambda l: Wbits[l], max_users=1, max_ctx=8)
    seq = np.concatenate([b.decode([0], [i], hidden=h[i:i + 1]) for i in range(6)])
    np.testing.assert_allclose(seq, full, rtol=1e-12, atol=1e-13)
    c = OracleStage(shape, 0, 2, lambda l: Wbits[l], max_users=1, max_ctx=8)
    chunked = np.concatenate([c.prefill(0, 0, hidden=h[:4]), c.prefill(0, 4, hidden=h[4:])])
    np.testing.assert_allclose(chunked, full, rtol=1e-12, atol=1e-13)


def test_stage_composition():
    shape = TINY
    Wbits = _tiny_weights(shape, 0, 3)
    h = rng(24).standard_normal((2, shape.hidden))
    whole = OracleStage(shape, 0, 3, lambda l: Wbits[l], max_users=2, max_ctx=4)
    first = OracleStage(shape, 0, 1, lambda l: Wbits[l], max_users=2, max_ctx=4)
    second = OracleStage(shape, 1, 3, lambda l: Wbits[l], max_users=2, max_ctx=4)
    y = whole.decode([0, 1], [0, 0], hidden=h)
    z = second.decode([0, 1], [0, 0], hidden=first.decode([0, 1], [0, 0], hidden=h))
    assert np.array_equal(y, z)


def test_batch_rows_are_independent():
    shape = TINY
    Wbits = _tiny_weights(shape, 0, 2)
    pre = rng(25).standard_normal((5, shape.hidden))
    h = rng(26).standard_normal((3, shape.hidden))
    batched = OracleStage(shape, 0, 2, lambda l: Wbits[l], max_users=3, max_ctx=8)
    batched.prefill(1, 0, hidden=pre)
    yb = batched.decode([0, 1, 2], [0, 5, 0], hidden=h)
    for row, (u, p) in enumerate([(0, 0), (1, 5), (2, 0)]):
        single = OracleStage(shape, 0, 2, lambda l: Wbits[l], max_users=3, max_ctx=8)
        if u == 1:
            single.prefill(1, 0, hidden=pre)
        y = single.decode([u], [p], hidden=h[row:row + 1])
        np.testing.assert_allclose(y[0], yb[row], rtol=1e-13, atol=1e-14)


def test_position_and_user_preconditions():
    shape = TINY
    Wbits = _tiny_weights(shape, 0, 1)
    s = OracleStage(shape, 0, 1, lambda l: Wbits[l], max_users=2, max_ctx=4)
    with pytest.raises(ValueError):
        s.decode([0], [1], hidden=np.zeros((1, shape.hidden)))
    with pytest.raises(ValueError):
        s.decode([0, 0], [0, 0], hidden=np.zeros((2, shape.hidden)))
    with pytest.raises(ValueError):
        s.decode([0], [0], tokens=np.array([1]))  # no head


# ---------------------------------------------------------------- head
def test_embedding_is_exact_gather():
    hb = synth.head_weights(TINY, 97)
    toks = np.array([0, 49, 7, 7])
    got = OracleStage(TINY, 0, 1, lambda l: synth.layer_weights(TINY, 97, l), hb)._input(toks, None)
    assert np.array_equal(got, bf16_to_f64(hb["embed"][toks]))


def test_argmax_planted_and_ties():
    V, H = 50, 16
    x = rng(27).standard_normal((1, H))
    g = np.ones(H)
    W = rng(28).standard_normal((V, H)) * 0.02
    xn = rms_norm(x, g, 1e-5)[0]
    W[31] = 10 * xn / np.linalg.norm(xn)
    assert argmax_lowest(head_logits(x, g, W, 1e-5))[0] == 31
    W[12] = W[31]  # exact duplicate at a lower index wins the tie
    assert argmax_lowest(head_logits(x, g, W, 1e-5))[0] == 12
    with pytest.raises(FloatingPointError):
        argmax_lowest(np.array([[0.0, np.nan]]))
