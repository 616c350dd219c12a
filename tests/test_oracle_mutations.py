"""Planted mistakes in the oracle must be caught by its pins.

Each case swaps one oracle function for a plausible wrong variant (on the CPU,
inside this process only) and checks that the scalar brute force then
disagrees with the oracle by far more than the pins' tolerance.
"""
import numpy as np
import pytest

import synth
from oracle import stage_oracle as so
from tests import brute

SHAPE = synth.ModelShape(n_layers=2, hidden=16, n_q_heads=4, n_kv_heads=2, head_dim=4, ffn=24, vocab=50,
                         rms_eps=1e-5, rope_theta=10000.0)


def _interleaved_rope(u, pos, theta):
    u = np.asarray(u, dtype=np.float64)
    hd = u.shape[-1]
    w = np.power(theta, -2.0 * np.arange(hd // 2) / hd)
    phi = np.asarray(pos, dtype=np.float64)[..., None, None] * w
    a, b = u[..., 0::2], u[..., 1::2]
    out = np.empty_like(u)
    out[..., 0::2] = a * np.cos(phi) - b * np.sin(phi)
    out[..., 1::2] = b * np.cos(phi) + a * np.sin(phi)
    return out


def _sign_flipped_rope(u, pos, theta):
    return _ORIG["rope"](u, -np.asarray(pos), theta)


def _strided_gqa(q, keys, values, n_kv_heads):
    N, nq, hd = q.shape
    out = np.empty((N, nq, hd))
    for n in range(N):
        for h in range(nq):
            g = h % n_kv_heads
            s = keys[n][:, g, :] @ q[n, h] / np.sqrt(hd)
            out[n, h] = so.softmax(s) @ values[n][:, g, :]
    return out.reshape(N, nq * hd)


def _drop_current_key(q, keys, values, n_kv_heads):
    keys = [k[:-1] if len(k) > 1 else k for k in keys]
    values = [v[:-1] if len(v) > 1 else v for v in values]
    return _ORIG["attention_rows"](q, keys, values, n_kv_heads)


def _eps_outside(x, g, eps):
    x = np.asarray(x, dtype=np.float64)
    return x / (np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps) * g


def _no_gain(x, g, eps):
    return _ORIG["rms_norm"](x, np.ones_like(g), eps)


def _swapped_gate_up(z, wg, wu, wd):
    return (so.silu(z @ wu.T) * (z @ wg.T)) @ wd.T


def _transposed_down(z, wg, wu, wd):
    a = so.silu(z @ wg.T) * (z @ wu.T)
    return a @ wd.reshape(wd.shape[1], wd.shape[0])


_ORIG = {"attention_rows": so.attention_rows, "rms_norm": so.rms_norm, "rope": so.rope}

MUTATIONS = {
    "rope_interleaved_pairs": ("rope", _interleaved_rope),
    "rope_sign": ("rope", _sign_flipped_rope),
    "gqa_strided_groups": ("attention_rows", _strided_gqa),
    "causal_drops_own_key": ("attention_rows", _drop_current_key),
    "rmsnorm_eps_outside_sqrt": ("rms_norm", _eps_outside),
    "rmsnorm_gain_dropped": ("rms_norm", _no_gain),
    "swiglu_gate_up_swapped": ("mlp_swiglu", _swapped_gate_up),
    "down_projection_transposed": ("mlp_swiglu", _transposed_down),
}


def _max_rel_gap():
    Wbits = {l: synth.layer_weights(SHAPE, 96, l) for l in range(2)}
    # small-magnitude rows make the eps placement visible as well
    h = np.random.default_rng(0).standard_normal((3, SHAPE.hidden)) * np.array([[1.0], [0.003], [1.0]])
    orc = so.OracleStage(SHAPE, 0, 2, lambda l: Wbits[l], max_users=1, max_ctx=8)
    got = orc.prefill(0, 0, hidden=h)
    br = brute.BruteStage(SHAPE, 0, 2, {l: {k: brute.widen(v) for k, v in w.items()} for l, w in Wbits.items()})
    want = np.array(br.forward(h.tolist(), [0, 0, 0], [0, 1, 2]))
    return float(np.max(np.abs(got - want) / np.max(np.abs(want), axis=-1, keepdims=True)))


def test_unmutated_oracle_agrees():
    assert _max_rel_gap() < 1e-10


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(so, attr, fn)
    assert _max_rel_gap() > 1e-6, name


def _decoder_layer_qk_norm_after_rope(x, w, shape, kv, layer, users, positions):
    """Planted mistake: the per-head q/k norms applied after RoPE instead of before."""
    x = np.asarray(x, dtype=np.float64)
    N, H = x.shape
    nq, nkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    pos = np.asarray(positions, dtype=np.int64)
    xn = so.rms_norm(x, w["attn_norm"], shape.rms_eps)
    q = so.rope((xn @ w["wq"].T).reshape(N, nq, hd), pos, shape.rope_theta)
    k = so.rope((xn @ w["wk"].T).reshape(N, nkv, hd), pos, shape.rope_theta)
    v = (xn @ w["wv"].T).reshape(N, nkv, hd)
    q = so.rms_norm(q, w["q_norm"], shape.rms_eps)
    k = so.rms_norm(k, w["k_norm"], shape.rms_eps)
    for n in range(N):
        kv.k[layer][users[n], pos[n]] = k[n]
        kv.v[layer][users[n], pos[n]] = v[n]
    keys = [kv.k[layer][users[n], : pos[n] + 1] for n in range(N)]
    vals = [kv.v[layer][users[n], : pos[n] + 1] for n in range(N)]
    x = x + so.attention_rows(q, keys, vals, nkv) @ w["wo"].T
    z = so.rms_norm(x, w["mlp_norm"], shape.rms_eps)
    return x + so.mlp_swiglu(z, w["wg"], w["wu"], w["wd"])


def test_qwen3_pin_catches_qk_norm_after_rope(monkeypatch):
    from tests import test_oracle_pins as pins
    pytest.importorskip("transformers")
    monkeypatch.setattr(so, "decoder_layer", _decoder_layer_qk_norm_after_rope)
    with pytest.raises(AssertionError):
        pins.test_qk_norm_stage_matches_transformers_qwen3_in_float64()
