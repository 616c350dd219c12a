"""GPU parity at the full workload shapes (8B-, 32B- and 70B-shaped stages), against the float64 oracle.

Each case uses the launch configuration the benchmark times: the stage's own
layer range, its batch and its (injected or prefilled) context.  Where the
oracle cannot follow every step in seconds, a case runs fewer steps or one
layer of the stage; each docstring says which.
"""
import numpy as np
import pytest

import synth
from oracle import OracleStage, bf16_to_f64, rms_norm
from tests.helpers import argmax_agrees, assert_hidden_close, plant_lm_rows

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(170)]


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


@pytest.fixture(scope="module")
def kf():
    from paper_2609_34045_amd import stage
    return stage


def dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def build(torch, kf, wl, lo, hi, users, max_ctx, contexts, head=False, cache_weights=True):
    """GPU stage + oracle on the same seeded weights, with KV injected for ``contexts``."""
    s = wl.shape
    layers = {l: synth.layer_weights(s, wl.cfg_id, l, wl.seed) for l in range(lo, hi)}
    hw = synth.head_weights(s, wl.cfg_id, wl.seed) if head else None
    g = kf.Stage(s, lo, hi, layers, hw)
    kv = g.kv(users, max_ctx)
    o = OracleStage(s, lo, hi, lambda l: layers[l], hw, max_users=users, max_ctx=max_ctx,
                    cache_weights=cache_weights)
    for u, n in enumerate(contexts):
        if n == 0:
            continue
        for l in range(lo, hi):
            kb, vb = synth.injected_kv(s, wl.cfg_id, l, u, n, wl.seed)
            kv.write(l, u, 0, dev(torch, kb.view(np.int16)), dev(torch, vb.view(np.int16)))
            o.kv.inject(l, u, 0, kb, vb)
        kv.set_len(u, n)
        o.kv.set_len(u, n)
    return g, kv, o, layers


def decode_steps(torch, g, kv, o, wl, users, steps, first_step=0):
    s = wl.shape
    worst = 0.0
    for i in range(steps):
        x = synth.hidden_states(wl.cfg_id, synth.STREAM_DECODE_HIDDEN, first_step + i, len(users), s.hidden, wl.seed)
        pos = [kv.len(u) for u in users]
        y = g.decode(kv, users, pos, hidden=dev(torch, x))
        ref = o.decode(users, pos, hidden=x)
        worst = max(worst, assert_hidden_close(host(y), ref, what=f"{wl.name} step {i}"))
    return worst


def test_8b_mid_stage_decode(torch, kf):
    """Layers [8,16) of the 8B shape, batch 1, KV injected for [0, 2048): 4 decode steps."""
    wl = synth.WORKLOADS["8b_mid"]
    g, kv, o, _ = build(torch, kf, wl, wl.layer_lo, wl.layer_hi, 1, 2048 + 72, wl.contexts)
    print("max row rel err", decode_steps(torch, g, kv, o, wl, [0], 4))
    kv.close()
    g.close()


@pytest.fixture(scope="module")
def head_stage(torch, kf):
    wl = synth.WORKLOADS["8b_head"]
    g, kv, o, layers = build(torch, kf, wl, wl.layer_lo, wl.layer_hi, 4, 4096 + 40, (0, 0, 0, 0), head=True)
    yield wl, g, kv, o
    kv.close()
    g.close()


def test_8b_head_argmax_on_identical_hidden(torch, head_stage):
    """Full LM head (V = 128256): greedy tokens on the same fp32 hidden rows equal the oracle's."""
    wl, g, kv, o = head_stage
    h = synth.hidden_states(wl.cfg_id, synth.STREAM_DECODE_HIDDEN, 900, 4, wl.shape.hidden, wl.seed)
    t_gpu, mx = g.head_argmax(dev(torch, h), with_max=True)
    lr = o.logits(h)
    lg = host(g.head_logits(dev(torch, h)))
    assert_hidden_close(lg, lr, rtol=1e-3, what="logits")
    assert np.array_equal(t_gpu.cpu().numpy(), np.argmax(lr, axis=1))
    np.testing.assert_allclose(mx.cpu().numpy(), lr.max(axis=1), rtol=1e-4)


def test_8b_head_planted_ties_at_full_vocab(torch, kf):
    """V = 128256: batch row 0 gets an exact tie between LM-head rows 1003 and 127000 (different
    workgroups, so the final reduction must keep the lower index), row 1 a tie inside one 8-row
    workgroup (72002 and 72007), row 2 a planted maximum in the last row (128255, the tail workgroup);
    row 3 is unplanted.  GPU tokens equal the oracle's, which are the lowest planted indices."""
    wl = synth.WORKLOADS["8b_head"]
    s = wl.shape
    hw = synth.head_weights(s, wl.cfg_id, wl.seed)
    h = synth.hidden_states(wl.cfg_id, synth.STREAM_DECODE_HIDDEN, 901, 4, s.hidden, wl.seed)
    xh = rms_norm(h.astype(np.float64), bf16_to_f64(hw["final_norm"]), s.rms_eps)
    plants = {0: [127000, 1003], 1: [72007, 72002], 2: [128255]}
    for b, rows in plants.items():
        hw = plant_lm_rows(hw, xh[b], rows)
    lw = synth.layer_weights(s, wl.cfg_id, 0, wl.seed)
    g = kf.Stage(s, 0, 1, {0: lw}, hw)
    o = OracleStage(s, 0, 1, {0: lw}.__getitem__, hw, max_users=1, max_ctx=4)
    t = g.head_argmax(dev(torch, h)).cpu().numpy()
    want = o.argmax(h)
    assert [int(want[b]) for b in plants] == [1003, 72002, 128255]
    assert np.array_equal(t, want), (t, want)
    g.sync()
    g.close()


def test_8b_head_planted_ties_on_kept_rows(torch, kf):
    """V = 128256 on the rows a batch-4 decode kept (the head stage's path, 12-row workgroups): the
    decode's output rows of one layer are taken from the oracle, and the LM head gets for row 0 an exact
    tie across workgroups (2000 and 90001), for row 1 a tie inside one 12-row workgroup (60002 and
    60010), for row 2 a planted maximum in the last row (128255); row 3 is unplanted.  GPU tokens equal
    the oracle's, which are the lowest planted indices."""
    wl = synth.WORKLOADS["8b_head"]
    s = wl.shape
    lw = synth.layer_weights(s, wl.cfg_id, 0, wl.seed)
    hw = synth.head_weights(s, wl.cfg_id, wl.seed)
    users, pos = [0, 1, 2, 3], [0, 0, 0, 0]
    toks = synth.tokens(wl.cfg_id, 7, 4, s.vocab, wl.seed)
    o = OracleStage(s, 0, 1, {0: lw}.__getitem__, hw, max_users=4, max_ctx=4)
    y_ref = o.decode(users, pos, tokens=toks)
    xh = rms_norm(y_ref, bf16_to_f64(hw["final_norm"]), s.rms_eps)
    plants = {0: [90001, 2000], 1: [60010, 60002], 2: [128255]}
    for b, rows in plants.items():
        hw = plant_lm_rows(hw, xh[b], rows)
    o = OracleStage(s, 0, 1, {0: lw}.__getitem__, hw, max_users=4, max_ctx=4)
    want = o.argmax(o.decode(users, pos, tokens=toks))
    assert [int(want[b]) for b in plants] == [2000, 60002, 128255]
    g = kf.Stage(s, 0, 1, {0: lw}, hw)
    kv = g.kv(4, 4)
    assert g.decode(kv, users, pos, tokens=dev(torch, toks), keep=True) is None
    t = g.head_argmax(None, rows=4).cpu().numpy()
    assert np.array_equal(t, want), (t, want)
    g.sync()
    kv.close()
    g.close()


def test_8b_head_prefill_then_teacher_forced_decode(torch, head_stage):
    """Embedding + layers [0,4) + head; token prefill of 16/64/128/256 tokens (one chunk per user),
    then 8 greedy steps at batch 4 where both sides consume the oracle's token."""
    wl, g, kv, o = head_stage
    s = wl.shape
    ctx = (16, 64, 128, 256)
    for u, n in enumerate(ctx):
        toks = synth.tokens(wl.cfg_id, 10 + u, n, s.vocab, wl.seed)
        y = g.prefill(kv, u, 0, tokens=dev(torch, toks))
        ref = o.prefill(u, 0, tokens=toks)
        assert_hidden_close(host(y), ref, what=f"prefill user {u}")
    users = [0, 1, 2, 3]
    tok = np.array([int(o.argmax(ref[-1:])[0])] * 4, dtype=np.int32)
    near = 0
    for step in range(8):
        pos = [kv.len(u) for u in users]
        y = g.decode(kv, users, pos, tokens=dev(torch, tok))
        ref = o.decode(users, pos, tokens=tok)
        assert_hidden_close(host(y), ref, what=f"decode step {step}")
        t_gpu = g.head_argmax(y).cpu().numpy()
        lr = o.logits(ref)
        t_ref = np.argmax(lr, axis=1)
        lg = host(g.head_logits(y))
        for b in range(4):
            assert argmax_agrees(int(t_gpu[b]), int(t_ref[b]), lr[b], lg[b])
            near += int(t_gpu[b] != t_ref[b])
        tok = t_ref.astype(np.int32)
    print("near ties", near)


def test_8b_head_ragged_full_contexts(torch, kf):
    """Layers [0,4) + head at the workload's ragged contexts {256, 1024, 2048, 4096} (KV injected):
    2 closed-loop greedy steps at batch 4."""
    wl = synth.WORKLOADS["8b_head"]
    g, kv, o, _ = build(torch, kf, wl, wl.layer_lo, wl.layer_hi, 4, 4096 + 8, wl.contexts, head=True)
    users = [0, 1, 2, 3]
    tok = synth.tokens(wl.cfg_id, 0, 4, wl.shape.vocab, wl.seed)
    for step in range(2):
        pos = [kv.len(u) for u in users]
        y = g.decode(kv, users, pos, tokens=dev(torch, tok))
        ref = o.decode(users, pos, tokens=tok)
        assert_hidden_close(host(y), ref, what=f"ragged step {step}")
        t_gpu = g.head_argmax(y).cpu().numpy()
        lr, lg = o.logits(ref), host(g.head_logits(y))
        t_ref = np.argmax(lr, axis=1)
        for b in range(4):
            assert argmax_agrees(int(t_gpu[b]), int(t_ref[b]), lr[b], lg[b])
        tok = t_ref.astype(np.int32)
    kv.close()
    g.close()


def test_32b_stage_decode_batch_1_and_4(torch, kf):
    """Layers [16,32) of the 32B shape at context 4096 (KV injected): 2 steps at batch 1, 2 at batch 4."""
    wl = synth.WORKLOADS["32b_b4"]
    g, kv, o, _ = build(torch, kf, wl, wl.layer_lo, wl.layer_hi, 4, 4096 + 8, wl.contexts)
    decode_steps(torch, g, kv, o, wl, [0], 2)
    decode_steps(torch, g, kv, o, wl, [3, 1, 2, 0], 2, first_step=10)
    kv.close()
    g.close()


def test_32b_two_layers_batch_2_and_3_ragged(torch, kf):
    """Layers [16,18) of the 32B shape with ragged contexts {4096, 1500, 333}: one step at batch 2 and
    one at batch 3 (the down projection's 10-row workgroups at these batches, fp16 inputs, and
    attention splits that end inside the shorter rows)."""
    wl = synth.WORKLOADS["32b_b4"]
    g, kv, o, _ = build(torch, kf, wl, 16, 18, 3, 4096 + 8, (4096, 1500, 333))
    print("max row rel err", decode_steps(torch, g, kv, o, wl, [2, 0], 1),
          decode_steps(torch, g, kv, o, wl, [1, 2, 0], 1, first_step=20))
    kv.close()
    g.close()


def test_70b_prefill_chunk_one_layer(torch, kf):
    """Layer 40 of the 70B shape: a 512-token prefill chunk at positions [3584, 4096) on top of an
    injected cache for [0, 3584) (all 512 output rows compared), then 2 decode steps."""
    wl = synth.WORKLOADS["70b"]
    s = wl.shape
    g, kv, o, _ = build(torch, kf, wl, 40, 41, 1, 4096 + 8, (3584,))
    h = synth.hidden_states(wl.cfg_id, synth.STREAM_PREFILL_HIDDEN, 7, 512, s.hidden, wl.seed)
    y = g.prefill(kv, 0, 3584, hidden=dev(torch, h))
    ref = o.prefill(0, 3584, hidden=h)
    print("prefill max row rel err", assert_hidden_close(host(y), ref, what="70B prefill chunk"))
    decode_steps(torch, g, kv, o, wl, [0], 2)
    kv.close()
    g.close()


def test_70b_stage_decode(torch, kf):
    """Layers [40,50) of the 70B shape, batch 1, KV injected for [0, 4096): one decode step
    (the oracle widens one layer at a time)."""
    wl = synth.WORKLOADS["70b"]
    g, kv, o, _ = build(torch, kf, wl, wl.layer_lo, wl.layer_hi, 1, 4096 + 8, (4096,), cache_weights=False)
    decode_steps(torch, g, kv, o, wl, [0], 1)
    kv.close()
    g.close()


def test_8b_long_context_decode(torch, kf):
    """Ragged contexts up to 32768 keys (64 splits of 512 keys per head) on one 8B-shaped layer."""
    wl = synth.WORKLOADS["8b_b4_32k"]
    g, kv, o, _ = build(torch, kf, wl, 8, 9, 4, 32800, wl.contexts, cache_weights=True)
    worst = decode_steps(torch, g, kv, o, wl, [0, 1, 2, 3], 2)
    worst = max(worst, decode_steps(torch, g, kv, o, wl, [0], 1, first_step=5))
    print("long-context max row rel err", worst)
    kv.close()
    g.close()
