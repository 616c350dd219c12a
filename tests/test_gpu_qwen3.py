"""GPU parity for Qwen3-style blocks (per-head q/k RMSNorm before RoPE), against the float64 oracle.

The tiny shape keeps the query width (8 x 64 = 512) different from the hidden
size (384); the full shapes are Qwen3-8B and Qwen3-32B blocks (the latter with
64 x 128 = 8192 query width against H = 5120) on a couple of layers.  Decode
runs the raw-q/k QKV epilogue plus the per-head norm kernel; prefill runs the
norm inside its RoPE kernel.  Every call goes through the C ABI.
"""
import numpy as np
import pytest

import synth
from oracle import OracleStage
from tests.helpers import SeededModel, argmax_agrees, assert_hidden_close

pytestmark = pytest.mark.gpu

TINY = synth.SHAPE_QWEN3_TINY
CFG = 11


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


@pytest.fixture(scope="module")
def st():
    from paper_2609_34045_amd import stage
    return stage


def dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def test_tiny_prefill_decode_and_head(torch, st):
    model = SeededModel(TINY, CFG)
    g = st.Stage(TINY, 0, 2, model.layer, model.head())
    kv = g.kv(2, 128)
    o = OracleStage(TINY, 0, 2, model.layer, model.head(), max_users=2, max_ctx=128)
    toks = synth.tokens(CFG, 0, 40, TINY.vocab)
    worst = 0.0
    pos = 0
    for n in (24, 16):  # chunked prefill from tokens
        y = g.prefill(kv, 0, pos, tokens=dev(torch, toks[pos:pos + n]))
        ref = o.prefill(0, pos, tokens=toks[pos:pos + n])
        worst = max(worst, assert_hidden_close(host(y), ref, what=f"prefill at {pos}"))
        pos += n
    h = synth.hidden_states(CFG, synth.STREAM_PREFILL_HIDDEN, 0, 9, TINY.hidden)  # a second user, ragged
    y = g.prefill(kv, 1, 0, hidden=dev(torch, h))
    worst = max(worst, assert_hidden_close(host(y), o.prefill(1, 0, hidden=h), what="user 1 prefill"))
    tok = int(toks[-1])
    for step in range(6):  # batch of the two users at different positions, greedy for user 0
        p = [kv.len(0), kv.len(1)]
        x1 = synth.hidden_states(CFG, synth.STREAM_DECODE_HIDDEN, step, 1, TINY.hidden)
        emb = o.head["embed"][tok][None, :]
        hin = np.concatenate([emb, x1]).astype(np.float32)
        y = g.decode(kv, [0, 1], p, hidden=dev(torch, hin))
        ref = o.decode([0, 1], p, hidden=hin)
        worst = max(worst, assert_hidden_close(host(y), ref, what=f"decode step {step}"))
        lg = host(g.head_logits(y))[0]
        lr = o.logits(ref)[0]
        t_gpu, t_ref = int(host(g.head_argmax(y))[0]), int(np.argmax(lr))
        assert argmax_agrees(t_gpu, t_ref, lr, lg)
        tok = t_ref
    print("qwen3 tiny max row rel err", worst)
    kv.close()
    g.close()


def _full(torch, st, shape, cfg_id, lo, hi, users, ctx, inject):
    layers = {l: synth.layer_weights(shape, cfg_id, l) for l in range(lo, hi)}
    g = st.Stage(shape, lo, hi, layers, None)
    kv = g.kv(users, ctx)
    o = OracleStage(shape, lo, hi, lambda l: layers[l], None, max_users=users, max_ctx=ctx)
    for u, n in enumerate(inject):
        for l in range(lo, hi):
            kb, vb = synth.injected_kv(shape, cfg_id, l, u, n)
            kv.write(l, u, 0, dev(torch, kb.view(np.int16)), dev(torch, vb.view(np.int16)))
            o.kv.inject(l, u, 0, kb, vb)
        kv.set_len(u, n)
        o.kv.set_len(u, n)
    return g, kv, o


@pytest.mark.parametrize("shape,cfg_id", [(synth.SHAPE_QWEN3_8B, 12), (synth.SHAPE_QWEN3_32B, 13)],
                         ids=["qwen3_8b", "qwen3_32b"])
def test_full_shape_decode_batch_and_prefill_chunk(torch, st, shape, cfg_id):
    g, kv, o = _full(torch, st, shape, cfg_id, 10, 12, 4, 1100, (1000, 300, 700, 0))
    worst = 0.0
    users = [0, 1, 2]
    for step in range(3):
        x = synth.hidden_states(cfg_id, synth.STREAM_DECODE_HIDDEN, step, 3, shape.hidden)
        pos = [kv.len(u) for u in users]
        y = g.decode(kv, users, pos, hidden=dev(torch, x))
        worst = max(worst, assert_hidden_close(host(y), o.decode(users, pos, hidden=x), what=f"decode {step}"))
    h = synth.hidden_states(cfg_id, synth.STREAM_PREFILL_HIDDEN, 0, 96, shape.hidden)  # user 3 from empty
    y = g.prefill(kv, 3, 0, hidden=dev(torch, h))
    worst = max(worst, assert_hidden_close(host(y), o.prefill(3, 0, hidden=h), what="prefill chunk"))
    x = synth.hidden_states(cfg_id, synth.STREAM_DECODE_HIDDEN, 9, 1, shape.hidden)
    y = g.decode(kv, [3], [96], hidden=dev(torch, x))
    worst = max(worst, assert_hidden_close(host(y), o.decode([3], [96], hidden=x), what="decode after prefill"))
    print(shape, "max row rel err", worst)
    kv.close()
    g.close()


@pytest.mark.timeout(170)
def test_qwen3_32b_prefill_chunk_as_benched(torch, st):
    """Layer 16 of the Qwen3-32B shape, the benchmark's chunk: 512 tokens at positions [3584, 4096)
    over an injected cache for [0, 3584) (all 512 rows compared), then one decode step."""
    wl = synth.WORKLOADS["qwen3_32b_b1"]
    shape, cfg_id = wl.shape, wl.cfg_id
    g, kv, o = _full(torch, st, shape, cfg_id, 16, 17, 1, 4096 + 8, (3584,))
    h = synth.hidden_states(cfg_id, synth.STREAM_PREFILL_HIDDEN, 7, 512, shape.hidden)
    y = g.prefill(kv, 0, 3584, hidden=dev(torch, h))
    worst = assert_hidden_close(host(y), o.prefill(0, 3584, hidden=h), what="qwen3-32b chunk")
    x = synth.hidden_states(cfg_id, synth.STREAM_DECODE_HIDDEN, 3, 1, shape.hidden)
    y = g.decode(kv, [0], [4096], hidden=dev(torch, x))
    worst = max(worst, assert_hidden_close(host(y), o.decode([0], [4096], hidden=x), what="decode after chunk"))
    print("qwen3-32b chunk max row rel err", worst)
    kv.close()
    g.close()


def test_tiny_paged_batch4_new_keys_inside_pages(torch, st):
    """Batch-4 decode of q/k-norm blocks over a paged cache whose pages are scattered.

    The contexts (3000 / 2000 / 2500 / 900 keys, injected one 64-position page
    per user in turn) make the batch's split-KV workgroups 80 keys long, so
    splits start inside pages, and over the steps each row's new key falls at
    different offsets of its 16-key block: the workgroup holding it normalises,
    rotates and stores it, and scores it in place of the stale cache row.
    """
    page = 64
    model = SeededModel(TINY, CFG)
    ctx = (3000, 2000, 2500, 900)
    max_ctx = max(ctx) + 8
    npages = sum((n + 5 + page - 1) // page for n in ctx)
    g = st.Stage(TINY, 0, 2, model.layer, None)
    kv = g.kv(4, max_ctx, pages=npages)
    o = OracleStage(TINY, 0, 2, model.layer, None, max_users=4, max_ctx=max_ctx)
    full = {(l, u): synth.injected_kv(TINY, CFG, l, u, n) for l in (0, 1) for u, n in enumerate(ctx)}
    for p0 in range(0, max(ctx), page):
        for u, n in enumerate(ctx):
            if p0 >= n:
                continue
            m = min(page, n - p0)
            for l in (0, 1):
                kb, vb = full[(l, u)]
                kv.write(l, u, p0, dev(torch, kb[p0:p0 + m].view(np.int16)), dev(torch, vb[p0:p0 + m].view(np.int16)))
            kv.set_len(u, p0 + m)
    for (l, u), (kb, vb) in full.items():
        o.kv.inject(l, u, 0, kb, vb)
    for u, n in enumerate(ctx):
        o.kv.set_len(u, n)
    worst = 0.0
    users = [1, 3, 0, 2]
    for step in range(5):
        pos = [kv.len(u) for u in users]
        x = synth.hidden_states(CFG, synth.STREAM_DECODE_HIDDEN, step, 4, TINY.hidden)
        y = g.decode(kv, users, pos, hidden=dev(torch, x))
        worst = max(worst, assert_hidden_close(host(y), o.decode(users, pos, hidden=x), what=f"decode {step}"))
    print("qwen3 tiny paged batch-4 max row rel err", worst)
    kv.close()
    g.close()
