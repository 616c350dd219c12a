"""Paged KV caches (kf_kv_create_paged) on the GPU against the float64 oracle.

The users' chunks are interleaved, so every user's pages lie scattered through
the pool; decode crosses page boundaries; a reset user's pages are lent to
another user with other contents; a request the pool cannot serve fails with
nothing changed.  The oracle keeps one dense cache per user: the pages are
bookkeeping the results must not see.  Every call goes through the C ABI.
"""
import numpy as np
import pytest

import synth
from oracle import OracleStage
from tests.helpers import SeededModel, assert_hidden_close

pytestmark = pytest.mark.gpu

TINY = synth.SHAPE_TINY
PAGE = 64


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


def pages_held(n):
    return (n + PAGE - 1) // PAGE


def test_tiny_interleaved_users_reset_and_reuse(torch, st):
    model = SeededModel(TINY, 31)
    g = st.Stage(TINY, 0, 2, model.layer, model.head())
    kv = g.kv(4, 512, pages=12)  # a reservation would take 4 x 8 pages
    o = OracleStage(TINY, 0, 2, model.layer, model.head(), max_users=4, max_ctx=512)
    assert kv.pages() == (12, 12)
    toks = {u: synth.tokens(31, u, 300, TINY.vocab) for u in range(4)}
    worst = 0.0
    # interleaved chunked prefill: users 0, 1, 2 take pages in turn
    for chunk in ((0, 40), (1, 70), (2, 25), (0, 60), (2, 90), (1, 30), (0, 29)):
        u, n = chunk
        p0 = kv.len(u)
        y = g.prefill(kv, u, p0, tokens=dev(torch, toks[u][p0:p0 + n]))
        worst = max(worst, assert_hidden_close(host(y), o.prefill(u, p0, tokens=toks[u][p0:p0 + n]),
                                               what=f"prefill user {u} at {p0}"))
    lens = {u: kv.len(u) for u in range(3)}
    assert lens == {0: 129, 1: 100, 2: 115}
    assert kv.pages() == (12, 12 - sum(pages_held(n) for n in lens.values()))
    # batched decode: users 1 and 2 cross position 128 and take a page each
    users = [0, 1, 2]
    for step in range(30):
        pos = [kv.len(u) for u in users]
        x = synth.hidden_states(31, synth.STREAM_DECODE_HIDDEN, step, 3, TINY.hidden)
        y = g.decode(kv, users, pos, hidden=dev(torch, x))
        worst = max(worst, assert_hidden_close(host(y), o.decode(users, pos, hidden=x), what=f"decode {step}"))
    # reset user 1: its pages go back to the pool and user 3 takes them
    free_before = kv.pages()[1]
    kv.set_len(1, 0)
    o.kv.set_len(1, 0)
    assert kv.pages()[1] == free_before + pages_held(130)
    y = g.prefill(kv, 3, 0, tokens=dev(torch, toks[3][:150]))
    worst = max(worst, assert_hidden_close(host(y), o.prefill(3, 0, tokens=toks[3][:150]), what="prefill user 3"))
    users = [3, 0, 2]
    for step in range(6):
        pos = [kv.len(u) for u in users]
        x = synth.hidden_states(31, synth.STREAM_DECODE_HIDDEN, 100 + step, 3, TINY.hidden)
        y = g.decode(kv, users, pos, hidden=dev(torch, x))
        worst = max(worst, assert_hidden_close(host(y), o.decode(users, pos, hidden=x), what=f"decode after reuse {step}"))
    # a request the pool cannot serve changes nothing
    free = kv.pages()[1]
    lens = [kv.len(u) for u in range(4)]
    with pytest.raises(st.KFError) as e:
        g.prefill(kv, 1, 0, tokens=dev(torch, toks[1][:(free + 1) * PAGE]))
    assert e.value.status == st.KF_ENOMEM
    with pytest.raises(st.KFError) as e:
        kv.set_len(1, (free + 1) * PAGE)
    assert e.value.status == st.KF_ENOMEM
    assert kv.pages()[1] == free and [kv.len(u) for u in range(4)] == lens
    # shrinking returns the pages past the new length
    kv.set_len(3, 64)
    o.kv.set_len(3, 64)
    assert kv.pages()[1] == free + pages_held(lens[3]) - 1
    x = synth.hidden_states(31, synth.STREAM_DECODE_HIDDEN, 200, 1, TINY.hidden)
    y = g.decode(kv, [3], [64], hidden=dev(torch, x))  # position 64 starts a new page
    worst = max(worst, assert_hidden_close(host(y), o.decode([3], [64], hidden=x), what="decode after shrink"))
    print("paged tiny max row rel err", worst)
    kv.close()
    g.close()


def test_write_read_round_trip_on_scattered_pages(torch, st):
    """kv.write / kv.read through the page table are exact (fp16 in, fp16 stored, fp32 out)."""
    model = SeededModel(TINY, 32)
    g = st.Stage(TINY, 0, 2, model.layer, None)
    kv = g.kv(3, 400, pages=20)
    rng = np.random.default_rng(5)
    data = {}
    for u, n in ((0, 100), (1, 64), (2, 200), (0, 150), (1, 1)):  # interleaved writes, users growing
        p0 = kv.len(u)
        k = rng.standard_normal((n, TINY.n_kv_heads, TINY.head_dim)).astype(np.float16)
        v = rng.standard_normal((n, TINY.n_kv_heads, TINY.head_dim)).astype(np.float16)
        kv.write(1, u, p0, dev(torch, k), dev(torch, v))  # float16 tensors: stored as they are
        kv.set_len(u, p0 + n)
        dk, dv = data.get(u, (np.zeros((0,) + k.shape[1:], np.float16),) * 2)
        data[u] = (np.concatenate([dk, k]), np.concatenate([dv, v]))
    for u, (k, v) in data.items():
        rk, rv = kv.read(1, u, 0, len(k))
        np.testing.assert_array_equal(rk.cpu().numpy(), k.astype(np.float32))
        np.testing.assert_array_equal(rv.cpu().numpy(), v.astype(np.float32))
    with pytest.raises(st.KFError):  # positions on pages user 1 does not hold
        kv.read(1, 1, 0, 200)
    kv.close()
    g.close()


def test_8b_shape_paged_decode_with_injected_contexts(torch, st):
    """Two 8B-shaped layers; contexts 1000 / 300 / 700 injected page by page in turn (scattered pages)."""
    shape, cfg_id = synth.SHAPE_8B, 33
    layers = {l: synth.layer_weights(shape, cfg_id, l) for l in (4, 5)}
    g = st.Stage(shape, 4, 6, layers, None)
    ctx = (1000, 300, 700)
    kv = g.kv(4, 1100, pages=40)
    o = OracleStage(shape, 4, 6, lambda l: layers[l], None, max_users=4, max_ctx=1100)
    full = {(l, u): synth.injected_kv(shape, cfg_id, l, u, n) for l in (4, 5) for u, n in enumerate(ctx)}
    for p0 in range(0, max(ctx), PAGE):
        for u, n in enumerate(ctx):
            if p0 >= n:
                continue
            m = min(PAGE, n - p0)
            for l in (4, 5):
                kb, vb = full[(l, u)]
                kv.write(l, u, p0, dev(torch, kb[p0:p0 + m].view(np.int16)), dev(torch, vb[p0:p0 + m].view(np.int16)))
            kv.set_len(u, p0 + m)
    for (l, u), (kb, vb) in full.items():
        o.kv.inject(l, u, 0, kb, vb)
    for u, n in enumerate(ctx):
        o.kv.set_len(u, n)
    assert kv.pages() == (40, 40 - sum(pages_held(n) for n in ctx))
    worst = 0.0
    users = [0, 1, 2]
    for step in range(3):
        pos = [kv.len(u) for u in users]
        x = synth.hidden_states(cfg_id, synth.STREAM_DECODE_HIDDEN, step, 3, shape.hidden)
        y = g.decode(kv, users, pos, hidden=dev(torch, x))
        worst = max(worst, assert_hidden_close(host(y), o.decode(users, pos, hidden=x), what=f"decode {step}"))
    h = synth.hidden_states(cfg_id, synth.STREAM_PREFILL_HIDDEN, 0, 96, shape.hidden)  # user 3 from empty
    y = g.prefill(kv, 3, 0, hidden=dev(torch, h))
    worst = max(worst, assert_hidden_close(host(y), o.prefill(3, 0, hidden=h), what="prefill chunk"))
    print("paged 8B max row rel err", worst)
    kv.close()
    g.close()


@pytest.mark.parametrize("which", ["tiny", "8b"])
def test_batch4_decode_with_splits_inside_pages(torch, st, which):
    """Batch-4 decode whose split-KV workgroups start inside cache pages.

    From batch 2 the matrix-core attention takes splits of any multiple of 16
    keys: about one workgroup per CU over the batch's keys.  These contexts make
    that 80 keys (tiny shape, 2 KV heads) or 96 keys (8B shape, 8 KV heads), so
    splits start at keys 16, 32 or 48 of a page, over scattered pages.
    """
    if which == "tiny":
        shape, cfg_id, lays, ctx = TINY, 35, (0, 1), (3000, 2000, 2500, 900)
    else:
        shape, cfg_id, lays, ctx = synth.SHAPE_8B, 36, (6, 7), (1200, 500, 900, 60)
    layers = {l: synth.layer_weights(shape, cfg_id, l) for l in lays}
    max_ctx = max(ctx) + 8
    npages = sum(pages_held(n + 3) for n in ctx)
    g = st.Stage(shape, lays[0], lays[-1] + 1, layers, None)
    kv = g.kv(4, max_ctx, pages=npages)
    o = OracleStage(shape, lays[0], lays[-1] + 1, lambda l: layers[l], None, max_users=4, max_ctx=max_ctx)
    full = {(l, u): synth.injected_kv(shape, cfg_id, l, u, n) for l in lays for u, n in enumerate(ctx)}
    for p0 in range(0, max(ctx), PAGE):  # page by page, users in turn: every user's pages scattered
        for u, n in enumerate(ctx):
            if p0 >= n:
                continue
            m = min(PAGE, n - p0)
            for l in lays:
                kb, vb = full[(l, u)]
                kv.write(l, u, p0, dev(torch, kb[p0:p0 + m].view(np.int16)), dev(torch, vb[p0:p0 + m].view(np.int16)))
            kv.set_len(u, p0 + m)
    for (l, u), (kb, vb) in full.items():
        o.kv.inject(l, u, 0, kb, vb)
    for u, n in enumerate(ctx):
        o.kv.set_len(u, n)
    worst = 0.0
    users = [2, 0, 3, 1]
    for step in range(3):
        pos = [kv.len(u) for u in users]
        x = synth.hidden_states(cfg_id, synth.STREAM_DECODE_HIDDEN, step, 4, shape.hidden)
        y = g.decode(kv, users, pos, hidden=dev(torch, x))
        worst = max(worst, assert_hidden_close(host(y), o.decode(users, pos, hidden=x), what=f"decode {step}"))
    print(f"splits inside pages ({which}) max row rel err", worst)
    kv.close()
    g.close()
