"""kf_stage_prefill_noalloc against kf_stage_prefill: the same chunks through both entry points.

The no-allocation variant runs the same kernels over a static per-device scratch
array instead of the stage's own grown workspace, so its outputs and cache
contents must equal the allocating call's bit for bit; both are also held to the
float64 oracle's tolerance.  Two calls in a row, the second smaller, check that
nothing carried over in the shared array affects the next call.
"""
import numpy as np
import pytest

import synth
from oracle import OracleStage
from tests.helpers import SeededModel, assert_hidden_close

pytestmark = pytest.mark.gpu


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


def both(torch, g, kv_a, kv_b, user, pos0, **inp):
    """The chunk through kf_stage_prefill (cache kv_a) and kf_stage_prefill_noalloc (cache kv_b)."""
    src = inp.get("hidden", inp.get("tokens"))
    out_b = torch.empty((src.shape[0], g.shape.hidden), dtype=torch.float32, device="cuda")
    a = g.prefill(kv_a, user, pos0, **inp)
    b = g.prefill(kv_b, user, pos0, out=out_b, noalloc=True, **inp)
    g.sync()
    return a, b


def test_tiny_head_two_chunks(torch, st):
    """Tiny stage with the head: a 96-token token chunk for user 0, then a smaller 40-token hidden chunk
    for user 1; outputs and every cached key and value equal the allocating call's."""
    shape, cfg = synth.SHAPE_TINY, 1
    model = SeededModel(shape, cfg)
    g = st.Stage(shape, 0, 2, model.layer, model.head())
    kv_a, kv_b = g.kv(2, 160), g.kv(2, 160)
    o = OracleStage(shape, 0, 2, model.layer, model.head(), max_users=2, max_ctx=160)
    toks = synth.tokens(cfg, 30, 96, shape.vocab)
    a, b = both(torch, g, kv_a, kv_b, 0, 0, tokens=dev(torch, toks))
    assert torch.equal(a, b)
    assert_hidden_close(host(b), o.prefill(0, 0, tokens=toks), what="no-alloc token chunk")
    h = synth.hidden_states(cfg, synth.STREAM_PREFILL_HIDDEN, 31, 40, shape.hidden)
    a, b = both(torch, g, kv_a, kv_b, 1, 0, hidden=dev(torch, h))
    assert torch.equal(a, b)
    assert_hidden_close(host(b), o.prefill(1, 0, hidden=h), what="no-alloc hidden chunk")
    for user, n in ((0, 96), (1, 40)):
        assert kv_a.len(user) == kv_b.len(user) == n
        for l in range(2):
            ka, va = kv_a.read(l, user, 0, n)
            kb, vb = kv_b.read(l, user, 0, n)
            assert torch.equal(ka, kb) and torch.equal(va, vb)
    for x in (kv_a, kv_b, g):
        x.close()


def test_8b_layer_full_chunk_then_smaller(torch, st):
    """One 8B-shaped layer: a 512-token chunk (90 MiB of scratch) at [0, 512), then a 100-token chunk
    continuing the same user at [512, 612); then a 2048-token chunk, whose workspace exceeds the
    scratch, is refused with KF_ERANGE and changes nothing."""
    wl = synth.WORKLOADS["8b_mid"]
    shape = wl.shape
    lw = synth.layer_weights(shape, wl.cfg_id, 8, wl.seed)
    g = st.Stage(shape, 8, 9, {8: lw})
    kv_a, kv_b = g.kv(1, 2800), g.kv(1, 2800)
    o = OracleStage(shape, 8, 9, {8: lw}.__getitem__, None, max_users=1, max_ctx=2800)
    pos = 0
    for n in (512, 100):
        h = synth.hidden_states(wl.cfg_id, synth.STREAM_PREFILL_HIDDEN, 40 + n, n, shape.hidden, wl.seed)
        a, b = both(torch, g, kv_a, kv_b, 0, pos, hidden=dev(torch, h))
        assert torch.equal(a, b), f"chunk of {n}"
        assert_hidden_close(host(b), o.prefill(0, pos, hidden=h), what=f"no-alloc chunk of {n}")
        pos += n
    ka, va = kv_a.read(8, 0, 0, pos)
    kb, vb = kv_b.read(8, 0, 0, pos)
    assert torch.equal(ka, kb) and torch.equal(va, vb)
    big = torch.zeros((2048, shape.hidden), dtype=torch.float32, device="cuda")
    with pytest.raises(st.KFError) as e:
        g.prefill(kv_b, 0, pos, hidden=big, out=big, noalloc=True)
    assert e.value.status == st.KF_ERANGE and "scratch" in e.value.message
    assert kv_b.len(0) == pos
    g.sync()
    for x in (kv_a, kv_b, g):
        x.close()
