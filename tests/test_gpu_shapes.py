"""Every query-group size the decode attention is built for, against the float64 oracle.

The decode attention is instantiated per G = n_q_heads / n_kv_heads (1 to 8) and
head_dim (64, 128); the workload shapes reach G = 4, 5 and 8.  Small two-layer
stages with the head cover the rest, G = 1 (multi-head attention, the degenerate
case) included, and one Qwen3-style variant: chunked prefill from tokens,
ragged batched decode, and the head's greedy token.  Every call goes through the
C ABI.
"""
import numpy as np
import pytest

import synth
from oracle import OracleStage
from tests.helpers import SeededModel, argmax_agrees, assert_hidden_close

pytestmark = pytest.mark.gpu

CASES = [  # (n_q_heads, n_kv_heads, head_dim, qk_norm)
    (4, 4, 64, False),    # G = 1
    (4, 2, 128, False),   # G = 2
    (6, 2, 64, False),    # G = 3
    (12, 2, 128, False),  # G = 6
    (14, 2, 64, False),   # G = 7
    (6, 3, 128, True),    # G = 2, per-head q/k norms, query width 768 against hidden 256
]


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


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("nq,nkv,hd,qkn", CASES, ids=[f"g{c[0] // c[1]}_hd{c[2]}{'_qknorm' if c[3] else ''}" for c in CASES])
def test_group_size(torch, st, nq, nkv, hd, qkn):
    shape = synth.ModelShape(2, 256, nq, nkv, hd, 512, 300, 1e-5, 1e4, qk_norm=qkn)
    cfg = 50 + nq + nkv + hd // 64
    model = SeededModel(shape, cfg)
    g = st.Stage(shape, 0, 2, model.layer, model.head())
    kv = g.kv(3, 200)
    o = OracleStage(shape, 0, 2, model.layer, model.head(), max_users=3, max_ctx=200)
    worst = 0.0
    for u, n in ((0, 70), (1, 5), (2, 130)):  # prompts: several splits, one tiny, several key blocks
        toks = synth.tokens(cfg, u, n, shape.vocab)
        for c0 in range(0, n, 48):
            part = toks[c0:c0 + 48]
            y = g.prefill(kv, u, c0, tokens=torch.from_numpy(part).cuda())
            worst = max(worst, assert_hidden_close(host(y), o.prefill(u, c0, tokens=part), what=f"prefill {u}@{c0}"))
    for step, users in enumerate(([0, 1, 2], [2, 0], [1], [0, 1, 2])):
        pos = [kv.len(u) for u in users]
        x = synth.hidden_states(cfg, synth.STREAM_DECODE_HIDDEN, step, len(users), shape.hidden)
        y = g.decode(kv, users, pos, hidden=torch.from_numpy(x).cuda())
        ref = o.decode(users, pos, hidden=x)
        worst = max(worst, assert_hidden_close(host(y), ref, what=f"decode {step}"))
        lg = host(g.head_logits(y))
        lr = o.logits(ref)
        tg = host(g.head_argmax(y)).astype(np.int64)
        for b in range(len(users)):
            assert argmax_agrees(int(tg[b]), int(np.argmax(lr[b])), lr[b], lg[b])
    print(f"G={nq // nkv} hd={hd} qk_norm={qkn} max row rel err", worst)
    kv.close()
    g.close()


@pytest.mark.parametrize("ffn,T", [(16384, 512), (16384, 300), (1408, 512)], ids=["f16384_t512", "f16384_t300", "f1408_t512"])
def test_prefill_swiglu_tile_widths(torch, st, ffn, T):
    """The SwiGLU projection's two tile widths, against the float64 oracle.

    Its tiles are 256 rows by 224 or 256 columns (7 or 8 blocks of 16 gate
    and 16 up rows), whichever fills whole rounds of the chip in fewer
    tile-times.  The workload shapes all take 224; an FFN of 16384 at a
    512-token chunk (2 x 128 tiles of 256 columns, exactly one round) takes
    256, and a 300-token chunk the same with a ragged row tile.  FFN 1408
    ends in a partial column tile.  One layer, a prefill from hidden rows on
    an empty cache; every output row is compared.
    """
    shape = synth.ModelShape(1, 256, 4, 2, 64, ffn, 300, 1e-5, 1e4)
    cfg = 60 + ffn % 97
    model = SeededModel(shape, cfg)
    g = st.Stage(shape, 0, 1, model.layer, None)
    kv = g.kv(1, T)
    h = synth.hidden_states(cfg, synth.STREAM_PREFILL_HIDDEN, 0, T, shape.hidden)
    y = g.prefill(kv, 0, 0, hidden=torch.from_numpy(h).cuda())
    o = OracleStage(shape, 0, 1, model.layer, None, max_users=1, max_ctx=T)
    err = assert_hidden_close(host(y), o.prefill(0, 0, hidden=h), what=f"prefill ffn {ffn} T {T}")
    print(f"ffn={ffn} T={T} prefill max row rel err", err)
    kv.close()
    g.close()


@pytest.mark.parametrize("T", [300, 512], ids=["t300", "t512"])
def test_prefill_splitk_tile_widths(torch, st, T):
    """The split-K projections' three tile widths, against the float64 oracle.

    A split-K launch takes tiles of 256 rows by 256, 160 or 128 columns,
    whichever covers its grid in the fewest weighted tile-times.  At H 6144,
    32 query heads and 8 KV heads of 128, FFN 8192, the QKV projection (6144
    columns: the last 160-column tile is partial) takes 160 columns in 3 K
    slices, the output projection 128 columns in 2, the down projection 256
    in 4; their slices meet in the RoPE and row-norm kernels and in the
    output store.  300 tokens end in a partial row tile.  One layer, a
    prefill from hidden rows on an empty cache; every output row is compared.
    """
    shape = synth.ModelShape(1, 6144, 32, 8, 128, 8192, 300, 1e-5, 1e4)
    cfg = 77
    model = SeededModel(shape, cfg)
    g = st.Stage(shape, 0, 1, model.layer, None)
    kv = g.kv(1, T)
    h = synth.hidden_states(cfg, synth.STREAM_PREFILL_HIDDEN, 0, T, shape.hidden)
    y = g.prefill(kv, 0, 0, hidden=torch.from_numpy(h).cuda())
    o = OracleStage(shape, 0, 1, model.layer, None, max_users=1, max_ctx=T)
    err = assert_hidden_close(host(y), o.prefill(0, 0, hidden=h), what=f"prefill T {T}")
    print(f"split-K tile widths T={T} prefill max row rel err", err)
    kv.close()
    g.close()
