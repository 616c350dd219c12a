"""Edge cases at the largest sizes the library accepts, against the float64 oracle.

A cache of max_ctx = 1,048,576 positions (the maximum) decoded at its last
slot: the attention then runs the largest split (1024 keys per workgroup) and
the most splits per row (1024), so the output projection's merge takes its
longest loops.  Over a million random keys the softmax is nearly flat and the
attention output nearly zero, which would hide a lost split; so two "needle"
keys, at positions 3 and 700,001 (different splits and pages), are aligned
with the token's own rotated queries (computed on the host from the oracle's
definitions) and dominate every head.  The output is then the mean of the
needles' values, which moves the hidden row by tens of percent: a wrong page,
split or merge weight exceeds the tolerance.  Both the reserved and the paged
cache are checked; one position more is refused.  Every call goes through the
C ABI.
"""
import numpy as np
import pytest

import synth
from oracle import OracleStage
from oracle.stage_oracle import bf16_to_f64, rms_norm, rope
from tests.helpers import SeededModel, assert_hidden_close

pytestmark = pytest.mark.gpu

TINY = synth.SHAPE_TINY
MAX_CTX = 1 << 20


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


def to_bf16(a: np.ndarray) -> np.ndarray:
    """float64 -> bf16 bit patterns, round to nearest even (finite values)."""
    b = np.asarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)


@pytest.mark.parametrize("paged", [False, True], ids=["reserved", "paged"])
def test_decode_at_the_last_slot_of_the_largest_cache(torch, st, paged):
    cfg_id = 41
    model = SeededModel(TINY, cfg_id)
    g = st.Stage(TINY, 0, 1, model.layer, None)
    n = MAX_CTX - 1
    kv = g.kv(1, MAX_CTX, pages=MAX_CTX // 64 if paged else None)
    kb, vb = synth.injected_kv(TINY, cfg_id, 0, 0, n)
    x = synth.hidden_states(cfg_id, synth.STREAM_DECODE_HIDDEN, 0, 1, TINY.hidden)
    # needles: key = 400 x the unit mean direction of each KV group's rotated queries at position n
    w = {k: bf16_to_f64(v) for k, v in model.layer(0).items()}
    nq, nkv, hd = TINY.n_q_heads, TINY.n_kv_heads, TINY.head_dim
    q = rope((rms_norm(x, w["attn_norm"], TINY.rms_eps) @ w["wq"].T).reshape(1, nq, hd), np.array([n]),
             TINY.rope_theta)[0]
    grp = nq // nkv
    rng = np.random.default_rng(7)
    for j in (3, 700_001):
        for kh in range(nkv):
            qg = q[kh * grp:(kh + 1) * grp]
            u = (qg / np.linalg.norm(qg, axis=1, keepdims=True)).sum(0)
            kb[j, kh] = to_bf16(400.0 * u / np.linalg.norm(u))
            vb[j, kh] = to_bf16(2.0 * rng.standard_normal(hd))
    # what the needles alone add to the row: W_o times the mean of their values, per head's KV group
    o = np.concatenate([(bf16_to_f64(vb[3, h // grp]) + bf16_to_f64(vb[700_001, h // grp])) / 2 for h in range(nq)])
    share = np.max(np.abs(o @ w["wo"].T)) / np.max(np.abs(x))
    assert share > 0.2  # large enough that a lost or misweighted needle breaks the 1e-2 bound
    kv.write(0, 0, 0, torch.from_numpy(kb.view(np.int16)).cuda(), torch.from_numpy(vb.view(np.int16)).cuda())
    kv.set_len(0, n)
    o = OracleStage(TINY, 0, 1, model.layer, None, max_users=1, max_ctx=MAX_CTX)
    o.kv.inject(0, 0, 0, kb, vb)
    o.kv.set_len(0, n)
    del kb, vb
    y = g.decode(kv, [0], [n], hidden=torch.from_numpy(x).cuda())
    err = assert_hidden_close(y.float().cpu().numpy().astype(np.float64), o.decode([0], [n], hidden=x),
                              what="decode over 1,048,576 keys")
    print("max-context row rel err", err, "needle share of the row", share)
    assert kv.len(0) == MAX_CTX
    with pytest.raises(st.KFError) as e:  # the cache is full
        g.decode(kv, [0], [MAX_CTX], hidden=torch.from_numpy(x).cuda())
    assert e.value.status == st.KF_ERANGE
    if paged:
        assert kv.pages() == (MAX_CTX // 64, 0)
    kv.close()
    with pytest.raises(st.KFError) as e:
        g.kv(1, MAX_CTX + 1)
    assert e.value.status == st.KF_ERANGE
    g.close()


def test_prefill_with_late_dominant_keys(torch, st):
    """Chunked prefill over an injected cache whose later keys dominate chosen queries.

    The prefill attention keeps, per query, a reference maximum for its
    exponentials and moves it only when a key block's maximum exceeds it by
    more than 8 (log2 units), so probabilities may reach 2^8 and O is rescaled
    only on such a jump.  Random keys never jump that far, so four needles per
    target query are planted in the cache, aligned with that query's rotated
    vector (computed on the host from the oracle's definitions), at scores
    7.5, 15, 12 and 17 log2 units above the query's largest ordinary score:
    the first stays under the threshold (probabilities near 2^7.5), the
    second moves the reference, the third and fourth sit in the second key
    split (a fresh reference there, a jump, then a rise under the threshold),
    so the merge of the two splits weighs references set both ways.  The last
    two needles carry most of the weight between them, and the needles move
    the target rows by tens of percent, so a misweighted needle or split
    breaks the 1e-2 bound.  Targets sit in both 128-query tiles and both KV
    groups; every row of the chunk is compared with the oracle.
    """
    cfg_id = 43
    model = SeededModel(TINY, cfg_id)
    nq, nkv, hd = TINY.n_q_heads, TINY.n_kv_heads, TINY.head_dim
    grp = nq // nkv
    n0, T = 1024, 256
    kb, vb = synth.injected_kv(TINY, cfg_id, 0, 0, n0)
    h = synth.hidden_states(cfg_id, synth.STREAM_PREFILL_HIDDEN, 0, T, TINY.hidden)
    w = {k: bf16_to_f64(v) for k, v in model.layer(0).items()}
    q = rope((rms_norm(h, w["attn_norm"], TINY.rms_eps) @ w["wq"].T).reshape(T, nq, hd), n0 + np.arange(T),
             TINY.rope_theta)
    log2e = 1.0 / np.log(2.0)
    rng = np.random.default_rng(11)
    kb0, vb0 = kb.copy(), vb.copy()
    for i, head in ((3, 0), (140, 6)):  # (query of the chunk, query head): both tiles, both KV groups
        g_kv = head // grp
        qv = q[i, head]
        ordinary = np.max(bf16_to_f64(kb[:, g_kv]) @ qv) / np.sqrt(hd) * log2e  # largest random score, log2 units
        for pos, delta in ((100, 7.5), (400, 15.0), (700, 12.0), (900, 17.0)):
            alpha = (ordinary + delta) / log2e * np.sqrt(hd) / np.linalg.norm(qv)
            kb[pos, g_kv] = to_bf16(alpha * qv / np.linalg.norm(qv))
            vb[pos, g_kv] = to_bf16(4.0 * rng.standard_normal(hd))

    def oracle(k_bits, v_bits):
        o = OracleStage(TINY, 0, 1, model.layer, None, max_users=1, max_ctx=n0 + T)
        o.kv.inject(0, 0, 0, k_bits, v_bits)
        o.kv.set_len(0, n0)
        return o.prefill(0, n0, hidden=h)

    ref = oracle(kb, vb)
    plain = oracle(kb0, vb0)
    for i in (3, 140):  # the needles move the target rows far beyond the tolerance
        assert np.max(np.abs(ref[i] - plain[i])) > 0.2 * np.max(np.abs(plain[i]))
    g = st.Stage(TINY, 0, 1, model.layer, None)
    kv = g.kv(1, n0 + T)
    kv.write(0, 0, 0, torch.from_numpy(kb.view(np.int16)).cuda(), torch.from_numpy(vb.view(np.int16)).cuda())
    kv.set_len(0, n0)
    y = g.prefill(kv, 0, n0, hidden=torch.from_numpy(h).cuda())
    err = assert_hidden_close(y.float().cpu().numpy().astype(np.float64), ref, what="prefill with needles")
    print("needle prefill max row rel err", err)
    kv.close()
    g.close()


def test_weight_matrices_beyond_the_fp16_range_are_refused(torch, st):
    """The stage keeps its matrices in fp16: a finite bf16 weight fp16 cannot hold fails init.

    65280 is the largest bf16 value below the fp16 maximum (65504) and is kept;
    65536 would become infinite.  Gains stay bf16 and take any finite value.
    """
    model = SeededModel(TINY, 41)
    base = {l: model.layer(l) for l in range(2)}

    def with_value(kind, value, layer=1, at=5):
        w = base[layer][kind].copy()
        w.flat[at] = to_bf16(np.array([value]))[0]
        return {l: ({**base[l], kind: w} if l == layer else base[l]) for l in range(2)}

    for kind in ("wq", "wd"):
        for v in (65536.0, -1.0e6):
            with pytest.raises(st.KFError) as e:
                st.Stage(TINY, 0, 2, with_value(kind, v), None)
            assert e.value.status == st.KF_EINVAL and "fp16" in e.value.message, (kind, v)
    head = dict(model.head())
    lm = head["lm_head"].copy()
    lm.flat[7] = to_bf16(np.array([1.0e5]))[0]
    with pytest.raises(st.KFError) as e:
        st.Stage(TINY, 0, 2, base, {**head, "lm_head": lm})
    assert e.value.status == st.KF_EINVAL
    g = st.Stage(TINY, 0, 2, with_value("wu", -65280.0), None)
    g.close()
    g = st.Stage(TINY, 0, 2, with_value("mlp_norm", 1.0e6), None)  # a gain: stays bf16
    g.close()
