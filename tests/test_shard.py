"""The safetensors shard loader (kf_shard_*): byte-range reads of a stage's share of a checkpoint.

CPU only: headers, the stage's tensor list, positioned reads and the tensors held
between fetches are host code.  Checkpoints are written by the safetensors package
from the seeded synthetic weights under Hugging Face Llama / Qwen3 names; every
fetched tensor must equal the array it was written from, and the bytes read must
equal the stage's share (paper, Section VI: shards fetched by byte range, shared
tensors not re-read after a replan).
"""
import dataclasses
import json
import struct

import numpy as np
import pytest

import synth
from tests import st_files

KINDS = {0: "attn_norm", 1: "wq", 2: "wk", 3: "wv", 4: "wo", 5: "mlp_norm", 6: "wg", 7: "wu", 8: "wd", 9: "embed",
         10: "final_norm", 11: "lm_head", 12: "q_norm", 13: "k_norm"}


@pytest.fixture(scope="module")
def sh():
    from paper_2609_34045_amd import shard
    return shard


@pytest.fixture(scope="module")
def kf():
    from paper_2609_34045_amd import stage
    return stage


def tiny_model(shape, cfg, n):
    return {l: synth.layer_weights(shape, cfg, l) for l in range(n)}, synth.head_weights(shape, cfg)


@pytest.fixture()
def two_files(tmp_path):
    """Layers 0-1 and the embedding in one file; layers 2-3, the final norm, the LM head and an unrelated
    fp32 tensor in the other."""
    shape = dataclasses.replace(synth.SHAPE_TINY, n_layers=4)
    layers, head = tiny_model(shape, 1, 4)
    a = st_files.checkpoint_tensors({0: layers[0], 1: layers[1]}, {"embed": head["embed"]})
    b = st_files.checkpoint_tensors({2: layers[2], 3: layers[3]},
                                    {"final_norm": head["final_norm"], "lm_head": head["lm_head"]})
    import torch
    b["model.rotary_emb.inv_freq"] = torch.arange(32, dtype=torch.float32)
    pa, pb = str(tmp_path / "model-00001-of-00002.safetensors"), str(tmp_path / "model-00002-of-00002.safetensors")
    st_files.save(pa, a)
    st_files.save(pb, b)
    return shape, layers, head, [pa, pb]


def block_bytes(shape):
    return shape.block_bytes()


def head_bytes(shape):
    return 2 * (2 * shape.vocab * shape.hidden + shape.hidden)


def check_fetched(got, layers, head):
    for layer, kind, arr in got:
        name = KINDS[kind]
        want = head[name] if layer < 0 else layers[layer][name]
        assert np.array_equal(arr, np.ascontiguousarray(want).reshape(-1)), (layer, name)


def test_fetch_reads_exactly_the_stage_share(sh, kf, two_files):
    shape, layers, head, paths = two_files
    with sh.Checkpoint(paths) as ck:
        assert ck.stats() == (0, 0)  # opening reads headers only
        total, fetch, n = ck.plan(shape, 1, 3, False)
        assert total == fetch == 2 * block_bytes(shape) and n == 18
        got = ck.fetch(shape, 1, 3, False)
        check_fetched(got, layers, head)
        assert sorted({l for l, _, _ in got}) == [1, 2]
        assert ck.stats() == (total, total)
        # a replan to [2, 4) with the head re-reads nothing it holds: layer 3 and the head only
        total2, fetch2, _ = ck.plan(shape, 2, 4, True)
        assert total2 == 2 * block_bytes(shape) + head_bytes(shape)
        bb, bh, _ = kf.stage_bytes(shape, 2, 4, True, 0, 0)  # the stage's own byte sizes (eq. (2)'s betas)
        assert total2 == 2 * bb + bh
        assert fetch2 == block_bytes(shape) + head_bytes(shape)
        check_fetched(ck.fetch(shape, 2, 4, True), layers, head)
        assert ck.stats()[0] == total + fetch2
        assert ck.plan(shape, 2, 4, True)[1] == 0
        ck.release(2, 4, True)  # layer 1 dropped
        assert ck.stats()[1] == total2
        assert ck.plan(shape, 1, 2, False)[1] == block_bytes(shape)
        ck.release()
        assert ck.stats()[1] == 0


def test_qwen3_names_and_tied_embeddings(sh, kf, tmp_path):
    shape = synth.SHAPE_QWEN3_TINY
    layers, head = tiny_model(shape, 11, 2)
    path = str(tmp_path / "qwen3.safetensors")
    st_files.save(path, st_files.checkpoint_tensors(layers, {"embed": head["embed"], "final_norm": head["final_norm"]}))
    with sh.Checkpoint(path) as ck:
        with pytest.raises(kf.KFError) as e:
            ck.plan(shape, 0, 2, True)
        assert e.value.status == kf.KF_EINVAL and "lm_head.weight" in e.value.message
        total, fetch, n = ck.plan(shape, 0, 2, True, tied=True)
        assert n == 2 * 11 + 3
        assert total == 2 * block_bytes(shape) + 2 * (shape.vocab * shape.hidden + shape.hidden)  # one shared matrix
        got = ck.fetch(shape, 0, 2, True, tied=True)
        tied_head = dict(head, lm_head=head["embed"])
        check_fetched(got, layers, tied_head)
        assert ck.stats()[0] == total


def write_raw(path, header: dict, data: bytes, pad: int = 0):
    h = json.dumps(header).encode() + b" " * pad
    with open(path, "wb") as f:
        f.write(struct.pack("<Q", len(h)) + h + data)


def test_malformed_files_are_refused(sh, kf, tmp_path):
    p = str(tmp_path / "bad.safetensors")
    good = {"x": {"dtype": "BF16", "shape": [2, 2], "data_offsets": [0, 8]}}
    write_raw(p, good, b"\0" * 8, pad=5)
    sh.Checkpoint(p).close()  # a space-padded header is valid
    cases = [
        ({"x": {"dtype": "BF16", "shape": [2, 2], "data_offsets": [0, 8]}}, b"\0" * 4),   # range past the end
        ({"x": {"dtype": "BF16", "shape": [2, 3], "data_offsets": [0, 8]}}, b"\0" * 8),   # size != shape
        ({"x": {"dtype": "BF16", "shape": [2, 2]}}, b"\0" * 8),                           # no offsets
        ({"x": {"dtype": "BF16", "shape": [2, 2], "data_offsets": [8, 0]}}, b"\0" * 8),   # reversed
    ]
    for hdr, data in cases:
        write_raw(p, hdr, data)
        with pytest.raises(kf.KFError) as e:
            sh.Checkpoint(p)
        assert e.value.status == kf.KF_EINVAL
    with open(p, "wb") as f:  # not JSON
        f.write(struct.pack("<Q", 5) + b"{oops")
    with pytest.raises(kf.KFError):
        sh.Checkpoint(p)
    with open(p, "wb") as f:  # header length beyond the file
        f.write(struct.pack("<Q", 1 << 20) + b"{}")
    with pytest.raises(kf.KFError):
        sh.Checkpoint(p)
    with pytest.raises(kf.KFError):
        sh.Checkpoint(str(tmp_path / "missing.safetensors"))
    q = str(tmp_path / "dup.safetensors")
    write_raw(q, good, b"\0" * 8)
    write_raw(p, good, b"\0" * 8)
    with pytest.raises(kf.KFError) as e:
        sh.Checkpoint([p, q])
    assert "twice" in e.value.message


def test_wrong_dtype_shape_or_missing_layer(sh, kf, tmp_path):
    shape = dataclasses.replace(synth.SHAPE_TINY, n_layers=4)
    layers, head = tiny_model(shape, 1, 2)
    t = st_files.checkpoint_tensors(layers, None)
    t["model.layers.1.mlp.up_proj.weight"] = t["model.layers.1.mlp.up_proj.weight"].float()
    t["model.layers.0.self_attn.o_proj.weight"] = t["model.layers.0.self_attn.o_proj.weight"][:, :256].contiguous()
    path = str(tmp_path / "m.safetensors")
    st_files.save(path, t)
    with sh.Checkpoint(path) as ck:
        with pytest.raises(kf.KFError) as e:
            ck.plan(shape, 1, 2, False)
        assert e.value.status == kf.KF_EUNSUPPORTED and "up_proj" in e.value.message
        with pytest.raises(kf.KFError) as e:
            ck.fetch(shape, 0, 1, False)
        assert e.value.status == kf.KF_EINVAL and "o_proj" in e.value.message
        with pytest.raises(kf.KFError) as e:
            ck.plan(shape, 2, 3, False)
        assert "model.layers.2." in e.value.message
        assert ck.stats() == (0, 0)  # a failed fetch holds nothing


@pytest.mark.gpu
def test_stage_from_checkpoint_equals_stage_from_arrays(sh, kf, two_files):
    """A head stage built by kf_shard_stage_init decodes bit-identically to one built from the arrays."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    shape, layers, head, paths = two_files
    with sh.Checkpoint(paths) as ck:
        a = ck.stage(shape, 0, 2, True)
    b = kf.Stage(shape, 0, 2, layers, head)
    ka, kb = a.kv(2, 32), b.kv(2, 32)
    toks = torch.from_numpy(synth.tokens(1, 3, 2, shape.vocab)).cuda()
    ya = a.decode(ka, [0, 1], [0, 0], tokens=toks)
    yb = b.decode(kb, [0, 1], [0, 0], tokens=toks)
    assert torch.equal(ya, yb)
    assert torch.equal(a.head_argmax(ya), b.head_argmax(yb))
    for x in (ka, kb, a, b):
        x.close()
