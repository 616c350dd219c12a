"""The C-ABI library: it loads, exports every declared entry point, and its host-only checks.

No compute call is made here (no GPU in this environment): only calls that
return before touching a device.
"""
import ctypes
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in sorted(os.listdir(os.path.join(ROOT, "include")))
           if h.endswith(".h")]


@pytest.fixture(scope="module")
def lib():
    from paper_2609_34045_amd import stage
    return stage.load_library()


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(kf_[a-z_]+)\s*\(", text))
    return sorted(names)


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("kf_stage_init", "kf_stage_prefill", "kf_stage_decode", "kf_head_logits", "kf_head_argmax",
              "kf_kv_create", "kf_stage_bytes", "kf_last_error", "kf_partition", "kf_plan", "kf_probe_bandwidth"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    from paper_2609_34045_amd import planner, ring, shard, stage
    names = declared_functions()
    assert set(names) == set(stage.EXPORTS) | set(planner.EXPORTS) | set(ring.EXPORTS) | set(shard.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_abi_version(lib):
    assert lib.kf_abi_version() == 5


def _comment_before(text: str, name: str) -> str:
    """The block comment that ends closest above the declaration of `name`."""
    at = re.search(r"\bkf_status\s+" + name + r"\s*\(", text).start()
    return text[:at][text[:at].rfind("/*"):]


@pytest.mark.parametrize("name", ["kf_stage_init", "kf_stage_decode", "kf_stage_prefill", "kf_head_logits",
                                  "kf_head_argmax", "kf_kv_create", "kf_stage_bytes"])
def test_boundary_declarations_cite_the_paper(name):
    """Each call of the stage boundary names the passage of the paper that defines it."""
    text = open(os.path.join(ROOT, "include", "kafila_stage.h")).read()
    assert re.search(r"Section [IVX]+(-[A-D])?", _comment_before(text, name)), name


def test_stage_bytes_matches_shape_arithmetic():
    from paper_2609_34045_amd import stage
    s = synth.SHAPE_8B
    bb, bh, res = stage.stage_bytes(s, 8, 16, False, 1, 2112)
    assert bb == 436_224_000 == s.block_bytes()
    assert bh == 0
    bb, bh, res_h = stage.stage_bytes(s, 0, 4, True, 4, 4160)
    assert bh == 2 * (2 * 128256 * 4096 + 4096)
    kv = 2 * 4 * 4 * 8 * 4160 * 128 * 2
    assert res_h >= 4 * bb + bh + kv
    assert res_h < 4 * bb + bh + kv + 64 * 2**20  # workspaces stay small
    assert stage.stage_bytes(synth.SHAPE_70B, 40, 50, False, 1, 4160)[0] == 1_711_308_800
    assert stage.stage_bytes(synth.SHAPE_32B, 16, 32, False, 1, 4160)[0] == 975_196_160


def _cfg(**kw):
    from paper_2609_34045_amd import stage
    base = dict(n_layers=4, hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=64, ffn=1408, vocab=100,
                rms_eps=1e-5, rope_theta=1e4)
    base.update(kw)
    return stage.ModelConfig(**base)


@pytest.mark.parametrize("kw,lo,hi,code", [
    (dict(), 2, 2, 1),            # empty range
    (dict(), -1, 2, 1),
    (dict(), 0, 5, 1),            # beyond n_layers
    (dict(head_dim=96), 0, 1, 6),
    (dict(n_q_heads=6, n_kv_heads=4), 0, 1, 1),
    (dict(n_q_heads=32, n_kv_heads=2), 0, 1, 6),   # 16 query heads per KV head
    (dict(hidden=520), 0, 1, 6),
])
def test_init_rejects_before_touching_the_device(lib, kw, lo, hi, code):
    from paper_2609_34045_amd import stage
    cfg = _cfg(**kw)
    ws = stage.Weights(None, 0)
    out = ctypes.c_void_p(123)
    st = lib.kf_stage_init(ctypes.byref(cfg), lo, hi, 0, ctypes.byref(ws), None, ctypes.byref(out))
    assert st == code, lib.kf_last_error()
    assert out.value is None
    assert lib.kf_last_error()


def test_init_reports_missing_and_misshapen_tensors(lib):
    from paper_2609_34045_amd import stage
    import numpy as np
    cfg = _cfg()
    a = np.zeros(512, dtype=np.uint16)
    t = (stage.Tensor * 1)(stage.Tensor(0, 0, a.ctypes.data, 511))
    out = ctypes.c_void_p()
    st = lib.kf_stage_init(ctypes.byref(cfg), 0, 1, 0, ctypes.byref(stage.Weights(t, 1)), None, ctypes.byref(out))
    assert st == 1 and b"numel" in lib.kf_last_error()
    t = (stage.Tensor * 1)(stage.Tensor(0, 0, a.ctypes.data, 512))
    st = lib.kf_stage_init(ctypes.byref(cfg), 0, 1, 0, ctypes.byref(stage.Weights(t, 1)), None, ctypes.byref(out))
    assert st == 1 and b"missing" in lib.kf_last_error()
    t = (stage.Tensor * 1)(stage.Tensor(-1, 9, a.ctypes.data, 100 * 512))
    st = lib.kf_stage_init(ctypes.byref(cfg), 0, 1, 0, ctypes.byref(stage.Weights(t, 1)), None, ctypes.byref(out))
    assert st == 1 and b"head" in lib.kf_last_error()


def _layer_tensors(stage, shape, layer, keep):
    import numpy as np
    items = []
    kinds = dict(stage.LAYER_KINDS, **(stage.QK_NORM_KINDS if shape.qk_norm else {}))
    for name, kind in kinds.items():
        a = np.zeros(int(np.prod(shape.tensor_shape(name))), dtype=np.uint16)
        keep.append(a)
        items.append(stage.Tensor(layer, kind, a.ctypes.data, a.size))
    return items


def test_qk_norm_tensors_are_checked_before_touching_the_device(lib):
    """q/k norm gains are required exactly when the config sets qk_norm (host-side checks only)."""
    from paper_2609_34045_amd import stage
    import numpy as np
    shape = synth.SHAPE_QWEN3_TINY
    keep = []
    full = _layer_tensors(stage, shape, 0, keep)
    out = ctypes.c_void_p()
    cfg = stage.ModelConfig.of(shape)
    # a Qwen3-style config without its two gains: missing tensor (kind 12)
    no_gains = [t for t in full if t.kind < 12]
    st = lib.kf_stage_init(ctypes.byref(cfg), 0, 1, 0, ctypes.byref(stage.Weights((stage.Tensor * 9)(*no_gains), 9)),
                           None, ctypes.byref(out))
    assert st == 1 and b"missing tensor: layer 0 kind 12" in lib.kf_last_error()
    # gains given to a config without qk_norm
    plain = stage.ModelConfig.of(shape)
    plain.qk_norm = 0
    st = lib.kf_stage_init(ctypes.byref(plain), 0, 1, 0, ctypes.byref(stage.Weights((stage.Tensor * 11)(*full), 11)),
                           None, ctypes.byref(out))
    assert st == 1 and b"without qk_norm" in lib.kf_last_error()
    # a gain of the wrong length
    bad = list(full)
    a = np.zeros(shape.head_dim + 1, dtype=np.uint16)
    bad[-1] = stage.Tensor(0, 13, a.ctypes.data, a.size)
    st = lib.kf_stage_init(ctypes.byref(cfg), 0, 1, 0, ctypes.byref(stage.Weights((stage.Tensor * 11)(*bad), 11)),
                           None, ctypes.byref(out))
    assert st == 1 and b"numel" in lib.kf_last_error()
    # qk_norm must be 0 or 1
    odd = stage.ModelConfig.of(shape)
    odd.qk_norm = 2
    st = lib.kf_stage_init(ctypes.byref(odd), 0, 1, 0, ctypes.byref(stage.Weights(None, 0)), None, ctypes.byref(out))
    assert st == 1 and b"qk_norm" in lib.kf_last_error()


def test_qk_norm_block_bytes_include_the_gains():
    from paper_2609_34045_amd import stage
    for shape in (synth.SHAPE_QWEN3_TINY, synth.SHAPE_QWEN3_8B, synth.SHAPE_QWEN3_32B):
        bb = stage.stage_bytes(shape, 0, 1, False, 1, 64)[0]
        assert bb == shape.block_bytes()
        plain = synth.ModelShape(**{**shape.__dict__, "qk_norm": False})
        assert bb == plain.block_bytes() + 2 * 2 * shape.head_dim
    # Qwen3-8B-shaped block: q 4096x4096, k and v 1024x4096, o 4096x4096, three 12288x4096, gains
    assert synth.SHAPE_QWEN3_8B.block_bytes() == 2 * (2 * 4096 * 4096 + 2 * 1024 * 4096 + 3 * 12288 * 4096 + 2 * 4096 + 2 * 128)


def test_null_handles_are_rejected(lib):
    n = ctypes.c_int32()
    assert lib.kf_kv_len(None, 0, ctypes.byref(n)) == 1
    assert lib.kf_stage_sync(None) == 1
    assert lib.kf_stage_destroy(None) == 1
    assert lib.kf_kv_destroy(None) == 1
    assert lib.kf_stage_decode(None, None, 1, None, None, None, None, None, 0) == 1
    assert lib.kf_head_argmax(None, 1, None, 0, None, None) == 1


def test_ring_rejects_before_touching_the_device(lib):
    """Ring argument checks that return before any stage or device is touched."""
    from paper_2609_34045_amd import ring
    r = ring._lib()
    out = ctypes.c_void_p(123)
    P = ctypes.c_void_p
    assert r.kf_ring_create(0, (P * 1)(), (P * 1)(), 1, 1, 0, ctypes.byref(out)) == 1
    assert out.value is None and b"n_members" in lib.kf_last_error()
    assert r.kf_ring_create(1, None, None, 1, 1, 0, ctypes.byref(out)) == 1
    assert r.kf_ring_create(1, (P * 1)(), (P * 1)(), 0, 1, 0, ctypes.byref(out)) == 1
    assert b"max_groups" in lib.kf_last_error()
    assert r.kf_ring_create(1, (P * 1)(), (P * 1)(), 65, 1, 0, ctypes.byref(out)) == 1
    assert r.kf_ring_create(1, (P * 1)(), (P * 1)(), 4, 0, 0, ctypes.byref(out)) == 1
    assert b"max_prefill" in lib.kf_last_error()
    assert r.kf_ring_create(1, (P * 1)(), (P * 1)(), 4, 8, 2, ctypes.byref(out)) == 1  # fp16 hand-off
    assert r.kf_ring_create(1, (P * 1)(), (P * 1)(), 4, 8, 0, ctypes.byref(out)) == 1  # NULL stage
    assert b"stages[0]" in lib.kf_last_error()
    assert r.kf_ring_create(1, (P * 1)(), (P * 1)(), 4, 8, 0, None) == 1
    one = (ctypes.c_int32 * 1)(1)
    assert r.kf_ring_generate(None, 1, one, one, P(8), 1, P(8), None) == 1
    assert r.kf_ring_prefill(None, 0, 1, P(8), P(8)) == 1
    assert r.kf_ring_sync(None) == 1
    assert r.kf_ring_destroy(None) == 1
    assert lib.kf_stage_describe(None, None, None, None, None, None, None) == 1
    assert lib.kf_kv_describe(None, None, None, None) == 1


def test_paged_kv_rejects_before_touching_the_device(lib):
    out = ctypes.c_void_p(123)
    assert lib.kf_kv_create_paged(None, 1, 64, 4, ctypes.byref(out)) == 1
    assert out.value is None
    assert lib.kf_kv_create_paged(ctypes.c_void_p(8), 1, 64, 0, ctypes.byref(out)) == 1  # no pages
    assert b"n_pages" in lib.kf_last_error() and out.value is None
    assert lib.kf_kv_pages(None, None, None) == 1


def test_kernel_classes_match_the_header():
    from paper_2609_34045_amd import stage
    text = open(os.path.join(ROOT, "include", "kafila_stage.h")).read()
    count = int(re.search(r"KF_K_COUNT\s*=\s*(\d+)", text).group(1))
    assert len(stage.KERNEL_CLASSES) == count
    assert int(re.search(r"#define KF_K_ALL (0x[0-9a-fA-F]+)", text).group(1), 16) == (1 << count) - 1
    names = re.findall(r"KF_K_([A-Z_]+)\s*=\s*(\d+),", text)
    for name, idx in names:
        assert stage.KERNEL_CLASSES[int(idx)] == name.lower(), name
