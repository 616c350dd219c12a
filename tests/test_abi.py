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
    from paper_2609_34045_amd import planner, stage
    names = declared_functions()
    assert set(names) == set(stage.EXPORTS) | set(planner.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_abi_version(lib):
    assert lib.kf_abi_version() == 1


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


def test_null_handles_are_rejected(lib):
    n = ctypes.c_int32()
    assert lib.kf_kv_len(None, 0, ctypes.byref(n)) == 1
    assert lib.kf_stage_sync(None) == 1
    assert lib.kf_stage_destroy(None) == 1
    assert lib.kf_kv_destroy(None) == 1
    assert lib.kf_stage_decode(None, None, 1, None, None, None, None, None, 0) == 1
    assert lib.kf_head_argmax(None, 1, None, 0, None, None) == 1
