"""Python binding of the safetensors shard loader (``include/kafila_shard.h``).

Argument marshalling only: header parsing, the stage's tensor list and the
byte-range reads run in ``libkafila_stage.so``.
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import stage as _st

EXPORTS = ("kf_shard_open", "kf_shard_close", "kf_shard_plan", "kf_shard_fetch", "kf_shard_stage_init",
           "kf_shard_release", "kf_shard_stats")
KF_SHARD_TIED_EMBEDDINGS = 1


def _lib():
    lib = _st.load_library()
    if not getattr(lib, "_kf_shard_sigs", False):
        P, I32, I64P = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64)
        cfgp = ctypes.POINTER(_st.ModelConfig)
        sig = {
            "kf_shard_open": (I32, [ctypes.POINTER(ctypes.c_char_p), I32, ctypes.POINTER(P)]),
            "kf_shard_close": (I32, [P]),
            "kf_shard_plan": (I32, [P, cfgp, I32, I32, I32, I32, I64P, I64P, ctypes.POINTER(ctypes.c_int32)]),
            "kf_shard_fetch": (I32, [P, cfgp, I32, I32, I32, I32, ctypes.POINTER(_st.Weights)]),
            "kf_shard_stage_init": (I32, [P, cfgp, I32, I32, I32, I32, P, ctypes.POINTER(P)]),
            "kf_shard_release": (I32, [P, I32, I32, I32]),
            "kf_shard_stats": (I32, [P, I64P, I64P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        lib._kf_shard_sigs = True
    return lib


class Checkpoint:
    """A checkpoint in one or more safetensors files; only the headers are read when it is opened."""

    def __init__(self, paths):
        lib = _lib()
        if isinstance(paths, str):
            paths = [paths]
        arr = (ctypes.c_char_p * len(paths))(*[p.encode() for p in paths])
        h = ctypes.c_void_p()
        _st._check(lib.kf_shard_open(arr, len(paths), ctypes.byref(h)), "kf_shard_open")
        self.handle, self._lib = h, lib

    def close(self):
        if self.handle:
            _st._check(self._lib.kf_shard_close(self.handle), "kf_shard_close")
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def plan(self, shape, lo: int, hi: int, has_head: bool, tied: bool = False):
        """(stage bytes, bytes a fetch would read now, tensors) of a stage of layers [lo, hi)."""
        cfg = _st.ModelConfig.of(shape)
        a, b, n = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32()
        _st._check(self._lib.kf_shard_plan(self.handle, ctypes.byref(cfg), lo, hi, int(has_head),
                                           KF_SHARD_TIED_EMBEDDINGS if tied else 0, ctypes.byref(a), ctypes.byref(b),
                                           ctypes.byref(n)), "kf_shard_plan")
        return a.value, b.value, n.value

    def fetch(self, shape, lo: int, hi: int, has_head: bool, tied: bool = False):
        """Read what the stage lacks; returns [(layer, kind, bf16 bits as a numpy copy)] for every stage tensor."""
        cfg = _st.ModelConfig.of(shape)
        w = _st.Weights()
        _st._check(self._lib.kf_shard_fetch(self.handle, ctypes.byref(cfg), lo, hi, int(has_head),
                                            KF_SHARD_TIED_EMBEDDINGS if tied else 0, ctypes.byref(w)), "kf_shard_fetch")
        out = []
        for i in range(w.count):
            t = w.tensors[i]
            buf = (ctypes.c_uint16 * t.numel).from_address(t.bf16)
            out.append((t.layer, t.kind, np.frombuffer(buf, dtype=np.uint16).copy()))
        return out

    def stage(self, shape, lo: int, hi: int, has_head: bool, tied: bool = False, stream=None) -> "_st.Stage":
        """kf_shard_stage_init: fetch, then create the stage on the current device."""
        import torch
        cfg = _st.ModelConfig.of(shape)
        if stream is None:
            stream = torch.cuda.current_stream()
        h = ctypes.c_void_p()
        _st._check(self._lib.kf_shard_stage_init(self.handle, ctypes.byref(cfg), lo, hi, int(has_head),
                                                 KF_SHARD_TIED_EMBEDDINGS if tied else 0,
                                                 ctypes.c_void_p(stream.cuda_stream), ctypes.byref(h)),
                   "kf_shard_stage_init")
        return _st.Stage.adopt(shape, lo, hi, has_head, h, stream)

    def release(self, lo: int = 0, hi: int = 0, has_head: bool = False):
        _st._check(self._lib.kf_shard_release(self.handle, lo, hi, int(has_head)), "kf_shard_release")

    def stats(self):
        """(tensor bytes read from the files so far, bytes held now)."""
        r, h = ctypes.c_int64(), ctypes.c_int64()
        _st._check(self._lib.kf_shard_stats(self.handle, ctypes.byref(r), ctypes.byref(h)), "kf_shard_stats")
        return r.value, h.value
