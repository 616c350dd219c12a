"""Python binding of the ring (``include/kafila_ring.h``): argument marshalling only.

Stages chained head first, each on its own stream, serve several request groups
at once (Section III's ring; Section VII-C's concurrent users).  Every step runs in
``libkafila_stage.so``: the stages' kernels, and the ring's ordering of their work
across streams.
"""
from __future__ import annotations

import ctypes

from . import stage as _stage

EXPORTS = ("kf_ring_create", "kf_ring_destroy", "kf_ring_prefill", "kf_ring_generate", "kf_ring_sync")

_configured = None


def _lib():
    global _configured
    lib = _stage.load_library()
    if _configured is lib:
        return lib
    I32, P, VP = ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p
    I32P = ctypes.POINTER(I32)
    sig = {
        "kf_ring_create": (I32, [I32, ctypes.POINTER(P), ctypes.POINTER(P), I32, I32, I32, ctypes.POINTER(P)]),
        "kf_ring_destroy": (I32, [P]),
        "kf_ring_prefill": (I32, [P, I32, I32, VP, VP]),
        "kf_ring_generate": (I32, [P, I32, I32P, I32P, VP, I32, VP, VP]),
        "kf_ring_sync": (I32, [P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _configured = lib
    return lib


class Ring:
    """``stages`` (head stage first, consecutive layer ranges) with their ``kvs``, on one device.

    Give each stage its own stream for the members to overlap.  ``io`` is the
    hand-off element type (torch.float32 or torch.bfloat16).
    """

    def __init__(self, stages, kvs, max_groups: int = 4, max_prefill: int = 512, io=None):
        import torch
        io = torch.float32 if io is None else io
        if io not in (torch.float32, torch.bfloat16):
            raise TypeError("the hand-off dtype is float32 or bfloat16")
        if len(stages) != len(kvs):
            raise ValueError("one KV cache per stage")
        lib = _lib()
        self.stages, self.kvs = list(stages), list(kvs)
        self.max_groups, self.max_prefill = max_groups, max_prefill
        m = len(stages)
        st = (ctypes.c_void_p * max(m, 1))(*[s.handle for s in stages])
        kv = (ctypes.c_void_p * max(m, 1))(*[k.handle for k in kvs])
        h = ctypes.c_void_p()
        dtype = _stage.KF_F32 if io == torch.float32 else _stage.KF_BF16
        _stage._check(lib.kf_ring_create(m, st, kv, max_groups, max_prefill, dtype, ctypes.byref(h)), "kf_ring_create")
        self.handle, self._lib, self.io = h, lib, io

    def close(self):
        if self.handle:
            _stage._check(self._lib.kf_ring_destroy(self.handle), "kf_ring_destroy")
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def sync(self):
        _stage._check(self._lib.kf_ring_sync(self.handle), "kf_ring_sync")

    def prefill(self, user: int, tokens):
        """Prompt chunk ``tokens`` (device int32 [n], ready) through every member; the next token, int32 [1]."""
        import torch
        _stage._require_device(tokens, "tokens")
        if tokens.dtype != torch.int32:
            raise TypeError("tokens must be int32")
        nxt = torch.empty(1, dtype=torch.int32, device=tokens.device)
        _stage._check(self._lib.kf_ring_prefill(self.handle, user, tokens.numel(), _stage._ptr(tokens), _stage._ptr(nxt)),
                      "kf_ring_prefill")
        self._in_use(tokens, nxt)
        return nxt

    def generate(self, groups, tokens_in, steps: int, out=None, hidden_out=None):
        """``groups``: lists of user ids; ``tokens_in``: device int32 [U] in the same order (ready).

        Returns device int32 [steps, U]: the tokens sampled at each step.  ``hidden_out`` (optional device
        tensor [steps, U, H] of the ring's io dtype) receives the hidden rows each token was sampled from.
        """
        import torch
        sizes = [len(g) for g in groups]
        users = [u for g in groups for u in g]
        U = len(users)
        _stage._require_device(tokens_in, "tokens_in")
        if tokens_in.dtype != torch.int32 or tokens_in.numel() != U:
            raise ValueError(f"tokens_in must be int32 with {U} entries")
        if out is None:
            out = torch.empty((max(steps, 0), U), dtype=torch.int32, device=tokens_in.device)
        gs = (ctypes.c_int32 * max(len(sizes), 1))(*sizes)
        us = (ctypes.c_int32 * max(U, 1))(*users)
        if hidden_out is not None:
            _stage._require_device(hidden_out, "hidden_out")
            if tuple(hidden_out.shape) != (steps, U, self.stages[0].shape.hidden) or hidden_out.dtype != self.io:
                raise ValueError("hidden_out must be [steps, U, H] of the ring's hand-off dtype")
        _stage._check(self._lib.kf_ring_generate(self.handle, len(sizes), gs, us, _stage._ptr(tokens_in), steps,
                                                 _stage._ptr(out), _stage._ptr(hidden_out)), "kf_ring_generate")
        self._in_use(tokens_in, out, *([hidden_out] if hidden_out is not None else []))
        return out

    def _in_use(self, *tensors):
        # The ring reads and writes these on the head stage's stream (every other
        # member's work is ordered before that stream's last work): keep torch's
        # allocator from reusing their memory before that stream gets there.
        s = self.stages[0].stream
        for t in tensors:
            t.record_stream(s)
