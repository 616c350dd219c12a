"""Python binding of the stage library (``include/kafila_stage.h``).

Argument marshalling only: every step of the forward pass runs in the HIP
kernels of ``libkafila_stage.so``.  torch provides device memory (tensors are
passed by ``data_ptr()``) and the stream.  The library must have been built
(``python -m paper_2609_34045_amd.build``); importing this module without it
raises, there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# KF_STAGE_LIB selects another build of the same library (e.g. a tuning variant).
LIB_PATH = os.environ.get("KF_STAGE_LIB", os.path.join(HERE, "libkafila_stage.so"))

KF_OK, KF_EINVAL, KF_ENOMEM, KF_ERANGE, KF_ESTATE, KF_EDEVICE, KF_EUNSUPPORTED = range(7)
STATUS_NAMES = {0: "KF_OK", 1: "KF_EINVAL", 2: "KF_ENOMEM", 3: "KF_ERANGE", 4: "KF_ESTATE", 5: "KF_EDEVICE",
                6: "KF_EUNSUPPORTED"}
KF_F32, KF_BF16, KF_F16 = 0, 1, 2
MAX_BATCH = 4

LAYER_KINDS = {"attn_norm": 0, "wq": 1, "wk": 2, "wv": 3, "wo": 4, "mlp_norm": 5, "wg": 6, "wu": 7, "wd": 8}
QK_NORM_KINDS = {"q_norm": 12, "k_norm": 13}  # per-head q / k RMSNorm gains of qk_norm blocks
HEAD_KINDS = {"embed": 9, "final_norm": 10, "lm_head": 11}

EXPORTS = ("kf_abi_version", "kf_last_error", "kf_stage_bytes", "kf_stage_init", "kf_stage_destroy",
           "kf_stage_set_stream", "kf_stage_sync", "kf_kv_create", "kf_kv_destroy", "kf_kv_len", "kf_kv_set_len",
           "kf_kv_write", "kf_kv_read", "kf_stage_decode", "kf_stage_prefill", "kf_head_logits", "kf_head_argmax",
           "kf_stage_profile", "kf_stage_profile_read", "kf_stage_describe", "kf_kv_describe",
           "kf_kv_create_paged", "kf_kv_pages", "kf_stage_set_flags", "kf_stage_get_flags",
           "kf_stage_prefill_noalloc")
PREFILL_SCRATCH_BYTES = 144 << 20  # KF_PREFILL_SCRATCH_BYTES: the no-allocation prefill's workspace limit
KF_STAGE_ORDERED = 1  # batch-1 decode adds the heads' output projections in a fixed order

# kf_kernel_class
KERNEL_CLASSES = ("prep", "qkv", "attn", "oproj", "gateup", "down", "lmhead", "argmax", "pf_norm", "pf_qkv", "pf_rope",
                  "pf_attn", "pf_oproj", "pf_gateup", "pf_down", "pf_store", "qknorm")


class KFError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


class ModelConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float),
                ("qk_norm", ctypes.c_int32)]

    @classmethod
    def of(cls, shape) -> "ModelConfig":
        return cls(shape.n_layers, shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn,
                   shape.vocab, shape.rms_eps, shape.rope_theta, int(getattr(shape, "qk_norm", False)))


class Tensor(ctypes.Structure):
    _fields_ = [("layer", ctypes.c_int32), ("kind", ctypes.c_int32), ("bf16", ctypes.c_void_p), ("numel", ctypes.c_int64)]


class Weights(ctypes.Structure):
    _fields_ = [("tensors", ctypes.POINTER(Tensor)), ("count", ctypes.c_int32)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load the built library once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2609_34045_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, I64, VP = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    I32P, I64P = ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64)
    sig = {
        "kf_abi_version": (I32, []),
        "kf_last_error": (ctypes.c_char_p, []),
        "kf_stage_bytes": (I32, [ctypes.POINTER(ModelConfig), I32, I32, I32, I32, I32, I64P, I64P, I64P]),
        "kf_stage_init": (I32, [ctypes.POINTER(ModelConfig), I32, I32, I32, ctypes.POINTER(Weights), VP,
                                ctypes.POINTER(P)]),
        "kf_stage_destroy": (I32, [P]),
        "kf_stage_set_stream": (I32, [P, VP]),
        "kf_stage_sync": (I32, [P]),
        "kf_kv_create": (I32, [P, I32, I32, ctypes.POINTER(P)]),
        "kf_kv_destroy": (I32, [P]),
        "kf_kv_len": (I32, [P, I32, I32P]),
        "kf_kv_set_len": (I32, [P, I32, I32]),
        "kf_kv_write": (I32, [P, I32, I32, I32, I32, VP, VP, I32]),
        "kf_kv_read": (I32, [P, I32, I32, I32, I32, VP, VP]),
        "kf_stage_decode": (I32, [P, P, I32, I32P, I32P, VP, VP, VP, I32]),
        "kf_stage_prefill": (I32, [P, P, I32, I32, I32, VP, VP, VP, I32]),
        "kf_stage_prefill_noalloc": (I32, [P, P, I32, I32, I32, VP, VP, VP, I32]),
        "kf_head_logits": (I32, [P, I32, VP, I32, VP]),
        "kf_head_argmax": (I32, [P, I32, VP, I32, VP, VP]),
        "kf_stage_profile": (I32, [P, I32]),
        "kf_stage_profile_read": (I32, [P, I32, I64P, ctypes.POINTER(ctypes.c_double)]),
        "kf_stage_describe": (I32, [P, ctypes.POINTER(ModelConfig), I32P, I32P, I32P, ctypes.POINTER(VP), I32P]),
        "kf_kv_describe": (I32, [P, ctypes.POINTER(P), I32P, I32P]),
        "kf_kv_create_paged": (I32, [P, I32, I32, I32, ctypes.POINTER(P)]),
        "kf_kv_pages": (I32, [P, I32P, I32P]),
        "kf_stage_set_flags": (I32, [P, I32]),
        "kf_stage_get_flags": (I32, [P, I32P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, where: str):
    if status != KF_OK:
        raise KFError(status, where, _lib.kf_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _io_dtype(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return KF_F32
    if t.dtype == torch.bfloat16:
        return KF_BF16
    raise TypeError(f"hidden states must be float32 or bfloat16, not {t.dtype}")


def _require_device(t, what: str):
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")


def stage_bytes(shape, lo: int, hi: int, has_head: bool, max_users: int, max_ctx: int):
    """(beta_block, beta_head, resident) bytes of a stage; host-only arithmetic in the library."""
    lib = load_library()
    cfg = ModelConfig.of(shape)
    bb, bh, rs = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(lib.kf_stage_bytes(ctypes.byref(cfg), lo, hi, int(has_head), max_users, max_ctx, ctypes.byref(bb),
                              ctypes.byref(bh), ctypes.byref(rs)), "kf_stage_bytes")
    return bb.value, bh.value, rs.value


class Stage:
    """Layers ``[lo, hi)`` of a model (and the head if ``head_weights`` is given) on the current device.

    ``layer_weights`` maps each held layer index to a dict of bf16 bit arrays
    (numpy uint16, row-major [out, in]) named attn_norm, wq, wk, wv, wo, mlp_norm,
    wg, wu, wd (plus q_norm and k_norm when the shape has qk_norm);
    ``head_weights`` holds embed, final_norm and lm_head.
    """

    def __init__(self, shape, lo: int, hi: int, layer_weights, head_weights=None, stream=None):
        import torch
        lib = load_library()
        self.shape, self.lo, self.hi = shape, lo, hi
        self.has_head = head_weights is not None
        self._cfg = ModelConfig.of(shape)
        keep, items = [], []
        for l in range(lo, hi):
            w = layer_weights[l] if not callable(layer_weights) else layer_weights(l)
            kinds = dict(LAYER_KINDS, **(QK_NORM_KINDS if self._cfg.qk_norm else {}))
            for name, kind in kinds.items():
                a = np.ascontiguousarray(w[name], dtype=np.uint16)
                keep.append(a)
                items.append(Tensor(l, kind, a.ctypes.data, a.size))
        if self.has_head:
            for name, kind in HEAD_KINDS.items():
                a = np.ascontiguousarray(head_weights[name], dtype=np.uint16)
                keep.append(a)
                items.append(Tensor(-1, kind, a.ctypes.data, a.size))
        arr = (Tensor * len(items))(*items)
        ws = Weights(arr, len(items))
        if stream is None:
            stream = torch.cuda.current_stream()
        self.stream = stream
        handle = ctypes.c_void_p()
        _check(lib.kf_stage_init(ctypes.byref(self._cfg), lo, hi, int(self.has_head), ctypes.byref(ws),
                                 ctypes.c_void_p(stream.cuda_stream), ctypes.byref(handle)), "kf_stage_init")
        self.handle = handle
        self._lib = lib

    @classmethod
    def adopt(cls, shape, lo: int, hi: int, has_head: bool, handle, stream) -> "Stage":
        """A Stage object for a kf_stage the library created elsewhere (e.g. kf_shard_stage_init)."""
        self = cls.__new__(cls)
        self.shape, self.lo, self.hi, self.has_head = shape, lo, hi, bool(has_head)
        self._cfg = ModelConfig.of(shape)
        self.stream, self.handle, self._lib = stream, handle, load_library()
        return self

    # -- lifetime
    def close(self):
        if self.handle:
            _check(self._lib.kf_stage_destroy(self.handle), "kf_stage_destroy")
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def set_stream(self, stream):
        _check(self._lib.kf_stage_set_stream(self.handle, ctypes.c_void_p(stream.cuda_stream)), "kf_stage_set_stream")
        self.stream = stream

    def sync(self):
        _check(self._lib.kf_stage_sync(self.handle), "kf_stage_sync")

    def set_flags(self, flags: int):
        """KF_STAGE_* behaviour flags (kf_stage_set_flags)."""
        _check(self._lib.kf_stage_set_flags(self.handle, int(flags)), "kf_stage_set_flags")

    def flags(self) -> int:
        f = ctypes.c_int32()
        _check(self._lib.kf_stage_get_flags(self.handle, ctypes.byref(f)), "kf_stage_get_flags")
        return f.value

    def describe(self) -> dict:
        """The library's own record of the stage (kf_stage_describe)."""
        cfg, lo, hi, head, dev = ModelConfig(), ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        st = ctypes.c_void_p()
        _check(self._lib.kf_stage_describe(self.handle, ctypes.byref(cfg), ctypes.byref(lo), ctypes.byref(hi),
                                           ctypes.byref(head), ctypes.byref(st), ctypes.byref(dev)), "kf_stage_describe")
        return {"config": cfg, "lo": lo.value, "hi": hi.value, "has_head": bool(head.value), "stream": st.value or 0,
                "device": dev.value}

    def profile(self, enable, classes=None):
        """Start (clearing earlier records) or stop per-kernel HIP-event timing.

        ``classes``: names from KERNEL_CLASSES to record (default: all).
        """
        mask = 0
        if enable:
            all_classes = (1 << len(KERNEL_CLASSES)) - 1
            mask = all_classes if classes is None else sum(1 << KERNEL_CLASSES.index(c) for c in classes)
        _check(self._lib.kf_stage_profile(self.handle, mask), "kf_stage_profile")

    def profile_read(self) -> dict:
        """{kernel class: (launches, total ms)} for classes with recorded launches."""
        out = {}
        for i, name in enumerate(KERNEL_CLASSES):
            n, t = ctypes.c_int64(), ctypes.c_double()
            _check(self._lib.kf_stage_profile_read(self.handle, i, ctypes.byref(n), ctypes.byref(t)),
                   "kf_stage_profile_read")
            if n.value:
                out[name] = (n.value, t.value)
        return out

    def kv(self, max_users: int, max_ctx: int, pages: int | None = None) -> "KV":
        """A KV cache; with ``pages`` a paged cache of that many 64-position pages shared by the users."""
        return KV(self, max_users, max_ctx, pages)

    # -- compute
    def decode(self, kv: "KV", users, positions, tokens=None, hidden=None, out=None, keep: bool = False):
        """kf_stage_decode; with ``keep`` (a stage that holds the head) the output rows stay in the stage
        for ``head_logits(None, rows)`` / ``head_argmax(None, rows)`` and None is returned."""
        import torch
        B = len(users)
        u = (ctypes.c_int32 * max(B, 1))(*users)
        p = (ctypes.c_int32 * max(B, 1))(*positions)
        if len(positions) != B:
            raise ValueError("users and positions differ in length")
        src = hidden if hidden is not None else tokens
        if hidden is not None:
            _require_device(hidden, "hidden")
            io = _io_dtype(hidden)
            odt = hidden.dtype
        else:
            io, odt = KF_F32, torch.float32
        if tokens is not None:
            _require_device(tokens, "tokens")
            if tokens.dtype != torch.int32:
                raise TypeError("tokens must be int32")
        if keep:
            if out is not None:
                raise ValueError("keep and out exclude each other")
        elif out is None:
            out = torch.empty((B, self.shape.hidden), dtype=odt, device=src.device if src is not None else "cuda")
        else:
            _require_device(out, "out")
            if _io_dtype(out) != io:
                raise TypeError("out dtype must match the hidden input dtype")
        _check(self._lib.kf_stage_decode(self.handle, kv.handle, B, u, p, _ptr(tokens), _ptr(hidden), _ptr(out), io),
               "kf_stage_decode")
        return out

    def prefill(self, kv: "KV", user: int, pos0: int, tokens=None, hidden=None, out=None, noalloc: bool = False):
        """kf_stage_prefill, or with ``noalloc`` kf_stage_prefill_noalloc (the library allocates nothing;
        pass ``out`` as well to keep the call free of allocations on the Python side too)."""
        import torch
        src = hidden if hidden is not None else tokens
        n = 0 if src is None else int(src.shape[0])
        if hidden is not None:
            _require_device(hidden, "hidden")
            io, odt = _io_dtype(hidden), hidden.dtype
        else:
            io, odt = KF_F32, torch.float32
        if tokens is not None:
            _require_device(tokens, "tokens")
            if tokens.dtype != torch.int32:
                raise TypeError("tokens must be int32")
        if out is None:
            out = torch.empty((max(n, 1), self.shape.hidden), dtype=odt, device=src.device if src is not None else "cuda")
        fn, name = ((self._lib.kf_stage_prefill_noalloc, "kf_stage_prefill_noalloc") if noalloc
                    else (self._lib.kf_stage_prefill, "kf_stage_prefill"))
        _check(fn(self.handle, kv.handle, user, pos0, n, _ptr(tokens), _ptr(hidden), _ptr(out), io), name)
        return out

    def _head_rows(self, hidden, rows):
        """(rows, dtype code, device) of a head call; hidden None means the rows the last decode kept."""
        if hidden is None:
            if rows is None:
                raise ValueError("rows is needed when hidden is None (the rows the last decode kept)")
            return int(rows), KF_F32, "cuda"
        _require_device(hidden, "hidden")
        return int(hidden.shape[0]), _io_dtype(hidden), hidden.device

    def head_logits(self, hidden, out=None, rows: int | None = None):
        import torch
        n, dt, dev = self._head_rows(hidden, rows)
        if out is None:
            out = torch.empty((n, self.shape.vocab), dtype=torch.float32, device=dev)
        _check(self._lib.kf_head_logits(self.handle, n, _ptr(hidden), dt, _ptr(out)), "kf_head_logits")
        return out

    def head_argmax(self, hidden, with_max: bool = False, rows: int | None = None):
        import torch
        n, dt, dev = self._head_rows(hidden, rows)
        tok = torch.empty((n,), dtype=torch.int32, device=dev)
        mx = torch.empty((n,), dtype=torch.float32, device=dev) if with_max else None
        _check(self._lib.kf_head_argmax(self.handle, n, _ptr(hidden), dt, _ptr(tok), _ptr(mx)), "kf_head_argmax")
        return (tok, mx) if with_max else tok


class KV:
    """A KV reservation of ``max_users`` users x ``max_ctx`` positions for every layer of a stage."""

    def __init__(self, stage: Stage, max_users: int, max_ctx: int, pages: int | None = None):
        self.stage, self.max_users, self.max_ctx = stage, max_users, max_ctx
        self._lib = stage._lib
        h = ctypes.c_void_p()
        if pages is None:
            _check(self._lib.kf_kv_create(stage.handle, max_users, max_ctx, ctypes.byref(h)), "kf_kv_create")
        else:
            _check(self._lib.kf_kv_create_paged(stage.handle, max_users, max_ctx, pages, ctypes.byref(h)),
                   "kf_kv_create_paged")
        self.handle = h

    def close(self):
        if self.handle:
            _check(self._lib.kf_kv_destroy(self.handle), "kf_kv_destroy")
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def len(self, user: int) -> int:
        n = ctypes.c_int32()
        _check(self._lib.kf_kv_len(self.handle, user, ctypes.byref(n)), "kf_kv_len")
        return n.value

    def set_len(self, user: int, n: int):
        _check(self._lib.kf_kv_set_len(self.handle, user, n), "kf_kv_set_len")

    def pages(self):
        """(pages in the cache, free pages); a reserved cache reports -1 free pages."""
        t, f = ctypes.c_int32(), ctypes.c_int32()
        _check(self._lib.kf_kv_pages(self.handle, ctypes.byref(t), ctypes.byref(f)), "kf_kv_pages")
        return t.value, f.value

    def describe(self) -> dict:
        owner, mu, mc = ctypes.c_void_p(), ctypes.c_int32(), ctypes.c_int32()
        _check(self._lib.kf_kv_describe(self.handle, ctypes.byref(owner), ctypes.byref(mu), ctypes.byref(mc)),
               "kf_kv_describe")
        return {"stage": owner.value, "max_users": mu.value, "max_ctx": mc.value}

    def write(self, layer: int, user: int, pos0: int, k, v):
        """k, v: device tensors [n, nkv, hd]: float32, float16, bfloat16, or int16 holding bf16 bits."""
        import torch
        _require_device(k, "k")
        _require_device(v, "v")
        if k.dtype != v.dtype:
            raise TypeError("k and v dtypes differ")
        if k.dtype == torch.float32:
            dt = KF_F32
        elif k.dtype == torch.float16:
            dt = KF_F16
        elif k.dtype in (torch.bfloat16, torch.int16):
            dt = KF_BF16
        else:
            raise TypeError("k/v dtype")
        _check(self._lib.kf_kv_write(self.handle, layer, user, pos0, int(k.shape[0]), _ptr(k), _ptr(v), dt),
               "kf_kv_write")

    def read(self, layer: int, user: int, pos0: int, n: int):
        """Returns (k, v) as float32 device tensors [n, nkv, hd] (exact copies of the fp16 cache)."""
        import torch
        s = self.stage.shape
        k = torch.empty((n, s.n_kv_heads, s.head_dim), dtype=torch.float32, device="cuda")
        v = torch.empty_like(k)
        _check(self._lib.kf_kv_read(self.handle, layer, user, pos0, n, _ptr(k), _ptr(v)), "kf_kv_read")
        return k, v
