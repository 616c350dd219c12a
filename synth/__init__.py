"""Seeded synthetic inputs for the stage workloads.

This package is shared by the CPU oracle's tests, the GPU parity tests and
the benchmark.  It generates numbers only (weights, hidden states, token ids,
injected KV) from a counter-based generator written in C (``synth.c``); it
holds none of the stage's arithmetic and imports neither the oracle nor the
HIP package.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB = os.path.join(_HERE, "libsynth.so")


def build(force: bool = True) -> str:
    """Compile ``libsynth.so`` next to its source with gcc."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm", "-lpthread"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        lib.synth_key.restype = ctypes.c_uint64
        lib.synth_key.argtypes = [ctypes.c_uint64] + [ctypes.c_int64] * 4
        lib.synth_normal_bf16.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_double, ctypes.c_double,
                                          ctypes.c_void_p, ctypes.c_int]
        lib.synth_normal_f32.argtypes = lib.synth_normal_bf16.argtypes
        lib.synth_uniform_i32.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int]
        _lib = lib
    return _lib


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def key(seed: int, cfg: int, stream: int, layer: int, kind: int) -> int:
    return int(_load().synth_key(seed, cfg, stream, layer, kind))


def normal_bf16(k: int, shape, mean: float = 0.0, std: float = 1.0) -> np.ndarray:
    """bf16 bit patterns (uint16) of mean + std * N(0,1), round to nearest even."""
    out = np.empty(shape, dtype=np.uint16)
    _load().synth_normal_bf16(k, out.size, mean, std, out.ctypes.data, _threads())
    return out


def normal_f32(k: int, shape, mean: float = 0.0, std: float = 1.0) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    _load().synth_normal_f32(k, out.size, mean, std, out.ctypes.data, _threads())
    return out


def uniform_i32(k: int, shape, modulus: int) -> np.ndarray:
    out = np.empty(shape, dtype=np.int32)
    _load().synth_uniform_i32(k, out.size, modulus, out.ctypes.data, _threads())
    return out


# Streams (second coordinate after the config id).
STREAM_WEIGHTS, STREAM_PREFILL_HIDDEN, STREAM_DECODE_HIDDEN, STREAM_TOKENS, STREAM_KV = 0, 1, 2, 3, 4

# Tensor kinds (generator coordinate); names follow the decoder-layer notation.
LAYER_KINDS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wg", "wu", "wd")
HEAD_KINDS = ("embed", "final_norm", "lm_head")
QK_NORM_KINDS = ("q_norm", "k_norm")  # per-head RMSNorm gains of q and k (Qwen3-style blocks)
KIND_ID = {n: i for i, n in enumerate(LAYER_KINDS + HEAD_KINDS + QK_NORM_KINDS)}
GAIN_KINDS = ("attn_norm", "mlp_norm", "final_norm", "q_norm", "k_norm")


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rms_eps: float = 1e-5
    rope_theta: float = 1e4
    qk_norm: bool = False  # RMSNorm over each q and k head (gains [head_dim]) before RoPE, as in Qwen3

    def layer_kinds(self):
        return LAYER_KINDS + (QK_NORM_KINDS if self.qk_norm else ())

    def tensor_shape(self, kind: str):
        H, hd, F = self.hidden, self.head_dim, self.ffn
        return {
            "attn_norm": (H,), "mlp_norm": (H,), "final_norm": (H,), "q_norm": (hd,), "k_norm": (hd,),
            "wq": (self.n_q_heads * hd, H), "wk": (self.n_kv_heads * hd, H), "wv": (self.n_kv_heads * hd, H),
            "wo": (H, self.n_q_heads * hd), "wg": (F, H), "wu": (F, H), "wd": (H, F),
            "embed": (self.vocab, H), "lm_head": (self.vocab, H),
        }[kind]

    def block_bytes(self) -> int:
        return sum(2 * int(np.prod(self.tensor_shape(k))) for k in self.layer_kinds())


@dataclass(frozen=True)
class Workload:
    """One stage workload: a layer range of a model shape, optional head, and its inputs."""
    cfg_id: int
    name: str
    shape: ModelShape
    layer_lo: int
    layer_hi: int
    has_head: bool
    batch: int
    contexts: tuple          # per-row context length already in the cache when decode starts
    decode_steps: int
    prefill_chunk: int = 0   # tokens per prefill chunk (0 = no prefill in the workload)
    seed: int = 0
    notes: str = ""
    extra: dict = field(default_factory=dict)


SHAPE_TINY = ModelShape(2, 512, 8, 2, 64, 1408, 1000, 1e-5, 1e4)
SHAPE_8B = ModelShape(32, 4096, 32, 8, 128, 14336, 128256, 1e-5, 5e5)
SHAPE_32B = ModelShape(64, 5120, 40, 8, 128, 27648, 152064, 1e-5, 1e6)
SHAPE_70B = ModelShape(80, 8192, 64, 8, 128, 28672, 128256, 1e-5, 5e5)
# Qwen3-style blocks (per-head q/k RMSNorm; query width nq*hd may differ from H), the
# family the paper serves.  The tiny shape keeps nq*hd (512) != H (384) on purpose.
SHAPE_QWEN3_TINY = ModelShape(2, 384, 8, 2, 64, 1024, 1000, 1e-6, 1e6, qk_norm=True)
SHAPE_QWEN3_8B = ModelShape(36, 4096, 32, 8, 128, 12288, 151936, 1e-6, 1e6, qk_norm=True)
SHAPE_QWEN3_32B = ModelShape(64, 5120, 64, 8, 128, 25600, 151936, 1e-6, 1e6, qk_norm=True)

WORKLOADS = {
    "tiny": Workload(1, "tiny", SHAPE_TINY, 0, 2, False, 1, (128,), 16, prefill_chunk=128,
                     notes="KV built by prefill of 128 N(0,1) hidden states, then 16 decode steps"),
    "8b_mid": Workload(2, "8b_mid", SHAPE_8B, 8, 16, False, 1, (2048,), 64,
                       notes="layers [8,16) of 32, KV injected for [0,2048)"),
    "8b_head": Workload(3, "8b_head", SHAPE_8B, 0, 4, True, 4, (256, 1024, 2048, 4096), 32,
                        notes="embedding + layers [0,4) + final norm + LM head, ragged batch 4"),
    "32b_b1": Workload(4, "32b_b1", SHAPE_32B, 16, 32, False, 1, (4096,), 64,
                       notes="layers [16,32) of 64, KV injected for [0,4096)"),
    "32b_b4": Workload(4, "32b_b4", SHAPE_32B, 16, 32, False, 4, (4096, 4096, 4096, 4096), 64,
                       notes="layers [16,32) of 64, four users at context 4096"),
    "70b": Workload(5, "70b", SHAPE_70B, 40, 50, False, 1, (4096,), 64, prefill_chunk=512,
                    notes="layers [40,50) of 80; prefill chunks of 512 into 4096, then 64 decode steps"),
    # long declared context: the KV reads (134 MB per layer) are a quarter of the step
    "8b_mid_32k": Workload(8, "8b_mid_32k", SHAPE_8B, 8, 16, False, 1, (32768,), 64,
                           notes="layers [8,16) of 32, KV injected for [0,32768)"),
    "8b_b4_32k": Workload(9, "8b_b4_32k", SHAPE_8B, 8, 16, False, 4, (32768, 16384, 8192, 1024), 32,
                          notes="layers [8,16) of 32, four users up to 32768 keys"),
    # Qwen3-style blocks (the paper's served family), same roles as 8b_mid / 32b_b1
    "qwen3_8b_mid": Workload(6, "qwen3_8b_mid", SHAPE_QWEN3_8B, 9, 18, False, 1, (2048,), 64,
                             notes="layers [9,18) of 36, KV injected for [0,2048)"),
    "qwen3_32b_b1": Workload(7, "qwen3_32b_b1", SHAPE_QWEN3_32B, 16, 32, False, 1, (4096,), 64, prefill_chunk=512,
                             notes="layers [16,32) of 64, KV injected for [0,4096)"),
}


def layer_weights(shape: ModelShape, cfg_id: int, layer: int, seed: int = 0) -> dict:
    """bf16 bit patterns of one decoder layer's tensors, row-major [out, in].

    Projections are N(0, 0.02^2); RMSNorm gains are 1 + N(0, 0.02^2).  Keys use the
    global layer index, so a layer has the same weights in every stage that holds it.
    """
    out = {}
    for kind in shape.layer_kinds():
        k = key(seed, cfg_id, STREAM_WEIGHTS, layer, KIND_ID[kind])
        mean = 1.0 if kind in GAIN_KINDS else 0.0
        out[kind] = normal_bf16(k, shape.tensor_shape(kind), mean, 0.02)
    return out


def head_weights(shape: ModelShape, cfg_id: int, seed: int = 0) -> dict:
    out = {}
    for kind in HEAD_KINDS:
        k = key(seed, cfg_id, STREAM_WEIGHTS, -1, KIND_ID[kind])
        mean = 1.0 if kind in GAIN_KINDS else 0.0
        out[kind] = normal_bf16(k, shape.tensor_shape(kind), mean, 0.02)
    return out


def hidden_states(cfg_id: int, stream: int, step: int, rows: int, hidden: int, seed: int = 0) -> np.ndarray:
    """fp32 N(0,1) hidden inputs, [rows, hidden]; ``step`` indexes the call."""
    return normal_f32(key(seed, cfg_id, stream, step, 0), (rows, hidden), 0.0, 1.0)


def tokens(cfg_id: int, step: int, rows: int, vocab: int, seed: int = 0) -> np.ndarray:
    return uniform_i32(key(seed, cfg_id, STREAM_TOKENS, step, 0), (rows,), vocab)


def injected_kv(shape: ModelShape, cfg_id: int, layer: int, user: int, n: int, seed: int = 0):
    """bf16 K and V for positions [0, n) of one user, [n, n_kv_heads, head_dim] each.

    Scale 0.02*sqrt(hidden): a unit-RMS hidden state projected by N(0, 0.02^2) weights.
    """
    std = 0.02 * float(np.sqrt(shape.hidden))
    shp = (n, shape.n_kv_heads, shape.head_dim)
    k = normal_bf16(key(seed, cfg_id, STREAM_KV, layer, 2 * user), shp, 0.0, std)
    v = normal_bf16(key(seed, cfg_id, STREAM_KV, layer, 2 * user + 1), shp, 0.0, std)
    return k, v


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32 (a 16-bit shift)."""
    return (bits.astype(np.uint32) << 16).view(np.float32)
