"""Shared test helpers: seeded weights for both sides, error metrics, the argmax rule."""
from __future__ import annotations

import numpy as np

import synth

# Per-row tolerance on hidden states: max_i |gpu_i - oracle_i| / max_i |oracle_i|.
HIDDEN_RTOL = 1e-2


def row_rel_err(gpu: np.ndarray, ref: np.ndarray) -> np.ndarray:
    gpu = np.asarray(gpu, dtype=np.float64).reshape(ref.shape[0], -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(ref.shape[0], -1)
    return np.max(np.abs(gpu - ref), axis=1) / np.max(np.abs(ref), axis=1)


def assert_hidden_close(gpu, ref, rtol: float = HIDDEN_RTOL, what: str = ""):
    err = row_rel_err(gpu, ref)
    assert np.all(np.isfinite(np.asarray(gpu, dtype=np.float64))), f"{what}: non-finite GPU output"
    assert float(err.max()) <= rtol, f"{what}: max row relative error {err.max():.3e} > {rtol}"
    return float(err.max())


def argmax_agrees(t_gpu: int, t_ref: int, logits_ref: np.ndarray, logits_gpu: np.ndarray) -> bool:
    """Greedy-token rule: equal tokens, or a near tie within the logits' own error.

    A differing token is accepted only if the oracle's logit gap between the two
    tokens is at most twice the largest |gpu - oracle| logit difference.
    """
    if t_gpu == t_ref:
        return True
    gap = float(logits_ref[t_ref] - logits_ref[t_gpu])
    tol = 2.0 * float(np.max(np.abs(np.asarray(logits_gpu, np.float64) - logits_ref)))
    return gap <= tol


class SeededModel:
    """bf16 weights of a model shape from the seeded generator, cached per layer."""

    def __init__(self, shape, cfg_id: int, seed: int = 0, cache: bool = True):
        self.shape, self.cfg_id, self.seed = shape, cfg_id, seed
        self._cache = {} if cache else None
        self._head = None

    def layer(self, l: int) -> dict:
        if self._cache is None:
            return synth.layer_weights(self.shape, self.cfg_id, l, self.seed)
        if l not in self._cache:
            self._cache[l] = synth.layer_weights(self.shape, self.cfg_id, l, self.seed)
        return self._cache[l]

    def head(self) -> dict:
        if self._head is None:
            self._head = synth.head_weights(self.shape, self.cfg_id, self.seed)
        return self._head


def f32_to_bf16_bits(a) -> np.ndarray:
    """float values to bf16 bit patterns, rounded to nearest even (finite inputs)."""
    u = np.asarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def plant_lm_rows(head: dict, xhat: np.ndarray, rows, scale: float = 10.0) -> dict:
    """A copy of the head weights whose LM-head rows `rows` all hold scale * xhat / |xhat| (bf16),
    so that their logits on the normalised hidden row xhat are equal and far above the others."""
    h = dict(head)
    lm = np.array(head["lm_head"], copy=True)
    bits = f32_to_bf16_bits(scale * xhat / np.linalg.norm(xhat))
    for r in rows:
        lm[r] = bits
    h["lm_head"] = lm
    return h
