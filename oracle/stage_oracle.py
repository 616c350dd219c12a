"""Plain float64 CPU oracle of one pipeline stage (test infrastructure only).

Kafila divides a model's contiguous chain of transformer blocks among the
members of a ring; a member's *stage* maps the hidden state of each token
through its block range, and the member holding the *head* also embeds the
token before its blocks and unembeds and samples after the model's last block
(paper Section III, "The Kafila Session Model", and Fig. 1; the per-stage cost
of eq. (2) in Section V-A counts one block's bytes per assigned block plus the
head's bytes).  The paper does not define the block itself: it serves Qwen3
models decoded greedily at a fixed seed (Section VI-A).  This oracle therefore
writes out the textbook pre-norm decoder layer (RMSNorm, grouped-query
attention with rotary position embedding, SwiGLU MLP, no biases) and a greedy
head, with every reading of the unstated details listed here:

* RMSNorm: ``x / sqrt(mean(x^2) + eps) * g``; eps inside the square root, gain
  applied after normalisation.
* RoPE: rotate-half pairs ``(i, i + hd/2)`` at angle ``p * theta^(-2i/hd)``,
  full head dimension rotated, angles in float64.
* GQA: query head ``h`` reads KV head ``h // (n_q / n_kv)`` (contiguous groups).
* Causality: a token at position ``p`` attends keys ``0..p`` inclusive; its own
  key and value are appended to the cache before attention.  The position is
  also the cache slot (append-only).
* Head: untied embedding and output projection; greedy argmax, lowest index on
  ties.
* Qwen3-style blocks (the family the paper serves) add an RMSNorm over each q
  and each k head vector (gains of length head_dim, the layer's eps) after the
  projections and before RoPE; their query width nq * head_dim may differ from
  the hidden size.  Pinned against transformers' Qwen3 model in float64.
* Rows of a batch are independent users with their own cache and position.

Everything is float64.  Weights arrive as bf16 bit patterns and are widened
exactly.  There is no blocking, fusion or reordering beyond the definition.
Parity pins: each function is checked in ``tests/test_oracle_pins.py`` against
closed forms, invariants, library routines (torch CPU, transformers' Llama
layer, and its Qwen3 model for the q/k-norm variant) and a separately
written scalar brute force.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

F64 = np.float64


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns (uint16) as float64 (row blocks widened on threads)."""
    bits = np.asarray(bits)
    if bits.dtype != np.uint16:
        raise TypeError("bf16 tensors are passed as uint16 bit patterns")
    if bits.size < (1 << 22) or bits.ndim == 0:
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(F64)
    out = np.empty(bits.shape, dtype=F64)
    flat_in, flat_out = bits.reshape(-1), out.reshape(-1)
    step = 1 << 21

    def one(i):
        out_blk = flat_out[i:i + step]
        out_blk[:] = (flat_in[i:i + step].astype(np.uint32) << 16).view(np.float32)

    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(one, range(0, flat_in.size, step)))
    return out


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * g."""
    x = np.asarray(x, dtype=F64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, dtype=F64)


def rope(u: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half RoPE.

    u: [..., n_heads, hd]; pos: integer positions broadcastable to u.shape[:-2].
    For i < hd/2 with w_i = theta^(-2i/hd) and phi = pos * w_i:
      out_i        = u_i cos(phi) - u_{i+hd/2} sin(phi)
      out_{i+hd/2} = u_{i+hd/2} cos(phi) + u_i sin(phi)
    """
    u = np.asarray(u, dtype=F64)
    hd = u.shape[-1]
    half = hd // 2
    i = np.arange(half, dtype=F64)
    omega = np.power(F64(theta), -2.0 * i / hd)
    phi = np.asarray(pos, dtype=F64)[..., None, None] * omega  # [..., 1, half]
    c, s = np.cos(phi), np.sin(phi)
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def softmax(s: np.ndarray) -> np.ndarray:
    """Softmax over the last axis with max subtraction."""
    s = np.asarray(s, dtype=F64)
    e = np.exp(s - np.max(s, axis=-1, keepdims=True))
    return e / np.sum(e, axis=-1, keepdims=True)


def silu(u: np.ndarray) -> np.ndarray:
    return u / (1.0 + np.exp(-u))


def mlp_swiglu(z: np.ndarray, wg: np.ndarray, wu: np.ndarray, wd: np.ndarray) -> np.ndarray:
    """down( silu(z Wg^T) * (z Wu^T) ); weights row-major [out, in]."""
    return (silu(z @ wg.T) * (z @ wu.T)) @ wd.T


def attention_rows(q: np.ndarray, keys: list, values: list, n_kv_heads: int) -> np.ndarray:
    """GQA attention for a list of query rows.

    q: [N, n_q, hd]; keys[n], values[n]: [len_n, n_kv, hd] (the keys row n may see).
    Query head h reads KV head h // (n_q / n_kv); the query heads of one KV head
    are scored together.  Returns [N, n_q * hd].
    """
    N, nq, hd = q.shape
    group = nq // n_kv_heads
    out = np.empty((N, nq, hd), dtype=F64)
    for n in range(N):
        K, V = keys[n], values[n]
        for g in range(n_kv_heads):
            hs = slice(g * group, (g + 1) * group)
            s = (q[n, hs] @ K[:, g, :].T) / np.sqrt(F64(hd))  # [group, len]
            out[n, hs] = softmax(s) @ V[:, g, :]
    return out.reshape(N, nq * hd)


class OracleKV:
    """Per-layer, per-user key/value cache in float64 with append-only lengths."""

    def __init__(self, layers, max_users: int, max_ctx: int, n_kv_heads: int, head_dim: int):
        self.layers = list(layers)
        self.max_users, self.max_ctx = max_users, max_ctx
        self.k = {l: np.zeros((max_users, max_ctx, n_kv_heads, head_dim), F64) for l in self.layers}
        self.v = {l: np.zeros((max_users, max_ctx, n_kv_heads, head_dim), F64) for l in self.layers}
        self.len = np.zeros(max_users, dtype=np.int64)

    def inject(self, layer: int, user: int, pos0: int, k_bits: np.ndarray, v_bits: np.ndarray):
        """Write bf16 K/V (post-rotation keys), [n, n_kv, hd], at positions pos0.. of one user."""
        n = k_bits.shape[0]
        self.k[layer][user, pos0:pos0 + n] = bf16_to_f64(k_bits)
        self.v[layer][user, pos0:pos0 + n] = bf16_to_f64(v_bits)

    def set_len(self, user: int, n: int):
        self.len[user] = n


def decoder_layer(x, w, shape, kv: OracleKV, layer: int, users, positions):
    """One pre-norm decoder layer over rows ``x`` [N, H].

    Row n belongs to ``users[n]`` at ``positions[n]``.  All rows' keys and values
    are written to the cache first; row n then attends its user's keys
    ``0..positions[n]``.  Rows of one user must be at consecutive positions
    (a prefill chunk), rows of different users are independent (a batch).
    ``w`` maps tensor names to float64 arrays.
    """
    x = np.asarray(x, dtype=F64)
    N, H = x.shape
    nq, nkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    pos = np.asarray(positions, dtype=np.int64)
    xn = rms_norm(x, w["attn_norm"], shape.rms_eps)
    q = (xn @ w["wq"].T).reshape(N, nq, hd)
    k = (xn @ w["wk"].T).reshape(N, nkv, hd)
    v = (xn @ w["wv"].T).reshape(N, nkv, hd)
    if "q_norm" in w:  # Qwen3-style: each q and k head is RMS-normalised (gain over head_dim) before RoPE
        q = rms_norm(q, w["q_norm"], shape.rms_eps)
        k = rms_norm(k, w["k_norm"], shape.rms_eps)
    q = rope(q, pos, shape.rope_theta)
    k = rope(k, pos, shape.rope_theta)
    for n in range(N):
        kv.k[layer][users[n], pos[n]] = k[n]
        kv.v[layer][users[n], pos[n]] = v[n]
    keys = [kv.k[layer][users[n], : pos[n] + 1] for n in range(N)]
    vals = [kv.v[layer][users[n], : pos[n] + 1] for n in range(N)]
    o = attention_rows(q, keys, vals, nkv)
    x = x + o @ w["wo"].T
    z = rms_norm(x, w["mlp_norm"], shape.rms_eps)
    return x + mlp_swiglu(z, w["wg"], w["wu"], w["wd"])


def embed(tokens, e_bits_or_f64) -> np.ndarray:
    e = e_bits_or_f64
    rows = e[np.asarray(tokens, dtype=np.int64)]
    return bf16_to_f64(rows) if rows.dtype == np.uint16 else np.asarray(rows, dtype=F64)


def head_logits(x, final_norm, lm_head, eps: float) -> np.ndarray:
    """logits = RMSNorm(x; g_f) W_lm^T."""
    return rms_norm(x, final_norm, eps) @ lm_head.T


def argmax_lowest(logits: np.ndarray) -> np.ndarray:
    """Greedy token per row; the lowest index wins ties (numpy's first occurrence)."""
    logits = np.asarray(logits)
    if not np.all(np.isfinite(logits)):
        raise FloatingPointError("non-finite logits")
    return np.argmax(logits, axis=-1).astype(np.int64)


def _widen(wbits: dict) -> dict:
    return {k: (bf16_to_f64(v) if v.dtype == np.uint16 else np.asarray(v, F64)) for k, v in wbits.items()}


class OracleStage:
    """A contiguous layer range ``[lo, hi)`` plus, optionally, the head.

    ``layer_weights(l)`` returns layer l's tensors (bf16 bit patterns or float64);
    ``head_weights`` is a dict with embed, final_norm and lm_head when the stage
    has the head.  With ``cache_weights`` False the layer tensors are widened
    on every use (bounded memory at full model shapes).
    """

    def __init__(self, shape, lo: int, hi: int, layer_weights, head_weights=None,
                 max_users: int = 1, max_ctx: int = 256, cache_weights: bool = True):
        if not (0 <= lo < hi <= shape.n_layers):
            raise ValueError("layer range")
        self.shape, self.lo, self.hi = shape, lo, hi
        self._lw, self._cache = layer_weights, {} if cache_weights else None
        self.head = _widen(head_weights) if head_weights is not None else None
        self.kv = OracleKV(range(lo, hi), max_users, max_ctx, shape.n_kv_heads, shape.head_dim)

    def weights(self, l: int) -> dict:
        if self._cache is None:
            return _widen(self._lw(l))
        if l not in self._cache:
            self._cache[l] = _widen(self._lw(l))
        return self._cache[l]

    def _run(self, x, users, positions):
        for l in range(self.lo, self.hi):
            x = decoder_layer(x, self.weights(l), self.shape, self.kv, l, users, positions)
        return x

    def _input(self, tokens, hidden):
        if (tokens is None) == (hidden is None):
            raise ValueError("exactly one of tokens / hidden")
        if tokens is not None:
            if self.head is None:
                raise ValueError("token input needs the head")
            return embed(tokens, self.head["embed"])
        return np.asarray(hidden, dtype=F64)

    def decode(self, users, positions, tokens=None, hidden=None) -> np.ndarray:
        """One token for each of ``len(users)`` users; returns hidden_out [B, H]."""
        users, positions = list(users), list(positions)
        if len(set(users)) != len(users):
            raise ValueError("users must be distinct")
        for u, p in zip(users, positions):
            if p != self.kv.len[u]:
                raise ValueError("position must equal the user's cache length")
        x = self._run(self._input(tokens, hidden), users, positions)
        for u in users:
            self.kv.len[u] += 1
        return x

    def prefill(self, user: int, pos0: int, tokens=None, hidden=None) -> np.ndarray:
        """A chunk of consecutive tokens of one user from ``pos0``; returns [T, H]."""
        if pos0 != self.kv.len[user]:
            raise ValueError("pos0 must equal the user's cache length")
        x = self._input(tokens, hidden)
        T = x.shape[0]
        x = self._run(x, [user] * T, list(range(pos0, pos0 + T)))
        self.kv.len[user] += T
        return x

    def logits(self, hidden) -> np.ndarray:
        if self.head is None:
            raise ValueError("no head")
        return head_logits(hidden, self.head["final_norm"], self.head["lm_head"], self.shape.rms_eps)

    def argmax(self, hidden) -> np.ndarray:
        return argmax_lowest(self.logits(hidden))
