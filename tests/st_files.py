"""Synthetic safetensors checkpoints for the shard-loader tests (test infrastructure).

Tensors are the seeded synthetic weights, named as in Hugging Face Llama / Qwen3
checkpoints and written with the safetensors package's own writer, so the loader
is checked against the format as that library produces it.
"""
from __future__ import annotations

import numpy as np

LAYER_NAMES = {"attn_norm": "input_layernorm.weight", "wq": "self_attn.q_proj.weight",
               "wk": "self_attn.k_proj.weight", "wv": "self_attn.v_proj.weight", "wo": "self_attn.o_proj.weight",
               "mlp_norm": "post_attention_layernorm.weight", "wg": "mlp.gate_proj.weight",
               "wu": "mlp.up_proj.weight", "wd": "mlp.down_proj.weight", "q_norm": "self_attn.q_norm.weight",
               "k_norm": "self_attn.k_norm.weight"}
HEAD_NAMES = {"embed": "model.embed_tokens.weight", "final_norm": "model.norm.weight", "lm_head": "lm_head.weight"}


def bf16_tensor(bits: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)


def checkpoint_tensors(layers: dict, head: dict | None) -> dict:
    """{HF name: torch bf16 tensor} for layer index -> synth layer dict, plus the head."""
    out = {}
    for l, w in layers.items():
        for k, v in w.items():
            out[f"model.layers.{l}.{LAYER_NAMES[k]}"] = bf16_tensor(v)
    if head:
        for k, v in head.items():
            out[HEAD_NAMES[k]] = bf16_tensor(v)
    return out


def save(path: str, tensors: dict):
    from safetensors.torch import save_file
    save_file(tensors, path, metadata={"format": "pt"})
