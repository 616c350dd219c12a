"""CPU oracle of one pipeline stage's forward pass (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  The product path (the HIP library and its
binding) never imports, links or calls it.
"""
from .stage_oracle import (  # noqa: F401
    OracleKV,
    OracleStage,
    argmax_lowest,
    attention_rows,
    bf16_to_f64,
    decoder_layer,
    embed,
    head_logits,
    mlp_swiglu,
    rms_norm,
    rope,
    silu,
    softmax,
)
