"""CPU reference (fp64) for the cached-context action decoder.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by the smoke check and by
the benchmark's CPU-baseline leg, never by the product package.  It shares no
code with the GPU library (see ``decoder.py`` for what it computes and the
passages of the paper it follows).
"""
from .decoder import (  # noqa: F401
    ActionContext, Config, Params, apply_rope, bin_embedding, bin_logits,
    causal_attention, decoder_layer, embed_ids, forward, full_decode, full_step,
    greedy, linear, rms_norm, rope_frequencies, silu, softmax,
)
