"""Turns seeded workload arrays into the fp64 reference's inputs (tests only)."""
import numpy as np

import oracle.decoder as D
from paper_2508_10259_amd import workload as W


class _Decoded:
    """Layer-indexable fp64 view of an encoded stack (host numpy or device-drawn),
    each layer decoded once and kept."""

    def __init__(self, stack, dtype):
        self.stack, self.dtype = stack, dtype
        self.cache = {}

    def __getitem__(self, l):
        if l not in self.cache:
            x = self.stack[l]
            if not isinstance(self.stack, W.DeviceStack):  # device stacks hand out fp32 already
                x = W.to_f32(x, self.dtype)
            self.cache[l] = np.asarray(x, dtype=np.float64)
        return self.cache[l]


def oracle_config(spec):
    return D.Config(spec.n_layers, spec.d_model, spec.n_heads, spec.head_dim, spec.d_ffn,
                    spec.vocab, spec.n_bins, spec.rms_eps, spec.rope_theta)


def oracle_params(w):
    spec = w.spec
    arrays = {n: _Decoded(getattr(w, n), spec.dtype) for n in W.MATRICES}
    arrays.update(g_attn=w.g_attn, g_ffn=w.g_ffn, g_final=w.g_final,
                  embed=W.to_f32(w.embed, spec.dtype), head_bins=W.to_f32(w.head_bins, spec.dtype))
    return D.Params(oracle_config(spec), **arrays)


def prefix_f64(p, spec, prefix):
    """Prefix embeddings: patch rows, then embedding rows of the instruction ids (ids first when
    the prefix says so)."""
    pt = prefix.patches
    if hasattr(pt, "cpu"):  # drawn on the device
        pt = pt.float().cpu().numpy()
        x = pt.astype(np.float64)
    else:
        x = W.to_f32(pt, spec.dtype).astype(np.float64)
    t = D.embed_ids(p, prefix.text_ids)
    return np.concatenate([t, x] if getattr(prefix, "text_first", False) else [x, t], axis=0)
