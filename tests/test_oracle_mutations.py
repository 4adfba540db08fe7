"""Plant plausible mistakes in a copy of the fp64 reference and require the pins to catch each.

Every mutation is applied to a fresh, private copy of the reference module on
the CPU; the real module is never touched.
"""
import importlib.util
import math
import sys

import numpy as np
import pytest

import oracle.decoder as D_real
from oracle_pins import ALL_PINS


def _fresh():
    spec = importlib.util.spec_from_file_location("oracle_decoder_copy", D_real.__file__)
    m = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = m  # dataclasses resolve annotations through sys.modules
    spec.loader.exec_module(m)
    return m


def _rope_sign(m):
    def apply_rope(x, positions, theta):
        dh = x.shape[-1]; half = dh // 2
        ang = np.outer(np.asarray(positions, float), m.rope_frequencies(dh, theta))[:, None, :]
        c, s = np.cos(ang), np.sin(ang)
        a, b = x[..., :half], x[..., half:]
        return np.concatenate([a * c + b * s, -a * s + b * c], axis=-1)
    m.apply_rope = apply_rope


def _rope_interleaved(m):
    def apply_rope(x, positions, theta):
        dh = x.shape[-1]
        ang = np.outer(np.asarray(positions, float), m.rope_frequencies(dh, theta))[:, None, :]
        c, s = np.cos(ang), np.sin(ang)
        a, b = x[..., 0::2], x[..., 1::2]
        out = np.empty_like(x)
        out[..., 0::2], out[..., 1::2] = a * c - b * s, a * s + b * c
        return out
    m.apply_rope = apply_rope


def _rope_freq(m):
    m.rope_frequencies = lambda dh, theta: theta ** (-np.arange(dh // 2, dtype=float) / dh)


def _rms_no_eps(m):
    m.rms_norm = lambda x, g, eps: x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) * g


def _rms_eps_outside(m):
    m.rms_norm = lambda x, g, eps: x / (np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps) * g


def _rms_no_gain(m):
    m.rms_norm = lambda x, g, eps: x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def _silu_relu(m):
    m.silu = lambda z: np.maximum(z, 0.0)


def _silu_sigmoid(m):
    m.silu = lambda z: 1.0 / (1.0 + np.exp(-z))


def _attn_no_scale(m):
    orig = m.causal_attention
    m.causal_attention = lambda q, k, v, qp, kp: orig(q * math.sqrt(q.shape[-1]), k, v, qp, kp)


def _attn_noncausal(m):
    orig = m.causal_attention
    m.causal_attention = lambda q, k, v, qp, kp: orig(q, k, v, np.full_like(np.asarray(qp), 10 ** 9), kp)


def _attn_excludes_self(m):
    orig = m.causal_attention
    m.causal_attention = lambda q, k, v, qp, kp: orig(q, k, v, np.asarray(qp) - 1, kp)


def _heads_strided(m):
    m.split_heads = lambda x, cfg: x.reshape(x.shape[0], cfg.head_dim, cfg.n_heads).transpose(0, 2, 1)


def _layer_variant(m, variant):
    def decoder_layer(p, l, h, positions, k_past, v_past):
        cfg = p.cfg
        u = m.rms_norm(h, p.layer("g_attn", l), cfg.rms_eps)
        wq, wk = ("w_k", "w_q") if variant == "qk_swap" else ("w_q", "w_k")
        q = m.split_heads(m.linear(p.layer(wq, l), u), cfg)
        k = m.split_heads(m.linear(p.layer(wk, l), u), cfg)
        v = m.split_heads(m.linear(p.layer("w_v", l), u), cfg)
        q = m.apply_rope(q, positions, cfg.rope_theta)
        if variant != "k_unrotated":
            k = m.apply_rope(k, positions, cfg.rope_theta)
        k_all = np.concatenate([k_past, k]); v_all = np.concatenate([v_past, v])
        o = m.causal_attention(q, k_all, v_all, positions, np.arange(k_all.shape[0]))
        att = m.linear(p.layer("w_o", l), o.reshape(h.shape[0], cfg.d_model))
        h = att if variant == "no_attn_residual" else h + att
        g_ffn = p.layer("g_attn" if variant == "ffn_uses_attn_gain" else "g_ffn", l)
        u = m.rms_norm(h, g_ffn, cfg.rms_eps)
        gate, up = m.linear(p.layer("w_gate", l), u), m.linear(p.layer("w_up", l), u)
        if variant == "gate_up_swap":
            gate, up = up, gate
        y = m.linear(p.layer("w_down", l), m.silu(gate) * up)
        h = y if variant == "no_ffn_residual" else h + y
        return h, k_all, v_all
    m.decoder_layer = decoder_layer


def _positions_restart(m):
    orig = m.decoder_layer
    m.decoder_layer = lambda p, l, h, pos, kp, vp: orig(p, l, h, np.asarray(pos) - np.asarray(pos)[0], kp, vp)


def _bin_id(m):
    m.bin_embedding = lambda p, b: p.layer("embed", int(b))


def _argmax_last(m):
    m.greedy = lambda z: int(len(z) - 1 - np.argmax(np.asarray(z)[::-1]))


def _no_commit(m):
    def _extend(self, b, x):
        m.forward(self.p, x, start=int(self.lens[b]), past=self.kv[b])
    m.ActionContext._extend = _extend


def _keep_actions(m):
    orig_step = m.ActionContext.step

    def step(self, new, n_actions, forced=None):
        t, z = orig_step(self, new, n_actions, forced)
        for b in range(self.batch):
            for j in range(n_actions - 1):
                self._extend(b, m.bin_embedding(self.p, t[b, j])[None])
        return t, z
    m.ActionContext.step = step


def _text_id_offset(m):
    m.embed_ids = lambda p, ids: np.stack([p.layer("embed", (int(i) + p.cfg.n_bins) % p.cfg.vocab) for i in ids]) \
        if len(ids) else np.zeros((0, p.cfg.d_model))


def _text_id_off_by_one(m):
    m.embed_ids = lambda p, ids: np.stack([p.layer("embed", (int(i) + 1) % p.cfg.vocab) for i in ids]) \
        if len(ids) else np.zeros((0, p.cfg.d_model))


def _forced_ignored(m):
    full, step = m.full_decode, m.ActionContext.step
    m.full_decode = lambda p, seq, n_actions, forced=None: full(p, seq, n_actions, None)
    m.ActionContext.step = lambda self, new, n_actions, forced=None: step(self, new, n_actions, None)


def _build_rows_all(m):
    orig = m.ActionContext.build_rows

    def build_rows(self, rows, prefixes):  # also re-runs every other row on the first new prefix
        orig(self, range(self.batch), [prefixes[0]] * self.batch)
        orig(self, rows, prefixes)
    m.ActionContext.build_rows = build_rows


def _invalidate_rows_keeps_length(m):
    def invalidate_rows(self, rows):
        for b in rows:
            self.row_valid[int(b)] = False
    m.ActionContext.invalidate_rows = invalidate_rows


def _append_no_commit(m):
    m.ActionContext.append = lambda self, new: None


MUTATIONS = {
    "rope_sign": _rope_sign, "rope_interleaved": _rope_interleaved, "rope_freq": _rope_freq,
    "rms_no_eps": _rms_no_eps, "rms_eps_outside": _rms_eps_outside, "rms_no_gain": _rms_no_gain,
    "silu_relu": _silu_relu, "silu_sigmoid": _silu_sigmoid,
    "attn_no_scale": _attn_no_scale, "attn_noncausal": _attn_noncausal,
    "attn_excludes_self": _attn_excludes_self, "heads_strided": _heads_strided,
    "qk_swap": lambda m: _layer_variant(m, "qk_swap"),
    "k_unrotated": lambda m: _layer_variant(m, "k_unrotated"),
    "no_attn_residual": lambda m: _layer_variant(m, "no_attn_residual"),
    "no_ffn_residual": lambda m: _layer_variant(m, "no_ffn_residual"),
    "ffn_uses_attn_gain": lambda m: _layer_variant(m, "ffn_uses_attn_gain"),
    "gate_up_swap": lambda m: _layer_variant(m, "gate_up_swap"),
    "positions_restart": _positions_restart, "bin_id": _bin_id, "argmax_last": _argmax_last,
    "no_commit": _no_commit, "keep_actions": _keep_actions,
    "text_id_offset": _text_id_offset, "text_id_off_by_one": _text_id_off_by_one,
    "forced_ignored": _forced_ignored, "build_rows_all": _build_rows_all,
    "invalidate_rows_keeps_length": _invalidate_rows_keeps_length, "append_no_commit": _append_no_commit,
}


def test_unmutated_copy_passes():
    m = _fresh()
    for pin in ALL_PINS:
        pin(m)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name):
    m = _fresh()
    MUTATIONS[name](m)
    caught = []
    for pin in ALL_PINS:
        try:
            pin(m)
        except Exception as e:  # noqa: BLE001 - any failure counts as caught
            caught.append(f"{pin.__name__}: {type(e).__name__}")
    assert caught, f"mutation {name} slipped past every pin"
