"""fp64 CPU reference for the cached-context action decoder.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call
this module; only the tests, the smoke check and the CPU-baseline leg of the
benchmark do.  It shares no code with the GPU library.

What it computes
----------------
The action-context mechanism of the paper (section 3.2.1, "Constructing the
Action Context") keeps the intermediate state of one inference -- for the
transformer that is the per-layer key/value cache -- and reuses it in the
next inference instead of recomputing it; after an inference the unseen KV
is added to the pool.  Its exception handler (section 3.3, "Handler", common
part) discards the current slice and re-infers from freshly collected
environment data.  Reuse removes redundant work but does not change the
result, so the plain definition the cached path must reproduce is "run the
whole decoder over the whole sequence again".  Two implementations follow:

* ``full_step``     -- the definition: every decoded token recomputes the
                       entire sequence from scratch.
* ``ActionContext`` -- the paper's mechanism: per-row K/V kept across steps,
                       only new tokens computed, new observation K/V added
                       after the step, fed-back action tokens dropped.

The decoder itself is not defined by the paper (its models are named but
never specified).  The workloads fix a Llama-style pre-norm decoder:
RMSNorm, rotary position embedding (rotate-half pairing), multi-head causal
attention, SwiGLU feed-forward, no biases, and an action head restricted to
the last ``n_bins`` vocabulary ids (the action bins).  Readings where the
text is silent: RMSNorm epsilon from the config, gains applied after
normalisation, RoPE frequencies base^(-2i/head_dim), causal attention over
the whole prefix, greedy argmax with the lowest index winning ties.

Every computation is fp64 NumPy; weights of any storage type are widened to
fp64 when used.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np

F64 = np.float64


@dataclass(frozen=True)
class Config:
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    n_bins: int
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0


class Params:
    """Weights as seen by the reference: fp64 views, drawn lazily per layer.

    ``w_q, w_k, w_v, w_o`` are ``[n_layers, d, d]``; ``w_gate, w_up`` are
    ``[n_layers, F, d]``; ``w_down`` is ``[n_layers, d, F]`` (each matrix maps
    ``in -> out`` as ``y = W @ x``).  ``g_attn, g_ffn`` are ``[n_layers, d]``,
    ``g_final`` ``[d]``, ``embed`` ``[vocab, d]`` and ``head_bins`` the last
    ``n_bins`` rows of the output head, ``[n_bins, d]``.  Each entry may be
    anything indexable by layer that yields a float array.
    """

    def __init__(self, cfg: Config, **arrays):
        self.cfg = cfg
        self.arrays = arrays

    def layer(self, name: str, l: int) -> np.ndarray:
        return np.asarray(self.arrays[name][l], dtype=F64)

    def get(self, name: str) -> np.ndarray:
        return np.asarray(self.arrays[name], dtype=F64)


# ----------------------------------------------------------------------------
# building blocks


def linear(w: np.ndarray, x: np.ndarray) -> np.ndarray:
    """``y[t] = W @ x[t]`` for every token row of ``x``."""
    return x @ w.T


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def silu(z: np.ndarray) -> np.ndarray:
    """z * sigmoid(z)."""
    return z / (1.0 + np.exp(-z))


def rope_frequencies(head_dim: int, theta: float) -> np.ndarray:
    """theta_i = base^(-2i/head_dim), i < head_dim/2."""
    i = np.arange(head_dim // 2, dtype=F64)
    return theta ** (-2.0 * i / head_dim)


def apply_rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half RoPE.  ``x`` is ``[T, H, dh]``, ``positions`` ``[T]``.

    The pair (i, i + dh/2) of a head vector at position t is rotated by the
    angle t * theta_i.
    """
    dh = x.shape[-1]
    half = dh // 2
    ang = np.outer(np.asarray(positions, dtype=F64), rope_frequencies(dh, theta))[:, None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def softmax(s: np.ndarray) -> np.ndarray:
    """Softmax over the last axis; ``-inf`` entries get weight 0."""
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                     q_pos: np.ndarray, k_pos: np.ndarray) -> np.ndarray:
    """Multi-head scaled dot-product attention; query t sees keys at positions <= t.

    ``q`` is ``[Tq, H, dh]``, ``k, v`` are ``[Tk, H, dh]``.  Returns ``[Tq, H, dh]``.
    """
    dh = q.shape[-1]
    qh = np.transpose(q, (1, 0, 2))          # [H, Tq, dh]
    kh = np.transpose(k, (1, 2, 0))          # [H, dh, Tk]
    vh = np.transpose(v, (1, 0, 2))          # [H, Tk, dh]
    s = np.matmul(qh, kh) / math.sqrt(dh)    # [H, Tq, Tk]
    visible = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]
    s = np.where(visible[None], s, -np.inf)
    p = softmax(s)
    return np.transpose(np.matmul(p, vh), (1, 0, 2))


def split_heads(x: np.ndarray, cfg: Config) -> np.ndarray:
    return x.reshape(x.shape[0], cfg.n_heads, cfg.head_dim)


def decoder_layer(p: Params, l: int, h: np.ndarray, positions: np.ndarray,
                  k_past: np.ndarray, v_past: np.ndarray):
    """One pre-norm decoder layer over new tokens ``h`` ``[T, d]``.

    ``k_past, v_past`` ``[Tp, H, dh]`` hold the (already rotated) keys and
    values of positions 0..Tp-1; the new tokens sit at ``positions``.
    Returns (h_out, k_all, v_all) where k_all/v_all include the new tokens.
    """
    cfg = p.cfg
    u = rms_norm(h, p.layer("g_attn", l), cfg.rms_eps)
    q = split_heads(linear(p.layer("w_q", l), u), cfg)
    k = split_heads(linear(p.layer("w_k", l), u), cfg)
    v = split_heads(linear(p.layer("w_v", l), u), cfg)
    q = apply_rope(q, positions, cfg.rope_theta)
    k = apply_rope(k, positions, cfg.rope_theta)
    k_all = np.concatenate([k_past, k], axis=0)
    v_all = np.concatenate([v_past, v], axis=0)
    o = causal_attention(q, k_all, v_all, positions, np.arange(k_all.shape[0]))
    h = h + linear(p.layer("w_o", l), o.reshape(h.shape[0], cfg.d_model))
    u = rms_norm(h, p.layer("g_ffn", l), cfg.rms_eps)
    a = silu(linear(p.layer("w_gate", l), u)) * linear(p.layer("w_up", l), u)
    h = h + linear(p.layer("w_down", l), a)
    return h, k_all, v_all


def empty_kv(cfg: Config) -> np.ndarray:
    return np.zeros((0, cfg.n_heads, cfg.head_dim), dtype=F64)


def forward(p: Params, x: np.ndarray, start: int = 0,
            past: Optional[List[Tuple[np.ndarray, np.ndarray]]] = None):
    """Run every layer over tokens ``x`` ``[T, d]`` at positions start..start+T-1.

    ``past`` (one (K, V) pair per layer, ``start`` positions long) is the
    cached context; ``None`` means an empty context (``start`` must be 0).
    Returns (h_final [T, d], kv list covering positions 0..start+T-1).
    """
    cfg = p.cfg
    h = np.asarray(x, dtype=F64)
    positions = np.arange(start, start + h.shape[0])
    if past is None:
        assert start == 0
        past = [(empty_kv(cfg), empty_kv(cfg)) for _ in range(cfg.n_layers)]
    kv = []
    for l in range(cfg.n_layers):
        assert past[l][0].shape[0] == start
        h, k_all, v_all = decoder_layer(p, l, h, positions, past[l][0], past[l][1])
        kv.append((k_all, v_all))
    return h, kv


def bin_logits(p: Params, h_last: np.ndarray) -> np.ndarray:
    """Final RMSNorm, then the output head restricted to the last ``n_bins`` ids.

    ``h_last`` is ``[d]`` or ``[R, d]``; returns ``[n_bins]`` or ``[R, n_bins]``.
    Rows V-n_bins..V-1 of the head are exactly those slices of the full
    vocabulary logits.
    """
    cfg = p.cfg
    u = rms_norm(np.asarray(h_last, dtype=F64), p.get("g_final"), cfg.rms_eps)
    return u @ p.get("head_bins").T


def greedy(logits: np.ndarray) -> int:
    """argmax over bins; the lowest index wins ties."""
    return int(np.argmax(logits))


def bin_embedding(p: Params, b: int) -> np.ndarray:
    """Embedding of action bin ``b`` = vocabulary id V - n_bins + b."""
    cfg = p.cfg
    return p.layer("embed", cfg.vocab - cfg.n_bins + int(b))


def embed_ids(p: Params, ids: Sequence[int]) -> np.ndarray:
    return np.stack([p.layer("embed", int(i)) for i in ids]) if len(ids) else \
        np.zeros((0, p.cfg.d_model), dtype=F64)


# ----------------------------------------------------------------------------
# the definition: full recomputation for every decoded token


def full_decode(p: Params, seq: np.ndarray, n_actions: int,
                forced: Optional[Sequence[int]] = None):
    """Greedy decoding of ``n_actions`` bins after sequence ``seq`` ``[T, d]``.

    Each token's logits come from a fresh forward pass over the committed
    sequence followed by the bins fed back so far.  ``forced[j]`` (teacher
    forcing) replaces the fed-back bin j while the reported choice stays the
    argmax.  Returns (tokens [A] int, logits [A, n_bins]).
    """
    toks, logs = [], []
    x = np.asarray(seq, dtype=F64)
    for j in range(n_actions):
        h, _ = forward(p, x)
        z = bin_logits(p, h[-1])
        a = greedy(z)
        toks.append(a)
        logs.append(z)
        if j + 1 < n_actions:
            fb = a if forced is None else int(forced[j])
            x = np.concatenate([x, bin_embedding(p, fb)[None]], axis=0)
    return np.array(toks, dtype=np.int64), np.stack(logs)


def full_step(p: Params, seqs: List[np.ndarray], new: Optional[List[Optional[np.ndarray]]],
              n_actions: int, forced: Optional[np.ndarray] = None):
    """One action step over a batch of rows, by full recomputation.

    Row b commits ``new[b]`` (observation tokens) onto ``seqs[b]`` and then
    decodes greedily.  Returns (tokens [B, A], logits [B, A, n_bins], seqs').
    """
    out_t, out_z, out_s = [], [], []
    for b, s in enumerate(seqs):
        s = np.asarray(s, dtype=F64)
        if new is not None and new[b] is not None and len(new[b]):
            s = np.concatenate([s, np.asarray(new[b], dtype=F64)], axis=0)
        t, z = full_decode(p, s, n_actions, None if forced is None else forced[b])
        out_t.append(t)
        out_z.append(z)
        out_s.append(s)
    return np.stack(out_t), np.stack(out_z), out_s


# ----------------------------------------------------------------------------
# the action context: cached K/V reused across steps


class ActionContext:
    """Per-row cached context with build / step / invalidate.

    ``build`` computes and keeps every layer's K/V for each row's prefix and
    the final hidden state of the last position.  ``step`` first adds the new
    observation tokens to the context (computing only them, against the
    cached K/V), then decodes ``n_actions`` bins: the first bin's logits come
    from the kept last hidden state; each later bin costs one forward pass of
    a single fed-back token against the cache.  Fed-back tokens are not kept.
    ``invalidate`` discards everything; stepping an invalid context is an error.

    The exception handler's common part (paper section 3.3, "Handler")
    discards a slice and re-infers from fresh environment data; for one robot
    of a batch that is ``invalidate_rows`` followed by ``build_rows``, which
    leave the other rows' contexts as they are.  Every row must hold a context
    before the batch steps.  ``append`` is the post-inference insert of new
    observation tokens alone (section 3.2.1), without decoding.
    """

    def __init__(self, p: Params, batch: int):
        self.p = p
        self.batch = batch
        self.kv: List[Optional[list]] = [None] * batch
        self.h_last: List[Optional[np.ndarray]] = [None] * batch
        self.lens = np.zeros(batch, dtype=np.int64)
        self.row_valid = np.zeros(batch, dtype=bool)

    @property
    def valid(self) -> bool:
        return bool(np.all(self.row_valid))

    def _build_row(self, b: int, x: np.ndarray) -> None:
        x = np.asarray(x, dtype=F64)
        assert x.shape[0] > 0
        h, kv = forward(self.p, x)
        self.kv[b], self.h_last[b], self.lens[b] = kv, h[-1].copy(), x.shape[0]
        self.row_valid[b] = True

    def build(self, prefixes: Sequence[np.ndarray]) -> None:
        assert len(prefixes) == self.batch
        for b, x in enumerate(prefixes):
            self._build_row(b, x)

    def build_rows(self, rows: Sequence[int], prefixes: Sequence[np.ndarray]) -> None:
        assert len(rows) == len(prefixes)
        for b, x in zip(rows, prefixes):
            self._build_row(int(b), x)

    def invalidate(self) -> None:
        self.invalidate_rows(range(self.batch))

    def invalidate_rows(self, rows: Sequence[int]) -> None:
        for b in rows:
            b = int(b)
            self.kv[b], self.h_last[b], self.lens[b] = None, None, 0
            self.row_valid[b] = False

    def append(self, new: Sequence[Optional[np.ndarray]]) -> None:
        if not self.valid:
            raise RuntimeError("append on an invalid action context")
        for b in range(self.batch):
            if new[b] is not None and len(new[b]):
                self._extend(b, np.asarray(new[b], dtype=F64))

    def _extend(self, b: int, x: np.ndarray) -> None:
        h, kv = forward(self.p, x, start=int(self.lens[b]), past=self.kv[b])
        self.kv[b], self.h_last[b] = kv, h[-1].copy()
        self.lens[b] += x.shape[0]

    def step(self, new: Optional[Sequence[Optional[np.ndarray]]], n_actions: int,
             forced: Optional[np.ndarray] = None):
        """Returns (tokens [B, A], logits [B, A, n_bins])."""
        if not self.valid:
            raise RuntimeError("step on an invalid action context")
        toks = np.zeros((self.batch, n_actions), dtype=np.int64)
        logs = np.zeros((self.batch, n_actions, self.p.cfg.n_bins), dtype=F64)
        for b in range(self.batch):
            if new is not None and new[b] is not None and len(new[b]):
                self._extend(b, np.asarray(new[b], dtype=F64))
            kv, h, pos = self.kv[b], self.h_last[b], int(self.lens[b])
            for j in range(n_actions):
                z = bin_logits(self.p, h)
                a = greedy(z)
                toks[b, j], logs[b, j] = a, z
                if j + 1 < n_actions:
                    fb = a if forced is None else int(forced[b][j])
                    hs, kv = forward(self.p, bin_embedding(self.p, fb)[None], start=pos, past=kv)
                    h, pos = hs[-1], pos + 1
        return toks, logs

    def lengths(self) -> np.ndarray:
        return self.lens.copy()
