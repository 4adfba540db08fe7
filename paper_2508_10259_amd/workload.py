"""Seeded synthetic inputs for the cached-context action decoder.

This module holds random inputs and shapes only: model dimensions, weight
draws, prefix and observation embeddings, instruction token ids and ragged
prefix lengths.  It computes no part of the decoder itself.  The GPU path and
the CPU reference both consume what it returns, and neither depends on the
other.

Every stream is keyed by an explicit tuple (seed, purpose, indices) through
``numpy.random.SeedSequence``, so any single matrix, row or step can be
regenerated alone and in any order.

Value encoding: ``f32`` arrays are ``numpy.float32``; ``bf16`` arrays are
``numpy.uint16`` bit patterns produced by round-to-nearest-even from an fp32
draw.  ``bf16_bits_to_f32`` widens them exactly.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# ----------------------------------------------------------------------------
# value encoding


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even).

    Inputs must be finite; the draws below always are.
    """
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_f32(values: np.ndarray, dtype: str) -> np.ndarray:
    """Decode an encoded array (``f32`` or ``bf16`` bits) to fp32."""
    if dtype == "bf16":
        return bf16_bits_to_f32(values)
    return np.asarray(values, dtype=np.float32)


def encode(x: np.ndarray, dtype: str) -> np.ndarray:
    """Encode fp32 draws in the storage type of a model."""
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    return np.ascontiguousarray(x, dtype=np.float32)


# ----------------------------------------------------------------------------
# model shapes


@dataclass(frozen=True)
class ModelSpec:
    """Dimensions of a Llama-style pre-norm decoder with a 256-bin action head."""

    name: str
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    n_bins: int
    dtype: str  # "f32" or "bf16": storage of weights, embeddings and K/V
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    init_std: float = 0.02

    def __post_init__(self):
        assert self.n_heads * self.head_dim == self.d_model
        assert self.head_dim % 2 == 0
        assert 0 < self.n_bins <= self.vocab
        assert self.dtype in ("f32", "bf16")

    @property
    def matmul_params(self) -> int:
        return self.n_layers * (4 * self.d_model ** 2 + 3 * self.d_model * self.d_ffn)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def kv_bytes_per_token(self) -> int:
        return self.n_layers * 2 * self.d_model * self.elem_bytes


MODELS: Dict[str, ModelSpec] = {
    # 2 layers, d=256, 4 heads of 64, SwiGLU 1024, 256-id vocabulary (all ids are bins), fp32
    "tiny": ModelSpec("tiny", 2, 256, 4, 64, 1024, 256, 256, "f32"),
    # 12 layers, d=1024, 16 heads of 64, FFN 4096, 256-id vocabulary (all ids are bins), bf16
    "mid": ModelSpec("mid", 12, 1024, 16, 64, 4096, 256, 256, "bf16"),
    # 32 layers, d=4096, 32 heads of 128, FFN 11008, vocab 32000 (last 256 ids are bins), bf16
    "7b": ModelSpec("7b", 32, 4096, 32, 128, 11008, 32000, 256, "bf16"),
}

MATRICES = ("w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down")


def matrix_shape(spec: ModelSpec, name: str) -> Tuple[int, int]:
    d, f = spec.d_model, spec.d_ffn
    return {
        "w_q": (d, d), "w_k": (d, d), "w_v": (d, d), "w_o": (d, d),
        "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f),
        "embed": (spec.vocab, d), "head": (spec.vocab, d),
    }[name]


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(k) for k in key]))


# purpose tags inside SeedSequence keys
_T_MAT, _T_EMB, _T_HEAD, _T_PATCH, _T_IDS, _T_OBS, _T_LENS, _T_TIE = range(1, 9)


def draw_matrix(spec: ModelSpec, seed: int, layer: int, name: str) -> np.ndarray:
    """One weight matrix ``[out, in]`` drawn N(0, init_std) in fp32, then encoded."""
    shape = matrix_shape(spec, name)
    idx = MATRICES.index(name)
    x = _rng(seed, _T_MAT, layer, idx).standard_normal(shape, dtype=np.float32)
    x *= np.float32(spec.init_std)
    return encode(x, spec.dtype)


def draw_table(spec: ModelSpec, seed: int, name: str, rows: Optional[slice] = None) -> np.ndarray:
    """``embed`` or ``head`` table ``[vocab, d]``; ``rows`` selects a row range.

    The table is drawn in blocks of 256 rows with a stream per block, so a
    row range costs only the blocks it touches.
    """
    tag = _T_EMB if name == "embed" else _T_HEAD
    v, d = spec.vocab, spec.d_model
    rows = rows if rows is not None else slice(0, v)
    r0, r1 = rows.start or 0, rows.stop if rows.stop is not None else v
    out = []
    blk = 256
    for b0 in range((r0 // blk) * blk, r1, blk):
        nb = min(blk, v - b0)
        x = _rng(seed, tag, b0 // blk).standard_normal((nb, d), dtype=np.float32)
        x *= np.float32(spec.init_std)
        lo, hi = max(r0, b0) - b0, min(r1, b0 + nb) - b0
        out.append(x[lo:hi])
    return encode(np.concatenate(out, axis=0), spec.dtype)


class LayerStack:
    """Lazy ``[n_layers, out, in]`` view of one weight kind: ``stack[l]`` draws layer l."""

    def __init__(self, spec: ModelSpec, seed: int, name: str, cache: bool = True):
        self.spec, self.seed, self.name = spec, seed, name
        self.shape = (spec.n_layers,) + matrix_shape(spec, name)
        self._cache: Dict[int, np.ndarray] = {} if cache else None

    def __len__(self):
        return self.spec.n_layers

    def __getitem__(self, layer: int) -> np.ndarray:
        if self._cache is not None and layer in self._cache:
            return self._cache[layer]
        m = draw_matrix(self.spec, self.seed, layer, self.name)
        if self._cache is not None:
            self._cache[layer] = m
        return m


@dataclass
class Weights:
    """Encoded weights of one model.

    ``w_*`` are ``LayerStack`` (or arrays ``[n_layers, out, in]``), gains are
    fp32 ones (``[n_layers, d]`` / ``[d]``), ``embed`` and ``head`` are the
    full ``[vocab, d]`` tables unless ``head_rows`` restricts the head to
    its last ``n_bins`` rows (the only ones the action decoder reads).
    """

    spec: ModelSpec
    seed: int
    w_q: object
    w_k: object
    w_v: object
    w_o: object
    w_gate: object
    w_up: object
    w_down: object
    g_attn: np.ndarray
    g_ffn: np.ndarray
    g_final: np.ndarray
    embed: np.ndarray
    head_bins: np.ndarray  # last n_bins rows of the head, [n_bins, d]

    def stack(self, name: str) -> np.ndarray:
        """Materialise ``[n_layers, out, in]`` for one matrix kind."""
        s = getattr(self, name)
        if isinstance(s, np.ndarray):
            return s
        return np.stack([s[l] for l in range(self.spec.n_layers)])


def make_weights(spec: ModelSpec, seed: int = 0, lazy: Optional[bool] = None) -> Weights:
    """All weights of ``spec`` from ``seed``; matrices N(0, 0.02), gains 1.0."""
    if lazy is None:
        lazy = spec.matmul_params > 400_000_000
    mats = {}
    for name in MATRICES:
        st = LayerStack(spec, seed, name, cache=not lazy)
        mats[name] = st if lazy else np.stack([st[l] for l in range(spec.n_layers)])
    d = spec.d_model
    return Weights(
        spec=spec, seed=seed, **mats,
        g_attn=np.ones((spec.n_layers, d), np.float32),
        g_ffn=np.ones((spec.n_layers, d), np.float32),
        g_final=np.ones((d,), np.float32),
        embed=draw_table(spec, seed, "embed"),
        head_bins=draw_table(spec, seed, "head", slice(spec.vocab - spec.n_bins, spec.vocab)),
    )


# ----------------------------------------------------------------------------
# device-side draws for the 7B-parameter model (numpy draws ~30 M normals/s,
# minutes for 6.5 G weights): torch's CUDA Philox generator, one stream per
# (seed, purpose, indices) key, same N(0, std) recipe, rounded to bf16 by
# torch (round to nearest even).  The CPU reference receives host copies.


def _key_seed(*key: int) -> int:
    return int(np.random.SeedSequence([int(k) for k in key]).generate_state(1, dtype=np.uint64)[0] >> 1)


def device_normal(shape, std, dtype: str, device, *key: int):
    """torch tensor on `device`: N(0, std) drawn in fp32 from the stream `key`, in `dtype`."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(_key_seed(*key))
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(torch.bfloat16) if dtype == "bf16" else x


class DeviceStack:
    """``[n_layers, out, in]`` device tensor of one matrix kind; ``stack[l]`` gives a host
    fp32 numpy copy of layer l (for the CPU reference)."""

    def __init__(self, t):
        self.t = t
        self.shape = tuple(t.shape)

    def __len__(self):
        return self.shape[0]

    def __getitem__(self, layer: int) -> np.ndarray:
        return self.t[layer].float().cpu().numpy()


def make_device_weights(spec: ModelSpec, seed: int = 0, device="cuda") -> Weights:
    """All weights of ``spec`` drawn on the device (matrices N(0, 0.02), gains 1.0).
    Matrix fields are DeviceStack; tables are host arrays in the model dtype encoding."""
    import torch
    d = spec.d_model
    mats = {}
    for idx, name in enumerate(MATRICES):
        out_, in_ = matrix_shape(spec, name)
        t = torch.empty((spec.n_layers, out_, in_), device=device,
                        dtype=torch.bfloat16 if spec.dtype == "bf16" else torch.float32)
        for l in range(spec.n_layers):
            t[l].copy_(device_normal((out_, in_), spec.init_std, spec.dtype, device, seed, _T_MAT, l, idx))
        mats[name] = DeviceStack(t)

    def table(tag, rows):
        x = device_normal((rows, d), spec.init_std, spec.dtype, device, seed, tag)
        if spec.dtype == "bf16":
            return x.view(torch.int16).cpu().numpy().view(np.uint16)
        return x.cpu().numpy()
    return Weights(
        spec=spec, seed=seed, **mats,
        g_attn=np.ones((spec.n_layers, d), np.float32),
        g_ffn=np.ones((spec.n_layers, d), np.float32),
        g_final=np.ones((d,), np.float32),
        embed=table(_T_EMB, spec.vocab),
        head_bins=table(_T_HEAD, spec.n_bins),
    )


# ----------------------------------------------------------------------------
# episodes: prefixes, per-step observation tokens, ragged lengths


@dataclass(frozen=True)
class Workload:
    """A synthetic VLA-shaped decode workload.

    ``prefix_lens`` is either a fixed ``(n_patch, n_text)`` pair for every row,
    or ``None`` with ``ragged=(lo, hi, n_text)``: per row L_b ~ U{lo..hi},
    made of (L_b - n_text) patch embeddings followed by n_text instruction ids.
    """

    name: str
    model: str
    batch: int
    n_actions: int
    steps: int
    prefix: Optional[Tuple[int, int]] = None
    ragged: Optional[Tuple[int, int, int]] = None
    new_per_step: int = 0
    invalidate_every: int = 0
    recompute_each_step: bool = False
    capacity: int = 0  # 0: derived
    # rows in `shared[0]` groups (row b in group b % shared[0]): every row of a group starts with
    # the group's instruction (shared[1] ids) and scene (shared[2] patch embeddings), then its own
    # patches; ragged lengths count all of it
    shared: Optional[Tuple[int, int, int]] = None

    @property
    def spec(self) -> ModelSpec:
        return MODELS[self.model]

    def max_prefix(self) -> int:
        if self.prefix is not None:
            return sum(self.prefix)
        return self.ragged[1]

    def derived_capacity(self, steps_between_builds: Optional[int] = None, extra_new: int = 0) -> int:
        """Smallest 64-multiple that fits the longest row of one build window."""
        if self.capacity:
            return self.capacity
        w = steps_between_builds if steps_between_builds is not None else (
            self.invalidate_every or (1 if self.recompute_each_step else self.steps))
        need = self.max_prefix() + w * (self.new_per_step + extra_new) + self.n_actions - 1
        return (need + 63) // 64 * 64


WORKLOADS: Dict[str, Workload] = {
    # tiny fp32 decoder, cached prefix of 64 N(0,1) embeddings, 7 action tokens, batch 1
    "tiny-b1": Workload("tiny-b1", "tiny", 1, 7, 100, prefix=(64, 0)),
    # mid-size bf16 decoder, 256 patches + 24 instruction ids, 7 action tokens, batch 8, 500 steps
    "mid-b8": Workload("mid-b8", "mid", 8, 7, 500, prefix=(256, 24)),
    # 7B bf16 decoder, 256 patches + 32 instruction ids, 7 action tokens, batch 1, 200 steps
    "7b-b1": Workload("7b-b1", "7b", 1, 7, 200, prefix=(256, 32)),
    # 7B, batch 64, ragged prefixes U{200..400}, 16 new observation tokens per step,
    # every row invalidated and rebuilt every 20 steps
    "7b-b64-ragged": Workload("7b-b64-ragged", "7b", 64, 7, 200, ragged=(200, 400, 32),
                              new_per_step=16, invalidate_every=20, capacity=768),
    # 7B, action chunking: 56 tokens per step against a 600-token prefix, batch 16
    "7b-chunk56-b16": Workload("7b-chunk56-b16", "7b", 16, 56, 50, prefix=(568, 32)),
    # as 7b-b64-ragged, with the 64 rows in 8 tasks: a row's prefix is its task's 32 instruction
    # ids and 224 scene patches, then U{0..144} patches of its own (lengths U{256..400})
    "7b-b64-shared": Workload("7b-b64-shared", "7b", 64, 7, 200, ragged=(256, 400, 32), new_per_step=16,
                              invalidate_every=20, capacity=768, shared=(8, 32, 224)),
}


def prefix_lengths(wl: Workload, seed: int, epoch: int) -> np.ndarray:
    """Per-row prefix lengths L_b for build ``epoch``."""
    if wl.prefix is not None:
        return np.full(wl.batch, sum(wl.prefix), dtype=np.int32)
    lo, hi, _ = wl.ragged
    return _rng(seed, _T_LENS, epoch).integers(lo, hi + 1, size=wl.batch).astype(np.int32)


def _n_text(wl: Workload) -> int:
    return wl.prefix[1] if wl.prefix is not None else wl.ragged[2]


def text_id_range(spec: ModelSpec) -> Tuple[int, int]:
    """Instruction ids are drawn from the non-bin ids, or from all ids when every id is a bin."""
    if spec.vocab > spec.n_bins:
        return 0, spec.vocab - spec.n_bins
    return 0, spec.vocab


@dataclass
class Prefix:
    """One row's prefix: ``patches`` [n_patch, d] (encoded) then ``text_ids`` [n_text], or the ids
    first when ``text_first``."""

    patches: np.ndarray
    text_ids: np.ndarray
    text_first: bool = False

    @property
    def length(self) -> int:
        return self.patches.shape[0] + self.text_ids.shape[0]


def _shared_prefix(wl: Workload, seed: int, epoch: int, row: int, length: int, device=None) -> Prefix:
    spec = wl.spec
    groups, n_text, n_scene = wl.shared
    g = row % groups
    lo, hi = text_id_range(spec)
    ids = _rng(seed, _T_IDS, epoch, 1 << 20, g).integers(lo, hi, size=n_text).astype(np.int32)
    own = length - n_text - n_scene
    if device is None:
        scene = _rng(seed, _T_PATCH, epoch, 1 << 20, g).standard_normal((n_scene, spec.d_model), dtype=np.float32)
        mine = _rng(seed, _T_PATCH, epoch, row).standard_normal((own, spec.d_model), dtype=np.float32)
        return Prefix(encode(np.concatenate([scene, mine]), spec.dtype), ids, text_first=True)
    import torch
    scene = device_normal((n_scene, spec.d_model), 1.0, spec.dtype, device, seed, _T_PATCH, epoch, 1 << 20, g)
    mine = device_normal((own, spec.d_model), 1.0, spec.dtype, device, seed, _T_PATCH, epoch, row)
    return Prefix(torch.cat([scene, mine]), ids, text_first=True)


def make_prefix(wl: Workload, seed: int, epoch: int, row: int, length: Optional[int] = None) -> Prefix:
    spec = wl.spec
    if length is None:
        length = int(prefix_lengths(wl, seed, epoch)[row])
    if wl.shared:
        return _shared_prefix(wl, seed, epoch, row, length)
    n_text = min(_n_text(wl), length)
    n_patch = length - n_text
    x = _rng(seed, _T_PATCH, epoch, row).standard_normal((n_patch, spec.d_model), dtype=np.float32)
    lo, hi = text_id_range(spec)
    ids = _rng(seed, _T_IDS, epoch, row).integers(lo, hi, size=n_text).astype(np.int32)
    return Prefix(encode(x, spec.dtype), ids)


def make_prefixes(wl: Workload, seed: int, epoch: int) -> List[Prefix]:
    lens = prefix_lengths(wl, seed, epoch)
    return [make_prefix(wl, seed, epoch, b, int(lens[b])) for b in range(wl.batch)]


def make_prefix_device(wl: Workload, seed: int, epoch: int, row: int, length: Optional[int] = None,
                       device="cuda") -> Prefix:
    """As make_prefix, with the patch embeddings drawn on the device (a torch tensor)."""
    spec = wl.spec
    if length is None:
        length = int(prefix_lengths(wl, seed, epoch)[row])
    if wl.shared:
        return _shared_prefix(wl, seed, epoch, row, length, device)
    n_text = min(_n_text(wl), length)
    x = device_normal((length - n_text, spec.d_model), 1.0, spec.dtype, device, seed, _T_PATCH, epoch, row)
    lo, hi = text_id_range(spec)
    ids = _rng(seed, _T_IDS, epoch, row).integers(lo, hi, size=n_text).astype(np.int32)
    return Prefix(x, ids)


def make_observation_device(spec: ModelSpec, seed: int, step: int, n_rows: int, n: int, device="cuda"):
    """[n_rows * n, d] fresh N(0,1) observation embeddings for all rows of one step, on the device."""
    return device_normal((n_rows * n, spec.d_model), 1.0, spec.dtype, device, seed, _T_OBS, step, 1 << 20)


def make_observation(spec: ModelSpec, seed: int, step: int, row: int, n: int) -> np.ndarray:
    """``n`` fresh N(0,1) observation embeddings for one row at one step (encoded)."""
    x = _rng(seed, _T_OBS, step, row).standard_normal((n, spec.d_model), dtype=np.float32)
    return encode(x, spec.dtype)


_T_FLOW = 9


def make_flow_head(spec: ModelSpec, action_dim: int, seed: int = 0):
    """Weights of a flow-matching action head (encoded in the model dtype): w_in [d][a] with
    N(0, 1/a) entries (unit-scale token embeddings from unit-scale latents), w_t [d] N(0, 1),
    w_out [a][d] N(0, 0.02)."""
    d = spec.d_model
    w_in = _rng(seed, _T_FLOW, 1).standard_normal((d, action_dim), dtype=np.float32) / np.float32(np.sqrt(action_dim))
    w_t = _rng(seed, _T_FLOW, 2).standard_normal((d,), dtype=np.float32)
    w_out = _rng(seed, _T_FLOW, 3).standard_normal((action_dim, d), dtype=np.float32) * np.float32(0.02)
    return encode(w_in, spec.dtype), encode(w_t, spec.dtype), encode(w_out, spec.dtype)


def make_latent(seed: int, key: int, rows: int, n_tokens: int, action_dim: int) -> np.ndarray:
    """N(0, 1) action latents [rows][n_tokens][action_dim] (fp32): the noise of a cold start."""
    return _rng(seed, _T_FLOW, 100, key).standard_normal((rows, n_tokens, action_dim), dtype=np.float32)


def random_gaussian(shape: Sequence[int], seed: int, *key: int, dtype: str = "f32",
                    std: float = 1.0) -> np.ndarray:
    """A generic seeded N(0, std) array, encoded in ``dtype`` (for kernel-level tests)."""
    x = _rng(seed, _T_TIE, *key).standard_normal(tuple(shape), dtype=np.float32) * np.float32(std)
    return encode(x, dtype)
