"""Shared helpers of the GPU parity tests: device set-up through the C ABI,
the fp64 reference on the same seeded inputs, and the comparison metrics."""
from __future__ import annotations

import sys
from dataclasses import dataclass
from typing import List, Optional

import numpy as np

from paper_2508_10259_amd import workload as W
import oracle.decoder as D
from ref_bridge import oracle_params, prefix_f64


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


@dataclass
class Compare:
    max_abs: float
    strict: float  # fraction of GPU choices equal to the reference argmax
    band: float    # fraction of GPU choices within `tol` of the reference maximum
    n: int


def compare(z_ref: np.ndarray, z_gpu: np.ndarray, t_gpu: np.ndarray, tol: float) -> Compare:
    z_ref = np.asarray(z_ref, dtype=np.float64)
    err = float(np.max(np.abs(z_ref - z_gpu))) if z_ref.size else 0.0
    ref_arg = np.argmax(z_ref, axis=-1)
    strict = float(np.mean(ref_arg == t_gpu))
    picked = np.take_along_axis(z_ref, t_gpu[..., None].astype(np.int64), axis=-1)[..., 0]
    band = float(np.mean(picked >= np.max(z_ref, axis=-1) - tol))
    return Compare(err, strict, band, int(t_gpu.size))


def small_spec(dtype="bf16", n_layers=2, d=256, H=4, F=512, V=300, n_bins=256, name="small") -> W.ModelSpec:
    return W.ModelSpec(name, n_layers, d, H, d // H, F, V, n_bins, dtype)


class Pair:
    """The same seeded model on the device (through the C ABI) and in the fp64 reference."""

    def __init__(self, spec: W.ModelSpec, seed: int = 0, device="cuda", gains: bool = False):
        from paper_2508_10259_amd.runtime import DeviceModel
        self.spec = spec
        self.w = W.make_weights(spec, seed)
        if gains:  # RMSNorm gains 1 + 0.25 N(0,1) instead of the workloads' 1.0
            L, d = spec.n_layers, spec.d_model
            self.w.g_attn = (1 + 0.25 * W.random_gaussian((L, d), seed, 1, dtype="f32")).astype(np.float32)
            self.w.g_ffn = (1 + 0.25 * W.random_gaussian((L, d), seed, 2, dtype="f32")).astype(np.float32)
            self.w.g_final = (1 + 0.25 * W.random_gaussian((d,), seed, 3, dtype="f32")).astype(np.float32)
        self.p = oracle_params(self.w)
        self.dev = DeviceModel(self.w, device)

    def prefixes_f64(self, prefixes: List[W.Prefix]) -> List[np.ndarray]:
        return [prefix_f64(self.p, self.spec, pr) for pr in prefixes]

    def obs_f64(self, x: np.ndarray) -> np.ndarray:
        return W.to_f32(x, self.spec.dtype).astype(np.float64)


def gpu_new_tokens(spec: W.ModelSpec, news: List[Optional[np.ndarray]], device="cuda"):
    """Packed device tensor and per-row lengths of per-row observation tokens."""
    import torch
    from paper_2508_10259_amd.runtime import to_device
    lens = [0 if x is None else x.shape[0] for x in news]
    if sum(lens) == 0:
        return None, lens
    packed = np.concatenate([x for x in news if x is not None and x.shape[0] > 0], axis=0)
    return to_device(packed, spec.dtype, device), lens


class ForcedRef:
    """One row of the fp64 reference stepped with given fed-back bins.

    A step's logits come from one forward pass over the step's new tokens followed by the
    embedding-table rows (vocab - n_bins + bin) of the bins fed back after actions 0..A-2:
    the logits of action j are those of the sequence's last committed token (j = 0) or of
    the j-th fed-back token -- the teacher-forced decoding that ``pin_forced_decoding``
    pins to the reference's own step.  New tokens are committed, fed-back ones dropped
    (``pin_lifecycle``).  Feeding the GPU's own choices back makes both sides follow one
    trajectory, so a near-tie flip cannot cascade while every position is still compared.
    """

    def __init__(self, p, prefix: np.ndarray):
        self.p = p
        h, self.kv = D.forward(p, np.asarray(prefix, dtype=np.float64))
        self.h_last = h[-1].copy()
        self.len = prefix.shape[0]

    def step(self, new: Optional[np.ndarray], fed) -> np.ndarray:
        """Logits [A, n_bins]; fed = the A bins chosen (the last one is not fed back)."""
        p = self.p
        A = len(fed)
        n_new = 0 if new is None else int(new.shape[0])
        parts = ([] if n_new == 0 else [np.asarray(new, dtype=np.float64)]) + \
            [D.bin_embedding(p, int(f))[None] for f in fed[:A - 1]]
        if not parts:
            return D.bin_logits(p, self.h_last[None])
        h, kv = D.forward(p, np.concatenate(parts, axis=0), start=self.len, past=self.kv)
        hs = [self.h_last] + list(h[:A - 1]) if n_new == 0 else list(h[n_new - 1:n_new - 1 + A])
        z = D.bin_logits(p, np.stack(hs))
        if n_new:
            self.len += n_new
            self.kv = [(k[:self.len], v[:self.len]) for k, v in kv]
            self.h_last = h[n_new - 1].copy()
        return z


def percentiles(errs) -> str:
    e = np.abs(np.concatenate([np.ravel(x) for x in errs]))
    q = np.percentile(e, [50, 90, 99, 99.9, 100])
    return "p50 {:.2e} p90 {:.2e} p99 {:.2e} p99.9 {:.2e} max {:.2e}".format(*q)
