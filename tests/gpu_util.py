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
