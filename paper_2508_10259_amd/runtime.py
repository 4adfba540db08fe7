"""Torch-facing wrapper over the C ABI.

PyTorch only provides device memory and the stream; every step of the
decoder runs in ``libams.so``.  ``DeviceModel`` uploads encoded weights and
creates the model handle; ``DeviceContext`` owns a context workspace and
exposes build / step / invalidate.
"""
from __future__ import annotations

import atexit
import ctypes as C
import weakref
from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import capi
from .workload import MATRICES, ModelSpec, Prefix, Weights


# Handles still open when the interpreter exits are released by an exit hook
# (contexts first, then models) while the HIP runtime that owns their streams
# and graphs is certainly up, not left to object finalisation at shutdown.
_live_contexts: "weakref.WeakSet" = weakref.WeakSet()
_live_models: "weakref.WeakSet" = weakref.WeakSet()


@atexit.register
def _release_live_handles() -> None:
    for group in (_live_contexts, _live_models):
        for obj in list(group):
            try:
                obj.close()
            except Exception:
                pass


def torch_dtype(dtype: str) -> torch.dtype:
    return torch.float32 if dtype == "f32" else torch.bfloat16


def to_device(values: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """Encoded numpy array (fp32, or bf16 bit patterns) -> device tensor."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(values).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(values, dtype=np.float32))
    return t.to(device)


def _stream(stream=None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def model_cfg(spec: ModelSpec) -> capi.ModelCfg:
    return capi.ModelCfg(spec.n_layers, spec.d_model, spec.n_heads, spec.head_dim, spec.d_ffn, spec.vocab,
                         spec.n_bins, spec.rms_eps, spec.rope_theta,
                         capi.AMS_F32 if spec.dtype == "f32" else capi.AMS_BF16)


class DeviceModel:
    """Weights on the device plus the library's packed copy."""

    def __init__(self, w: Weights, device="cuda", keep_source: bool = False):
        self.lib = capi.load()
        self.spec = spec = w.spec
        self.device = torch.device(device)
        td = torch_dtype(spec.dtype)
        src = {}
        for name in MATRICES:
            stack = getattr(w, name)
            if hasattr(stack, "t"):  # drawn on the device already
                src[name] = stack.t
                continue
            t = torch.empty((spec.n_layers,) + tuple(stack[0].shape), dtype=td, device=device)
            for l in range(spec.n_layers):
                t[l].copy_(to_device(stack[l], spec.dtype, device))
            src[name] = t
        src["g_attn"] = torch.from_numpy(w.g_attn).to(device)
        src["g_ffn"] = torch.from_numpy(w.g_ffn).to(device)
        src["g_final"] = torch.from_numpy(w.g_final).to(device)
        self.embed = to_device(w.embed, spec.dtype, device)
        src["embed"] = self.embed
        src["head_bins"] = to_device(w.head_bins, spec.dtype, device)
        self.cfg = model_cfg(spec)
        wts = capi.Weights(**{k: v.data_ptr() for k, v in src.items()})
        nbytes = self.lib.ams_model_workspace_bytes(C.byref(self.cfg))
        if nbytes == 0:
            raise ValueError("invalid model configuration")
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
        h = C.c_void_p()
        capi.check(self.lib.ams_model_create(C.byref(self.cfg), C.byref(wts), self.ws.data_ptr(), nbytes,
                                             _stream(), C.byref(h)), "ams_model_create")
        torch.cuda.current_stream().synchronize()
        self.handle = h
        _live_models.add(self)
        # the packed copy is all the library reads afterwards, except `embed`
        self.source = src if keep_source else {"embed": self.embed}

    def embed_ids(self, ids: torch.Tensor, out: torch.Tensor) -> None:
        assert ids.dtype == torch.int32 and ids.is_contiguous() and out.is_contiguous()
        capi.check(self.lib.ams_embed_ids(self.handle, ids.data_ptr(), ids.numel(), out.data_ptr(), _stream()),
                   "ams_embed_ids")

    def pack_prefixes(self, prefixes: Sequence[Prefix]) -> Tuple[torch.Tensor, List[int]]:
        """Packed prefix rows: each row's patch embeddings, then its instruction
        ids embedded on the device by the library."""
        spec = self.spec
        lens = [p.length for p in prefixes]
        out = torch.empty((sum(lens), spec.d_model), dtype=torch_dtype(spec.dtype), device=self.device)
        o = 0
        for p in prefixes:
            n_p, n_t = p.patches.shape[0], len(p.text_ids)
            po, to = (o + n_t, o) if p.text_first else (o, o + n_p)
            if n_p:
                src = p.patches if isinstance(p.patches, torch.Tensor) else to_device(p.patches, spec.dtype, self.device)
                out[po:po + n_p].copy_(src)
            if n_t:
                ids = torch.from_numpy(p.text_ids.astype(np.int32)).to(self.device)
                self.embed_ids(ids, out[to:to + n_t])
            o += p.length
        return out, lens

    def close(self):
        if getattr(self, "handle", None):
            self.lib.ams_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class DeviceContext:
    """Per-row cached context: K/V slab + activations in one workspace."""

    def __init__(self, model: DeviceModel, batch: int, capacity: int, max_pass_tokens: int = 0,
                 n_pages: Optional[int] = None, share_prefix: bool = False):
        """n_pages / share_prefix: a paged context (ams_ctx_create_paged) with that many K/V pages per
        layer (0: a page for every position) whose rows share prefix pages when share_prefix."""
        self.lib, self.model, self.batch, self.capacity = model.lib, model, batch, capacity
        self.share_prefix = bool(share_prefix)
        paged = n_pages is not None or share_prefix
        flags = capi.AMS_CTX_SHARE_PREFIX if share_prefix else 0
        if paged:
            nbytes = self.lib.ams_ctx_workspace_bytes_paged(C.byref(model.cfg), batch, capacity, max_pass_tokens,
                                                            n_pages or 0, flags)
        else:
            nbytes = self.lib.ams_ctx_workspace_bytes(C.byref(model.cfg), batch, capacity, max_pass_tokens)
        if nbytes == 0:
            raise ValueError("invalid context arguments")
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=model.device)
        self.n_pages = n_pages or batch * (capacity // 64)
        h = C.c_void_p()
        if paged:
            capi.check(self.lib.ams_ctx_create_paged(model.handle, batch, capacity, max_pass_tokens, n_pages or 0,
                                                     flags, self.ws.data_ptr(), nbytes, C.byref(h)),
                       "ams_ctx_create_paged")
        else:
            capi.check(self.lib.ams_ctx_create(model.handle, batch, capacity, max_pass_tokens, self.ws.data_ptr(),
                                               nbytes, C.byref(h)), "ams_ctx_create")
        self.handle = h
        self._keep = []
        _live_contexts.add(self)

    def build(self, prefix: torch.Tensor, lens: Sequence[int]) -> None:
        assert prefix.is_contiguous()
        capi.check(self.lib.ams_ctx_build(self.handle, prefix.data_ptr(), capi.int_array(lens), _stream()),
                   "ams_ctx_build")

    def step(self, n_actions: int, new: Optional[torch.Tensor] = None, new_lens: Optional[Sequence[int]] = None,
             tokens: Optional[torch.Tensor] = None, logits: Optional[torch.Tensor] = None, want_logits: bool = True,
             forced: Optional[torch.Tensor] = None):
        """Returns (tokens [B, A] int32, logits [B, A, n_bins] fp32 or None) on the device."""
        B, nb = self.batch, self.model.spec.n_bins
        dev = self.model.device
        if tokens is None:
            tokens = torch.empty((B, n_actions), dtype=torch.int32, device=dev)
        if logits is None and want_logits:
            logits = torch.empty((B, n_actions, nb), dtype=torch.float32, device=dev)
        nl = capi.int_array(new_lens) if new_lens is not None else None
        capi.check(self.lib.ams_ctx_step(self.handle, new.data_ptr() if new is not None else None, nl, n_actions,
                                         tokens.data_ptr(), logits.data_ptr() if logits is not None else None,
                                         forced.data_ptr() if forced is not None else None, _stream()),
                   "ams_ctx_step")
        return tokens, logits

    def build_rows(self, rows: Sequence[int], prefix: torch.Tensor, lens: Sequence[int]) -> None:
        """Rebuild only `rows` (strictly increasing) from their new prefixes, packed in that order."""
        assert prefix.is_contiguous()
        capi.check(self.lib.ams_ctx_build_rows(self.handle, capi.int_array(rows), len(rows), prefix.data_ptr(),
                                               capi.int_array(lens), _stream()), "ams_ctx_build_rows")

    def invalidate_rows(self, rows: Sequence[int]) -> None:
        capi.check(self.lib.ams_ctx_invalidate_rows(self.handle, capi.int_array(rows), len(rows)),
                   "ams_ctx_invalidate_rows")

    def append(self, new: torch.Tensor, new_lens: Sequence[int]) -> None:
        """Commit new observation tokens without decoding actions."""
        capi.check(self.lib.ams_ctx_append(self.handle, new.data_ptr() if new is not None else None,
                                           capi.int_array(new_lens), _stream()), "ams_ctx_append")

    def invalidate(self) -> None:
        capi.check(self.lib.ams_ctx_invalidate(self.handle), "ams_ctx_invalidate")

    def pages(self):
        """(page table [batch][capacity/64], reference counts [n_pages], pages in use) as numpy / int."""
        pt = np.zeros((self.batch, self.capacity // 64), dtype=np.int32)
        refs = np.zeros(self.n_pages, dtype=np.int32)
        used = C.c_int32()
        capi.check(self.lib.ams_ctx_pages(self.handle, pt.ctypes.data, refs.ctypes.data, C.byref(used)),
                   "ams_ctx_pages")
        return pt, refs, int(used.value)

    def flow(self, head: "DeviceFlowHead", x: torch.Tensor, tau0: float, n_steps: int) -> torch.Tensor:
        """Euler-integrate every row's action latent x [batch][n_tokens][action_dim] (fp32, in place)."""
        assert x.dtype == torch.float32 and x.is_contiguous() and x.shape[0] == self.batch
        capi.check(self.lib.ams_ctx_flow(self.handle, C.byref(head.c), x.data_ptr(), C.c_float(tau0), n_steps,
                                         _stream()), "ams_ctx_flow")
        return x

    def row_host_bytes(self, length: int) -> int:
        return int(self.lib.ams_ctx_row_host_bytes(self.handle, length))

    def offload_rows(self, rows: Sequence[int], host: Sequence[torch.Tensor]) -> None:
        """Move rows' contexts into pinned host tensors (torch pin_memory, >= row_host_bytes)."""
        ptrs = (C.c_void_p * len(rows))(*[h.data_ptr() for h in host])
        capi.check(self.lib.ams_ctx_offload_rows(self.handle, capi.int_array(rows), len(rows), ptrs, _stream()),
                   "ams_ctx_offload_rows")

    def reload_rows(self, rows: Sequence[int], host: Sequence[torch.Tensor]) -> None:
        ptrs = (C.c_void_p * len(rows))(*[h.data_ptr() for h in host])
        capi.check(self.lib.ams_ctx_reload_rows(self.handle, capi.int_array(rows), len(rows), ptrs, _stream()),
                   "ams_ctx_reload_rows")

    def row_states(self) -> List[int]:
        arr = (C.c_int32 * self.batch)()
        capi.check(self.lib.ams_ctx_row_states(self.handle, arr), "ams_ctx_row_states")
        return list(arr)

    def lengths(self) -> List[int]:
        arr = (C.c_int32 * self.batch)()
        capi.check(self.lib.ams_ctx_lengths(self.handle, arr), "ams_ctx_lengths")
        return list(arr)

    @property
    def state(self) -> int:
        return self.lib.ams_ctx_state(self.handle)

    @property
    def persistent_decode(self) -> bool:
        """True when a step's action decode runs as one persistent launch."""
        return self.lib.ams_ctx_persistent_decode(self.handle) == 1

    def close(self):
        if getattr(self, "handle", None):
            self.lib.ams_ctx_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def index_hash(data: torch.Tensor, seg_bytes: int, ws: Optional[torch.Tensor] = None,
               out: Optional[torch.Tensor] = None):
    """Two-phase hash (ams_index_hash) of a contiguous device tensor's bytes.  Returns
    (out [1] int64 tensor holding the uint64 index value, ws: the phase-1 segment hashes)."""
    lib = capi.load()
    assert data.is_cuda and data.is_contiguous()
    n = data.numel() * data.element_size()
    need = lib.ams_index_hash_workspace_bytes(n, seg_bytes)
    if need == 0:
        raise ValueError("invalid index hash sizes")
    if ws is None:
        ws = torch.empty(need // 8, dtype=torch.int64, device=data.device)
    if out is None:
        out = torch.empty(1, dtype=torch.int64, device=data.device)
    capi.check(lib.ams_index_hash(data.data_ptr(), n, seg_bytes, ws.data_ptr(), ws.numel() * 8, out.data_ptr(),
                                  _stream()), "ams_index_hash")
    return out, ws


class DeviceFlowHead:
    """A flow-matching action head's weights on the device (model dtype): w_in [d][a], w_t [d],
    w_out [a][d], from encoded numpy arrays."""

    def __init__(self, spec, w_in: np.ndarray, w_t: np.ndarray, w_out: np.ndarray, n_tokens: int, device="cuda"):
        self.t = [to_device(w, spec.dtype, device) for w in (w_in, w_t, w_out)]
        a = w_in.shape[1]
        self.c = capi.FlowHead(self.t[0].data_ptr(), self.t[1].data_ptr(), self.t[2].data_ptr(), a, n_tokens)
        self.action_dim, self.n_tokens = a, n_tokens
