"""ctypes declarations of ``include/ams.h`` (argument marshalling only).

``load()`` returns the loaded ``libams.so`` with every function typed.  It
raises if the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libams.so")

AMS_OK, AMS_EINVAL, AMS_ESTATE, AMS_ECAPACITY, AMS_ENODEV, AMS_EHIP, AMS_ENOMEM = 0, -1, -2, -3, -4, -5, -6
AMS_F32, AMS_BF16 = 0, 1
AMS_CTX_SHARE_PREFIX = 1
STATE_EMPTY, STATE_READY, STATE_INVALID, STATE_OFFLOADED = 0, 1, 2, 3


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("head_dim", C.c_int32), ("d_ffn", C.c_int32), ("vocab", C.c_int32),
                ("n_bins", C.c_int32), ("rms_eps", C.c_float), ("rope_theta", C.c_float),
                ("dtype", C.c_int32)]


class Weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down",
                                          "g_attn", "g_ffn", "g_final", "embed", "head_bins")]


class FlowHead(C.Structure):
    _fields_ = [("w_in", C.c_void_p), ("w_t", C.c_void_p), ("w_out", C.c_void_p), ("action_dim", C.c_int32),
                ("n_tokens", C.c_int32)]


# name -> (restype, argtypes)
SIGNATURES = {
    "ams_status_str": (C.c_char_p, [C.c_int32]),
    "ams_last_error": (C.c_char_p, []),
    "ams_device_count": (C.c_int32, []),
    "ams_model_workspace_bytes": (C.c_size_t, [C.POINTER(ModelCfg)]),
    "ams_model_create": (C.c_int32, [C.POINTER(ModelCfg), C.POINTER(Weights), C.c_void_p, C.c_size_t,
                                     C.c_void_p, C.POINTER(C.c_void_p)]),
    "ams_model_destroy": (None, [C.c_void_p]),
    "ams_embed_ids": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p]),
    "ams_index_hash_workspace_bytes": (C.c_size_t, [C.c_size_t, C.c_int32]),
    "ams_index_hash": (C.c_int32, [C.c_void_p, C.c_size_t, C.c_int32, C.c_void_p, C.c_size_t, C.c_void_p,
                                   C.c_void_p]),
    "ams_index_hash_noalloc": (C.c_int32, [C.c_void_p, C.c_size_t, C.c_int32, C.c_void_p, C.c_void_p]),
    "ams_ctx_workspace_bytes": (C.c_size_t, [C.POINTER(ModelCfg), C.c_int32, C.c_int32, C.c_int32]),
    "ams_ctx_create": (C.c_int32, [C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_size_t,
                                   C.POINTER(C.c_void_p)]),
    "ams_ctx_destroy": (None, [C.c_void_p]),
    "ams_ctx_workspace_bytes_paged": (C.c_size_t, [C.POINTER(ModelCfg), C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                                   C.c_int32]),
    "ams_ctx_create_paged": (C.c_int32, [C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                         C.c_void_p, C.c_size_t, C.POINTER(C.c_void_p)]),
    "ams_ctx_pages": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_void_p, C.POINTER(C.c_int32)]),
    "ams_ctx_build": (C.c_int32, [C.c_void_p, C.c_void_p, C.POINTER(C.c_int32), C.c_void_p]),
    "ams_ctx_step": (C.c_int32, [C.c_void_p, C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.c_void_p,
                                 C.c_void_p, C.c_void_p, C.c_void_p]),
    "ams_ctx_invalidate": (C.c_int32, [C.c_void_p]),
    "ams_ctx_row_host_bytes": (C.c_size_t, [C.c_void_p, C.c_int32]),
    "ams_ctx_offload_rows": (C.c_int32, [C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.POINTER(C.c_void_p),
                                         C.c_void_p]),
    "ams_ctx_reload_rows": (C.c_int32, [C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.POINTER(C.c_void_p),
                                        C.c_void_p]),
    "ams_ctx_row_states": (C.c_int32, [C.c_void_p, C.POINTER(C.c_int32)]),
    "ams_ctx_flow": (C.c_int32, [C.c_void_p, C.POINTER(FlowHead), C.c_void_p, C.c_float, C.c_int32, C.c_void_p]),
    "ams_tier_plan": (C.c_int32, [C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                  C.c_int64, C.c_void_p, C.POINTER(C.c_int64)]),
    "ams_ctx_build_rows": (C.c_int32, [C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.c_void_p,
                                       C.POINTER(C.c_int32), C.c_void_p]),
    "ams_ctx_invalidate_rows": (C.c_int32, [C.c_void_p, C.POINTER(C.c_int32), C.c_int32]),
    "ams_ctx_append": (C.c_int32, [C.c_void_p, C.c_void_p, C.POINTER(C.c_int32), C.c_void_p]),
    "ams_ctx_lengths": (C.c_int32, [C.c_void_p, C.POINTER(C.c_int32)]),
    "ams_ctx_state": (C.c_int32, [C.c_void_p]),
    "ams_ctx_persistent_decode": (C.c_int32, [C.c_void_p]),
}

_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2508_10259_amd.build`")
    lib = C.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


class AmsError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = load()
        self.status = status
        super().__init__(f"{where}: {lib.ams_status_str(status).decode()}: {lib.ams_last_error().decode()}")


def check(status: int, where: str) -> None:
    if status != AMS_OK:
        raise AmsError(status, where)


def int_array(values) -> C.Array:
    vals = [int(v) for v in values]
    return (C.c_int32 * len(vals))(*vals)
