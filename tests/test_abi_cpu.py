"""The C ABI on the CPU: the library loads, exports every function ``include/ams.h``
declares, and rejects bad arguments before touching a device.  The host-only
bookkeeping (state machine, pass planner, layouts) is compiled with g++ and
address/undefined-behaviour sanitizers and run."""
import ctypes as C
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ams.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2508_10259_amd import capi
    if not os.path.exists(capi.LIB_PATH):
        from paper_2508_10259_amd.build import build
        build()
    return capi.load()


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ams_[a-z_]+)\s*\(", src)))


def test_every_declared_function_is_exported(lib):
    names = header_functions()
    assert len(names) >= 15
    out = subprocess.run(["nm", "-D", "--defined-only", os.path.join(ROOT, "paper_2508_10259_amd", "libams.so")],
                         stdout=subprocess.PIPE, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (ams_\w+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    from paper_2508_10259_amd.capi import SIGNATURES
    assert sorted(SIGNATURES) == names


def _cfg(**kw):
    from paper_2508_10259_amd.capi import ModelCfg
    base = dict(n_layers=12, d_model=1024, n_heads=16, head_dim=64, d_ffn=4096, vocab=256, n_bins=256,
                rms_eps=1e-5, rope_theta=10000.0, dtype=1)
    base.update(kw)
    return ModelCfg(**base)


def test_status_strings(lib):
    assert lib.ams_status_str(0) == b"AMS_OK"
    assert lib.ams_status_str(-3) == b"AMS_ECAPACITY"
    assert lib.ams_status_str(99) == b"AMS_UNKNOWN"


def test_workspace_sizes(lib):
    c = _cfg()
    mb = lib.ams_model_workspace_bytes(C.byref(c))
    params = 12 * (4 * 1024 ** 2 + 3 * 1024 * 4096)
    # fp16 compute: row-major and fragment-ordered copies of every layer matrix
    assert params * 4 <= mb <= params * 4 + 64 * 1024 * 1024
    mb32 = lib.ams_model_workspace_bytes(C.byref(_cfg(dtype=0)))
    assert params * 4 <= mb32 <= params * 4 + 64 * 1024 * 1024
    kb = lib.ams_ctx_workspace_bytes(C.byref(c), 8, 320, 0)
    assert kb >= 12 * 2 * 8 * 320 * 1024 * 2
    assert kb % 256 == 0
    for bad in (dict(head_dim=96, n_heads=1024 // 96), dict(d_ffn=1000), dict(n_bins=0), dict(vocab=100),
                dict(rms_eps=0.0), dict(dtype=7), dict(rope_theta=1.0), dict(n_layers=0)):
        assert lib.ams_model_workspace_bytes(C.byref(_cfg(**bad))) == 0, bad
    assert lib.ams_ctx_workspace_bytes(C.byref(c), 0, 320, 0) == 0
    assert lib.ams_ctx_workspace_bytes(C.byref(c), 8, 100, 0) == 0
    assert lib.ams_ctx_workspace_bytes(C.byref(c), 8, 320, 64) == 0
    assert lib.ams_model_workspace_bytes(None) == 0


def test_invalid_arguments_rejected_before_device(lib):
    from paper_2508_10259_amd import capi
    c = _cfg()
    w = capi.Weights()
    out = C.c_void_p()
    assert lib.ams_model_create(None, C.byref(w), None, 0, None, C.byref(out)) == capi.AMS_EINVAL
    bad = _cfg(head_dim=96)
    assert lib.ams_model_create(C.byref(bad), C.byref(w), None, 0, None, C.byref(out)) == capi.AMS_EINVAL
    assert b"head_dim" in lib.ams_last_error()
    assert lib.ams_model_create(C.byref(c), C.byref(w), None, 0, None, C.byref(out)) == capi.AMS_EINVAL
    assert lib.ams_model_create(C.byref(c), C.byref(w), C.c_void_p(0x1001), 1 << 40, None,
                                C.byref(out)) == capi.AMS_EINVAL  # misaligned
    assert lib.ams_model_create(C.byref(c), C.byref(w), C.c_void_p(0x1000), 16, None,
                                C.byref(out)) == capi.AMS_ENOMEM
    assert lib.ams_model_create(C.byref(c), C.byref(w), C.c_void_p(0x1000), 1 << 40, None,
                                C.byref(out)) == capi.AMS_EINVAL  # NULL weights
    assert out.value is None
    assert lib.ams_ctx_create(None, 1, 64, 0, None, 0, C.byref(out)) == capi.AMS_EINVAL
    assert lib.ams_ctx_build(None, None, None, None) == capi.AMS_EINVAL
    assert lib.ams_ctx_step(None, None, None, 7, None, None, None, None) == capi.AMS_EINVAL
    assert lib.ams_ctx_invalidate(None) == capi.AMS_EINVAL
    assert lib.ams_ctx_lengths(None, None) == capi.AMS_EINVAL
    assert lib.ams_ctx_state(None) == capi.AMS_EINVAL
    assert lib.ams_ctx_persistent_decode(None) == capi.AMS_EINVAL
    assert lib.ams_embed_ids(None, None, 3, None, None) == capi.AMS_EINVAL
    lib.ams_ctx_destroy(None)
    lib.ams_model_destroy(None)


def test_no_device_is_reported(lib):
    from paper_2508_10259_amd import capi
    if lib.ams_device_count() > 0:
        pytest.skip("a gfx950 device is present")
    c = _cfg()
    ptrs = {n: 0x10000 for n, _ in capi.Weights._fields_}
    w = capi.Weights(**ptrs)
    out = C.c_void_p()
    st = lib.ams_model_create(C.byref(c), C.byref(w), C.c_void_p(0x100000), 1 << 40, None, C.byref(out))
    assert st == capi.AMS_ENODEV, lib.ams_last_error()
    assert out.value is None


def test_host_state_under_sanitizers(tmp_path):
    exe = str(tmp_path / "state_test")
    src = os.path.join(ROOT, "tests", "cpp", "state_test.cpp")
    inc = os.path.join(ROOT, "paper_2508_10259_amd", "csrc", "host")
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
                    "-fno-sanitize-recover=all", f"-I{inc}", src, "-o", exe], check=True)
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    assert "state_test: ok" in r.stdout


def test_index_hash_rejects_before_device(lib):
    from paper_2508_10259_amd import capi
    assert lib.ams_index_hash_workspace_bytes(100, 16) == 7 * 8
    assert lib.ams_index_hash_workspace_bytes(4096, 4096) == 8
    assert lib.ams_index_hash_workspace_bytes(4097, 4096) == 16
    for n, s in ((0, 16), (10, 8), (10, 24), (10, 65552)):
        assert lib.ams_index_hash_workspace_bytes(n, s) == 0
    out = C.c_void_p(256)
    assert lib.ams_index_hash(C.c_void_p(256), 0, 16, C.c_void_p(256), 8, out, None) == capi.AMS_EINVAL
    assert lib.ams_index_hash(C.c_void_p(256), 100, 20, C.c_void_p(256), 64, out, None) == capi.AMS_EINVAL
    assert lib.ams_index_hash(C.c_void_p(257), 100, 16, C.c_void_p(256), 64, out, None) == capi.AMS_EINVAL
    assert lib.ams_index_hash(C.c_void_p(256), 100, 16, C.c_void_p(256), 48, out, None) == capi.AMS_ENOMEM
    assert b"workspace" in lib.ams_last_error()
