"""Single-kernel checks through the test-only probe ABI (libams_probe.so).

Each kernel is compared element by element with its plain definition in
fp64 NumPy on the same fp16/fp32 inputs (fp16 is the compute type of
bf16-stored models): GEMM with each epilogue at token
counts on both sides of the skinny/tiled switch and ragged tile tails,
RMSNorm, the decode GEMV with RMSNorm fused, and the action head's argmax
with planted exact ties.
"""
import ctypes as C
import os

import numpy as np
import pytest

from paper_2508_10259_amd import workload as W
from gpu_util import log

pytestmark = pytest.mark.gpu

EPI_STORE, EPI_RESID, EPI_SWIGLU = 0, 1, 2


@pytest.fixture(scope="module")
def probe():
    import torch
    from paper_2508_10259_amd.build import PROBE_LIB
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(PROBE_LIB):
        pytest.fail("libams_probe.so missing: run the build first")
    lib = C.CDLL(PROBE_LIB)
    return lib


CT = {"f32": 0, "f16": 2}  # compute types of the probe ABI


def _rand(shape, *key, dtype="f16", std=1.0):
    x = W.random_gaussian(shape, *key, dtype="f32", std=std)
    return x.astype(np.float16) if dtype == "f16" else x


def _dev(x, dtype):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _f(x, dtype):
    return np.asarray(x).astype(np.float64)


def _stream():
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _silu(z):
    return z / (1.0 + np.exp(-z))


def _unpack_gu(Wp, F):
    """Inverse of the 16-row gate/up interleave used by the packed weights."""
    gate = np.empty((F,) + Wp.shape[1:], Wp.dtype)
    up = np.empty_like(gate)
    for blk in range(F // 16):
        gate[16 * blk:16 * blk + 16] = Wp[32 * blk:32 * blk + 16]
        up[16 * blk:16 * blk + 16] = Wp[32 * blk + 16:32 * blk + 32]
    return gate, up


@pytest.mark.parametrize("dtype", ["f16", "f32"])
@pytest.mark.parametrize("epi", [EPI_STORE, EPI_RESID, EPI_SWIGLU])
@pytest.mark.parametrize("M", [1, 3, 16, 17, 40, 64, 65, 130, 257])
@pytest.mark.parametrize("K", [384, 1024])
def test_gemm(probe, dtype, epi, M, K):
    import torch
    N = 256
    log(f"gemm dtype={dtype} epi={epi} M={M} N={N} K={K}")
    u = _rand((M, K), 1, M, K, dtype=dtype)
    Wt = _rand((N, K), 2, N, K, dtype=dtype, std=0.05)
    ud, Wd = _dev(u, dtype), _dev(Wt, dtype)
    y = _f(u, dtype) @ _f(Wt, dtype).T
    if epi == EPI_SWIGLU:
        out = torch.zeros((M, N // 2), dtype=torch.float32 if dtype == "f32" else torch.float16, device="cuda")
        ldo = N // 2
    else:
        h0 = W.random_gaussian((M, N), 3, M, dtype="f32")
        out = torch.from_numpy(h0.copy() if epi == EPI_RESID else np.zeros_like(h0)).cuda()
        ldo = N
    # the decode GEMV (fp16, M <= 64) can also write the fp16 copy of updated residual rows
    with16 = epi == EPI_RESID and dtype == "f16" and M <= 64
    out16 = torch.full((M, N), 7.0, dtype=torch.float16, device="cuda") if with16 else None
    rc = probe.ams_probe_gemm(CT[dtype], epi, C.c_void_p(ud.data_ptr()), C.c_void_p(Wd.data_ptr()),
                              M, N, K, C.c_void_p(out.data_ptr()), ldo,
                              C.c_void_p(out16.data_ptr() if with16 else None), _stream())
    assert rc == 0
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    if with16:
        assert torch.equal(out16, out.half()), "fp16 residual copy differs from the fp32 rows"
    elif dtype == "f32" or epi != EPI_RESID or M > 64:
        # any other configuration rejects the fp16 copy before launching
        spare = torch.empty((M, N), dtype=torch.float16, device="cuda")
        assert probe.ams_probe_gemm(CT[dtype], epi, C.c_void_p(ud.data_ptr()), C.c_void_p(Wd.data_ptr()), M, N, K,
                                    C.c_void_p(out.data_ptr()), ldo, C.c_void_p(spare.data_ptr()), _stream()) != 0
    if epi == EPI_STORE:
        ref = y
    elif epi == EPI_RESID:
        ref = h0.astype(np.float64) + y
    else:
        g, up = _unpack_gu(y.T, N // 2)
        ref = (_silu(g) * up).T
    scale = max(1.0, float(np.max(np.abs(ref))))
    tol = (1e-5 if dtype == "f32" else 2e-5) * scale * np.sqrt(K / 128)
    if epi == EPI_SWIGLU and dtype == "f16":
        tol = max(tol, 2 ** -11 * float(np.max(np.abs(ref))))
    err = float(np.max(np.abs(got - ref)))
    assert err <= tol, f"max abs err {err:.3e} > {tol:.3e}"


@pytest.mark.parametrize("dtype", ["f16", "f32"])
@pytest.mark.parametrize("d", [384, 4096])
def test_rmsnorm(probe, dtype, d):
    import torch
    M, eps = 5, 1e-5
    h = W.random_gaussian((M, d), 4, d, dtype="f32") * 3.0
    hd = torch.from_numpy(h).cuda()
    out = torch.empty((M, d), dtype=torch.float32 if dtype == "f32" else torch.float16, device="cuda")
    rc = probe.ams_probe_rmsnorm(CT[dtype], C.c_void_p(hd.data_ptr()), M, d, C.c_float(eps),
                                 C.c_void_p(out.data_ptr()), _stream())
    assert rc == 0
    torch.cuda.synchronize()
    h64 = h.astype(np.float64)
    ref = h64 / np.sqrt(np.mean(h64 * h64, axis=-1, keepdims=True) + eps)
    got = out.float().cpu().numpy()
    tol = 1e-5 * np.max(np.abs(ref)) if dtype == "f32" else 2 ** -11 * np.max(np.abs(ref))
    assert np.max(np.abs(got - ref)) <= tol


@pytest.mark.parametrize("dtype", ["f16", "f32"])
@pytest.mark.parametrize("n_bins", [256, 100])
def test_argmax_feed_ties(probe, dtype, n_bins):
    """Lowest-index argmax with exact planted ties, logits copied out, forced/clamped feed."""
    import torch
    B, d, A, j, ldl = 4, 256, 3, 1, 320
    lg = W.random_gaussian((B, ldl), 9, dtype="f32")
    lg[0, 3] = lg[0, 7] = lg[0, 90] = 10.0     # ties: lowest index 3 wins
    lg[1, n_bins - 1] = lg[1, n_bins - 2] = 9.0
    lg[2, :n_bins] = 1.5                        # all equal: bin 0
    lg[:, n_bins:] = 100.0                      # padding beyond n_bins never wins
    emb = _rand((n_bins, d), 7, n_bins, dtype=dtype)
    lgd, embd = torch.from_numpy(lg).cuda(), _dev(emb, dtype)
    tok = torch.full((B, A), -1, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, A, n_bins), dtype=torch.float32, device="cuda")
    forced = torch.tensor([[0, 5, 0], [0, n_bins + 7, 0], [0, -3, 0], [0, 2, 0]], dtype=torch.int32, device="cuda")
    h = torch.zeros((B, d), dtype=torch.float32, device="cuda")
    h16 = torch.zeros((B, d), dtype=torch.float16, device="cuda") if dtype == "f16" else None
    ref = np.argmax(lg[:, :n_bins], axis=-1)
    assert list(ref[:3]) == [3, n_bins - 2, 0]
    for use_forced in (False, True):
        rc = probe.ams_probe_argmax_feed(CT[dtype], C.c_void_p(lgd.data_ptr()), ldl, C.c_void_p(embd.data_ptr()), B, d,
                                         n_bins, A, j, C.c_void_p(tok.data_ptr()), C.c_void_p(out.data_ptr()),
                                         C.c_void_p(forced.data_ptr() if use_forced else None),
                                         C.c_void_p(h.data_ptr()), 1,
                                         C.c_void_p(h16.data_ptr() if h16 is not None else None), _stream())
        assert rc == 0
        torch.cuda.synchronize()
        assert np.array_equal(tok[:, j].cpu().numpy(), ref)
        assert np.array_equal(out[:, j].cpu().numpy(), lg[:, :n_bins])
        feed = forced[:, j].cpu().numpy().clip(0, n_bins - 1) if use_forced else ref
        assert np.array_equal(h.cpu().numpy(), _f(emb, dtype)[feed].astype(np.float32))
        if h16 is not None:
            assert np.array_equal(h16.cpu().numpy(), emb[feed])


@pytest.mark.parametrize("epi", [EPI_STORE, EPI_RESID, EPI_SWIGLU])
@pytest.mark.parametrize("M", [1, 5, 16])
@pytest.mark.parametrize("K", [256, 1024, 4096])
def test_gemv_rmsnorm(probe, epi, M, K):
    """Fused RMSNorm GEMV on the fp16 residual copy x: y = W (x / rms(x)) with the statistic
    from the same fp16 values; fp16 products are exact in the fp32 accumulator, so the bound
    is the accumulation (and, for SwiGLU, the fp16 output rounding)."""
    import torch
    N, eps = 256, 1e-5
    log(f"gemv_rmsnorm epi={epi} M={M} K={K}")
    x = (W.random_gaussian((M, K), 21, M, K, dtype="f32") * 4.0).astype(np.float16)
    Wt = _rand((N, K), 23, K, dtype="f16", std=0.05)
    x64 = x.astype(np.float64)
    rs = 1.0 / np.sqrt(np.mean(x64 * x64, axis=-1, keepdims=True) + eps)
    y = (x64 * rs) @ _f(Wt, "f16").T
    with16 = epi == EPI_RESID
    if epi == EPI_SWIGLU:
        out = torch.zeros((M, N // 2), dtype=torch.float16, device="cuda")
        ldo = N // 2
        gg, up = _unpack_gu(y.T, N // 2)
        ref = (_silu(gg) * up).T
    else:
        h0 = W.random_gaussian((M, N), 24, M, dtype="f32")
        out = torch.from_numpy(h0.copy() if epi == EPI_RESID else np.zeros_like(h0)).cuda()
        ldo = N
        ref = y + (h0 if epi == EPI_RESID else 0.0)
    out16 = torch.zeros((M, N), dtype=torch.float16, device="cuda") if with16 else None
    xd, wd = torch.from_numpy(x).cuda(), _dev(Wt, "f16")  # keep both alive across the launch
    rc = probe.ams_probe_gemv_rmsnorm(2, epi, C.c_void_p(xd.data_ptr()), C.c_float(eps), C.c_void_p(wd.data_ptr()),
                                      M, N, K, C.c_void_p(out.data_ptr()), ldo,
                                      C.c_void_p(out16.data_ptr() if with16 else None), _stream())
    assert rc == 0
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    scale = max(1.0, float(np.max(np.abs(ref))))
    tol = 2e-5 * scale * np.sqrt(K / 128)
    if epi == EPI_SWIGLU:
        tol = max(tol, 2 ** -11 * float(np.max(np.abs(ref))))
    err = float(np.max(np.abs(got - ref)))
    assert err <= tol, f"max abs err {err:.3e} > {tol:.3e}"
    if with16:
        assert torch.equal(out16, out.half())
