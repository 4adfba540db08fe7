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


def _frag(Wt):
    """MFMA fragment order of W [N][K]: 16-row strip s, 128-column chunk c and 32-column
    step i form one block of 64 lanes x 8 values, lane l holding row 16 s + l % 16 and
    columns 128 c + 32 i + 8 (l / 16) .. + 8 (the layout the wide decode GEMM and the
    persistent decode read)."""
    N, K = Wt.shape
    return np.ascontiguousarray(Wt.reshape(N // 16, 16, K // 128, 4, 4, 8).transpose(0, 2, 3, 4, 1, 5)).reshape(N, K)


def _pair(x):
    """fp16 pair of x: hi = fp16(x), lo = fp16(x - hi)."""
    hi = x.astype(np.float16)
    return hi, (x.astype(np.float64) - hi.astype(np.float64)).astype(np.float16)


def _ptr(t):
    return C.c_void_p(t.data_ptr() if t is not None else None)


@pytest.mark.parametrize("dtype", ["f16", "f32"])
@pytest.mark.parametrize("epi", [EPI_STORE, EPI_RESID, EPI_SWIGLU])
@pytest.mark.parametrize("M", [1, 3, 8, 9, 16, 17, 40, 64, 65, 130, 257])
@pytest.mark.parametrize("K", [384, 1024])
@pytest.mark.parametrize("pair", [False, True])
def test_gemm(probe, dtype, epi, M, K, pair):
    """GEMM with each epilogue against the exact product of its inputs.  `pair`: the fp16 decode
    GEMV form, whose input is hi + lo (lo = the rounding error of hi) and whose residual / SwiGLU
    outputs also come as fp16 pairs."""
    import torch
    if pair and (dtype != "f16" or M > 64):
        pytest.skip("fp16 pairs belong to the fp16 decode GEMV (M <= 64)")
    N = 256
    log(f"gemm dtype={dtype} epi={epi} M={M} N={N} K={K} pair={pair}")
    x = W.random_gaussian((M, K), 1, M, K, dtype="f32")
    if pair:
        u, ulo = _pair(x)
        xin = u.astype(np.float64) + ulo.astype(np.float64)
    else:
        u, ulo = (x.astype(np.float16) if dtype == "f16" else x), None
        xin = _f(u, dtype)
    Wt = _rand((N, K), 2, N, K, dtype=dtype, std=0.05)
    ud, Wd = _dev(u, dtype), _dev(Wt, dtype)
    ulod = _dev(ulo, dtype) if pair else None
    y = xin @ _f(Wt, dtype).T
    if epi == EPI_SWIGLU:
        out = torch.zeros((M, N // 2), dtype=torch.float32 if dtype == "f32" else torch.float16, device="cuda")
        ldo = N // 2
    else:
        h0 = W.random_gaussian((M, N), 3, M, dtype="f32")
        out = torch.from_numpy(h0.copy() if epi == EPI_RESID else np.zeros_like(h0)).cuda()
        ldo = N
    # fp16 outputs beside the residual rows (and the rounding error of SwiGLU's fp16 output)
    with16 = epi == EPI_RESID and dtype == "f16" and M <= 64
    o16 = torch.full((M, N), 7.0, dtype=torch.float16, device="cuda") if with16 else None
    olo = None
    if pair and epi == EPI_RESID:
        olo = torch.full((M, N), 7.0, dtype=torch.float16, device="cuda")
    elif pair and epi == EPI_SWIGLU:
        olo = torch.full((M, N // 2), 7.0, dtype=torch.float16, device="cuda")
    rc = probe.ams_probe_gemm(CT[dtype], epi, _ptr(ud), _ptr(ulod), _ptr(Wd), M, N, K, _ptr(out), ldo, _ptr(o16),
                              _ptr(olo), _stream())
    assert rc == 0
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    if with16:
        assert torch.equal(o16, out.half()), "fp16 residual copy differs from the fp32 rows"
        if pair:
            assert torch.equal(olo, (out - out.half().float()).half()), "lo part is not the rounding error"
    elif not pair and (dtype == "f32" or epi != EPI_RESID or M > 64):
        # any other configuration rejects the fp16 copy before launching
        spare = torch.empty((M, N), dtype=torch.float16, device="cuda")
        assert probe.ams_probe_gemm(CT[dtype], epi, _ptr(ud), C.c_void_p(None), _ptr(Wd), M, N, K, _ptr(out), ldo,
                                    _ptr(spare), C.c_void_p(None), _stream()) != 0
    if epi == EPI_STORE:
        ref = y
    elif epi == EPI_RESID:
        ref = h0.astype(np.float64) + y
    else:
        g, up = _unpack_gu(y.T, N // 2)
        ref = (_silu(g) * up).T
        if pair:  # the SwiGLU value as the fp16 pair carries it
            got = got + olo.float().cpu().numpy().astype(np.float64)
    scale = max(1.0, float(np.max(np.abs(ref))))
    tol = (1e-5 if dtype == "f32" else 2e-5) * scale * np.sqrt(K / 128)
    if epi == EPI_SWIGLU and dtype == "f16" and not pair:
        tol = max(tol, 2 ** -11 * float(np.max(np.abs(ref))))
    err = float(np.max(np.abs(got - ref)))
    assert err <= tol, f"max abs err {err:.3e} > {tol:.3e}"


@pytest.mark.parametrize("dtype", ["f16", "f32"])
@pytest.mark.parametrize("d", [384, 4096])
@pytest.mark.parametrize("pair", [False, True])
def test_rmsnorm(probe, dtype, d, pair):
    import torch
    if pair and dtype != "f16":
        pytest.skip("fp16 pairs only")
    M, eps = 5, 1e-5
    h = W.random_gaussian((M, d), 4, d, dtype="f32") * 3.0
    hd = torch.from_numpy(h).cuda()
    out = torch.empty((M, d), dtype=torch.float32 if dtype == "f32" else torch.float16, device="cuda")
    lo = torch.empty((M, d), dtype=torch.float16, device="cuda") if pair else None
    rc = probe.ams_probe_rmsnorm(CT[dtype], C.c_void_p(hd.data_ptr()), M, d, C.c_float(eps),
                                 C.c_void_p(out.data_ptr()), _ptr(lo), _stream())
    assert rc == 0
    torch.cuda.synchronize()
    h64 = h.astype(np.float64)
    ref = h64 / np.sqrt(np.mean(h64 * h64, axis=-1, keepdims=True) + eps)
    got = out.float().cpu().numpy().astype(np.float64)
    if pair:
        got = got + lo.float().cpu().numpy()
        tol = 2e-6 * np.max(np.abs(ref))
    else:
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
    h16lo = torch.full((B, d), 5.0, dtype=torch.float16, device="cuda") if dtype == "f16" else None
    ref = np.argmax(lg[:, :n_bins], axis=-1)
    assert list(ref[:3]) == [3, n_bins - 2, 0]
    for use_forced in (False, True):
        rc = probe.ams_probe_argmax_feed(CT[dtype], C.c_void_p(lgd.data_ptr()), ldl, C.c_void_p(embd.data_ptr()), B, d,
                                         n_bins, A, j, C.c_void_p(tok.data_ptr()), C.c_void_p(out.data_ptr()),
                                         C.c_void_p(forced.data_ptr() if use_forced else None),
                                         C.c_void_p(h.data_ptr()), 1,
                                         _ptr(h16), _ptr(h16lo), _stream())
        assert rc == 0
        torch.cuda.synchronize()
        assert np.array_equal(tok[:, j].cpu().numpy(), ref)
        assert np.array_equal(out[:, j].cpu().numpy(), lg[:, :n_bins])
        feed = forced[:, j].cpu().numpy().clip(0, n_bins - 1) if use_forced else ref
        assert np.array_equal(h.cpu().numpy(), _f(emb, dtype)[feed].astype(np.float32))
        if h16 is not None:  # fp16 pair of the fed row: (embedding, 0)
            assert np.array_equal(h16.cpu().numpy(), emb[feed])
            assert not h16lo.float().abs().sum().item()


@pytest.mark.parametrize("epi", [EPI_STORE, EPI_RESID, EPI_SWIGLU])
@pytest.mark.parametrize("M", [1, 5, 8, 9, 16])
@pytest.mark.parametrize("K", [256, 1024, 4096])
@pytest.mark.parametrize("pair", [False, True])
def test_gemv_rmsnorm(probe, epi, M, K, pair):
    """Fused RMSNorm GEMV on the fp16 copy x = hi of the residual rows (or the pair x = hi + lo):
    y = W x / rms(hi), the statistic taken from hi; fp16 products are exact in the fp32
    accumulator, so the bound is the accumulation (and, for plain SwiGLU, the fp16 output
    rounding)."""
    import torch
    N, eps = 256, 1e-5
    log(f"gemv_rmsnorm epi={epi} M={M} K={K} pair={pair}")
    h = W.random_gaussian((M, K), 21, M, K, dtype="f32") * 4.0
    if pair:
        hi, lo = _pair(h)
        x64 = hi.astype(np.float64) + lo.astype(np.float64)
    else:
        hi, lo = h.astype(np.float16), None
        x64 = hi.astype(np.float64)
    Wt = _rand((N, K), 23, K, dtype="f16", std=0.05)
    h64 = hi.astype(np.float64)
    rs = 1.0 / np.sqrt(np.mean(h64 * h64, axis=-1, keepdims=True) + eps)
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
    o16 = torch.zeros((M, N), dtype=torch.float16, device="cuda") if with16 else None
    olo = None
    if pair and epi != EPI_STORE:
        olo = torch.zeros(tuple(out.shape), dtype=torch.float16, device="cuda")
    hd, wd = torch.from_numpy(hi).cuda(), _dev(Wt, "f16")  # keep every input alive across the launch
    lod = torch.from_numpy(lo).cuda() if pair else None
    rc = probe.ams_probe_gemv_rmsnorm(2, epi, _ptr(hd), _ptr(lod), C.c_float(eps), _ptr(wd), M, N, K, _ptr(out), ldo,
                                      _ptr(o16), _ptr(olo), _stream())
    assert rc == 0
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    if pair and epi == EPI_SWIGLU:
        got = got + olo.float().cpu().numpy()
    scale = max(1.0, float(np.max(np.abs(ref))))
    tol = 2e-5 * scale * np.sqrt(K / 128)
    if epi == EPI_SWIGLU and not pair:
        tol = max(tol, 2 ** -11 * float(np.max(np.abs(ref))))
    err = float(np.max(np.abs(got - ref)))
    assert err <= tol, f"max abs err {err:.3e} > {tol:.3e}"
    if with16:
        assert torch.equal(o16, out.half())
        if pair:
            assert torch.equal(olo, (out - out.half().float()).half())


def _rope_tab(cap, dh, theta=10000.0):
    half = dh // 2
    ang = np.arange(cap)[:, None] * theta ** (-2.0 * np.arange(half)[None, :] / dh)
    return np.stack([np.cos(ang), np.sin(ang)], axis=-1).astype(np.float32)  # [cap][half][2]


def _to_pages(X, perm):
    """Logical K or V [B][H][cap][dh] -> a page pool [B * cap/64][H][64][dh] in which row b's
    page i (positions 64i .. 64i+63) sits at pool page perm[b * cap/64 + i]."""
    B, H, cap, dh = X.shape
    ppr = cap // 64
    pool = np.zeros((B * ppr, H, 64, dh), X.dtype)
    for b in range(B):
        for i in range(ppr):
            pool[perm[b * ppr + i]] = X[b, :, 64 * i:64 * (i + 1)]
    return pool


def _from_pages(pool, perm, B, cap):
    ppr = cap // 64
    X = np.zeros((B, pool.shape[1], cap, pool.shape[3]), pool.dtype)
    for b in range(B):
        for i in range(ppr):
            X[b, :, 64 * i:64 * (i + 1)] = pool[perm[b * ppr + i]]
    return X


def _round(x, dtype):
    return x.astype(np.float16).astype(np.float64) if dtype == "f16" else x.astype(np.float32).astype(np.float64)


@pytest.mark.parametrize("dtype,dh,cap,lens,jpos,splits", [
    ("f32", 64, 512, [300, 17], 0, 1),        # two block rounds per wave
    ("f32", 128, 512, [301, 0, 128], 2, 1),   # three rounds; an empty cached prefix
    ("f16", 64, 1024, [700, 5], 1, 1),        # two rounds of 512 keys
    ("f16", 128, 1024, [600, 63, 64, 65], 0, 1),
    ("f16", 128, 320, [294], 0, 5),           # split keys, merged
    ("f16", 64, 256, [2, 130], 0, 4),         # splits beyond a short row stay empty
    ("f32", 64, 512, [260, 3], 5, 8),
])
def test_attn_decode(probe, dtype, dh, cap, lens, jpos, splits):
    """Decode attention of one fed-back token per row against the plain definition: the
    query and the new key rotated (rotate-half RoPE), the new key and value rounded to the
    slab type and appended at p = lens[b] + jpos, softmax(K q / sqrt(dh)) V over keys 0..p.
    The rows' 64-position K/V pages sit in the pool in a random order (page table)."""
    import torch
    B, H = len(lens), 2
    d, half = H * dh, dh // 2
    log(f"attn_decode {dtype} dh={dh} cap={cap} lens={lens} jpos={jpos} splits={splits}")
    np_t = np.float16 if dtype == "f16" else np.float32
    qkv = W.random_gaussian((B, 3 * d), 31, dh, cap, dtype="f32")
    K = W.random_gaussian((B, H, cap, dh), 32, dh, cap, dtype="f32").astype(np_t)
    V = W.random_gaussian((B, H, cap, dh), 33, dh, cap, dtype="f32").astype(np_t)
    tab = _rope_tab(cap, dh)
    # the K/V pages of the rows scattered over the pool in a random order
    perm = np.random.default_rng(cap + dh).permutation(B * (cap // 64)).astype(np.int32)
    pt_d = torch.from_numpy(perm).cuda()
    qkv_d, K_d, V_d = _dev(qkv, dtype), _dev(_to_pages(K, perm), dtype), _dev(_to_pages(V, perm), dtype)
    tab_d = _dev(tab, "f32")
    lens_d = torch.tensor(lens, dtype=torch.int32, device="cuda")
    part = torch.zeros((B * H * (cap // 64) * (dh + 2),), dtype=torch.float32, device="cuda")
    o = torch.zeros((B, d), dtype=torch.float16 if dtype == "f16" else torch.float32, device="cuda")
    olo = torch.zeros((B, d), dtype=torch.float16, device="cuda") if dtype == "f16" else None  # rounding error of o
    # the rows dispatched longest first, as the engine orders them (ranks by decreasing length,
    # ties by row index); the output does not depend on the order
    order = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    assert probe.ams_probe_len_order(_ptr(lens_d), B, _ptr(order), _stream()) == 0
    torch.cuda.synchronize()
    assert order.cpu().numpy().tolist() == sorted(range(B), key=lambda b: (-lens[b], b))
    rc = probe.ams_probe_attn_decode(CT[dtype], C.c_void_p(qkv_d.data_ptr()), C.c_void_p(lens_d.data_ptr()), jpos,
                                     B, H, dh, cap, _ptr(pt_d), splits, C.c_void_p(tab_d.data_ptr()),
                                     C.c_void_p(K_d.data_ptr()),
                                     C.c_void_p(V_d.data_ptr()), C.c_void_p(part.data_ptr()),
                                     C.c_void_p(o.data_ptr()), _ptr(olo), _ptr(order), _stream())
    assert rc == 0
    torch.cuda.synchronize()
    got = o.float().cpu().numpy().astype(np.float64)
    if olo is not None:  # the output as the fp16 pair carries it
        got = got + olo.float().cpu().numpy()
    K_after = _from_pages(K_d.cpu().numpy(), perm, B, cap)
    V_after = _from_pages(V_d.cpu().numpy(), perm, B, cap)
    for b in range(B):
        p = lens[b] + jpos
        cs = tab[p].astype(np.float64)  # [half][2]
        for h in range(H):
            x = qkv[b].astype(np.float64)
            q, k, v = (x[j * d + h * dh:j * d + (h + 1) * dh] for j in range(3))
            rot = lambda z: np.concatenate([z[:half] * cs[:, 0] - z[half:] * cs[:, 1],
                                            z[:half] * cs[:, 1] + z[half:] * cs[:, 0]])
            # the kernel appended the new token's K/V at p; it rotates in fp32, so the stored key
            # is the rounded exact rotation up to fp32 rounding of the two products (bounded by
            # their magnitudes, as they may cancel) plus one unit of the slab type
            ulp = 2.0 ** -10 if dtype == "f16" else 2.0 ** -23
            k_st, v_st = K_after[b, h, p].astype(np.float64), V_after[b, h, p].astype(np.float64)
            k_def = rot(k)
            ak, ac, asn = np.abs(k), np.abs(cs[:, 0]), np.abs(cs[:, 1])
            terms = np.concatenate([ak[:half] * ac + ak[half:] * asn, ak[:half] * asn + ak[half:] * ac])
            assert np.all(np.abs(k_st - k_def) <= ulp * np.abs(k_def) + 2.0 ** -22 * terms)
            assert np.array_equal(v_st, _round(v, dtype))
            k_new, v_new = k_st, v_st
            Kc = np.concatenate([K[b, h, :p].astype(np.float64), k_new[None]])
            Vc = np.concatenate([V[b, h, :p].astype(np.float64), v_new[None]])
            s = Kc @ (rot(q) / np.sqrt(dh))
            w = np.exp(s - s.max())
            ref = (w / w.sum()) @ Vc
            g = got[b, h * dh:(h + 1) * dh]
            tol = 5e-6 * np.max(np.abs(ref)) + 1e-6
            assert np.all(np.abs(g - ref) <= tol), (b, h, float(np.max(np.abs(g - ref))))
    mask = np.ones(K.shape[:3], bool)
    for b in range(B):
        mask[b, :, lens[b] + jpos] = False
    assert np.array_equal(K_after[mask], K[mask]) and np.array_equal(V_after[mask], V[mask])


@pytest.mark.parametrize("dh,segs", [
    (128, [(0, 300, 16), (1, 0, 5), (2, 470, 1), (3, 37, 16)]),   # extension-sized: keys split over waves
    (64, [(0, 280, 16), (1, 0, 16), (2, 129, 3)]),
    (128, [(0, 60, 17), (1, 0, 40), (2, 200, 70)]),               # longer segments: 64-query tiles
    (64, [(1, 33, 100), (0, 0, 1)]),
])
def test_attn_prefill(probe, dh, segs):
    """Causal attention of packed segments (row b, first position p0, n tokens) over keys
    0..p0+n-1 of each row's slab, fp16: q rotated (rotate-half RoPE) and scaled, against
    softmax(K q) V in float64 on the same fp16 slab values."""
    import torch
    B, H, cap = 4, 2, 512
    d, half = H * dh, dh // 2
    log(f"attn_prefill dh={dh} segs={segs}")
    n_tok = sum(n for _, _, n in segs)
    qkv = W.random_gaussian((n_tok, 3 * d), 71, dh, n_tok, dtype="f32")
    K = W.random_gaussian((B, H, cap, dh), 72, dh, dtype="f32").astype(np.float16)
    V = W.random_gaussian((B, H, cap, dh), 73, dh, dtype="f32").astype(np.float16)
    tab = _rope_tab(cap, dh)
    off = np.cumsum([0] + [n for _, _, n in segs]).astype(np.int32)
    perm = np.random.default_rng(dh + n_tok).permutation(B * (cap // 64)).astype(np.int32)
    pt_d = torch.from_numpy(perm).cuda()
    rows = torch.tensor([b for b, _, _ in segs], dtype=torch.int32, device="cuda")
    pos = torch.tensor([p for _, p, _ in segs], dtype=torch.int32, device="cuda")
    offd = torch.from_numpy(off).cuda()
    qkv_d, tab_d = _dev(qkv, "f32"), _dev(tab, "f32")
    K_d, V_d = _dev(_to_pages(K, perm), "f16"), _dev(_to_pages(V, perm), "f16")
    o = torch.full((n_tok, d), float("nan"), dtype=torch.float16, device="cuda")
    max_len = max(n for _, _, n in segs)
    max_end = max(p + n for _, p, n in segs)
    rc = probe.ams_probe_attn_prefill(CT["f16"], _ptr(qkv_d), _ptr(rows), _ptr(pos), _ptr(offd), len(segs), n_tok,
                                      max_len, max_end, H, dh, cap, _ptr(pt_d), _ptr(tab_d), _ptr(K_d), _ptr(V_d),
                                      _ptr(o),
                                      _stream())
    assert rc == 0
    torch.cuda.synchronize()
    got = o.float().cpu().numpy().astype(np.float64)
    for si, (b, p0, n) in enumerate(segs):
        for i in range(n):
            t, p = off[si] + i, p0 + i
            cs = tab[p].astype(np.float64)
            for h in range(H):
                q = qkv[t, h * dh:(h + 1) * dh].astype(np.float64)
                qr = np.concatenate([q[:half] * cs[:, 0] - q[half:] * cs[:, 1],
                                     q[:half] * cs[:, 1] + q[half:] * cs[:, 0]]) / np.sqrt(dh)
                qr = qr.astype(np.float16).astype(np.float64)  # the MFMA input is fp16
                s_ = K[b, h, :p + 1].astype(np.float64) @ qr
                w = np.exp(s_ - s_.max())
                ref = (w / w.sum()) @ V[b, h, :p + 1].astype(np.float64)
                # P enters P.V in fp16 (relative 2^-11), the output is fp16
                tol = 2e-3 * np.max(np.abs(V[b, h, :p + 1])) + 1e-3 * np.max(np.abs(ref))
                err = float(np.max(np.abs(got[t, h * dh:(h + 1) * dh] - ref)))
                assert err <= tol, (si, i, h, err, tol)



@pytest.mark.parametrize("dh,segs", [
    (128, [(0, 300, 16), (1, 0, 5), (2, 470, 1), (0, 316, 16)]),
    (64, [(0, 280, 16), (1, 0, 16), (2, 129, 3)]),
    (128, [(1, 60, 40), (2, 200, 70), (0, 1000, 24)]),
])
def test_kv_append_tab(probe, dh, segs):
    """The fp16 K/V append from a pass's token tables against k_kv_append on the same inputs:
    v bitwise, k within one fp16 unit (the same rotation, possibly contracted differently),
    every other slot of the page pools untouched."""
    import torch
    B, cap, d = 3, 1024, 512
    H = d // dh
    log(f"kv_append_tab dh={dh} segs={segs}")
    n_tok = sum(n for _, _, n in segs)
    off = np.cumsum([0] + [n for _, _, n in segs]).astype(np.int32)
    qkv = W.random_gaussian((n_tok, 3 * d), 85, n_tok, dh, dtype="f32")
    tab = _rope_tab(cap, dh)
    perm = np.random.default_rng(86 + dh).permutation(B * (cap // 64)).astype(np.int32)
    pt_d = torch.from_numpy(perm).cuda()
    rows = torch.tensor([b for b, _, _ in segs], dtype=torch.int32, device="cuda")
    pos = torch.tensor([p for _, p, _ in segs], dtype=torch.int32, device="cuda")
    offd = torch.from_numpy(off).cuda()
    qkv_d, tab_d = _dev(qkv, "f32"), _dev(tab, "f32")
    pool = W.random_gaussian((B * (cap // 64) * H * 64 * dh,), 87, dh, dtype="f32").astype(np.float16)
    KA, VA, KB, VB = (_dev(pool, "f16") for _ in range(4))
    tb = torch.zeros((n_tok,), dtype=torch.int64, device="cuda")
    tp = torch.zeros((n_tok,), dtype=torch.int32, device="cuda")
    max_len = max(n for _, _, n in segs)
    max_end = max(p + n for _, p, n in segs)
    assert probe.ams_probe_kv_append(CT["f16"], _ptr(qkv_d), _ptr(rows), _ptr(pos), _ptr(offd), len(segs), n_tok,
                                     max_len, max_end, H, dh, cap, _ptr(pt_d), _ptr(tab_d), _ptr(KA), _ptr(VA),
                                     _stream()) == 0
    assert probe.ams_probe_kv_append_tab(_ptr(qkv_d), _ptr(rows), _ptr(pos), _ptr(offd), len(segs), n_tok, H, dh,
                                         cap, _ptr(pt_d), _ptr(tab_d), _ptr(KB), _ptr(VB), _ptr(tb), _ptr(tp),
                                         _stream()) == 0
    torch.cuda.synchronize()
    assert torch.equal(VA, VB)
    ka, kb = KA.float().cpu().numpy(), KB.float().cpu().numpy()
    ulp = np.spacing(np.maximum(np.abs(ka), np.abs(kb)).astype(np.float16)).astype(np.float32)
    assert bool(np.all(np.abs(ka - kb) <= ulp))
    # the appended slots changed, the rest of the pools did not
    assert not torch.equal(KA, _dev(pool, "f16"))
    changed = (KB.cpu().numpy() != pool) | (VB.cpu().numpy() != pool)
    assert int(changed.sum()) <= 2 * n_tok * d

@pytest.mark.parametrize("dh,segs", [
    (128, [(0, 0, 200), (1, 37, 60), (2, 500, 41)]),
    (64, [(2, 63, 130), (0, 0, 1), (1, 250, 128)]),
])
def test_gemm_qkv_kv(probe, dh, segs):
    """The QKV projection with the K/V append in its epilogue: q columns bitwise those of the
    256 x 256-tile GEMM, v bitwise and k within one fp16 unit of what k_kv_append writes from
    that GEMM's output (the same rotation, possibly contracted differently), every other slot
    of the page pools untouched; sampled k and v against the fp64 product rotated by RoPE."""
    import torch
    B, cap, d = 3, 1024, 512
    H, half = d // dh, dh // 2
    log(f"gemm_qkv_kv dh={dh} segs={segs}")
    n_tok = sum(n for _, _, n in segs)
    off = np.cumsum([0] + [n for _, _, n in segs]).astype(np.int32)
    u = _rand((n_tok, d), 81, n_tok, dh)
    Wt = _rand((3 * d, d), 82, d, dh, std=0.05)
    tab = _rope_tab(cap, dh)
    perm = np.random.default_rng(83 + dh).permutation(B * (cap // 64)).astype(np.int32)
    pt_d = torch.from_numpy(perm).cuda()
    rows = torch.tensor([b for b, _, _ in segs], dtype=torch.int32, device="cuda")
    pos = torch.tensor([p for _, p, _ in segs], dtype=torch.int32, device="cuda")
    offd = torch.from_numpy(off).cuda()
    ud, Wd, tab_d = _dev(u, "f16"), _dev(Wt, "f16"), _dev(tab, "f32")
    pool = W.random_gaussian((B * (cap // 64) * H * 64 * dh,), 84, dh, dtype="f32").astype(np.float16)
    KA, VA, KB, VB = (_dev(pool, "f16") for _ in range(4))
    qa = torch.zeros((n_tok, 3 * d), dtype=torch.float32, device="cuda")
    qb = torch.zeros_like(qa)
    tb = torch.zeros((n_tok,), dtype=torch.int64, device="cuda")
    tp = torch.zeros((n_tok,), dtype=torch.int32, device="cuda")
    assert probe.ams_probe_qkv_kv(_ptr(ud), _ptr(Wd), d, _ptr(qa), _ptr(rows), _ptr(pos), _ptr(offd), len(segs), n_tok,
                                  H, dh, cap, _ptr(pt_d), _ptr(tab_d), _ptr(KA), _ptr(VA), _ptr(tb), _ptr(tp),
                                  _stream()) == 0
    assert probe.ams_probe_gemm_big(EPI_STORE, _ptr(ud), _ptr(Wd), n_tok, 3 * d, d, _ptr(qb), 3 * d, 256,
                                    _stream()) == 0
    max_len, max_end = max(n for _, _, n in segs), max(p + n for _, p, n in segs)
    assert probe.ams_probe_kv_append(CT["f16"], _ptr(qb), _ptr(rows), _ptr(pos), _ptr(offd), len(segs), n_tok,
                                     max_len, max_end, H, dh, cap, _ptr(pt_d), _ptr(tab_d), _ptr(KB), _ptr(VB),
                                     _stream()) == 0
    torch.cuda.synchronize()
    assert torch.equal(qa[:, :d], qb[:, :d])
    assert torch.equal(VA, VB)
    ka, kb_ = KA.cpu().numpy(), KB.cpu().numpy()
    diff = np.abs(ka.astype(np.float64) - kb_.astype(np.float64))
    ulp = np.abs(np.spacing(kb_.astype(np.float16))).astype(np.float64)
    assert bool(np.all(diff <= ulp)), float(np.max(diff / ulp))
    # sampled tokens against the definition
    Kp = _from_pages(ka.reshape(-1, H, 64, dh), perm, B, cap)
    Vp = _from_pages(VA.cpu().numpy().reshape(-1, H, 64, dh), perm, B, cap)
    uf, wf = _f(u, "f16"), _f(Wt, "f16")
    for si, (b, p0, n) in enumerate(segs):
        for i in sorted({0, n // 2, n - 1}):
            t, p = off[si] + i, p0 + i
            y = uf[t] @ wf.T
            cs = tab[p].astype(np.float64)
            for h in range(H):
                k = y[d + h * dh:d + (h + 1) * dh]
                kr = np.concatenate([k[:half] * cs[:, 0] - k[half:] * cs[:, 1], k[:half] * cs[:, 1] + k[half:] * cs[:, 0]])
                v = y[2 * d + h * dh:2 * d + (h + 1) * dh]
                tol = 2.0 ** -10 * np.abs(kr) + 1e-5 * max(1.0, float(np.max(np.abs(y))))
                assert bool(np.all(np.abs(Kp[b, h, p].astype(np.float64) - kr) <= tol)), (si, i, h)
                tol = 2.0 ** -10 * np.abs(v) + 1e-5 * max(1.0, float(np.max(np.abs(y))))
                assert bool(np.all(np.abs(Vp[b, h, p].astype(np.float64) - v) <= tol)), (si, i, h)


def test_qkv_fusable(probe):
    """The fused K/V append rides on the 256 x 256-tile QKV GEMM only: the 7B build's 19,712
    tokens take it, the 1,024-token extension (256 x 192 tiles) and a one-row build (128 x 128
    tiles) do not, nor head dims other than 64 and 128."""
    assert probe.ams_probe_qkv_fusable(19712, 12288, 128, 4096) == 1
    assert probe.ams_probe_qkv_fusable(1024, 12288, 128, 4096) == 0
    assert probe.ams_probe_qkv_fusable(288, 12288, 128, 4096) == 0
    assert probe.ams_probe_qkv_fusable(19712, 12288, 96, 4096) == 0


@pytest.mark.parametrize("M,N,K,splits", [(1024, 512, 1024, 4), (300, 256, 704, 3), (65, 768, 384, 6)])
def test_gemm_big_part(probe, M, N, K, splits):
    """Split-K form of the 256 x 256-tile GEMM: split s holds the product over its own range
    of 64-wide K steps (s*KT/S .. (s+1)*KT/S), against the exact fp16 products."""
    import torch
    log(f"gemm_big_part M={M} N={N} K={K} splits={splits}")
    u = _rand((M, K), 44, M, K)
    Wt = _rand((N, K), 45, N, K, std=0.05)
    part = torch.full((splits * M * N,), float("nan"), dtype=torch.float32, device="cuda")
    ud, Wd = _dev(u, "f16"), _dev(Wt, "f16")
    assert probe.ams_probe_gemm_big_part(_ptr(ud), _ptr(Wd), M, N, K, splits, _ptr(part), _stream()) == 0
    torch.cuda.synchronize()
    got = part.view(splits, M, N).cpu().numpy().astype(np.float64)
    KT = K // 64
    for sp in range(splits):
        k0, k1 = sp * KT // splits * 64, (sp + 1) * KT // splits * 64
        ref = _f(u[:, k0:k1], "f16") @ _f(Wt[:, k0:k1], "f16").T
        tol = 2e-5 * max(1.0, float(np.max(np.abs(ref)))) * np.sqrt(max(k1 - k0, 64) / 64)
        assert float(np.max(np.abs(got[sp] - ref))) <= tol, sp


@pytest.mark.parametrize("epi", [EPI_STORE, EPI_RESID, EPI_SWIGLU])
@pytest.mark.parametrize("M,N,K", [(1, 256, 64), (100, 256, 384), (256, 512, 1024), (300, 256, 384),
                                   (513, 768, 1024), (300, 576, 384), (1, 192, 64)])
@pytest.mark.parametrize("bn", [256, 192, 128])
def test_gemm_big(probe, epi, M, N, K, bn):
    """The 256 x 256-tile prefill GEMM (direct-to-LDS tiles, swizzled rows) on ragged token
    counts, against the exact product of its fp16 inputs; bn = 192 / 128: its 256 x 192 tiles
    (the store epilogue, N a multiple of 192) and 256 x 128 tiles."""
    import torch
    if N % bn or (bn == 192 and epi != EPI_STORE):
        pytest.skip("256 x 192 tiles serve the store epilogue; N must be a multiple of the tile width")
    log(f"gemm_big epi={epi} M={M} N={N} K={K} bn={bn}")
    u = _rand((M, K), 41, M, K)
    Wt = _rand((N, K), 42, N, K, std=0.05)
    y = _f(u, "f16") @ _f(Wt, "f16").T
    if epi == EPI_SWIGLU:
        out = torch.zeros((M, N // 2), dtype=torch.float16, device="cuda")
        ldo = N // 2
        g, up = _unpack_gu(y.T, N // 2)
        ref = (_silu(g) * up).T
    else:
        h0 = W.random_gaussian((M, N), 43, M, dtype="f32")
        out = torch.from_numpy(h0.copy() if epi == EPI_RESID else np.zeros_like(h0)).cuda()
        ldo = N
        ref = y + (h0.astype(np.float64) if epi == EPI_RESID else 0.0)
    ud, Wd = _dev(u, "f16"), _dev(Wt, "f16")
    rc = probe.ams_probe_gemm_big(epi, _ptr(ud), _ptr(Wd), M, N, K, _ptr(out), ldo, bn, _stream())
    assert rc == 0
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    scale = max(1.0, float(np.max(np.abs(ref))))
    tol = 2e-5 * scale * np.sqrt(K / 128)
    if epi == EPI_SWIGLU:
        tol = max(tol, 2 ** -11 * float(np.max(np.abs(ref))))
    err = float(np.max(np.abs(got - ref)))
    assert err <= tol, f"max abs err {err:.3e} > {tol:.3e}"


@pytest.mark.parametrize("M,N,epi", [(2560, 4608, EPI_STORE), (2300, 4608, EPI_STORE), (1024, 22016, EPI_SWIGLU),
                                     (1000, 22016, EPI_STORE)])
def test_gemm_tile_plans(probe, M, N, epi):
    """gemm() where the 256 x 256 tiles would leave a round of the CUs partly idle: at
    2,560 / 2,300 x 4,608 both tile widths take one round (10 x 18 = 180 tiles of 256 x 256,
    10 x 24 = 240 of 256 x 192), so it takes the narrower ones; at 1,024 / 1,000 x 22,016 the
    first 64 tile columns fill one round and the remaining 22 go to 256 x 128 tiles.  Against
    the exact product (SwiGLU over the interleaved gate / up rows)."""
    import torch
    K = 128
    log(f"gemm tile plan M={M} N={N} K={K} epi={epi}")
    u = _rand((M, K), 44, M, K)
    Wt = _rand((N, K), 45, N, K, std=0.05)
    y = _f(u, "f16") @ _f(Wt, "f16").T
    if epi == EPI_SWIGLU:
        g, up = _unpack_gu(y.T, N // 2)
        ref = (_silu(g) * up).T
        out = torch.zeros((M, N // 2), dtype=torch.float16, device="cuda")
        ldo = N // 2
    else:
        ref = y
        out = torch.zeros((M, N), dtype=torch.float32, device="cuda")
        ldo = N
    rc = probe.ams_probe_gemm(CT["f16"], epi, _ptr(_dev(u, "f16")), None, _ptr(_dev(Wt, "f16")), M, N, K,
                              _ptr(out), ldo, None, None, _stream())
    assert rc == 0
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    tol = 2e-5 * max(1.0, float(np.max(np.abs(ref))))
    if epi == EPI_SWIGLU:
        tol = max(tol, 2 ** -11 * float(np.max(np.abs(ref))))
    err = float(np.max(np.abs(got - ref)))
    assert err <= tol, f"max abs err {err:.3e} > {tol:.3e}"


@pytest.mark.parametrize("M", [1, 8, 16, 40, 64])
@pytest.mark.parametrize("K,splits", [(1024, 2), (4096, 4), (4096, 8), (1152, 3)])
@pytest.mark.parametrize("pair", [False, True])
def test_gemm_split_resid(probe, M, K, splits, pair):
    """Split-K decode GEMV: per-split partial sums reduced into the residual rows (splits added in
    order), against h + x W^T; the fp16 pair of the new rows as the unsplit residual epilogue."""
    import torch
    N = 256
    log(f"gemm_part M={M} K={K} splits={splits} pair={pair}")
    x = W.random_gaussian((M, K), 51, M, K, dtype="f32")
    if pair:
        u, ulo = _pair(x)
        xin = u.astype(np.float64) + ulo.astype(np.float64)
    else:
        u, ulo = x.astype(np.float16), None
        xin = u.astype(np.float64)
    Wt = _rand((N, K), 52, N, K, std=0.05)
    h0 = W.random_gaussian((M, N), 53, M, dtype="f32")
    ud, Wd = _dev(u, "f16"), _dev(Wt, "f16")
    ulod = _dev(ulo, "f16") if pair else None
    part = torch.full((splits * M * N,), float("nan"), dtype=torch.float32, device="cuda")
    h = torch.from_numpy(h0.copy()).cuda()
    o16 = torch.zeros((M, N), dtype=torch.float16, device="cuda")
    olo = torch.zeros((M, N), dtype=torch.float16, device="cuda") if pair else None
    assert probe.ams_probe_gemm_part(_ptr(ud), _ptr(ulod), _ptr(Wd), M, N, K, splits, _ptr(part), _stream()) == 0
    assert probe.ams_probe_part_resid(_ptr(part), splits, M, N, _ptr(h), _ptr(o16), _ptr(olo), _stream()) == 0
    torch.cuda.synchronize()
    ref = h0.astype(np.float64) + xin @ _f(Wt, "f16").T
    got = h.cpu().numpy().astype(np.float64)
    tol = 2e-5 * max(1.0, float(np.max(np.abs(ref)))) * np.sqrt(K / 128)
    assert float(np.max(np.abs(got - ref))) <= tol
    # each split covers its own K range: the partials add up to the product
    psum = part.view(splits, M, N).sum(0).cpu().numpy().astype(np.float64)
    assert float(np.max(np.abs(psum - (ref - h0)))) <= tol
    assert torch.equal(o16, h.half())
    if pair:
        assert torch.equal(olo, (h - h.half().float()).half())


@pytest.mark.parametrize("M,d,splits", [(1024, 4096, 4), (7, 1024, 8), (300, 5120, 3), (5, 12288, 2),
                                         (64, 4096, 8), (33, 1024, 5), (128, 4096, 16), (96, 5120, 7)])
def test_resid_norm(probe, M, d, splits):
    """The token passes' split-K residual reduction with the next RMSNorm in one pass: h and u
    bitwise equal to part_resid followed by rmsnorm, and u within fp16 rounding of the fp64
    definition RMSNorm(h + sum of the partial sums)."""
    import torch
    eps = 1e-5
    log(f"resid_norm M={M} d={d} splits={splits}")
    part = W.random_gaussian((splits, M, d), 95, M, d, dtype="f32")
    h0 = W.random_gaussian((M, d), 96, M, d, dtype="f32")
    pd = torch.from_numpy(part.reshape(-1).copy()).cuda()
    h1, h2 = torch.from_numpy(h0.copy()).cuda(), torch.from_numpy(h0.copy()).cuda()
    u1 = torch.zeros((M, d), dtype=torch.float16, device="cuda")
    u2 = torch.zeros_like(u1)
    assert probe.ams_probe_resid_norm(_ptr(pd), splits, M, d, _ptr(h1), C.c_float(eps), _ptr(u1), _stream()) == 0
    assert probe.ams_probe_part_resid(_ptr(pd), splits, M, d, _ptr(h2), None, None, _stream()) == 0
    assert probe.ams_probe_rmsnorm(CT["f16"], _ptr(h2), M, d, C.c_float(eps), _ptr(u2), None, _stream()) == 0
    torch.cuda.synchronize()
    assert torch.equal(h1, h2) and torch.equal(u1, u2)
    hn = h0.astype(np.float64) + part.astype(np.float64).sum(axis=0)
    rs = 1.0 / np.sqrt(np.mean(hn * hn, axis=1, keepdims=True) + eps)
    ref = hn * rs
    err = np.abs(u1.float().cpu().numpy() - ref)
    # fp16 rounding of the output (half an ulp, subnormals included), the fp32 sums of the
    # splits and the residual (their terms' magnitudes times n * 2^-24), and the fp32 norm
    terms = np.abs(h0).astype(np.float64) + np.abs(part).astype(np.float64).sum(axis=0)
    bound = 2.0 ** -11 * np.abs(ref) + 2.0 ** -25 + (splits + 1) * 2.0 ** -24 * terms * rs + 1e-6 * np.abs(ref)
    assert bool(np.all(err <= bound)), float(np.max(err - bound))


@pytest.mark.parametrize("B", [1, 2, 64, 300])
def test_len_order(probe, B):
    """The decode attention's dispatch order: the rows by decreasing length, ties by row index
    (lengths drawn from a narrow range so that ties occur), a permutation of [0, B)."""
    import torch
    lens = np.random.default_rng(B).integers(200, 230, B).astype(np.int32)
    lens_d = torch.from_numpy(lens).cuda()
    order = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    assert probe.ams_probe_len_order(_ptr(lens_d), B, _ptr(order), _stream()) == 0
    torch.cuda.synchronize()
    assert order.cpu().numpy().tolist() == sorted(range(B), key=lambda b: (-int(lens[b]), b))


@pytest.mark.parametrize("qsplits,norm", [(1, True), (4, True), (8, False)])
@pytest.mark.parametrize("splits", [1, 3])
def test_attn_decode_parts(probe, qsplits, norm, splits):
    """Decode attention fed the QKV projection's split-K partial sums (and the row sums of
    squares for its RMSNorm scale) gives, bit for bit, the output and the appended K/V of the
    attention fed the reduced projection (part_store with the same scale)."""
    import torch
    B, H, dh, cap, jpos, eps = 5, 4, 128, 256, 2, 1e-5
    d = H * dh
    lens = [3, 60, 64, 130, 190]
    log(f"attn_decode_parts qsplits={qsplits} norm={norm} splits={splits}")
    pq = W.random_gaussian((qsplits, B, 3 * d), 91, qsplits, dtype="f32")
    ssv = (np.random.default_rng(92).random((B, d // 128)) * 300 + 10).astype(np.float32)
    K = W.random_gaussian((B, H, cap, dh), 93, cap, dtype="f32").astype(np.float16)
    V = W.random_gaussian((B, H, cap, dh), 94, cap, dtype="f32").astype(np.float16)
    perm = np.random.default_rng(95).permutation(B * (cap // 64)).astype(np.int32)
    pt_d = torch.from_numpy(perm).cuda()
    tab_d = _dev(_rope_tab(cap, dh), "f32")
    lens_d = torch.tensor(lens, dtype=torch.int32, device="cuda")
    pq_d = torch.from_numpy(pq.reshape(-1).copy()).cuda()
    ss_d = torch.from_numpy(ssv).cuda() if norm else None
    qkv = torch.zeros((B, 3 * d), dtype=torch.float32, device="cuda")
    if norm:
        assert probe.ams_probe_part_store_norm(_ptr(pq_d), qsplits, B, 3 * d, _ptr(qkv), _ptr(ss_d), d,
                                               C.c_float(eps), _stream()) == 0
    else:
        assert probe.ams_probe_part_store(_ptr(pq_d), qsplits, B, 3 * d, _ptr(qkv), _stream()) == 0
    res = []
    for fused in (False, True):
        K_d, V_d = _dev(_to_pages(K, perm), "f16"), _dev(_to_pages(V, perm), "f16")
        part = torch.zeros((B * H * (cap // 64) * (dh + 2),), dtype=torch.float32, device="cuda")
        o = torch.zeros((B, d), dtype=torch.float16, device="cuda")
        olo = torch.zeros_like(o)
        if fused:
            rc = probe.ams_probe_attn_decode_parts(CT["f16"], _ptr(pq_d), qsplits, _ptr(ss_d), d // 128,
                                                   C.c_float(eps), _ptr(lens_d), jpos, B, H, dh, cap, _ptr(pt_d),
                                                   splits, _ptr(tab_d), _ptr(K_d), _ptr(V_d), _ptr(part), _ptr(o),
                                                   _ptr(olo), _stream())
        else:
            rc = probe.ams_probe_attn_decode(CT["f16"], _ptr(qkv), _ptr(lens_d), jpos, B, H, dh, cap, _ptr(pt_d),
                                             splits, _ptr(tab_d), _ptr(K_d), _ptr(V_d), _ptr(part), _ptr(o),
                                             _ptr(olo), None, _stream())
        assert rc == 0
        torch.cuda.synchronize()
        res.append((o, olo, K_d, V_d))
    for x, y in zip(res[0], res[1]):
        assert torch.equal(x, y)


@pytest.mark.parametrize("M", [12, 33, 64])
@pytest.mark.parametrize("splits", [1, 3])
def test_merge_norm(probe, M, splits):
    """Wide-path reductions that carry the RMSNorm: the residual reduction leaves the
    unnormalised fp16 pair and the sums of squares per 128 columns; the projection
    reductions (store, SwiGLU) divide each row by its rms, RMSNorm(h) W^T = (h W^T) / rms(h)."""
    import torch
    d, F, eps = 512, 512, 1e-5
    Nq = 3 * d
    log(f"merge_norm M={M} splits={splits}")
    pr = W.random_gaussian((splits, M, d), 71, M, splits, dtype="f32")
    h0 = W.random_gaussian((M, d), 72, M, dtype="f32")
    part = torch.from_numpy(pr.reshape(-1).copy()).cuda()
    h = torch.from_numpy(h0.copy()).cuda()
    o16 = torch.zeros((M, d), dtype=torch.float16, device="cuda")
    olo = torch.zeros((M, d), dtype=torch.float16, device="cuda")
    ss = torch.full((M, d // 128), float("nan"), dtype=torch.float32, device="cuda")
    assert probe.ams_probe_part_resid_ss(_ptr(part), splits, M, d, _ptr(h), _ptr(o16), _ptr(olo), _ptr(ss),
                                         _stream()) == 0
    torch.cuda.synchronize()
    hn = h.cpu().numpy().astype(np.float64)
    assert float(np.max(np.abs(hn - (h0 + pr.astype(np.float64).sum(0))))) <= 1e-5
    assert torch.equal(o16, h.half()) and torch.equal(olo, (h - h.half().float()).half())
    sq = (hn ** 2).reshape(M, d // 128, 128).sum(-1)
    assert np.allclose(ss.cpu().numpy(), sq, rtol=1e-5, atol=1e-5)
    rstd = 1.0 / np.sqrt((hn ** 2).mean(1, keepdims=True) + eps)
    # store: the summed partials of a projection of the unnormalised rows, scaled by 1/rms
    pq = W.random_gaussian((splits, M, Nq), 73, M, splits, dtype="f32")
    out = torch.zeros((M, Nq), dtype=torch.float32, device="cuda")
    assert probe.ams_probe_part_store_norm(_ptr(torch.from_numpy(pq.reshape(-1).copy()).cuda()), splits, M, Nq,
                                           _ptr(out), _ptr(ss), d, C.c_float(eps), _stream()) == 0
    torch.cuda.synchronize()
    ref = pq.astype(np.float64).sum(0) * rstd
    assert float(np.max(np.abs(out.cpu().numpy() - ref))) <= 2e-5 * max(1.0, float(np.max(np.abs(ref))))
    # SwiGLU: gate and up both scaled by 1/rms before the product
    pg = W.random_gaussian((splits, M, 2 * F), 74, M, splits, dtype="f32")
    a = torch.zeros((M, F), dtype=torch.float16, device="cuda")
    alo = torch.zeros((M, F), dtype=torch.float16, device="cuda")
    pgd = torch.from_numpy(pg.reshape(-1).copy()).cuda()
    assert probe.ams_probe_part_swiglu_norm(_ptr(pgd), splits, M, 2 * F, _ptr(a), _ptr(alo), _ptr(ss), d,
                                            C.c_float(eps), _stream()) == 0
    torch.cuda.synchronize()
    y = pg.astype(np.float64).sum(0) * rstd
    gg, up = _unpack_gu(y.T, F)
    ref = (_silu(gg) * up).T
    got = a.float().cpu().numpy().astype(np.float64) + alo.float().cpu().numpy()
    assert float(np.max(np.abs(got - ref))) <= 2e-5 * max(1.0, float(np.max(np.abs(ref))))
    # shapes the scaled reductions do not take are refused
    assert probe.ams_probe_part_store_norm(_ptr(pgd), splits, M, 384, _ptr(out), _ptr(ss), d, C.c_float(eps),
                                           _stream()) != 0


@pytest.mark.parametrize("N,K", [(16, 128), (48, 384), (1024, 4096), (4096, 11008), (22016, 4096)])
def test_frag_pack(probe, N, K):
    """frag_pack moves every 16 bytes of W to the block and lane its fragment-order formula
    names (bit for bit), checked against the NumPy transposition, which the smallest case also
    checks against the formula entry by entry; shapes off the 16 x 128 grid are refused."""
    import torch
    log(f"frag_pack N={N} K={K}")
    Wt = _rand((N, K), 91, N, K)
    ref = _frag(Wt).reshape(-1)
    if N * K <= 48 * 384:
        for s in range(N // 16):
            for c in range(K // 128):
                for i in range(4):
                    for ln in range(64):
                        o = (((s * (K // 128) + c) * 4 + i) * 64 + ln) * 8
                        col = 128 * c + 32 * i + 8 * (ln // 16)
                        assert np.array_equal(ref[o:o + 8], Wt[16 * s + ln % 16, col:col + 8])
    src = _dev(Wt, "f16")
    dst = torch.full((N * K,), float("nan"), dtype=torch.float16, device="cuda")
    assert probe.ams_probe_frag_pack(_ptr(src), N, K, _ptr(dst), _stream()) == 0
    torch.cuda.synchronize()
    assert np.array_equal(dst.cpu().numpy().view(np.uint16), ref.view(np.uint16))
    assert probe.ams_probe_frag_pack(_ptr(src), N - 8, K, _ptr(dst), _stream()) != 0
    assert probe.ams_probe_frag_pack(_ptr(src), N, K - 64, _ptr(dst), _stream()) != 0


@pytest.mark.parametrize("M", [5, 17, 33, 64])
@pytest.mark.parametrize("N,K,splits", [(256, 1024, 1), (384, 4096, 8), (256, 1152, 3), (2048, 4096, 8),
                                        (1024, 5120, 8), (1152, 1408, 4), (512, 512, 4)])
@pytest.mark.parametrize("pair", [False, True])
def test_gemm_wide(probe, M, N, K, splits, pair):
    """Wide decode GEMM (128 weight rows per workgroup, LDS-staged activations, weights in
    fragment order) and its reductions: partial sums per K split, store / residual / SwiGLU epilogues, against the
    exact products of the fp16 (pair) inputs.  The splits cover 1 to 8 chunks of 128, uneven
    splits (11 chunks over 4) and chunk counts that are not multiples of the kernel's two or
    three weight chunks in flight."""
    import torch
    log(f"gemm_wide M={M} N={N} K={K} splits={splits} pair={pair}")
    x = W.random_gaussian((M, K), 61, M, K, dtype="f32")
    if pair:
        u, ulo = _pair(x)
        xin = u.astype(np.float64) + ulo.astype(np.float64)
    else:
        u, ulo = x.astype(np.float16), None
        xin = u.astype(np.float64)
    Wt = _rand((N, K), 62, N, K, std=0.05)
    y = xin @ _f(Wt, "f16").T
    ud, Wd = _dev(u, "f16"), _dev(_frag(Wt), "f16")
    ulod = _dev(ulo, "f16") if pair else None
    part = torch.full((splits * M * N,), float("nan"), dtype=torch.float32, device="cuda")
    assert probe.ams_probe_gemm_wide(_ptr(ud), _ptr(ulod), _ptr(Wd), M, N, K, splits, _ptr(part), _stream()) == 0
    tol = 2e-5 * max(1.0, float(np.max(np.abs(y)))) * np.sqrt(K / 128)
    # store
    out = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    assert probe.ams_probe_part_store(_ptr(part), splits, M, N, _ptr(out), _stream()) == 0
    torch.cuda.synchronize()
    assert float(np.max(np.abs(out.cpu().numpy() - y))) <= tol
    # residual, with the fp16 pair of the new rows
    h0 = W.random_gaussian((M, N), 63, M, dtype="f32")
    h = torch.from_numpy(h0.copy()).cuda()
    o16 = torch.zeros((M, N), dtype=torch.float16, device="cuda")
    olo = torch.zeros((M, N), dtype=torch.float16, device="cuda")
    assert probe.ams_probe_part_resid(_ptr(part), splits, M, N, _ptr(h), _ptr(o16), _ptr(olo), _stream()) == 0
    torch.cuda.synchronize()
    assert float(np.max(np.abs(h.cpu().numpy() - (h0 + y)))) <= tol
    assert torch.equal(o16, h.half()) and torch.equal(olo, (h - h.half().float()).half())
    # SwiGLU over the packed gate/up rows, fp16 pair out
    a = torch.zeros((M, N // 2), dtype=torch.float16, device="cuda")
    alo = torch.zeros((M, N // 2), dtype=torch.float16, device="cuda")
    assert probe.ams_probe_part_swiglu(_ptr(part), splits, M, N, _ptr(a), _ptr(alo), _stream()) == 0
    torch.cuda.synchronize()
    gg, up = _unpack_gu(y.T, N // 2)
    ref = (_silu(gg) * up).T
    got = a.float().cpu().numpy().astype(np.float64) + alo.float().cpu().numpy()
    assert float(np.max(np.abs(got - ref))) <= max(tol, 4e-6 * float(np.max(np.abs(ref))))


@pytest.mark.parametrize("M", [5, 33, 64])
@pytest.mark.parametrize("N,K,splits", [(256, 1024, 1), (512, 4096, 8), (1152, 1408, 4), (2048, 1024, 3),
                                        (256, 2048, 16)])
def test_gemm_wide_reduce(probe, M, N, K, splits):
    """The wide decode GEMM with its reduction fused (the last split of each 128-row tile adds
    the partial sums in split order): store, SwiGLU and residual results equal those of the
    separate reduction kernels bit for bit, the residual's sums of squares per 128 columns
    match the new rows, the RMSNorm scale from given sums of squares matches the separate
    scaled reductions (or the closed form where they do not take the shape), and the tile
    counters are back at zero, so a second call gives the same results."""
    import torch
    log(f"gemm_wide_reduce M={M} N={N} K={K} splits={splits}")
    eps = 1e-5
    x = W.random_gaussian((M, K), 81, M, K, dtype="f32")
    u, ulo = _pair(x)
    Wt = _rand((N, K), 82, N, K, std=0.05)
    ud, ulod, Wd = _dev(u, "f16"), _dev(ulo, "f16"), _dev(_frag(Wt), "f16")
    part = torch.empty((splits * M * N,), dtype=torch.float32, device="cuda")
    assert probe.ams_probe_gemm_wide(_ptr(ud), _ptr(ulod), _ptr(Wd), M, N, K, splits, _ptr(part), _stream()) == 0
    part2 = torch.empty_like(part)
    cnt = torch.zeros((N // 128,), dtype=torch.int32, device="cuda")
    ss_in = torch.from_numpy((np.random.default_rng(M + N).random((M, K // 128)) * 50 + 1).astype(np.float32)).cuda()
    f = C.c_float(eps)

    def fused(epi, out=None, olo=None, ldo=0, h=None, o16=None, olo2=None, ss_out=None, ss=None):
        assert probe.ams_probe_gemm_wide_reduce(epi, _ptr(ud), _ptr(ulod), _ptr(Wd), M, N, K, splits, _ptr(part2),
                                                _ptr(cnt), _ptr(out), _ptr(olo), ldo, _ptr(h), _ptr(o16),
                                                _ptr(olo2), _ptr(ss_out), _ptr(ss), f, _stream()) == 0
        torch.cuda.synchronize()
        assert int(cnt.abs().sum()) == 0

    # store, without and with the RMSNorm scale
    ref = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    assert probe.ams_probe_part_store(_ptr(part), splits, M, N, _ptr(ref), _stream()) == 0
    for _ in range(2):
        out = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        fused(0, out=out, ldo=N)
        assert torch.equal(out, ref)
    out = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    fused(0, out=out, ldo=N, ss=ss_in)
    rstd = 1.0 / np.sqrt(ss_in.cpu().numpy().astype(np.float64).sum(1, keepdims=True) / K + eps)
    if N % 256 == 0 and K % 256 == 0:
        ref_n = torch.zeros_like(out)
        assert probe.ams_probe_part_store_norm(_ptr(part), splits, M, N, _ptr(ref_n), _ptr(ss_in), K, f,
                                               _stream()) == 0
        torch.cuda.synchronize()
        assert torch.equal(out, ref_n)
    want = ref.cpu().numpy().astype(np.float64) * rstd
    assert float(np.max(np.abs(out.cpu().numpy() - want))) <= 1e-6 * max(1.0, float(np.max(np.abs(want))))
    # SwiGLU (fp16 pair out)
    a = torch.zeros((M, N // 2), dtype=torch.float16, device="cuda")
    alo = torch.zeros_like(a)
    assert probe.ams_probe_part_swiglu(_ptr(part), splits, M, N, _ptr(a), _ptr(alo), _stream()) == 0
    a2, alo2 = torch.full_like(a, float("nan")), torch.full_like(alo, float("nan"))
    fused(2, out=a2, olo=alo2, ldo=N // 2)
    assert torch.equal(a, a2) and torch.equal(alo, alo2)
    if (N // 2) % 256 == 0 and K % 256 == 0:
        assert probe.ams_probe_part_swiglu_norm(_ptr(part), splits, M, N, _ptr(a), _ptr(alo), _ptr(ss_in), K, f,
                                                _stream()) == 0
        fused(2, out=a2, olo=alo2, ldo=N // 2, ss=ss_in)
        assert torch.equal(a, a2) and torch.equal(alo, alo2)
    # residual with the fp16 pair and the sums of squares per 128 columns
    h0 = torch.from_numpy(W.random_gaussian((M, N), 83, M, dtype="f32")).cuda()
    h, o16, olo = h0.clone(), torch.zeros((M, N), dtype=torch.float16, device="cuda"), None
    olo = torch.zeros_like(o16)
    assert probe.ams_probe_part_resid(_ptr(part), splits, M, N, _ptr(h), _ptr(o16), _ptr(olo), _stream()) == 0
    h2, o16b, olob = h0.clone(), torch.full_like(o16, float("nan")), torch.full_like(olo, float("nan"))
    ss2 = torch.full((M, N // 128), float("nan"), dtype=torch.float32, device="cuda")
    fused(1, h=h2, o16=o16b, olo2=olob, ss_out=ss2)
    assert torch.equal(h, h2) and torch.equal(o16, o16b) and torch.equal(olo, olob)
    hn = h2.cpu().numpy().astype(np.float64)
    assert np.allclose(ss2.cpu().numpy(), (hn ** 2).reshape(M, N // 128, 128).sum(-1), rtol=1e-5, atol=1e-5)
    # shapes and arguments it does not take are refused
    bad = probe.ams_probe_gemm_wide_reduce(3, _ptr(ud), _ptr(ulod), _ptr(Wd), M, N, K, splits, _ptr(part2),
                                           _ptr(cnt), _ptr(out), None, N, None, None, None, None, None, f, _stream())
    assert bad != 0
    bad = probe.ams_probe_gemm_wide_reduce(0, _ptr(ud), _ptr(ulod), _ptr(Wd), M, N, K, splits, _ptr(part2),
                                           None, _ptr(out), None, N, None, None, None, None, None, f, _stream())
    assert bad != 0


def test_peak_kernels(probe):
    """The measured-peak kernels compute what they claim: the stream copy reproduces its
    source, the stream read's per-thread sums add up to the source's sum, and each lane of the
    MFMA loop ends with 1024 x^2 iters (8 chains x 4 elements x 32 products of x * x per MFMA);
    sizes that are not whole 16-byte vectors are refused."""
    import torch
    log("peak kernels")
    n = (64 << 20) // 4
    src = torch.from_numpy(W.random_gaussian((n,), 95, dtype="f32")).cuda()
    dst = torch.zeros_like(src)
    assert probe.ams_probe_stream_copy(_ptr(src), _ptr(dst), C.c_size_t(4 * n), 1024, _stream()) == 0
    ones = torch.ones(n, dtype=torch.float32, device="cuda")
    out = torch.full((1024 * 256,), float("nan"), dtype=torch.float32, device="cuda")
    assert probe.ams_probe_stream_read(_ptr(ones), C.c_size_t(4 * n), _ptr(out), 1024, _stream()) == 0
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    assert float(out.double().sum()) == float(n)
    for shape in (0, 1):
        for x, iters in ((1.0, 1000), (0.5, 333)):
            m = torch.full((16 * 256,), float("nan"), dtype=torch.float32, device="cuda")
            assert probe.ams_probe_mfma_loop(shape, C.c_float(x), iters, _ptr(m), 16, _stream()) == 0
            torch.cuda.synchronize()
            assert bool((m == 1024.0 * x * x * iters).all()), (shape, x, iters)
    assert probe.ams_probe_mfma_loop(2, C.c_float(1.0), 10, _ptr(m), 16, _stream()) != 0
    probe.ams_probe_mfma_loop_flops.restype = C.c_double
    assert probe.ams_probe_mfma_loop_flops(1000, 16) == 16 * 4 * 1000 * 8 * 16 * 16 * 32 * 2
    assert probe.ams_probe_stream_copy(_ptr(src), _ptr(dst), C.c_size_t(4 * n - 4), 1024, _stream()) != 0
    assert probe.ams_probe_stream_read(_ptr(ones), C.c_size_t(12), _ptr(out), 1024, _stream()) != 0
