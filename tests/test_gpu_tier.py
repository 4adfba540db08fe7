"""The host tier through the C ABI: rows moved to pinned host memory and back (kernels writing
and reading the host images), dropped and recomputed, chosen by the eviction plan.

A row that went to host memory and came back decodes bit for bit as if it had stayed, also
when other rows took its pages meanwhile; the image's K/V are the reference's keys and values
of that row in the documented layout; a dropped and rebuilt row matches the reference."""
import numpy as np
import pytest

from paper_2508_10259_amd import workload as W
import oracle.decoder as D
import oracle.tier as T
from gpu_util import ForcedRef, Pair, compare, gpu_new_tokens, log, small_spec

pytestmark = pytest.mark.gpu

TOL = {"bf16": 3e-2, "f32": 1e-4}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _prefixes(spec, seed, lens):
    return [W.Prefix(W.make_observation(spec, seed, 0, b, n - min(4, n - 1)),
                     np.arange(min(4, n - 1), dtype=np.int32) * 5 % 40) for b, n in enumerate(lens)]


def _pinned(n):
    import torch
    return torch.empty(n, dtype=torch.uint8).pin_memory()


@pytest.mark.parametrize("dtype,B,d,H,F,paged", [
    ("bf16", 5, 256, 4, 512, False),   # persistent decode
    ("bf16", 12, 512, 8, 1536, True),  # wide decode, pooled pages reused while rows are away
    ("f32", 3, 256, 2, 512, True),
])
def test_offload_reload_roundtrip(dtype, B, d, H, F, paged):
    import torch
    from paper_2508_10259_amd import capi
    from paper_2508_10259_amd.runtime import DeviceContext
    spec = small_spec(dtype, 2, d, H, F)
    pair = Pair(spec, seed=41)
    lens = [int(x) for x in np.random.default_rng(B + d).integers(20, 180, size=B)]
    pre = _prefixes(spec, 41, lens)
    packed, plens = pair.dev.pack_prefixes(pre)
    cap = 256
    kw = dict(n_pages=B * cap // 64) if paged else {}
    ctx, twin = DeviceContext(pair.dev, B, cap, **kw), DeviceContext(pair.dev, B, cap, **kw)
    for c in (ctx, twin):
        c.build(packed, plens)
    news = [[W.make_observation(spec, 41, 10 + s, b, 1 + b % 3) for b in range(B)] for s in range(3)]
    A = 4

    def step(c, s):
        nt, nl = gpu_new_tokens(spec, news[s])
        return c.step(A, nt, nl)
    step(ctx, 0), step(twin, 0)
    away = [1, B - 1]
    lens_now = ctx.lengths()
    bufs = [_pinned(ctx.row_host_bytes(lens_now[r])) for r in away]
    ctx.offload_rows(away, bufs)
    assert [ctx.row_states()[r] for r in away] == [capi.STATE_OFFLOADED] * 2 and ctx.state == capi.STATE_INVALID
    assert all(ctx.lengths()[r] == 0 for r in away)
    with pytest.raises(capi.AmsError) as e:
        ctx.step(A)
    assert e.value.status == capi.AMS_ESTATE
    if paged:  # another row rebuilt meanwhile, longer: it takes freed pages
        ctx.invalidate_rows([0])
        twin.invalidate_rows([0])
        p0, l0 = pair.dev.pack_prefixes(_prefixes(spec, 42, [lens[0] + 60]))
        ctx.build_rows([0], p0, l0)
        twin.build_rows([0], p0, l0)
        assert ctx.pages()[2] == ctx.n_pages - 2 * (cap // 64)
    torch.cuda.synchronize()
    # the image: header, then every layer's K / V as [layer][K|V][head][len][dh]
    es = 4 if dtype == "f32" else 2
    img = bufs[0].numpy()
    L = lens_now[away[0]]
    assert img[:4].tobytes() == b"AMSR" and int(img[8:12].view(np.int32)[0]) == L
    kv = img[256:256 + 2 * spec.n_layers * L * d * es].view(np.float16 if es == 2 else np.float32)
    kv = kv.astype(np.float64).reshape(spec.n_layers, 2, H, L, d // H)
    ref_seq = np.concatenate([pair.prefixes_f64([pre[away[0]]])[0], pair.obs_f64(news[0][away[0]])])
    _, kv_ref = D.forward(pair.p, ref_seq)
    for l in range(spec.n_layers):
        for j in range(2):
            want = np.transpose(kv_ref[l][j], (1, 0, 2))  # [H][len][dh]
            err = np.max(np.abs(kv[l, j] - want))
            assert err <= (2e-2 if es == 2 else 1e-4) * max(1.0, np.max(np.abs(want))), (l, j, err)
    ctx.reload_rows(away, bufs)
    assert ctx.state == capi.STATE_READY and ctx.lengths() == twin.lengths()
    for s in (1, 2):
        t, z = step(ctx, s)
        t2, z2 = step(twin, s)
        torch.cuda.synchronize()
        assert np.array_equal(t.cpu().numpy(), t2.cpu().numpy()) and np.array_equal(z.cpu().numpy(), z2.cpu().numpy())
    log(f"roundtrip {dtype} B={B} paged={paged}: bitwise equal to the context that kept its rows")
    ctx.close()
    twin.close()


def test_tier_plan_drives_evictions():
    """Rows with priorities and last-use ticks: the plan picks the victims (the reference's plan);
    dropped rows are rebuilt from their kept inputs, offloaded rows reloaded; every row then
    matches the fp64 reference."""
    import ctypes as C
    import torch
    from paper_2508_10259_amd import capi
    from paper_2508_10259_amd.runtime import DeviceContext
    spec = small_spec("bf16", 2, 256, 4, 512)
    pair = Pair(spec, seed=43)
    B, cap = 8, 256
    lens = [int(x) for x in np.random.default_rng(43).integers(40, 190, size=B)]
    pre = _prefixes(spec, 43, lens)
    ctx = DeviceContext(pair.dev, B, cap, n_pages=B * cap // 64)
    ctx.build(*pair.dev.pack_prefixes(pre))
    prio = np.array([1, 0, 0, 2, 0, 1, 0, 2], np.int32)  # 0: cheap to recompute (vision-like)
    last = np.array([5, 9, 3, 1, 7, 2, 8, 4], np.int64)
    pages = np.full(B, cap // 64, np.int32)
    drop = (prio == 0).astype(np.int32)
    res, pin = np.ones(B, np.int32), np.zeros(B, np.int32)
    pin[6] = 1
    act = np.zeros(B, np.int32)
    freed = C.c_int64()
    lib = capi.load()
    assert lib.ams_tier_plan(B, prio.ctypes.data, last.ctypes.data, pages.ctypes.data, drop.ctypes.data,
                             res.ctypes.data, pin.ctypes.data, 14, act.ctypes.data, C.byref(freed)) == 0
    want, f = T.eviction_plan(prio.tolist(), last.tolist(), pages.tolist(), drop.astype(bool).tolist(),
                              res.astype(bool).tolist(), pin.astype(bool).tolist(), 14)
    assert act.tolist() == want and freed.value == f == 16
    dropped = [r for r in range(B) if act[r] == T.DROP]
    offl = [r for r in range(B) if act[r] == T.OFFLOAD]
    log(f"plan: drop {dropped}, offload {offl}")
    assert dropped == [1, 2, 4] and offl == [5]
    bufs = [_pinned(ctx.row_host_bytes(lens[r])) for r in offl]
    ctx.offload_rows(offl, bufs)
    ctx.invalidate_rows(dropped)
    assert ctx.pages()[2] == (B - 4) * (cap // 64)
    ctx.build_rows(dropped, *pair.dev.pack_prefixes([pre[r] for r in dropped]))
    ctx.reload_rows(offl, bufs)
    t, z = ctx.step(5)
    torch.cuda.synchronize()
    refs = [ForcedRef(pair.p, x) for x in pair.prefixes_f64(pre)]
    tc = t.cpu().numpy()
    z_ref = np.stack([refs[b].step(None, tc[b]) for b in range(B)])
    c = compare(z_ref, z.cpu().numpy(), tc, TOL["bf16"])
    log(f"after evictions: max_abs={c.max_abs:.2e} band={c.band:.3f}")
    assert c.max_abs <= TOL["bf16"] and c.band == 1.0
    ctx.close()
