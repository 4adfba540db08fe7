"""GPU path (through the C ABI) against the fp64 reference on the same seeded inputs.

Tolerances: logits max-abs 1e-4 on the fp32 path and 3e-2 on the bf16 path;
argmax agreement counted strictly (fp32) or within the logit tolerance of the
reference maximum (bf16, where several bins can be correct when the top
reference logits sit closer than the tolerance).  bf16 runs are
teacher-forced with the reference's choices so one near-tie cannot cascade.
"""
import numpy as np
import pytest

from paper_2508_10259_amd import workload as W
import oracle.decoder as D
from gpu_util import Pair, compare, gpu_new_tokens, log, small_spec

pytestmark = pytest.mark.gpu

TOL_F32, TOL_BF16 = 1e-4, 3e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _run(pair, wl_prefixes, news_per_step, n_actions, capacity, forced_from_ref, max_pass_tokens=0, seed_tag=""):
    """Builds and steps both sides; returns per-step (ref logits, gpu logits, gpu tokens)."""
    import torch
    from paper_2508_10259_amd.runtime import DeviceContext
    spec = pair.spec
    B = len(wl_prefixes)
    ref = D.ActionContext(pair.p, B)
    ref.build(pair.prefixes_f64(wl_prefixes))
    ctx = DeviceContext(pair.dev, B, capacity, max_pass_tokens)
    prefix, lens = pair.dev.pack_prefixes(wl_prefixes)
    ctx.build(prefix, lens)
    out = []
    for s, news in enumerate(news_per_step):
        log(f"{seed_tag} step {s}")
        rn = None if news is None else [None if x is None else pair.obs_f64(x) for x in news]
        t_ref, z_ref = ref.step(rn, n_actions)
        forced = torch.from_numpy(t_ref.astype(np.int32)).cuda() if forced_from_ref else None
        new_t, new_lens = gpu_new_tokens(spec, news) if news is not None else (None, None)
        t_gpu, z_gpu = ctx.step(n_actions, new_t, new_lens, forced=forced)
        torch.cuda.synchronize()
        out.append((z_ref, z_gpu.cpu().numpy(), t_gpu.cpu().numpy(), t_ref))
        assert ctx.lengths() == list(ref.lengths())
    ctx.close()
    return out


def test_tiny_fp32_free_running():
    """2-layer d=256 fp32 decoder, 64-token prefix, 7 actions: tokens equal, logits <= 1e-4."""
    wl = W.WORKLOADS["tiny-b1"]
    pair = Pair(wl.spec, seed=0)
    pre = W.make_prefixes(wl, 0, 0)
    news = [None] + [[W.make_observation(wl.spec, 0, s, 0, 1)] for s in range(1, 6)]
    res = _run(pair, pre, news, wl.n_actions, 128, forced_from_ref=False, seed_tag="tiny")
    for z_ref, z_gpu, t_gpu, t_ref in res:
        c = compare(z_ref, z_gpu, t_gpu, TOL_F32)
        log(f"tiny max_abs={c.max_abs:.2e} strict={c.strict}")
        assert c.max_abs <= TOL_F32
        assert np.array_equal(t_gpu, t_ref)


@pytest.mark.parametrize("n_layers,d,H,F", [(2, 256, 4, 512), (2, 256, 2, 512), (2, 512, 4, 1408)])
def test_small_bf16_ragged(n_layers, d, H, F):
    """bf16, ragged rows (1..150 tokens, tile tails), per-row new tokens incl. empty rows."""
    spec = small_spec("bf16", n_layers, d, H, F)
    pair = Pair(spec, seed=3)
    wl = W.Workload("small", "tiny", 4, 5, 3, ragged=(1, 150, 8))
    lens = [1, 37, 150, 64]
    pre = [W.Prefix(W.make_observation(spec, 5, 100, b, lens[b] - min(8, lens[b] - 1)),
                    np.arange(min(8, lens[b] - 1), dtype=np.int32) * 7 % 44) for b in range(4)]
    news = [None,
            [W.make_observation(spec, 5, 1, b, n) if n else None for b, n in enumerate([3, 0, 1, 70])],
            [W.make_observation(spec, 5, 2, b, 1) for b in range(4)]]
    res = _run(pair, pre, news, 5, 320, forced_from_ref=True, seed_tag="small")
    for z_ref, z_gpu, t_gpu, _ in res:
        c = compare(z_ref, z_gpu, t_gpu, TOL_BF16)
        log(f"small bf16 max_abs={c.max_abs:.2e} strict={c.strict:.3f} band={c.band:.3f}")
        assert c.max_abs <= TOL_BF16
        assert c.band == 1.0


@pytest.mark.parametrize("d,H,F", [(512, 8, 1536), (384, 6, 1024)])
def test_small_bf16_wide_rows(d, H, F):
    """12 ragged rows decode on the wide path (9-64 rows: LDS-staged GEMM + split-K
    reductions); d = 512 carries each layer's RMSNorm in the reductions (sums of squares
    per 256 columns), d = 384 (not a multiple of 256) takes the RMSNorm kernel instead.
    Gains drawn around 1 so that the folded gains matter."""
    spec = small_spec("bf16", 2, d, H, F)
    pair = Pair(spec, seed=11, gains=True)
    B = 12
    lens = [1, 5, 17, 33, 40, 64, 65, 90, 100, 128, 129, 150]
    pre = [W.Prefix(W.make_observation(spec, 12, 100, b, lens[b] - min(6, lens[b] - 1)),
                    np.arange(min(6, lens[b] - 1), dtype=np.int32) * 5 % 44) for b in range(B)]
    news = [None,
            [W.make_observation(spec, 12, 1, b, n) if n else None for b, n in enumerate([2, 0, 1, 3] * 3)]]
    res = _run(pair, pre, news, 5, 192, forced_from_ref=True, seed_tag=f"wide d={d}")
    for z_ref, z_gpu, t_gpu, _ in res:
        c = compare(z_ref, z_gpu, t_gpu, TOL_BF16)
        log(f"wide rows d={d} max_abs={c.max_abs:.2e} strict={c.strict:.3f} band={c.band:.3f}")
        assert c.max_abs <= TOL_BF16
        assert c.band == 1.0


def test_small_bf16_nonunit_gains():
    """RMSNorm gains drawn around 1 (folded into the packed weights by the library)."""
    spec = small_spec("bf16", 2, 256, 4, 512)
    pair = Pair(spec, seed=8, gains=True)
    pre = [W.Prefix(W.make_observation(spec, 9, 0, b, 30 + 20 * b), np.zeros(0, np.int32)) for b in range(3)]
    news = [None, [W.make_observation(spec, 9, 1, b, 2) for b in range(3)]]
    res = _run(pair, pre, news, 4, 128, forced_from_ref=True, seed_tag="gains")
    for z_ref, z_gpu, t_gpu, _ in res:
        c = compare(z_ref, z_gpu, t_gpu, TOL_BF16)
        log(f"gains max_abs={c.max_abs:.2e} band={c.band:.3f}")
        assert c.max_abs <= TOL_BF16 and c.band == 1.0


def test_multi_pass_build():
    """A build split over several passes (max_pass_tokens = capacity: passes [60] [57] [10, 33] [41])
    matches the reference; the single-pass build uses other GEMM kernels, so the two agree
    to rounding, not bitwise."""
    import torch
    from paper_2508_10259_amd.runtime import DeviceContext
    spec = small_spec("bf16")
    pair = Pair(spec, seed=4)
    lens = [60, 57, 10, 33, 41]
    pre = [W.Prefix(W.make_observation(spec, 6, 0, b, n), np.zeros(0, np.int32)) for b, n in enumerate(lens)]
    z_by_mpt = {}
    for mpt in (0, 64):
        res = _run(pair, pre, [None], 4, 64, forced_from_ref=True, max_pass_tokens=mpt, seed_tag=f"mpt={mpt}")
        z_ref, z_gpu, t_gpu, _ = res[0]
        c = compare(z_ref, z_gpu, t_gpu, TOL_BF16)
        log(f"multi-pass mpt={mpt} max_abs={c.max_abs:.2e} band={c.band:.3f}")
        assert c.max_abs <= TOL_BF16 and c.band == 1.0
        z_by_mpt[mpt] = z_gpu
    assert np.max(np.abs(z_by_mpt[0] - z_by_mpt[64])) <= TOL_BF16


def test_mid_bf16_full_size():
    """12-layer d=1024 bf16 decoder, 8 rows of 256 patches + 24 ids, 7 actions;
    parity variant with one fresh observation token per step, teacher-forced."""
    wl = W.WORKLOADS["mid-b8"]
    pair = Pair(wl.spec, seed=0)
    pre = W.make_prefixes(wl, 0, 0)
    news = [None] + [[W.make_observation(wl.spec, 0, s, b, 1) for b in range(wl.batch)] for s in (1, 2)]
    res = _run(pair, pre, news, wl.n_actions, 320, forced_from_ref=True, seed_tag="mid")
    worst = 0.0
    bands = []
    for z_ref, z_gpu, t_gpu, _ in res:
        c = compare(z_ref, z_gpu, t_gpu, TOL_BF16)
        log(f"mid max_abs={c.max_abs:.2e} strict={c.strict:.3f} band={c.band:.3f}")
        worst = max(worst, c.max_abs)
        bands.append(c.band)
    assert worst <= TOL_BF16
    assert min(bands) == 1.0


def test_determinism_and_lifecycle():
    """Same inputs twice -> bitwise equal; invalidate -> AMS_ESTATE; rebuild == fresh build."""
    import torch
    from paper_2508_10259_amd import capi
    from paper_2508_10259_amd.runtime import DeviceContext
    spec = small_spec("bf16")
    pair = Pair(spec, seed=5)
    pre = [W.Prefix(W.make_observation(spec, 7, 0, b, 40 + 9 * b), np.zeros(0, np.int32)) for b in range(3)]
    prefix, lens = pair.dev.pack_prefixes(pre)
    ctx = DeviceContext(pair.dev, 3, 128)
    ctx.build(prefix, lens)
    t1, z1 = ctx.step(6)
    t2, z2 = ctx.step(6)
    torch.cuda.synchronize()
    assert torch.equal(t1, t2) and torch.equal(z1, z2)
    ctx.invalidate()
    assert ctx.state == capi.STATE_INVALID and ctx.lengths() == [0, 0, 0]
    with pytest.raises(capi.AmsError) as e:
        ctx.step(6)
    assert e.value.status == capi.AMS_ESTATE
    ctx.build(prefix, lens)
    t3, z3 = ctx.step(6)
    torch.cuda.synchronize()
    assert torch.equal(t1, t3) and torch.equal(z1, z3)
    # capacity: 40+9*2 = 58 tokens + n_actions - 1 must fit 128
    with pytest.raises(capi.AmsError) as e:
        ctx.step(72)
    assert e.value.status == capi.AMS_ECAPACITY
    assert ctx.lengths() == lens
    t4, _ = ctx.step(71)  # exact fit: 58 + 71 - 1 = 128
    torch.cuda.synchronize()
    assert torch.equal(t4[:, :6], t1)
    ctx.close()


def test_7b_single_row_full_size():
    """7B decoder (32 layers, d=4096, 32 heads of 128, FFN 11008, vocab 32000, bins = last 256 ids),
    1 row of 256 patches + 32 instruction ids, 7 actions, plus one step with a fresh observation
    token; weights drawn on the device, reference on host copies; teacher-forced."""
    import torch
    from paper_2508_10259_amd.runtime import DeviceContext, DeviceModel
    from ref_bridge import oracle_params, prefix_f64
    wl = W.WORKLOADS["7b-b1"]
    spec = wl.spec
    log("7b: drawing weights on the device")
    w = W.make_device_weights(spec, seed=0)
    dev = DeviceModel(w)
    p = oracle_params(w)
    pre = W.make_prefixes(wl, 0, 0)
    ref = D.ActionContext(p, 1)
    log("7b: reference build")
    ref.build([prefix_f64(p, spec, pre[0])])
    ctx = DeviceContext(dev, 1, 320)
    prefix, lens = dev.pack_prefixes(pre)
    ctx.build(prefix, lens)
    obs = W.make_observation(spec, 0, 1, 0, 1)
    for s_, news in enumerate([None, [obs]]):
        log(f"7b: step {s_}")
        t_ref, z_ref = ref.step(None if news is None else [W.to_f32(obs, "bf16").astype(np.float64)], wl.n_actions)
        forced = torch.from_numpy(t_ref.astype(np.int32)).cuda()
        new_t, new_lens = gpu_new_tokens(spec, news) if news is not None else (None, None)
        t_gpu, z_gpu = ctx.step(wl.n_actions, new_t, new_lens, forced=forced)
        torch.cuda.synchronize()
        c = compare(z_ref, z_gpu.cpu().numpy(), t_gpu.cpu().numpy(), TOL_BF16)
        log(f"7b max_abs={c.max_abs:.2e} strict={c.strict:.3f} band={c.band:.3f}")
        assert c.max_abs <= TOL_BF16 and c.band == 1.0
    ctx.close()


def _rows_ref(p, spec, prefixes, rows):
    ref = D.ActionContext(p, len(rows))
    ref.build([prefix_f64_of(p, spec, prefixes[b]) for b in rows])
    return ref


def prefix_f64_of(p, spec, prefix):
    from ref_bridge import prefix_f64
    return prefix_f64(p, spec, prefix)


def test_7b_ragged_batch64_extension_and_rebuild(model_7b):
    """64 rows with prefixes U{200..400} (capacity 768); a step that appends 16 fresh observation
    tokens to every row, then invalidate + rebuild on the next epoch's prefixes and step again.
    The reference checks rows 0, 37 and 63 (one by one, teacher-forced); the other rows are fed
    bin 0."""
    import torch
    from paper_2508_10259_amd import capi
    from paper_2508_10259_amd.runtime import DeviceContext
    spec, dev, p = model_7b
    wl = W.WORKLOADS["7b-b64-ragged"]
    rows = [0, 37, 63]
    ctx = DeviceContext(dev, wl.batch, wl.capacity)
    for epoch in (0, 1):
        pre = W.make_prefixes(wl, 0, epoch)
        log(f"7b-b64 epoch {epoch}: lens {[p_.length for p_ in pre[:4]]}...")
        if epoch:
            ctx.invalidate()
            with pytest.raises(capi.AmsError):
                ctx.step(wl.n_actions)
        prefix, lens = dev.pack_prefixes(pre)
        ctx.build(prefix, lens)
        ref = _rows_ref(p, spec, pre, rows)
        news = [W.make_observation(spec, 0, 100 * epoch + 1, b, wl.new_per_step) for b in range(wl.batch)]
        t_ref, z_ref = ref.step([W.to_f32(news[b], "bf16").astype(np.float64) for b in rows], wl.n_actions)
        forced = np.zeros((wl.batch, wl.n_actions), np.int32)
        forced[rows] = t_ref
        new_t, new_lens = gpu_new_tokens(spec, news)
        t_gpu, z_gpu = ctx.step(wl.n_actions, new_t, new_lens, forced=torch.from_numpy(forced).cuda())
        torch.cuda.synchronize()
        assert ctx.lengths() == [l + wl.new_per_step for l in lens]
        c = compare(z_ref, z_gpu.cpu().numpy()[rows], t_gpu.cpu().numpy()[rows], TOL_BF16)
        log(f"7b-b64 epoch {epoch} max_abs={c.max_abs:.2e} strict={c.strict:.3f} band={c.band:.3f}")
        assert c.max_abs <= TOL_BF16 and c.band == 1.0
    ctx.close()


def test_7b_chunk56_batch16_and_recompute(model_7b):
    """16 rows of 568 patches + 32 ids, 56 greedy tokens per step (8 actions x 7 tokens):
    row 0 against the reference over all 56 positions (teacher-forced); then the
    recompute mode (invalidate + build + step) reproduces the cached step bit for bit."""
    import torch
    from paper_2508_10259_amd.runtime import DeviceContext
    spec, dev, p = model_7b
    wl = W.WORKLOADS["7b-chunk56-b16"]
    cap = wl.derived_capacity()
    pre = W.make_prefixes(wl, 0, 0)
    ctx = DeviceContext(dev, wl.batch, cap)
    prefix, lens = dev.pack_prefixes(pre)
    ctx.build(prefix, lens)
    log("7b-chunk56: reference row 0")
    ref = _rows_ref(p, spec, pre, [0])
    t_ref, z_ref = ref.step(None, wl.n_actions)
    forced = np.zeros((wl.batch, wl.n_actions), np.int32)
    forced[0] = t_ref[0]
    forced_d = torch.from_numpy(forced).cuda()
    t_gpu, z_gpu = ctx.step(wl.n_actions, forced=forced_d)
    torch.cuda.synchronize()
    c = compare(z_ref, z_gpu.cpu().numpy()[:1], t_gpu.cpu().numpy()[:1], TOL_BF16)
    log(f"7b-chunk56 max_abs={c.max_abs:.2e} strict={c.strict:.3f} band={c.band:.3f}")
    assert c.max_abs <= TOL_BF16 and c.band == 1.0
    ctx.invalidate()
    ctx.build(prefix, lens)
    t2, z2 = ctx.step(wl.n_actions, forced=forced_d)
    torch.cuda.synchronize()
    assert torch.equal(t2, t_gpu) and torch.equal(z2, z_gpu)
    ctx.close()


@pytest.mark.parametrize("H", [4, 2])
def test_persistent_decode_matches_per_kernel_decode(H, monkeypatch):
    """Up to 8 fp16 rows a step runs as one persistent launch (AMS_FUSED unset); the
    same step through the per-kernel decode (AMS_FUSED=0) must give the same tokens
    when teacher-forced and logits within rounding (both are checked against the
    reference elsewhere; this pins the two native paths to each other, including the
    split-K and key-split merges at head_dim 64 and 128)."""
    import torch
    from paper_2508_10259_amd.runtime import DeviceContext
    spec = small_spec("bf16", 2, 256, H, 512)
    pair = Pair(spec, seed=11)
    lens = [1, 45, 130, 64, 200]
    pre = [W.Prefix(W.make_observation(spec, 12, 0, b, n), np.zeros(0, np.int32)) for b, n in enumerate(lens)]
    prefix, plens = pair.dev.pack_prefixes(pre)
    g = torch.Generator().manual_seed(3)
    forced = [torch.randint(0, spec.n_bins, (len(lens), 6), generator=g, dtype=torch.int32).cuda() for _ in range(2)]
    res = {}
    for mode in ("1", "0"):
        monkeypatch.setenv("AMS_FUSED", mode)
        ctx = DeviceContext(pair.dev, len(lens), 320)
        assert ctx.persistent_decode == (mode == "1")
        ctx.build(prefix, plens)
        t, z = ctx.step(6, forced=forced[0])
        t2, z2 = ctx.step(6, forced=forced[1])
        torch.cuda.synchronize()
        res[mode] = (t.cpu().numpy(), z.cpu().numpy(), t2.cpu().numpy(), z2.cpu().numpy())
        ctx.close()
    (t1, z1, f1, y1), (t0, z0, f0, y0) = res["1"], res["0"]
    d = max(np.max(np.abs(z1 - z0)), np.max(np.abs(y1 - y0)))
    log(f"persistent vs per-kernel H={H}: max_abs={d:.2e}")
    assert d <= 2e-3
    assert np.isfinite(z1).all() and np.isfinite(y1).all()
    assert (t1 >= 0).all() and (f1 >= 0).all()  # -1 would mean a barrier wait gave up
    # teacher-forced: the argmax of each position, where the top two logits are apart
    for a, b, z in ((t1, t0, z0), (f1, f0, y0)):
        top2 = np.sort(z, axis=-1)[..., -2:]
        clear = (top2[..., 1] - top2[..., 0]) > 4e-3
        assert np.array_equal(a[clear], b[clear])
