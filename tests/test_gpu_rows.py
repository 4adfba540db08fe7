"""Row-level invalidate and rebuild inside a live batch, and append-only commits, through the
C ABI against the fp64 reference.

The exception handler's common part for one robot of a batch discards that row's context
and rebuilds it from fresh data while the other rows keep theirs.  Checked: every row's
logits against the reference (rebuilt rows against a fresh build of their new prefix),
the untouched rows bit for bit against a twin context that never saw the row operations,
and a staggered schedule in which a different subset of rows is rebuilt before every step.
"""
import numpy as np
import pytest

from paper_2508_10259_amd import workload as W
from gpu_util import ForcedRef, Pair, compare, gpu_new_tokens, log, small_spec

pytestmark = pytest.mark.gpu

TOL_F32, TOL_BF16 = 1e-4, 3e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _prefix(spec, seed, tag, b, n):
    n_text = min(4, n - 1)
    return W.Prefix(W.make_observation(spec, seed, tag, b, n - n_text), np.arange(n_text, dtype=np.int32) * 3 % 40)


CASES = [  # (dtype, batch, d, heads, ffn): persistent decode at 5 rows, wide GEMMs at 12, fp32 per-kernel
    ("bf16", 5, 256, 4, 512),
    ("bf16", 12, 512, 8, 1536),
    ("f32", 3, 256, 4, 512),
]


@pytest.mark.parametrize("dtype,B,d,H,F", CASES)
def test_invalidate_rebuild_rows(dtype, B, d, H, F):
    import torch
    from paper_2508_10259_amd import capi
    from paper_2508_10259_amd.runtime import DeviceContext
    spec = small_spec(dtype, 2, d, H, F)
    tol = TOL_F32 if dtype == "f32" else TOL_BF16
    pair = Pair(spec, seed=21)
    lens = [int(x) for x in np.random.default_rng(B).integers(5, 120, size=B)]
    pre = [_prefix(spec, 21, 0, b, lens[b]) for b in range(B)]
    rows = [1, B - 1]
    pre2 = {b: _prefix(spec, 21, 1, b, 30 + 7 * b) for b in rows}
    news = [[W.make_observation(spec, 21, 10 + s, b, 1 + (b + s) % 3) for b in range(B)] for s in range(3)]
    prefix, plens = pair.dev.pack_prefixes(pre)
    ctx = DeviceContext(pair.dev, B, 256)
    twin = DeviceContext(pair.dev, B, 256)
    refs = [ForcedRef(pair.p, x) for x in pair.prefixes_f64(pre)]
    ctx.build(prefix, plens)
    twin.build(prefix, plens)
    A = 4
    results = []

    def step(c, s, append_first):
        new_t, new_lens = gpu_new_tokens(spec, news[s])
        if append_first:
            c.append(new_t, new_lens)
            return c.step(A)
        return c.step(A, new_t, new_lens)

    for s in range(3):
        if s == 1:  # one robot's exception (two rows here): discard and rebuild from fresh data
            ctx.invalidate_rows(rows)
            assert ctx.state == capi.STATE_INVALID
            got = ctx.lengths()
            assert all(got[b] == 0 for b in rows) and all(got[b] > 0 for b in range(B) if b not in rows)
            with pytest.raises(capi.AmsError) as e:
                ctx.step(A)
            assert e.value.status == capi.AMS_ESTATE
            rp, rl = pair.dev.pack_prefixes([pre2[b] for b in rows])
            ctx.build_rows(rows, rp, rl)
            assert ctx.state == capi.STATE_READY
            for b in rows:
                refs[b] = ForcedRef(pair.p, pair.prefixes_f64([pre2[b]])[0])
        t, z = step(ctx, s, append_first=(s == 2))
        t2, z2 = step(twin, s, append_first=(s == 2))
        torch.cuda.synchronize()
        t, z, t2, z2 = t.cpu().numpy(), z.cpu().numpy(), t2.cpu().numpy(), z2.cpu().numpy()
        z_ref = np.stack([refs[b].step(pair.obs_f64(news[s][b]), t[b]) for b in range(B)])
        c = compare(z_ref, z, t, tol)
        log(f"rows {dtype} B={B} step {s}: max_abs={c.max_abs:.2e} strict={c.strict:.3f} band={c.band:.3f}")
        assert c.max_abs <= tol and c.band == 1.0
        assert ctx.lengths() == [r.len for r in refs]
        keep = [b for b in range(B) if b not in rows]
        assert np.array_equal(t[keep], t2[keep]) and np.array_equal(z[keep], z2[keep]), "untouched rows changed"
        results.append(c)
    ctx.close()
    twin.close()


def test_staggered_row_rebuilds():
    """Before every step a different subset of rows (row b when (step + b) % 3 == 0) is
    invalidated and rebuilt from a new prefix, the others extend by 1-2 observation tokens;
    every row against the reference at every step (12 rows: the wide decode path)."""
    import torch
    from paper_2508_10259_amd.runtime import DeviceContext
    spec = small_spec("bf16", 2, 512, 8, 1536)
    pair = Pair(spec, seed=22)
    B, A = 12, 5
    pre = [_prefix(spec, 22, 0, b, 20 + 9 * b) for b in range(B)]
    ctx = DeviceContext(pair.dev, B, 320)
    ctx.build(*pair.dev.pack_prefixes(pre))
    refs = [ForcedRef(pair.p, x) for x in pair.prefixes_f64(pre)]
    for s in range(1, 7):
        rows = [b for b in range(B) if (s + b) % 3 == 0]
        fresh = [_prefix(spec, 22, s, b, 10 + (5 * s + 3 * b) % 90) for b in rows]
        ctx.invalidate_rows(rows)
        rp, rl = pair.dev.pack_prefixes(fresh)
        ctx.build_rows(rows, rp, rl)
        for b, fp in zip(rows, pair.prefixes_f64(fresh)):
            refs[b] = ForcedRef(pair.p, fp)
        news = [W.make_observation(spec, 22, 100 + s, b, 1 + (b % 2)) for b in range(B)]
        new_t, new_lens = gpu_new_tokens(spec, news)
        t, z = ctx.step(A, new_t, new_lens)
        torch.cuda.synchronize()
        t, z = t.cpu().numpy(), z.cpu().numpy()
        z_ref = np.stack([refs[b].step(pair.obs_f64(news[b]), t[b]) for b in range(B)])
        c = compare(z_ref, z, t, TOL_BF16)
        log(f"staggered step {s} rebuilt {rows}: max_abs={c.max_abs:.2e} band={c.band:.3f}")
        assert c.max_abs <= TOL_BF16 and c.band == 1.0
        assert ctx.lengths() == [r.len for r in refs]
    ctx.close()
