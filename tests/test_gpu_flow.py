"""The flow-matching action head (cold start from noise, warm start from a stored latent)
through the C ABI against the fp64 reference, and the context left as it was."""
import numpy as np
import pytest

from paper_2508_10259_amd import workload as W
import oracle.flow as FL
from gpu_util import Pair, log, small_spec

pytestmark = pytest.mark.gpu

TOL = {"bf16": 3e-2, "f32": 1e-4}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _head(pair, a, T):
    from paper_2508_10259_amd.runtime import DeviceFlowHead
    spec = pair.spec
    w = W.make_flow_head(spec, a, 7)
    dec = [W.to_f32(x, spec.dtype).astype(np.float64) for x in w]
    return DeviceFlowHead(spec, *w, n_tokens=T), FL.FlowHead(*dec)


@pytest.mark.parametrize("dtype,B,d,H,F", [("bf16", 5, 256, 4, 512), ("bf16", 12, 512, 8, 1536), ("f32", 3, 256, 4, 512)])
def test_flow_cold_and_warm(dtype, B, d, H, F):
    import torch
    from paper_2508_10259_amd.runtime import DeviceContext
    spec = small_spec(dtype, 2, d, H, F)
    pair = Pair(spec, seed=51)
    lens = [int(x) for x in np.random.default_rng(B).integers(10, 160, size=B)]
    pre = [W.Prefix(W.make_observation(spec, 51, 0, b, n - 3), np.array([1, 5, 9], np.int32)) for b, n in enumerate(lens)]
    a, T = 7, 8
    dh, rh = _head(pair, a, T)
    ctx = DeviceContext(pair.dev, B, 256)
    twin = DeviceContext(pair.dev, B, 256)
    packed, plens = pair.dev.pack_prefixes(pre)
    ctx.build(packed, plens)
    twin.build(packed, plens)
    seqs = pair.prefixes_f64(pre)
    x0 = W.make_latent(51, 0, B, T, a)
    stored = W.make_latent(51, 1, B, T, a) * 0.5
    for name, init, tau0, K in (("cold", x0, 0.0, 6), ("warm", stored, 0.5, 3)):
        x = torch.from_numpy(init.copy()).cuda()
        ctx.flow(dh, x, tau0, K)
        torch.cuda.synchronize()
        got = x.cpu().numpy().astype(np.float64)
        want = np.stack([FL.sample(pair.p, rh, seqs[b], init[b], tau0, K) for b in range(B)])
        err = float(np.max(np.abs(got - want)))
        moved = float(np.max(np.abs(want - init)))
        log(f"flow {dtype} B={B} {name}: max_abs={err:.2e} (latent moved by up to {moved:.2f})")
        assert err <= TOL[dtype] and moved > 10 * TOL[dtype]
    # the context is unchanged: the next action step equals the twin's, bit for bit
    t1, z1 = ctx.step(4)
    t2, z2 = twin.step(4)
    torch.cuda.synchronize()
    assert ctx.lengths() == twin.lengths() == plens
    assert np.array_equal(t1.cpu().numpy(), t2.cpu().numpy()) and np.array_equal(z1.cpu().numpy(), z2.cpu().numpy())
    ctx.close()
    twin.close()


def test_flow_7b_warm_start(model_7b):
    """The 7B decoder, 16 rows of the 600-token action-chunking prefix: a warm start from a stored
    latent (tau0 = 0.6, 4 steps) of an 8 x 7 chunk, row 0 against the reference."""
    import torch
    from paper_2508_10259_amd.runtime import DeviceContext, DeviceFlowHead
    from ref_bridge import prefix_f64
    spec, dev, p = model_7b
    wl = W.WORKLOADS["7b-chunk56-b16"]
    pre = W.make_prefixes(wl, 0, 0)
    ctx = DeviceContext(dev, wl.batch, wl.derived_capacity())
    ctx.build(*dev.pack_prefixes(pre))
    a, T = 7, 8
    w = W.make_flow_head(spec, a, 3)
    dh = DeviceFlowHead(spec, *w, n_tokens=T)
    rh = FL.FlowHead(*[W.to_f32(x, "bf16").astype(np.float64) for x in w])
    stored = W.make_latent(0, 5, wl.batch, T, a)
    x = torch.from_numpy(stored.copy()).cuda()
    ctx.flow(dh, x, 0.6, 4)
    torch.cuda.synchronize()
    want = FL.sample(p, rh, prefix_f64(p, spec, pre[0]), stored[0], 0.6, 4)
    err = float(np.max(np.abs(x.cpu().numpy()[0] - want)))
    log(f"flow 7b warm start row 0: max_abs={err:.2e}")
    assert err <= TOL["bf16"]
    ctx.close()
