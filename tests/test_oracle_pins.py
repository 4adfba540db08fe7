"""The fp64 reference against closed forms, invariants, special cases and brute force."""
import numpy as np
import pytest

import oracle.decoder as D
from oracle_pins import ALL_PINS, tiny_params, _ctx_vs_full, _rand


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_pin(pin):
    pin(D)


def test_cached_equals_full_random_shapes():
    """Cached == full on a spread of small shapes (heads, dims, lengths, bins)."""
    shapes = [  # (layers, d, H, F, V, n_bins)
        (1, 4, 1, 6, 8, 8), (2, 8, 4, 16, 30, 5), (3, 12, 3, 10, 16, 16), (1, 16, 2, 40, 64, 7),
    ]
    for i, (nl, d, H, F, V, nb) in enumerate(shapes):
        p = tiny_params(D, key=100 + i, n_layers=nl, d=d, H=H, F=F, V=V, n_bins=nb)
        B = 1 + i % 3
        prefixes = [_rand((2 + 3 * b + i, d), 200 + i, b) for b in range(B)]
        news = [None, [(_rand((1 + b, d), 300 + i, b) if (b + i) % 2 == 0 else None) for b in range(B)]]
        _ctx_vs_full(D, p, prefixes, news, n_actions=3)


def test_cached_equals_full_tiny_workload():
    """The 2-layer d=256 fp32 workload shape with its seeded weights: cached == full to 1e-12."""
    from paper_2508_10259_amd import workload as W
    from ref_bridge import oracle_params
    wl = W.WORKLOADS["tiny-b1"]
    w = W.make_weights(wl.spec, seed=0)
    p = oracle_params(w)
    pre = [W.to_f32(W.make_prefix(wl, 0, 0, 0).patches, "f32")]
    obs = [[W.to_f32(W.make_observation(wl.spec, 0, s, 0, 1), "f32")] for s in range(2)]
    _ctx_vs_full(D, p, pre, [None] + obs, n_actions=7)


def test_prefix_bridge_text_rows():
    """The tests' prefix conversion feeds the reference the decoded patch rows followed by
    exactly the table rows of the instruction ids (the rows the GPU gathers on the device)."""
    from paper_2508_10259_amd import workload as W
    from ref_bridge import oracle_params, prefix_f64
    spec = W.ModelSpec("pin", 1, 128, 2, 64, 128, 300, 256, "bf16")
    w = W.make_weights(spec, seed=2)
    p = oracle_params(w)
    patches = W.random_gaussian((3, 128), 2, 5, dtype="bf16")
    ids = np.array([0, 43, 1, 17], np.int32)  # 43 = vocab - n_bins - 1
    x = prefix_f64(p, spec, W.Prefix(patches, ids))
    table = W.bf16_bits_to_f32(w.embed).astype(np.float64)
    assert x.shape == (7, 128)
    assert np.array_equal(x[:3], W.bf16_bits_to_f32(patches).astype(np.float64))
    assert np.array_equal(x[3:], table[ids])


def test_forced_ref_helper_matches_reference_step():
    """The GPU tests' batched teacher-forced helper equals the reference's own step with the
    same forced bins (to 1e-12), with and without new tokens, over several steps."""
    from gpu_util import ForcedRef
    p = tiny_params(D, key=13, V=20, n_bins=6)
    pre = _rand((5, 8), 90)
    ctx = D.ActionContext(p, 1)
    ctx.build([pre])
    fr = ForcedRef(p, pre)
    rng = np.random.default_rng(1)
    for s, n in enumerate([2, 0, 1, 0, 3]):
        new = _rand((n, 8), 91, s) if n else None
        fed = rng.integers(0, 6, size=4)
        t, z = ctx.step([new], 4, forced=fed[None])
        zf = fr.step(new, fed)
        err = float(np.max(np.abs(z[0] - zf)))
        assert err <= 1e-12, (s, err)
        assert fr.len == ctx.lengths()[0]
    assert ForcedRef(p, pre).step(None, [3]).shape == (1, 6)
