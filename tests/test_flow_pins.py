"""The flow-matching head of the reference against closed forms, a scalar-loop evaluation of
one Euler step, and the composition of integration intervals; planted mistakes in private
copies of it must be caught."""
import importlib.util
import math
import sys

import numpy as np
import pytest

import oracle.decoder as D
import oracle.flow as F_real
from oracle_pins import _bf_layer, _rand, tiny_params


def _head(key, d, a):
    return F_real.FlowHead(_rand((d, a), key, 1, std=0.5), _rand((d,), key, 2, std=0.5), _rand((a, d), key, 3, std=0.5))


def pin_zero_steps(F):
    p = tiny_params(D, key=20)
    x0 = _rand((3, 2), 21)
    assert np.array_equal(F.sample(p, _head(22, 8, 2), _rand((4, 8), 23), x0, 0.0, 0), x0)


def pin_zero_readout(F):
    """W_out = 0: the velocity vanishes and the latent stays."""
    p = tiny_params(D, key=24)
    fh = _head(25, 8, 3)
    fh.w_out = np.zeros_like(fh.w_out)
    x0 = _rand((2, 3), 26)
    assert np.array_equal(F.sample(p, fh, _rand((5, 8), 27), x0, 0.2, 4), x0)


def pin_one_step_scalar(F):
    """One Euler step from tau0 = 0.25 (dt = 0.75) on a 1-layer d=4 model with 3 cached tokens and
    2 action tokens of 2 values: embedding, the layer (scalar loops over the whole sequence, the
    action tokens last), RMS readout and the update, all written out."""
    p = tiny_params(D, key=28, n_layers=1, d=4, H=2, F=3, V=5, n_bins=3, theta=7.0)
    fh = _head(29, 4, 2)
    seq = _rand((3, 4), 30)
    x0 = _rand((2, 2), 31)
    tau = 0.25
    e = [[sum(fh.w_in[j][k] * x0[i][k] for k in range(2)) + tau * fh.w_t[j] for j in range(4)] for i in range(2)]
    hs = _bf_layer(p, 0, seq.tolist() + e)[3:]
    v = []
    for h in hs:
        r = 1.0 / math.sqrt(sum(t * t for t in h) / 4 + p.cfg.rms_eps)
        v.append([sum(fh.w_out[i][j] * h[j] * r for j in range(4)) for i in range(2)])
    want = [[x0[i][k] + 0.75 * v[i][k] for k in range(2)] for i in range(2)]
    got = F.sample(p, fh, seq, x0, tau, 1)
    assert np.max(np.abs(got - np.array(want))) <= 1e-13


def pin_composition(F):
    """Integrating [0, 1] in 8 steps equals 5 steps to tau = 5/8, then a warm start from that
    latent over the remaining 3 (same grid)."""
    p = tiny_params(D, key=32)
    fh = _head(33, 8, 3)
    seq = _rand((6, 8), 34)
    x0 = _rand((4, 3), 35)
    full = F.sample(p, fh, seq, x0, 0.0, 8)
    # the first 5 steps of the cold run, written as a run that stops early
    _, kv = D.forward(p, seq)
    x = x0.copy()
    for k in range(5):
        x = x + (1.0 / 8) * F.velocity(p, fh, kv, 6, x, k / 8)
    warm = F.sample(p, fh, seq, x, 5 / 8, 3)
    assert np.max(np.abs(full - warm)) <= 1e-12


def pin_action_tokens_causal(F):
    """The velocity of action token i does not depend on later action tokens."""
    p = tiny_params(D, key=36)
    fh = _head(37, 8, 2)
    seq = _rand((4, 8), 38)
    _, kv = D.forward(p, seq)
    x = _rand((3, 2), 39)
    y = x.copy()
    y[2] += 1.0
    v1, v2 = F.velocity(p, fh, kv, 4, x, 0.3), F.velocity(p, fh, kv, 4, y, 0.3)
    assert np.max(np.abs(v1[:2] - v2[:2])) == 0.0 and np.max(np.abs(v1[2] - v2[2])) > 1e-6


ALL = [pin_zero_steps, pin_zero_readout, pin_one_step_scalar, pin_composition, pin_action_tokens_causal]


@pytest.mark.parametrize("pin", ALL, ids=[p.__name__ for p in ALL])
def test_pin(pin):
    pin(F_real)


def _fresh():
    spec = importlib.util.spec_from_file_location("oracle.flow_copy", F_real.__file__,
                                                  submodule_search_locations=None)
    m = importlib.util.module_from_spec(spec)
    m.__package__ = "oracle"
    sys.modules[spec.name] = m
    spec.loader.exec_module(m)
    return m


def _no_tau(m):
    orig = m.velocity
    m.velocity = lambda p, fh, past, start, x, tau: orig(p, fh, past, start, x, 0.0)


def _gain_readout(m):
    orig = m.velocity

    def v(p, fh, past, start, x, tau):
        e = np.asarray(x, dtype=np.float64) @ fh.w_in.T + tau * fh.w_t
        h, _ = D.forward(p, e, start=start, past=past)
        return D.rms_norm(h, p.get("g_final"), p.cfg.rms_eps) @ fh.w_out.T
    m.velocity = v


def _positions_from_zero(m):
    def v(p, fh, past, start, x, tau):
        e = np.asarray(x, dtype=np.float64) @ fh.w_in.T + tau * fh.w_t
        h, _ = D.forward(p, e)  # forgets the cached context
        u = h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + p.cfg.rms_eps)
        return u @ fh.w_out.T
    m.velocity = v


def _dt_over_k(m):
    orig = m.sample

    def s(p, fh, seq, x0, tau0, n):
        if n <= 0:
            return orig(p, fh, seq, x0, tau0, n)
        x = np.asarray(x0, dtype=np.float64).copy()
        _, kv = D.forward(p, np.asarray(seq, dtype=np.float64))
        for k in range(n):
            x = x + (1.0 / n) * m.velocity(p, fh, kv, seq.shape[0], x, tau0 + k / n)
        return x
    m.sample = s


def _tau_end(m):
    orig = m.sample

    def s(p, fh, seq, x0, tau0, n):
        if n <= 0:
            return orig(p, fh, seq, x0, tau0, n)
        x = np.asarray(x0, dtype=np.float64).copy()
        _, kv = D.forward(p, np.asarray(seq, dtype=np.float64))
        dt = (1.0 - tau0) / n
        for k in range(n):
            x = x + dt * m.velocity(p, fh, kv, seq.shape[0], x, tau0 + (k + 1) * dt)
        return x
    m.sample = s


MUTATIONS = {"no_tau": _no_tau, "gain_readout": _gain_readout, "positions_from_zero": _positions_from_zero,
             "dt_over_k": _dt_over_k, "tau_end": _tau_end}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name):
    m = _fresh()
    MUTATIONS[name](m)
    caught = 0
    for pin in ALL:
        try:
            pin(m)
        except Exception:  # noqa: BLE001
            caught += 1
    assert caught, f"mutation {name} slipped past every pin"
