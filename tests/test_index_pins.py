"""The two-phase hash of the reference against closed forms and invariants, and planted
mistakes in private copies of it that the pins must catch."""
import importlib.util
import sys

import numpy as np
import pytest

import oracle.index as X_real
from index_pins import ALL_INDEX_PINS, P


@pytest.mark.parametrize("pin", ALL_INDEX_PINS, ids=[p.__name__ for p in ALL_INDEX_PINS])
def test_pin(pin):
    pin(X_real)


def _fresh():
    spec = importlib.util.spec_from_file_location("oracle_index_copy", X_real.__file__)
    m = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = m
    spec.loader.exec_module(m)
    return m


def _big_endian_units(m):
    orig = m.hash_func1
    m.hash_func1 = lambda seg, s: orig(bytes(b for i in range(0, len(seg) - 1, 2) for b in (seg[i + 1], seg[i]))
                                        + (seg[-1:] if len(seg) % 2 else b""), s)


def _no_length(m):
    orig = m.hash_func1

    def f(seg, s):
        a, b = m.unpack(orig(seg, s))
        return m._pack((a - len(seg)) % P, (b - len(seg)) % P)
    m.hash_func1 = f


def _ascending_powers(m):
    def f(seg, s):
        padded = bytes(seg) + b"\0" * (s - len(seg))
        u = [int(x) for x in np.frombuffer(padded, dtype="<u2")]
        out = []
        for r in m.R:
            poly = sum(x * pow(r, j, P) for j, x in enumerate(u)) % P
            out.append((poly * r + len(seg)) % P)
        return m._pack(*out)
    m.hash_func1 = f


def _phase2_no_length(m):
    orig = m.hash_func2
    m.hash_func2 = lambda hs, n: orig(hs, 0)


def _phase2_reversed(m):
    orig = m.hash_func2
    m.hash_func2 = lambda hs, n: orig(list(reversed(hs)), n)


def _one_base(m):
    m.R = (m.R[0], m.R[0])
    m.Q = (m.Q[0], m.Q[0])


def _short_segments(m):
    orig = m.segments
    m.segments = lambda data, s: orig(data, max(2, s - 2))


def _pages_unchained(m):
    m.page_keys = lambda data, s, pb: [m.two_phase_hash(bytes(data)[(k - 1) * pb:k * pb], s)
                                       for k in range(1, len(data) // pb + 1)]


def _sum_phase2(m):
    def f(hs, n):
        out = []
        for c, q in enumerate(m.Q):
            out.append((sum(m.unpack(h)[c] for h in hs) * q + n) % P)
        return m._pack(*out)
    m.hash_func2 = f


MUTATIONS = {
    "big_endian_units": _big_endian_units, "no_length": _no_length, "ascending_powers": _ascending_powers,
    "phase2_no_length": _phase2_no_length, "phase2_reversed": _phase2_reversed, "one_base": _one_base,
    "short_segments": _short_segments, "pages_unchained": _pages_unchained, "sum_phase2": _sum_phase2,
}


def test_unmutated_copy_passes():
    m = _fresh()
    for pin in ALL_INDEX_PINS:
        pin(m)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name):
    m = _fresh()
    MUTATIONS[name](m)
    caught = []
    for pin in ALL_INDEX_PINS:
        try:
            pin(m)
        except Exception as e:  # noqa: BLE001
            caught.append(pin.__name__)
    assert caught, f"mutation {name} slipped past every pin"
