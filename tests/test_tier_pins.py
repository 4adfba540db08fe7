"""The eviction plan of the reference against hand-worked cases and invariants, planted
mistakes in private copies of it, and the library's plan (ams_tier_plan) against it on
random inputs."""
import ctypes as C
import importlib.util
import sys

import numpy as np
import pytest

import oracle.tier as T_real


def _cases():
    # rows:        0   1   2   3   4
    prio = [1, 0, 0, 2, 0]
    last = [5, 9, 3, 1, 3]
    pages = [4, 2, 3, 8, 1]
    drop = [False, True, False, False, True]
    res = [True, True, True, True, False]  # row 4 is not resident
    pin = [False, False, False, False, False]
    return prio, last, pages, drop, res, pin


def pin_hand_worked(T):
    """Priority 0 first, LRU within it: row 2 (t=3) then row 1 (t=9), then row 0 (prio 1);
    row 4 is not resident; row 2 is offloaded, row 1 (droppable) dropped."""
    prio, last, pages, drop, res, pin = _cases()
    a, f = T.eviction_plan(prio, last, pages, drop, res, pin, 3)
    assert a == [T.KEEP, T.KEEP, T.OFFLOAD, T.KEEP, T.KEEP] and f == 3
    a, f = T.eviction_plan(prio, last, pages, drop, res, pin, 4)
    assert a == [T.KEEP, T.DROP, T.OFFLOAD, T.KEEP, T.KEEP] and f == 5
    a, f = T.eviction_plan(prio, last, pages, drop, res, pin, 6)
    assert a == [T.OFFLOAD, T.DROP, T.OFFLOAD, T.KEEP, T.KEEP] and f == 9
    a, f = T.eviction_plan(prio, last, pages, drop, res, pin, 0)
    assert a == [T.KEEP] * 5 and f == 0


def pin_pinned_and_shortfall(T):
    """Pinned rows are never taken; asking for more than the candidates hold takes them all."""
    prio, last, pages, drop, res, pin = _cases()
    pin = [False, False, True, False, False]
    a, f = T.eviction_plan(prio, last, pages, drop, res, pin, 100)
    assert a == [T.OFFLOAD, T.DROP, T.KEEP, T.OFFLOAD, T.KEEP] and f == 14


def pin_ties_by_row(T):
    """Equal priority and last use: the lower row index goes first."""
    a, f = T.eviction_plan([0, 0, 0], [2, 2, 2], [1, 1, 1], [False] * 3, [True] * 3, [False] * 3, 2)
    assert a == [T.OFFLOAD, T.OFFLOAD, T.KEEP] and f == 2


def pin_minimal_prefix(T):
    """The taken rows are a prefix of the (priority, last use, row) order, and dropping the last
    of them would leave fewer than the pages asked for."""
    rng = np.random.default_rng(0)
    for _ in range(50):
        n = int(rng.integers(1, 9))
        prio = rng.integers(0, 3, n).tolist()
        last = rng.integers(0, 20, n).tolist()
        pages = rng.integers(1, 6, n).tolist()
        res = (rng.random(n) < 0.8).tolist()
        pin = (rng.random(n) < 0.2).tolist()
        need = int(rng.integers(1, 20))
        a, f = T.eviction_plan(prio, last, pages, [False] * n, res, pin, need)
        order = sorted((r for r in range(n) if res[r] and not pin[r]), key=lambda r: (prio[r], last[r], r))
        taken = [r for r in order if a[r] != T.KEEP]
        assert taken == order[:len(taken)]
        assert f == sum(pages[r] for r in taken)
        if taken and f >= need:
            assert f - pages[taken[-1]] < need


ALL = [pin_hand_worked, pin_pinned_and_shortfall, pin_ties_by_row, pin_minimal_prefix]


@pytest.mark.parametrize("pin", ALL, ids=[p.__name__ for p in ALL])
def test_pin(pin):
    pin(T_real)


def _fresh():
    spec = importlib.util.spec_from_file_location("oracle_tier_copy", T_real.__file__)
    m = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = m
    spec.loader.exec_module(m)
    return m


def _mru(m):  # most recently used first
    orig = m.eviction_plan
    m.eviction_plan = lambda p, t, n, d, r, pn, need: orig(p, [-x for x in t], n, d, r, pn, need)


def _priority_reversed(m):
    orig = m.eviction_plan
    m.eviction_plan = lambda p, t, n, d, r, pn, need: orig([-x for x in p], t, n, d, r, pn, need)


def _ignore_pinned(m):
    orig = m.eviction_plan
    m.eviction_plan = lambda p, t, n, d, r, pn, need: orig(p, t, n, d, r, [False] * len(p), need)


def _drop_all(m):
    orig = m.eviction_plan
    m.eviction_plan = lambda p, t, n, d, r, pn, need: orig(p, t, n, [True] * len(p), r, pn, need)


def _one_extra(m):
    orig = m.eviction_plan

    def f(p, t, n, d, r, pn, need):
        return orig(p, t, n, d, r, pn, need + 1) if need > 0 else orig(p, t, n, d, r, pn, need)
    m.eviction_plan = f


MUTATIONS = {"mru": _mru, "priority_reversed": _priority_reversed, "ignore_pinned": _ignore_pinned,
             "drop_all": _drop_all, "one_extra": _one_extra}


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


def test_library_plan_matches_reference():
    """ams_tier_plan (the library's host-side planner) against the reference on random inputs."""
    from paper_2508_10259_amd import capi
    import os
    if not os.path.exists(capi.LIB_PATH):
        pytest.skip("library not built")
    lib = capi.load()
    rng = np.random.default_rng(1)
    for _ in range(300):
        n = int(rng.integers(1, 40))
        prio = rng.integers(0, 4, n).astype(np.int32)
        last = rng.integers(0, 10, n).astype(np.int64)
        pages = rng.integers(0, 13, n).astype(np.int32)
        drop = (rng.random(n) < 0.4).astype(np.int32)
        res = (rng.random(n) < 0.8).astype(np.int32)
        pin = (rng.random(n) < 0.1).astype(np.int32)
        need = int(rng.integers(0, 60))
        act = np.zeros(n, np.int32)
        freed = C.c_int64()
        st = lib.ams_tier_plan(n, prio.ctypes.data, last.ctypes.data, pages.ctypes.data, drop.ctypes.data,
                               res.ctypes.data, pin.ctypes.data, need, act.ctypes.data, C.byref(freed))
        assert st == 0
        a, f = T_real.eviction_plan(prio.tolist(), last.tolist(), pages.tolist(), drop.astype(bool).tolist(),
                                    res.astype(bool).tolist(), pin.astype(bool).tolist(), need)
        assert act.tolist() == a and freed.value == f
