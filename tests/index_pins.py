"""Pins of the two-phase hash (oracle/index.py) to facts other than itself: closed forms of
one-unit and unit-vector segments (reduced to Python's modular pow), the zero segment, the
linearity of a polynomial hash, phase 2 on one and two segments, the partition into segments,
sensitivity to every bit, length and segment order, independence from the order in which phase
1 runs, and the chain property of page keys.  ``test_index_pins.py`` runs them on the module,
``test_index_mutations.py`` on copies with planted mistakes."""
from __future__ import annotations

import numpy as np

P = (1 << 31) - 1


def _bytes(n, seed):
    return np.random.default_rng(seed).integers(0, 256, size=n, dtype=np.uint8).tobytes()


def pin_single_unit(X):
    """s = 2: one little-endian unit u = b0 + 256 b1, so each component is u r + 2; the two
    components use different bases, so they differ for a nonzero unit."""
    assert X.R[0] != X.R[1] and X.Q[0] != X.Q[1]
    assert all(1 < b < P for b in X.R + X.Q)
    h = X.unpack(X.two_phase_hash(bytes([9, 4]), 2))
    assert h[0] != h[1]
    for b0, b1 in ((5, 1), (0, 0), (255, 255), (7, 0)):
        h = X.hash_func1(bytes([b0, b1]), 2)
        u = b0 + 256 * b1
        for c in range(2):
            assert X.unpack(h)[c] == (u * X.R[c] + 2) % P


def pin_unit_position(X):
    """A 1 in unit j of an s-byte segment contributes r^(s/2 - j) (r^(s/2-1-j) times r)."""
    s = 8
    for j in range(4):
        seg = bytearray(s)
        seg[2 * j] = 1
        h = X.hash_func1(bytes(seg), s)
        for c in range(2):
            assert X.unpack(h)[c] == (pow(X.R[c], 4 - j, P) + s) % P, (j, c)


def pin_zero_segment_is_length(X):
    """A zero segment hashes to its unpadded length (padding adds nothing but the length)."""
    for n in (1, 2, 7, 16):
        h = X.hash_func1(bytes(n), 16)
        assert X.unpack(h) == (n, n)


def pin_linearity(X):
    """h(u + v) - |B| = (h(u) - |B|) + (h(v) - |B|) mod p for unit-wise sums below 2^16."""
    rng = np.random.default_rng(3)
    s = 64
    u = rng.integers(0, 1 << 15, size=s // 2, dtype=np.uint16)
    v = rng.integers(0, 1 << 15, size=s // 2, dtype=np.uint16)
    hu, hv, hw = (X.unpack(X.hash_func1(x.astype("<u2").tobytes(), s)) for x in (u, v, u + v))
    for c in range(2):
        assert (hw[c] - s) % P == ((hu[c] - s) + (hv[c] - s)) % P


def pin_phase2_closed_forms(X):
    """One segment: H = h q + N; two segments: H = h1 q^2 + h2 q + N (per component)."""
    h1 = X.hash_func1(b"\x01\x00", 2)
    h2 = X.hash_func1(b"\x00\x02", 2)
    H1 = X.hash_func2([h1], 2)
    H2 = X.hash_func2([h1, h2], 4)
    for c in range(2):
        q = X.Q[c]
        a, b = X.unpack(h1)[c], X.unpack(h2)[c]
        assert X.unpack(H1)[c] == (a * q + 2) % P
        assert X.unpack(H2)[c] == (a * pow(q, 2, P) + b * q + 4) % P
    assert X.two_phase_hash(b"\x01\x00\x00\x02", 2) == H2


def pin_partition(X):
    """ceil(N / s) segments of s bytes, the last shorter when s does not divide N."""
    d = _bytes(1000, 1)
    for s in (2, 64, 100, 1000, 4096):
        segs = X.segments(d, s)
        assert len(segs) == -(-1000 // s)
        assert all(len(g) == s for g in segs[:-1]) and 0 < len(segs[-1]) <= s
        assert b"".join(segs) == d


def pin_sensitivity(X):
    """Every single-bit flip, an appended zero byte, dropping the last byte and swapping two
    different segments all change the final hash; the same bytes give the same hash."""
    s = 32
    d = bytearray(_bytes(200, 2))
    H = X.two_phase_hash(bytes(d), s)
    assert X.two_phase_hash(bytes(d), s) == H
    for i in range(len(d)):
        for bit in (0, 7):
            e = bytearray(d)
            e[i] ^= 1 << bit
            assert X.two_phase_hash(bytes(e), s) != H, (i, bit)
    assert X.two_phase_hash(bytes(d) + b"\0", s) != H
    assert X.two_phase_hash(bytes(d[:-1]), s) != H
    sw = bytes(d[32:64] + d[0:32] + d[64:])
    assert X.two_phase_hash(sw, s) != H


def pin_phase1_order_free(X):
    """Phase 1 hashes every segment on its own: computing the segment hashes in any order and
    merging them in segment order gives Algorithm 1's result."""
    s = 48
    d = _bytes(1001, 4)
    segs = X.segments(d, s)
    order = np.random.default_rng(5).permutation(len(segs))
    hs = [None] * len(segs)
    for i in order:
        hs[i] = X.hash_func1(segs[i], s)
    assert hs == X.segment_hashes(d, s)
    assert X.hash_func2(hs, len(d)) == X.two_phase_hash(d, s)


def pin_page_key_chain(X):
    """Page m's key covers the bytes up to its end: two inputs agreeing on their first two pages
    share those keys and differ from the third on; a change in page 0 changes every key."""
    s, page = 16, 64
    a = bytearray(_bytes(64 * 5 + 10, 6))
    b = bytearray(a)
    b[2 * 64 + 5] ^= 0x10
    ka, kb = X.page_keys(bytes(a), s, page), X.page_keys(bytes(b), s, page)
    assert len(ka) == 5
    assert ka[:2] == kb[:2] and all(x != y for x, y in zip(ka[2:], kb[2:]))
    assert ka == [X.two_phase_hash(bytes(a[:m * page]), s) for m in range(1, 6)]
    c = bytearray(a)
    c[3] ^= 1
    assert all(x != y for x, y in zip(ka, X.page_keys(bytes(c), s, page)))


ALL_INDEX_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
