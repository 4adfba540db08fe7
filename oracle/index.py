"""Two-phase hashing for the action index, and the page keys built on it.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU-baseline
leg of the benchmark import this module; it shares no code with the GPU library.

What it computes
----------------
Paper section 3.2.3 ("Action Compression", "Virtual Action"): the system
serialises an input into bytes, hashes every segment of that byte string
independently (phase 1, parallel), then merges the segment hashes in order
into one final value (phase 2) that indexes the action for lookup and reuse;
Algorithm 1 ("Two-Phase Hashing for Action Index") states the two phases.  The
paper fixes only that the hash functions are modular calculations.  Readings
taken here (none is stated by the paper):

* modulus: the Mersenne prime p = 2^31 - 1; every hash is evaluated with two
  independent bases and the two 31-bit values are packed into one 64-bit
  integer, first base in the low 32 bits, second in the high 32 bits;
* HashFunc1(B_i): the segment, zero-padded to s bytes, is read as s/2
  little-endian 16-bit units u_0 .. u_{s/2-1}; with r the base,
  h = (sum_j u_j r^(s/2 - 1 - j)) r + |B_i|  (mod p), |B_i| the unpadded length;
* HashFunc2(h_1 .. h_k): with q the base, per 31-bit component,
  H = (sum_i h_i q^(k - i)) q + N  (mod p), N the input's length in bytes;
* s is even and at least 2.

The page key of a prefix (shared-prefix K/V pages) is the two-phase hash of
the prefix's bytes up to the end of that page: a page holds the K/V of its
tokens, which depend on every earlier token, so two rows may share a page
exactly when their inputs agree up to the page's end.
"""
from __future__ import annotations

from typing import List, Sequence

import numpy as np

P = (1 << 31) - 1
R = (0x2545F491, 0x1B873593)  # HashFunc1 bases
Q = (0x3C6EF372, 0x0A54FF53)  # HashFunc2 bases


def _pack(a: int, b: int) -> int:
    return int(a) | (int(b) << 32)


def unpack(h: int):
    return int(h) & 0xFFFFFFFF, int(h) >> 32


def _powers_desc(base: int, n: int) -> np.ndarray:
    """[base^(n-1), ..., base^1, base^0] mod p."""
    pw = np.empty(n, dtype=np.uint64)
    x = 1
    for e in range(n):
        pw[n - 1 - e] = x
        x = x * base % P
    return pw


_POW_CACHE = {}


def hash_func1(segment: bytes, s: int) -> int:
    """Phase-1 hash of one segment (at most s bytes), both components packed."""
    assert s >= 2 and s % 2 == 0 and 0 < len(segment) <= s
    padded = bytes(segment) + b"\0" * (s - len(segment))
    u = np.frombuffer(padded, dtype="<u2").astype(np.uint64)
    out = []
    for r in R:
        key = (r, s // 2)
        if key not in _POW_CACHE:
            _POW_CACHE[key] = _powers_desc(r, s // 2)
        poly = int(np.sum(u * _POW_CACHE[key] % np.uint64(P)) % np.uint64(P))
        out.append((poly * r + len(segment)) % P)
    return _pack(*out)


def hash_func2(seg_hashes: Sequence[int], n_bytes: int) -> int:
    """Phase-2 merge of the segment hashes, in order, with the input length."""
    out = []
    for c, q in enumerate(Q):
        acc = 0
        for h in seg_hashes:
            acc = (acc * q + unpack(h)[c]) % P
        out.append((acc * q + n_bytes) % P)
    return _pack(*out)


def segments(data: bytes, s: int) -> List[bytes]:
    """Partition into ceil(N / s) segments of s bytes, the last possibly shorter."""
    data = bytes(data)
    return [data[i:i + s] for i in range(0, len(data), s)]


def segment_hashes(data: bytes, s: int) -> List[int]:
    """Phase 1: every segment hashed on its own."""
    return [hash_func1(b, s) for b in segments(data, s)]


def two_phase_hash(data: bytes, s: int) -> int:
    """Algorithm 1: phase 1 over the segments, phase 2 over their hashes."""
    assert len(data) > 0
    return hash_func2(segment_hashes(data, s), len(data))


def page_keys(data: bytes, s: int, page_bytes: int) -> List[int]:
    """Key of every full page of a prefix: the two-phase hash of data[: m * page_bytes]
    for m = 1 .. floor(N / page_bytes) (page_bytes a multiple of s)."""
    assert page_bytes % s == 0
    return [two_phase_hash(bytes(data)[:m * page_bytes], s) for m in range(1, len(data) // page_bytes + 1)]
