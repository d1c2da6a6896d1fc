"""Pins for the oracle's token distance (App. H, byte-level edit distance).

The oracle's textbook DP is checked against things that do not reuse its
formula: closed forms, metric axioms, a breadth-first search over edit scripts
and a differently-structured recursive definition.
"""
import functools
import itertools
from collections import deque

import numpy as np


def bfs_edit_distance(s: bytes, t: bytes) -> int:
    """Fewest single-byte insertions, deletions or substitutions turning s into t.

    Breadth-first search over strings; an optimal script only ever writes bytes
    of t, so the alphabet is restricted to those.
    """
    alphabet = sorted(set(t))
    limit = len(s) + len(t)
    seen = {s}
    frontier = deque([(s, 0)])
    while frontier:
        cur, dist = frontier.popleft()
        if cur == t:
            return dist
        if dist >= limit:
            continue
        nxt = set()
        for p in range(len(cur)):
            nxt.add(cur[:p] + cur[p + 1:])  # delete
            for c in alphabet:
                nxt.add(cur[:p] + bytes([c]) + cur[p + 1:])  # substitute
        for p in range(len(cur) + 1):
            for c in alphabet:
                nxt.add(cur[:p] + bytes([c]) + cur[p:])  # insert
        for n in nxt:
            if n not in seen and len(n) <= max(len(s), len(t)) + 1:
                seen.add(n)
                frontier.append((n, dist + 1))
    raise AssertionError("unreachable")


def recursive_distance(s: bytes, t: bytes) -> int:
    """Suffix recursion (first characters), memoised: a different route to the same number."""

    @functools.lru_cache(maxsize=None)
    def go(a: int, b: int) -> int:
        if a == len(s):
            return len(t) - b
        if b == len(t):
            return len(s) - a
        if s[a] == t[b]:
            return go(a + 1, b + 1)
        return 1 + min(go(a + 1, b), go(a, b + 1), go(a + 1, b + 1))

    return go(0, 0)


def test_closed_forms(orc):
    rng = np.random.default_rng(11)
    for _ in range(300):
        s = rng.integers(32, 127, size=rng.integers(0, 12)).astype(np.uint8).tobytes()
        t = rng.integers(32, 127, size=rng.integers(0, 12)).astype(np.uint8).tobytes()
        d = orc.levenshtein(s, t)
        assert orc.levenshtein(s, s) == 0
        assert orc.levenshtein(s, b"") == len(s)
        assert orc.levenshtein(b"", t) == len(t)
        assert d == orc.levenshtein(t, s)
        assert abs(len(s) - len(t)) <= d <= max(len(s), len(t))
        if len(s) == len(t):
            assert d <= sum(a != b for a, b in zip(s, t))  # Hamming bound


def test_triangle_inequality(orc):
    rng = np.random.default_rng(12)
    for _ in range(300):
        a, b, c = (rng.integers(97, 101, size=rng.integers(0, 7)).astype(np.uint8).tobytes()
                   for _ in range(3))
        assert orc.levenshtein(a, c) <= orc.levenshtein(a, b) + orc.levenshtein(b, c)


def test_bfs_all_short_strings(orc):
    words = [bytes(w) for n in range(4) for w in itertools.product(b"abc", repeat=n)]
    for s in words:
        for t in words:
            assert orc.levenshtein(s, t) == bfs_edit_distance(s, t), (s, t)


def test_recursive_definition_random(orc):
    rng = np.random.default_rng(13)
    for _ in range(500):
        s = rng.integers(97, 101, size=rng.integers(0, 9)).astype(np.uint8).tobytes()
        t = rng.integers(97, 101, size=rng.integers(0, 9)).astype(np.uint8).tobytes()
        assert orc.levenshtein(s, t) == recursive_distance(s, t), (s, t)


def test_long_tokens_and_high_bytes(orc):
    # 64-byte tokens and bytes >= 0x80 (UTF-8 continuation bytes) and 0x00
    rng = np.random.default_rng(14)
    for _ in range(40):
        s = rng.integers(0, 256, size=rng.integers(40, 65)).astype(np.uint8).tobytes()
        t = bytearray(s)
        for _ in range(5):
            t[int(rng.integers(0, len(t)))] = int(rng.integers(0, 256))
        t = bytes(t)
        assert orc.levenshtein(s, t) == recursive_distance(s, t)


def test_fig2_token_distances(orc):
    # distances along the path printed in Fig. 2 (byte edit distance, App. H)
    assert orc.levenshtein(b"S", b"Scale") == 4
    assert orc.levenshtein(b"cal", b"Scale") == 2
    assert orc.levenshtein(b"ing", b"ing") == 0
    assert orc.levenshtein(b"Law", b"L") == 2
    assert orc.levenshtein(b"Law", b"aw") == 1
    # UTF-8: a two-byte character against its one-byte lookalike costs 2 edits on bytes
    assert orc.levenshtein("é".encode(), b"e") == 2
