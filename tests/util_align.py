"""Helpers for alignment tests: tiny vocabularies and brute-force warping paths."""
import itertools
import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def table(tokens):
    """CSR byte table for a list of bytes tokens (ids = list order)."""
    data = np.frombuffer(b"".join(tokens), dtype=np.uint8).copy() if tokens else np.zeros(0, np.uint8)
    off = np.zeros(len(tokens) + 1, np.int32)
    off[1:] = np.cumsum([len(t) for t in tokens])
    return data, off, max([len(t) for t in tokens] + [1])


def pairs_csr(pairs):
    """[(draft_ids, target_ids), ...] -> draft_ids, draft_off, target_ids, target_off."""
    def csr(lists):
        off = np.zeros(len(lists) + 1, np.int32)
        off[1:] = np.cumsum([len(l) for l in lists])
        flat = np.array([x for l in lists for x in l], np.int32)
        return flat, off

    di, do = csr([p[0] for p in pairs])
    ti, to = csr([p[1] for p in pairs])
    return di, do, ti, to


def w_eff(k, m, w):
    return max(k, m) if w < 0 else max(w, abs(k - m))


def all_paths(k, m, L):
    """Every monotone, continuous warping path from (1,1) to (k,m) inside |i-j| <= L.

    Yields lists of 1-based (i, j) cells.  Built backwards from (k, m) so that the
    order of generation follows predecessor choices.
    """
    def rec(i, j):
        if abs(i - j) > L:
            return
        if (i, j) == (1, 1):
            yield [(1, 1)]
            return
        for di, dj in ((1, 1), (1, 0), (0, 1)):
            pi, pj = i - di, j - dj
            if pi >= 1 and pj >= 1:
                for p in rec(pi, pj):
                    yield p + [(i, j)]

    yield from rec(k, m)


def step_code(path):
    """Backward step sequence: 0 = diagonal, 1 = from (i-1, j), 2 = from (i, j-1)."""
    codes = []
    for (i0, j0), (i1, j1) in zip(reversed(path[:-1]), reversed(path[1:])):
        codes.append({(1, 1): 0, (1, 0): 1, (0, 1): 2}[(i1 - i0, j1 - j0)])
    return codes


def brute_force(cost, k, m, L):
    """(C*, canonical optimal path) over all in-band paths; cost is a k x m array."""
    best, cands = None, []
    for p in all_paths(k, m, L):
        c = sum(int(cost[i - 1][j - 1]) for i, j in p)
        if best is None or c < best:
            best, cands = c, [p]
        elif c == best:
            cands.append(p)
    canon = min(cands, key=step_code)
    return best, canon


def check_path_invariants(path, k, m, L, cost_matrix, total):
    """Monotone, continuous, anchored, in band, length bounds, cost sums to C*."""
    assert path[0] == (0, 0) and path[-1] == (k - 1, m - 1)
    assert max(k, m) <= len(path) <= k + m - 1
    for (i0, j0), (i1, j1) in zip(path[:-1], path[1:]):
        assert (i1 - i0, j1 - j0) in ((1, 0), (0, 1), (1, 1))
    for i, j in path:
        assert abs(i - j) <= L
    assert sum(int(cost_matrix[i][j]) for i, j in path) == total


def check_map(mp, path, k, m):
    """One draft index per target position: the largest on the path in that column."""
    assert len(mp) == m
    for j in range(m):
        assert mp[j] == max(i for i, jj in path if jj == j)
    assert all(a <= b for a, b in zip(mp[:-1], mp[1:]))
    assert mp[-1] == k - 1


def unpack_path(path_flat, plen, draft_off, target_off, b):
    base = 2 * (int(draft_off[b]) + int(target_off[b]))
    seg = path_flat[base:base + 2 * int(plen[b])]
    return [(int(seg[2 * p]), int(seg[2 * p + 1])) for p in range(int(plen[b]))]


def enumerate_small_pairs(rng, n, kmax, mmax, nd, nt):
    return [(list(rng.integers(0, nd, size=rng.integers(1, kmax + 1))),
             list(rng.integers(0, nt, size=rng.integers(1, mmax + 1)))) for _ in range(n)]


def product_words(alphabet, max_len):
    return [bytes(w) for n in range(1, max_len + 1) for w in itertools.product(alphabet, repeat=n)]
