"""Property-based pins (hypothesis) for the oracle: alignment against brute force over every
in-band warping path, the exact inverse-CDF sampler against rational arithmetic, and the
string consistency of re-tokenisation, on generated inputs."""
from fractions import Fraction

import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from util_align import brute_force, check_map, check_path_invariants, pairs_csr, product_words, table, \
    unpack_path, w_eff

WORDS = product_words(b"abc", 2)  # 12 tokens of 1-2 bytes
SETTINGS = settings(max_examples=60, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])

seqs = st.lists(st.integers(0, len(WORDS) - 1), min_size=1, max_size=5)


@SETTINGS
@given(x=seqs, y=seqs, w=st.sampled_from([-1, 0, 1, 2, 4]))
def test_alignment_is_the_canonical_brute_force_optimum(orc, x, y, w):
    vd, vdo, vdl = table(WORDS)
    di, do, ti, to = pairs_csr([(x, y)])
    cost, plen, path, mp = orc.align(vd, vdo, vdl, vd, vdo, vdl, di, do, ti, to, w)
    k, m = len(x), len(y)
    cm = [[orc.levenshtein(WORDS[a], WORDS[c]) for c in y] for a in x]
    L = w_eff(k, m, w)
    best, canon = brute_force(cm, k, m, L)
    got = unpack_path(path, plen, do, to, 0)
    assert int(cost[0]) == best
    assert got == [(i - 1, j - 1) for i, j in canon]
    check_path_invariants(got, k, m, L, cm, best)
    check_map(list(mp[to[0]:to[1]]), got, k, m)


@SETTINGS
@given(weights=st.lists(st.integers(0, 1 << 20), min_size=2, max_size=9),
       k=st.integers(0, (1 << 24) - 1), tok=st.integers(0, 8), qv=st.floats(0.0, 1.0, width=32))
def test_sampler_against_rational_arithmetic(orc, weights, k, tok, qv):
    """token = first x whose Q62 prefix exceeds floor(u Z), u = k 2^-24, with R quantised by truncation."""
    if sum(weights) == 0:
        weights[0] = 1
    V = len(weights)
    tok %= V
    p0 = (np.array(weights, np.float64) / sum(weights)).astype(np.float32)
    p1 = p0[::-1].copy()
    u = np.float32(k * 2.0**-24)
    nacc, out, _, z = orc.verify(V, np.array([tok], np.int32), np.array([0, 1], np.int32),
                                 np.array([qv], np.float32), np.stack([p0, p1]), np.array([0.999999], np.float32),
                                 np.array([u], np.float32))
    r = int(nacc[0])
    row = p0 if r == 0 else p1
    R = [max(np.float32(0), np.float32(row[x] - (np.float32(qv) if (r == 0 and x == tok) else 0)))
         for x in range(V)]
    R = [min(v, np.float32(1)) for v in R]
    Rq = [int(Fraction(float(v)) * 2**62) for v in R]
    Z = sum(Rq)
    assert int(z[0]) == Z
    if Z == 0:
        assert int(out[0]) == int(np.argmax(row))
        return
    T = int(Fraction(float(u)) * Z)
    acc = 0
    for x in range(V):
        acc += Rq[x]
        if acc > T:
            assert int(out[0]) == x
            return
    raise AssertionError("no crossing")


@SETTINGS
@given(ids=st.lists(st.lists(st.integers(0, len(WORDS) - 1), max_size=6), min_size=1, max_size=4))
def test_retokenisation_spells_the_draft_string(orc, ids):
    """App. A.1: the proxy target tokens spell the draft string, each the longest possible."""
    targets = [b"a", b"b", b"c", b"ab", b"bca", b"cc", b"abc", b"ba"]
    vd, vdo, _ = table(WORDS)
    vt, vto, _ = table(targets)
    flat = np.array([x for s in ids for x in s], np.int32)
    off = np.array([0] + list(np.cumsum([len(s) for s in ids])), np.int32)
    got, goff = orc.retokenize(vd, vdo, vt, vto, flat, off)
    for b, s in enumerate(ids):
        S = b"".join(WORDS[i] for i in s)
        T = [targets[t] for t in got[goff[b]:goff[b + 1]]]
        assert b"".join(T) == S
        p = 0
        for t in T:
            assert not any(len(u) > len(t) and S.startswith(u, p) for u in targets)
            p += len(t)
