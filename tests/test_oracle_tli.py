"""Pins for the oracle's Token-Level Intersection proposal (App. D Alg. 3).

Alg. 3 defines q' over the target vocabulary: the draft's mass on tokens both vocabularies
hold, renormalised by the mass q puts on that intersection, and zero elsewhere; standard
speculative decoding (Alg. 4) then runs with p and q'.  The oracle takes each vocabulary as
a set of byte strings (the lowest id stands for a string held by several ids) and forms the
normaliser S as the Q62-truncated intersected mass, summed exactly and rounded once to fp32.

Pins: a hand-worked intersection, a brute-force intersection over random tiny vocabularies,
S and q' re-derived with exact rational arithmetic (fractions) and a brute-force nearest-fp32
search (a different method from the oracle's integer rounding), rounding cases a naive fp32
sum gets wrong, the truncation and empty-intersection readings, and the lossless law of
Alg. 4 run on q' (chi-square).
"""
from fractions import Fraction

import numpy as np
import pytest

from test_oracle_sd import draw
from test_oracle_verify import ALPHA, chi2_pvalue, dist, u24


def table(strings):
    data = b"".join(strings)
    off = np.zeros(len(strings) + 1, np.int32)
    off[1:] = np.cumsum([len(s) for s in strings])
    return np.frombuffer(data, np.uint8) if data else np.zeros(0, np.uint8), off


def nearest_f32(fr: Fraction) -> np.float32:
    """The fp32 nearest to fr (ties to the even significand), by comparing the neighbours of
    the fp64 rounding with exact rational arithmetic."""
    if fr == 0:
        return np.float32(0.0)
    c = np.float32(float(fr))
    cands = {c, np.nextafter(c, np.float32(0)), np.nextafter(c, np.float32(np.inf))}
    best = sorted(cands, key=lambda x: (abs(Fraction(float(x)) - fr),
                                        int(np.array(x, np.float32).view(np.uint32)) & 1))
    return best[0]


def brute_q_prime(d2t, q):
    """q' by exact rationals: S = nearest fp32 of the sum of floor(q * 2^62) / 2^62 over the
    intersection, q'(y) = fp32(q(x) / S)."""
    inter = [x for x in range(len(d2t)) if d2t[x] >= 0]
    rows = []
    for r in range(q.shape[0]):
        qc = [min(max(float(v), 0.0), 1.0) if v == v else 0.0 for v in q[r]]
        total = sum(Fraction(int(Fraction(qc[x]) * 2 ** 62), 2 ** 62) for x in inter)
        S = nearest_f32(total)
        rows.append({int(d2t[x]): (np.float32(qc[x]) / S if S != 0 else np.float32(0)) for x in inter})
    return rows


def test_intersection_by_hand(orc):
    D = [b"a", b"b", b"ab", b"a", b""]
    T = [b"b", b"c", b"a", b"ab", b"b", b"abc"]
    d2t, t2d = orc.vocab_intersection(*table(D), *table(T))
    # "a" -> 2, "b" -> 0 (lowest of the two "b"), "ab" -> 3; draft 3 repeats "a"; draft 4 is empty
    assert d2t.tolist() == [2, 0, 3, -1, -1]
    assert t2d.tolist() == [1, -1, 0, 2, -1, -1]


def test_intersection_leaves_out_tokens_beyond_the_declared_length(orc):
    D = [b"abc", b"ab"]
    T = [b"ab", b"abc"]
    d2t, t2d = orc.vocab_intersection(*table(D), *table(T), vd_max_bytes=3, vt_max_bytes=2)
    assert d2t.tolist() == [-1, 0]
    assert t2d.tolist() == [1, -1]


@pytest.mark.parametrize("seed", range(4))
def test_intersection_matches_brute_force(orc, seed):
    rng = np.random.default_rng(600 + seed)
    alpha = b"xyz"

    def vocab(n):
        return [bytes(rng.choice(list(alpha), size=int(rng.integers(0, 4)))) for _ in range(n)]

    D, T = vocab(40), vocab(30)
    d2t, t2d = orc.vocab_intersection(*table(D), *table(T))
    for x, s in enumerate(D):
        lowest_d = min(i for i in range(len(D)) if D[i] == s)
        hits = [y for y in range(len(T)) if T[y] == s]
        want = hits[0] if (s and lowest_d == x and hits) else -1
        assert d2t[x] == want, (x, s)
    for y, s in enumerate(T):
        lowest_t = min(i for i in range(len(T)) if T[i] == s)
        hits = [x for x in range(len(D)) if D[x] == s]
        want = hits[0] if (s and lowest_t == y and hits) else -1
        assert t2d[y] == want, (y, s)


def identity(v):
    return np.arange(v, dtype=np.int32), np.arange(v, dtype=np.int32)


def test_normaliser_is_rounded_once(orc):
    # 1 + 3 * 2^-24 lies halfway between two fp32 neighbours of 1: ties to even give 1 + 2^-22,
    # where adding the terms one by one in fp32 would give 1
    q = np.array([[1.0, 2.0 ** -24, 2.0 ** -24, 2.0 ** -24]], np.float32)
    out = orc.tli_proposal(*identity(4), q)
    S = np.float32(1 + 2.0 ** -22)
    assert out[0, 0] == np.float32(1.0) / S
    assert np.all(out[0, 1:] == np.float32(2.0 ** -24) / S)
    naive = np.float32(0)
    for v in q[0]:
        naive = np.float32(naive + v)
    assert naive == np.float32(1.0) and out[0, 0] != np.float32(1.0)


def test_mass_below_q62_leaves_the_normaliser_but_not_the_row(orc):
    q = np.array([[0.5, 2.0 ** -70, 0.0]], np.float32)
    out = orc.tli_proposal(*identity(3), q)
    assert out[0].tolist() == [1.0, 2.0 ** -69, 0.0]


def test_rows_without_intersected_mass_are_zero(orc):
    d2t = np.array([-1, 0, -1], np.int32)
    t2d = np.array([1, -1], np.int32)
    q = np.array([[0.7, 0.0, 0.3], [np.nan, -1.0, 0.5], [0.2, 0.3, 0.5]], np.float32)
    out = orc.tli_proposal(d2t, t2d, q)
    assert out[0].tolist() == [0.0, 0.0] and out[1].tolist() == [0.0, 0.0]
    assert out[2].tolist() == [1.0, 0.0]  # the only intersected token gets all the mass


@pytest.mark.parametrize("seed", range(3))
def test_proposal_matches_exact_rationals(orc, seed):
    rng = np.random.default_rng(610 + seed)
    V_d, V_t, n = 50, 40, 4
    perm = rng.permutation(V_t)
    d2t = np.full(V_d, -1, np.int32)
    t2d = np.full(V_t, -1, np.int32)
    for x in rng.choice(V_d, 25, replace=False):
        y = int(perm[len(np.nonzero(d2t >= 0)[0])])
        d2t[x], t2d[y] = y, x
    q = rng.random((n, V_d)).astype(np.float32) ** 3
    q /= q.sum(axis=1, keepdims=True)
    q[1, 3] = np.float32(2.0 ** -140)  # a subnormal-range term and an unnormalised value
    q[2, 5] = np.float32(1.5)
    out = orc.tli_proposal(d2t, t2d, q.astype(np.float32))
    want = brute_q_prime(d2t, q)
    for r in range(n):
        for y in range(V_t):
            assert out[r, y] == want[r].get(y, np.float32(0)), (r, y)


def test_proposal_sums_to_one_and_keeps_ratios(orc):
    rng = np.random.default_rng(620)
    V = 3000
    q = rng.random((3, V)).astype(np.float32)
    q /= q.sum(axis=1, keepdims=True)
    d2t = np.where(rng.random(V) < 0.6, np.arange(V), -1).astype(np.int32)
    t2d = d2t.copy()
    out = orc.tli_proposal(d2t, t2d, q)
    inter = d2t >= 0
    assert np.all(out[:, ~inter] == 0)
    assert np.allclose(out.sum(axis=1, dtype=np.float64), 1.0, atol=V * 2.0 ** -23)
    a, b = np.nonzero(inter)[0][:2]
    assert np.allclose(out[:, a] * q[:, b], out[:, b] * q[:, a], rtol=4e-7)


@pytest.mark.parametrize("seed", [0, 1])
def test_standard_sd_on_the_tli_proposal_follows_the_target(orc, seed):
    """Alg. 3 then Alg. 4: draft tokens drawn from q' over T, verified against p; the first
    emitted token follows p (the proposal only changes the accept rate)."""
    rng = np.random.default_rng(630 + seed)
    D = [b"a", b"b", b"c", b"ab", b"q", b"zz"]
    T = [b"b", b"a", b"x", b"ab", b"y"]
    d2t, t2d = orc.vocab_intersection(*table(D), *table(T))
    V_t, N = len(T), 200_000
    q = dist(rng, len(D))[None, :]
    qp = orc.tli_proposal(d2t, t2d, q)[0]
    p = np.stack([dist(rng, V_t), dist(rng, V_t)])
    xs = draw(rng, qp, N)
    off = np.arange(N + 1, dtype=np.int32)
    nacc, tok, _, _ = orc.sd_verify(V_t, xs, off, np.tile(qp, (N, 1)), np.tile(p, (N, 1)),
                                    u24(rng, N), u24(rng, N))
    first = np.where(nacc > 0, xs, tok)
    assert chi2_pvalue(np.bincount(first, minlength=V_t), p[0]) > ALPHA


def test_given_mass_replaces_the_normaliser(orc):
    """A drafter's S (App. D Alg. 3 normalises q' on the draft side): the computed S passed back
    gives the same rows bit for bit; twice S halves every entry exactly (a power-of-two scale of
    the divisor); zero, negative or NaN S gives a zero row; S is taken as given even where it
    differs from the intersected mass."""
    rng = np.random.default_rng(5)
    v_d, v_t = 50, 40
    d2t = np.full(v_d, -1, np.int32)
    t2d = np.full(v_t, -1, np.int32)
    xs, ys = rng.choice(v_d, 30, replace=False), rng.choice(v_t, 30, replace=False)
    d2t[xs], t2d[ys] = ys, xs
    q = rng.random((6, v_d)).astype(np.float32)
    q /= q.sum(axis=1, keepdims=True)
    base = orc.tli_proposal(d2t, t2d, q)
    S = np.array([np.float32(q[r][d2t >= 0].sum()) for r in range(6)], np.float32)
    S_exact = np.array([np.float32(np.clip(q[r], 0, 1)[d2t >= 0][0]) / base[r][d2t[d2t >= 0][0]]
                        for r in range(6)], np.float32)
    same = orc.tli_proposal(d2t, t2d, q, mass=np.array([orc.round_to_f32(
        sum(int(v) for v in np.floor(q[r][d2t >= 0].astype(np.float64) * 2.0 ** 62)), 62) for r in range(6)],
        np.float32))
    assert np.array_equal(same.view(np.uint32), base.view(np.uint32))
    doubled = orc.tli_proposal(d2t, t2d, q, mass=2 * S)
    assert np.array_equal(doubled, orc.tli_proposal(d2t, t2d, q, mass=S) / np.float32(2))
    dead = orc.tli_proposal(d2t, t2d, q, mass=np.float32([0.0, -1.0, np.nan, 0.5, 0.5, 0.5]))
    assert not dead[:3].any()
    inter_y = d2t[d2t >= 0]
    inter_x = np.nonzero(d2t >= 0)[0]
    assert np.array_equal(dead[3][inter_y], q[3][inter_x] / np.float32(0.5))
    assert not np.delete(dead[3], inter_y).any()
    assert np.allclose(S_exact, S, rtol=1e-6)
