"""Pins for the oracle's transfer, acceptance and residual sampling.

Sec. 3 "Standard Speculative Sampling", Sec. 4.2.2 (acceptance rule and first
rejection), Sec. 4.2.3 / Alg. 2 (sample after the accepted prefix), App. D
Alg. 4 (residual "modified distribution"), App. A.2 / Limitations (one-hot
transferred proposal).  Distributional claims are checked with chi-square
tests; the sampler itself is checked exactly against rational arithmetic.
"""
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

ALPHA = 1e-3


def batch_single_position(p0, p1, tok, qv, ua, us):
    """N independent streams with M=1: proposal `tok` with transferred mass qv.

    Rows per stream: target row 0 (= p0) and the bonus row 1 (= p1).
    """
    n = len(ua)
    V = len(p0)
    target_ids = np.full(n, tok, np.int32)
    target_off = np.arange(n + 1, dtype=np.int32)
    rows = np.empty((2 * n, V), np.float32)
    rows[0::2] = p0
    rows[1::2] = p1
    q = np.full(n, qv, np.float32)
    return V, target_ids, target_off, q, rows, np.asarray(ua, np.float32), np.asarray(us, np.float32)


def u24(rng, n):
    return (rng.integers(0, 1 << 24, size=n).astype(np.float64) * 2.0**-24).astype(np.float32)


def first_token(nacc, tok, proposal):
    return np.where(nacc >= 1, proposal, tok)


def chi2_pvalue(counts, probs):
    probs = np.asarray(probs, np.float64)
    keep = probs > 0
    assert counts[~keep].sum() == 0
    if keep.sum() == 1:
        return 1.0  # a single admissible outcome: the check above is the whole test
    exp = probs[keep] / probs[keep].sum() * counts.sum()
    return stats.chisquare(counts[keep], exp).pvalue


def dist(rng, V):
    p = rng.random(V).astype(np.float32) + np.float32(0.05)
    return (p / p.sum(dtype=np.float32)).astype(np.float32)


@pytest.mark.parametrize("seed", [0, 1])
def test_one_hot_full_mass_reproduces_target(orc, seed):
    """With transferred mass 1 the emitted first token is distributed exactly as P_t."""
    rng = np.random.default_rng(seed)
    V, N = 6, 400_000
    p0, p1 = dist(rng, V), dist(rng, V)
    tok = int(rng.integers(0, V))
    args = batch_single_position(p0, p1, tok, 1.0, u24(rng, N), u24(rng, N))
    nacc, out, _, _ = orc.verify(*args)
    ft = first_token(nacc, out, tok)
    assert chi2_pvalue(np.bincount(ft, minlength=V), p0) > ALPHA


@pytest.mark.parametrize("a", [0.05, 0.3, 0.9])
def test_one_hot_partial_mass_closed_form(orc, a):
    """With mass a in (0,1) the law is the closed form below, not P_t.

    If a <= p(t): t with probability 1.  Otherwise t with probability p(t)/a and
    x != t with probability (1 - p(t)/a) p(x) / sum_{y != t} p(y).
    """
    rng = np.random.default_rng(int(a * 100))
    V, N = 5, 400_000
    p0, p1 = dist(rng, V), dist(rng, V)
    tok = 2
    args = batch_single_position(p0, p1, tok, a, u24(rng, N), u24(rng, N))
    nacc, out, _, _ = orc.verify(*args)
    ft = first_token(nacc, out, tok)
    pt = float(p0[tok])
    acc = min(1.0, pt / a)
    law = np.array([(1 - acc) * float(p0[x]) / (1 - pt) for x in range(V)])
    law[tok] = acc
    assert chi2_pvalue(np.bincount(ft, minlength=V), law) > ALPHA
    # and the acceptance frequency itself
    assert abs((nacc == 1).mean() - acc) < 5 * np.sqrt(acc * (1 - acc) / N + 1e-12)


def test_bonus_row_when_everything_is_accepted(orc):
    rng = np.random.default_rng(3)
    V, N = 7, 300_000
    p0, p1 = dist(rng, V), dist(rng, V)
    tok = 4
    p0 = p0.copy()
    args = batch_single_position(p0, p1, tok, float(p0[tok]) * 0.5, u24(rng, N), u24(rng, N))
    nacc, out, _, _ = orc.verify(*args)
    assert np.all(nacc == 1)  # ratio 2 > u always
    assert chi2_pvalue(np.bincount(out, minlength=V), p1) > ALPHA


def test_dense_proposal_output_law_is_target(orc):
    """App. D Alg. 4 with a genuine dense proposal: the emitted token follows P_t exactly."""
    rng = np.random.default_rng(4)
    V, N = 5, 200_000
    p, qd = dist(rng, V), dist(rng, V)
    cdf = np.cumsum(qd.astype(np.float64))
    xs = np.minimum(np.searchsorted(cdf, rng.random(N), side="right"), V - 1)
    ua, us = u24(rng, N), u24(rng, N)
    out = np.array([orc.verify_dense(p, qd, int(x), float(a), float(s))[0]
                    for x, a, s in zip(xs, ua, us)])
    assert chi2_pvalue(np.bincount(out, minlength=V), p) > ALPHA


def test_expected_accept_count_closed_form(orc):
    """P(gamma >= j) = prod_{l <= j} min(1, P_t(t_l) / q_l) for independent uniforms."""
    rng = np.random.default_rng(5)
    V, M, N = 8, 4, 200_000
    rows = np.stack([dist(rng, V) for _ in range(M + 1)])
    toks = np.array([1, 3, 5, 7], np.int32)
    qs = np.array([0.5, 0.05, 0.2, 0.9], np.float32)
    ratio = np.minimum(1.0, rows[np.arange(M), toks].astype(np.float64) / qs)
    expect = sum(np.prod(ratio[:j + 1]) for j in range(M))
    target_ids = np.tile(toks, N)
    target_off = (np.arange(N + 1) * M).astype(np.int32)
    big = np.tile(rows, (N, 1)).astype(np.float32)
    q = np.tile(qs, N)
    nacc, _, _, _ = orc.verify(V, target_ids, target_off, q, big, u24(rng, N * M), u24(rng, N))
    se = nacc.std() / np.sqrt(N)
    assert abs(nacc.mean() - expect) < 5 * se


def test_accept_rule_edges(orc):
    V = 4
    p0 = np.array([0.0, 0.5, 0.25, 0.25], np.float32)
    p1 = np.array([0.25, 0.25, 0.25, 0.25], np.float32)
    # q = 0 -> accepted; P_t(t) = 0 -> rejected; NaN q -> rejected; u = 0 with ratio > 0 accepted
    cases = [(1, 0.0, 0.99, True), (0, 0.3, 0.0, False), (1, np.nan, 0.1, False), (2, 0.5, 0.0, True),
             (2, 0.25, 0.999999, True), (2, 0.26, 0.99, False)]
    for tok, qv, ua, acc in cases:
        args = batch_single_position(p0, p1, tok, qv, [ua], [0.5])
        nacc, _, _, _ = orc.verify(*args)
        assert int(nacc[0]) == (1 if acc else 0), (tok, qv, ua)


def _q62(row):
    return [int(Fraction(float(x)) * 2**62) for x in row]  # floor of exact value


def test_sampler_matches_exact_rational_inverse_cdf(orc):
    """token = first x with prefix(x) > floor(u * Z) where every quantity is exact."""
    rng = np.random.default_rng(6)
    V = 9
    for trial in range(20):
        p0, p1 = dist(rng, V), dist(rng, V)
        tok = int(rng.integers(0, V))
        qv = float(rng.uniform(0.05, 1.0))
        us = np.concatenate([u24(rng, 300), np.float32([0.0, 1 - 2**-24, 2**-24, 0.5])])
        ua = np.full(len(us), 0.999999, np.float32)  # force rejection unless ratio ~ 1
        args = batch_single_position(p0, p1, tok, qv, ua, us)
        nacc, out, _, z = orc.verify(*args)
        for n in range(len(us)):
            r = int(nacc[n])
            if r == 0:
                R = [max(np.float32(0), np.float32(p0[x] - (np.float32(qv) if x == tok else 0)))
                     for x in range(V)]
            else:
                R = list(p1)
            Rq = _q62(R)
            Z = sum(Rq)
            assert int(z[n]) == Z
            T = int(Fraction(float(us[n])) * Z)
            acc, want = 0, None
            for x in range(V):
                acc += Rq[x]
                if acc > T:
                    want = x
                    break
            assert int(out[n]) == want


def test_sampler_frequency_over_all_uniform_grid(orc):
    """Over the whole 2^-24 grid each token is hit floor-exactly R_q(x)/Z of the time."""
    rng = np.random.default_rng(9)
    V = 5
    p1 = dist(rng, V)
    Rq = _q62(list(p1))
    Z = sum(Rq)
    counts = []
    prefix = 0
    for x in range(V):
        lo, hi = prefix, prefix + Rq[x]
        # #{k in [0, 2^24): lo <= floor(k Z / 2^24) < hi} = ceil(hi 2^24 / Z) - ceil(lo 2^24 / Z)
        counts.append((-((-hi * 2**24) // Z)) - (-((-lo * 2**24) // Z)))
        prefix = hi
    assert sum(counts) == 2**24
    for x in range(V):
        assert abs(counts[x] - Fraction(Rq[x], Z) * 2**24) <= 1
    # the oracle agrees on a sample of grid points, including every bucket boundary
    ks = set(int(k) for k in rng.integers(0, 2**24, size=400))
    edge = 0
    for x in range(V):
        edge += counts[x]
        ks.update({max(0, edge - 1), min(2**24 - 1, edge)})
    ks = sorted(ks)
    us = np.array([k * 2.0**-24 for k in ks], np.float32)
    args = batch_single_position(p1, p1, 0, 0.0, np.zeros(len(us)), us)  # q = 0 -> accept -> bonus row
    nacc, out, _, _ = orc.verify(*args)
    assert np.all(nacc == 1)
    bounds = np.cumsum(counts)
    for k, o in zip(ks, out):
        assert int(o) == int(np.searchsorted(bounds, k, side="right"))


def test_exact_threshold_against_fractions(orc):
    rng = np.random.default_rng(10)
    for _ in range(2000):
        u = np.float32(rng.random())
        if rng.random() < 0.2:
            u = np.float32(rng.random() * 2.0 ** -int(rng.integers(20, 140)))
        Z = int(rng.integers(1, 2**63, dtype=np.uint64)) * (1 if rng.random() < 0.5 else 2) - 1
        Z = max(1, min(Z, 2**64 - 1))
        assert orc.threshold(float(u), Z) == min(int(Fraction(float(u)) * Z), Z - 1)
    assert orc.threshold(0.0, 10) == 0
    assert orc.threshold(-0.5, 10) == 0
    assert orc.threshold(1.0, 10) == 9


def test_residual_row_normalised(orc):
    rng = np.random.default_rng(12)
    V, N = 1000, 16
    p0, p1 = dist(rng, V), dist(rng, V)
    args = batch_single_position(p0, p1, 17, 0.9, u24(rng, N), u24(rng, N))
    nacc, out, res, z = orc.verify(*args, residual=True)
    for n in range(N):
        assert abs(float(res[n].sum(dtype=np.float64)) - 1.0) < V * 2.0**-23
        if nacc[n] == 0:
            assert res[n][17] == 0.0  # the rejected proposal carries no residual mass
        assert res[n][out[n]] > 0


def test_zero_mass_fallback_is_first_argmax(orc):
    V = 6
    p0 = np.array([0.0, 0.0, 1.0, 0.0, 0.0, 0.0], np.float32)  # all mass on the proposal
    p1 = np.zeros(V, np.float32)
    args = batch_single_position(p0, p1, 2, 2.0, [0.9], [0.3])  # q > 1: rejected, residual empty
    nacc, out, res, z = orc.verify(*args, residual=True)
    assert int(nacc[0]) == 0 and int(z[0]) == 0 and int(out[0]) == 2
    assert list(res[0]) == [0, 0, 1, 0, 0, 0]


def test_stream_sentinels(orc):
    V = 4
    p = np.full(V, 0.25, np.float32)
    rows = np.tile(p, (6, 1))
    target_ids = np.array([1, 9, 2, 1, 1], np.int32)  # stream 1 holds id 9 >= V
    target_off = np.array([0, 1, 2, 5], np.int32)  # stream 2 has M = 3 > max_m = 2
    q = np.full(5, 0.5, np.float32)
    nacc, out, _, _ = orc.verify(V, target_ids, target_off, q, rows, np.full(5, 0.1, np.float32),
                                 np.full(3, 0.5, np.float32), max_m=2)
    assert int(nacc[0]) == 1 and list(nacc[1:]) == [-1, -1] and list(out[1:]) == [-1, -1]


def test_transfer_gathers_emitted_token_probability(orc):
    rng = np.random.default_rng(13)
    Vd = 50
    draft_ids = np.array([3, 7, 11, 49, 0], np.int32)
    draft_off = np.array([0, 3, 5], np.int32)
    target_off = np.array([0, 4, 6], np.int32)
    mp = np.array([0, 1, 1, 2, 0, 1], np.int32)
    probs = rng.random((5, Vd)).astype(np.float32)
    q = orc.transfer(Vd, draft_ids, draft_off, target_off, mp, probs)
    want = [probs[0, 3], probs[1, 7], probs[1, 7], probs[2, 11], probs[3, 49], probs[4, 0]]
    assert np.array_equal(q, np.array(want, np.float32))
    bad = orc.transfer(Vd, draft_ids, draft_off, target_off, np.array([0, 3, -1, 2, 0, 1], np.int32), probs)
    assert np.isnan(bad[1]) and np.isnan(bad[2]) and bad[0] == probs[0, 3]
