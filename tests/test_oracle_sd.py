"""Pins for the oracle's standard speculative sampling with dense proposals.

App. D Alg. 4 (standard speculative decoding over one vocabulary): drafted tokens are
kept while u_j < p_j(x_j) / q_j(x_j), the next token comes from max(0, p_r - q_r) after
a rejection at r, or from the bonus row after full acceptance.  The theorem behind
Alg. 4 (Leviathan et al. 2023, Chen et al. 2023) fixes the law of every emitted token:
it is the target's.  These tests check that law with chi-square tests, the accept count
against its closed form, the sampler against exact rational arithmetic, and the
one-hot special case against the (separately pinned) transferred-proposal verifier.
"""
from fractions import Fraction

import numpy as np
import pytest

from test_oracle_verify import ALPHA, chi2_pvalue, dist, u24


def draw(rng, q, n):
    """n draws from the distribution q (the drafter's sampling, an input to Alg. 4)."""
    cdf = np.cumsum(q.astype(np.float64))
    return np.minimum(np.searchsorted(cdf, rng.random(n), side="right"), len(q) - 1).astype(np.int32)


def batch(prows, qrows, xs, ua, us):
    """N streams with the same M = len(qrows) positions: per-stream drafted tokens xs[N, M]."""
    N, M = xs.shape
    off = (np.arange(N + 1) * M).astype(np.int32)
    draft_probs = np.tile(qrows, (N, 1)).astype(np.float32)
    target_probs = np.tile(prows, (N, 1)).astype(np.float32)
    return (prows.shape[1], xs.reshape(-1).astype(np.int32), off, draft_probs, target_probs,
            np.asarray(ua, np.float32), np.asarray(us, np.float32))


def emitted(nacc, tok, xs, k):
    """The k-th emitted token of every stream with nacc >= k (drafted, else the sample)."""
    sel = nacc >= k
    return np.where(nacc[sel] > k, xs[sel, k], tok[sel])


@pytest.mark.parametrize("seed", [0, 1])
def test_first_emitted_token_follows_target(orc, seed):
    rng = np.random.default_rng(100 + seed)
    V, M, N = 5, 2, 200_000
    prows = np.stack([dist(rng, V) for _ in range(M + 1)])
    qrows = np.stack([dist(rng, V) for _ in range(M)])
    xs = np.stack([draw(rng, qrows[j], N) for j in range(M)], axis=1)
    nacc, tok, _, _ = orc.sd_verify(*batch(prows, qrows, xs, u24(rng, N * M), u24(rng, N)))
    first = emitted(nacc, tok, xs, 0)
    assert chi2_pvalue(np.bincount(first, minlength=V), prows[0]) > ALPHA


def test_second_emitted_token_follows_target_given_first_kept(orc):
    rng = np.random.default_rng(102)
    V, M, N = 4, 2, 300_000
    prows = np.stack([dist(rng, V) for _ in range(M + 1)])
    qrows = np.stack([dist(rng, V) for _ in range(M)])
    xs = np.stack([draw(rng, qrows[j], N) for j in range(M)], axis=1)
    nacc, tok, _, _ = orc.sd_verify(*batch(prows, qrows, xs, u24(rng, N * M), u24(rng, N)))
    second = emitted(nacc, tok, xs, 1)
    assert len(second) > N // 4
    assert chi2_pvalue(np.bincount(second, minlength=V), prows[1]) > ALPHA


def test_identical_proposal_keeps_everything_and_samples_the_bonus_row(orc):
    rng = np.random.default_rng(103)
    V, M, N = 6, 3, 100_000
    prows = np.stack([dist(rng, V) for _ in range(M + 1)])
    qrows = prows[:M].copy()  # q = p: every ratio is exactly 1 > u
    xs = np.stack([draw(rng, qrows[j], N) for j in range(M)], axis=1)
    nacc, tok, _, _ = orc.sd_verify(*batch(prows, qrows, xs, u24(rng, N * M), u24(rng, N)))
    assert np.all(nacc == M)
    assert chi2_pvalue(np.bincount(tok, minlength=V), prows[M]) > ALPHA


def test_expected_accept_count_closed_form(orc):
    """E[gamma] = sum_j prod_{l <= j} min(1, p_l(x_l) / q_l(x_l)) for fixed drafted tokens."""
    rng = np.random.default_rng(104)
    V, M, N = 8, 4, 200_000
    prows = np.stack([dist(rng, V) for _ in range(M + 1)])
    qrows = np.stack([dist(rng, V) for _ in range(M)])
    x = np.array([1, 3, 5, 7], np.int32)
    ratio = np.minimum(1.0, prows[np.arange(M), x].astype(np.float64) / qrows[np.arange(M), x])
    expect = sum(np.prod(ratio[:j + 1]) for j in range(M))
    xs = np.tile(x, (N, 1))
    nacc, _, _, _ = orc.sd_verify(*batch(prows, qrows, xs, u24(rng, N * M), u24(rng, N)))
    assert abs(nacc.mean() - expect) < 5 * nacc.std() / np.sqrt(N)


def test_one_hot_proposal_rows_equal_the_transferred_verifier(orc):
    """A dense row that is a_j at x_j and 0 elsewhere is the one-hot proposal of the
    transferred verifier: every output (gamma, token, Z, residual) must be identical."""
    rng = np.random.default_rng(105)
    V, M, N = 37, 3, 400
    prows = np.stack([dist(rng, V) for _ in range(M + 1)])
    xs = rng.integers(0, V, size=(N, M)).astype(np.int32)
    a = rng.uniform(0.01, 1.0, size=(N, M)).astype(np.float32)
    a[::7, 0] = prows[0, xs[::7, 0]] * 0.5  # some certain accepts
    ua, us = u24(rng, N * M), u24(rng, N)
    off = (np.arange(N + 1) * M).astype(np.int32)
    dense = np.zeros((N * M, V), np.float32)
    dense[np.arange(N * M), xs.reshape(-1)] = a.reshape(-1)
    target_probs = np.tile(prows, (N, 1)).astype(np.float32)
    n1, t1, r1, z1 = orc.sd_verify(V, xs.reshape(-1), off, dense, target_probs, ua, us, residual=True)
    n2, t2, r2, z2 = orc.verify(V, xs.reshape(-1), off, a.reshape(-1), target_probs, ua, us, residual=True)
    assert np.array_equal(n1, n2) and np.array_equal(t1, t2) and np.array_equal(z1, z2)
    assert np.array_equal(r1.view(np.uint32), r2.view(np.uint32))
    assert 0 < (n1 == 0).sum() < N  # both branches exercised


def _q62(row):
    return [int(Fraction(float(x)) * 2**62) for x in row]


def test_sampler_matches_exact_rational_inverse_cdf(orc):
    rng = np.random.default_rng(106)
    V, M = 11, 1
    for trial in range(10):
        prows = np.stack([dist(rng, V) for _ in range(M + 1)])
        qrows = np.stack([dist(rng, V) for _ in range(M)])
        us = np.concatenate([u24(rng, 200), np.float32([0.0, 1 - 2**-24, 2**-24, 0.5])])
        N = len(us)
        xs = np.tile(np.array([int(np.argmin(prows[0] / qrows[0]))], np.int32), (N, 1))
        ua = u24(rng, N)
        nacc, tok, _, z = orc.sd_verify(*batch(prows, qrows, xs, ua, us))
        for n in range(N):
            r = int(nacc[n])
            if r == 0:
                R = [max(np.float32(0), np.float32(prows[0][y] - qrows[0][y])) for y in range(V)]
            else:
                R = list(prows[1])
            Rq = _q62(R)
            Z = sum(Rq)
            assert int(z[n]) == Z
            T = int(Fraction(float(us[n])) * Z)
            acc, want = 0, None
            for y in range(V):
                acc += Rq[y]
                if acc > T:
                    want = y
                    break
            assert int(tok[n]) == want


def test_residual_row_is_normalised_and_zero_where_draft_dominates(orc):
    rng = np.random.default_rng(107)
    V, M, N = 300, 2, 50
    prows = np.stack([dist(rng, V) for _ in range(M + 1)])
    qrows = np.stack([dist(rng, V) for _ in range(M)])
    xs = rng.integers(0, V, size=(N, M)).astype(np.int32)
    nacc, tok, res, _ = orc.sd_verify(*batch(prows, qrows, xs, u24(rng, N * M), u24(rng, N)), residual=True)
    for n in range(N):
        assert abs(float(res[n].astype(np.float64).sum()) - 1.0) < V * 2**-23
        r = int(nacc[n])
        if r < M:
            assert np.all(res[n][qrows[r] >= prows[r]] == 0)
        assert res[n][tok[n]] > 0


def test_sentinels_and_empty_streams(orc):
    rng = np.random.default_rng(108)
    V = 6
    p = np.stack([dist(rng, V) for _ in range(6)])
    q = np.stack([dist(rng, V) for _ in range(3)])
    # stream 0: M = 0 (bonus row 0); stream 1: drafted id out of range; stream 2: M = 2 > max_m = 1
    ids = np.array([V, 1, 2], np.int32)
    off = np.array([0, 0, 1, 3], np.int32)
    # target rows: stream 0 -> row 0; stream 1 -> rows 1..2; stream 2 -> rows 3..5
    nacc, tok, _, z = orc.sd_verify(V, ids, off, q, p, u24(rng, 3), np.float32([0.3, 0.3, 0.3]), max_m=1)
    assert nacc.tolist()[1:] == [-1, -1] and tok.tolist()[1:] == [-1, -1]
    assert nacc[0] == 0 and 0 <= tok[0] < V and z[0] > 0
