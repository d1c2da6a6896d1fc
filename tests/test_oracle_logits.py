"""Pins for the oracle's verification from bf16 logits (the target softmax formed inside the
verification, with the sampling temperatures of App. F).

The specified base-2 exponential is checked against 2^z in float64 (a relative bound over a
dense grid, exact powers of two) and the per-logit probability against exp in float64; the
verification is checked against
laws computed independently in float64: with a one-hot proposal of mass 1 the emitted token
follows softmax(logit / T), and after a rejection it follows the closed form of the
transferred-proposal law (min(1, p/q) at the proposal, the rest in proportion); an exactly
representable softmax fixes the acceptance boundary; invalid streams give sentinels.  With
caller-supplied log-sum-exp values the same laws hold, and a normaliser that makes the softmax
exact fixes the boundary there too.
"""
import math

import numpy as np
import pytest

from test_oracle_verify import ALPHA, chi2_pvalue, u24


def bf16_bits(x):
    """Round fp32 values to bf16 (ties to even), returned as uint16 bit patterns."""
    b = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def bf16_value(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


def softmax64(x):
    x = np.asarray(x, np.float64)
    e = np.exp(x - x.max())
    return e / e.sum()


def row_lse(bits, row_it):
    """Each row's log-sum-exp of bf16 logit * inv_temp (NaN as -inf), in float64, rounded to fp32."""
    x = bf16_value(bits).astype(np.float32) * np.asarray(row_it, np.float32)[:, None]
    x = np.where(np.isnan(x), -np.inf, x).astype(np.float64)
    m = x.max(axis=1)
    with np.errstate(invalid="ignore", divide="ignore"):
        s = np.log(np.exp(x - np.where(np.isfinite(m), m, 0)[:, None]).sum(axis=1)) + m
    return s.astype(np.float32)


def ulps(a: np.float32, b: float) -> float:
    """|a - b| in units of the fp32 spacing at b."""
    return abs(float(a) - b) / float(np.spacing(np.float32(b)))


def test_exp2_relative_error_and_exact_points(orc):
    """The specified 2^z (degree-5 Taylor polynomial of 2^f on [-1/2, 1/2] after k = rint(z)):
    within 3.5e-6 of 2^z (float64) over [-1, 31], exactly 2^k at integers, held at the ends of
    [-1, 31] (NaN as -1)."""
    zs = np.concatenate([np.linspace(-1.0, 31.0, 64001), np.linspace(-1.0, 1.0, 4001)]).astype(np.float32)
    rel = max(abs(float(orc.exp2(z)) / 2.0 ** float(z) - 1.0) for z in zs)
    assert rel <= 3.5e-6, rel
    for k in range(-1, 32):
        assert orc.exp2(float(k)) == np.float32(2.0 ** k)
    assert orc.exp2(40.0) == orc.exp2(31.0) == np.float32(2.0 ** 31)
    assert orc.exp2(-7.0) == orc.exp2(-1.0) == np.float32(0.5)
    assert orc.exp2(float("nan")) == np.float32(0.5) and orc.exp2(float("-inf")) == np.float32(0.5)
    assert orc.exp2(float("inf")) == np.float32(2.0 ** 31)


def test_logit_prob_against_the_natural_softmax(orc):
    """With a caller's log-sum-exp L, P(x) approximates exp(x * it - L) (float64) within the
    exponential's error and the fp32 rounding of its arguments, is 0 where exp(x * it - L) is
    below 2^-31 and 1 above the normaliser."""
    rng = np.random.default_rng(9)
    for _ in range(2000):
        x = np.float32(rng.normal(0, 4))
        it = np.float32(rng.uniform(0.5, 2.0))
        L = np.float32(x * it + rng.uniform(0.0, 20.0))
        want = math.exp(float(x) * float(it) - float(L))
        got = float(orc.logit_prob(x, it, L))
        assert abs(got - want) <= 2e-5 * want + 2.0 ** -31, (x, it, L, got, want)
    assert orc.logit_prob(0.0, 1.0, 30.0) == 0.0  # exp(-30) < 2^-31 x 2^... : below the cut
    assert orc.logit_prob(5.0, 1.0, 0.0) == 1.0


def one_position_batch(rng, logits_rows, q, N, t=None):
    """N streams with M = 1 over the same two rows (position 0 and the bonus row)."""
    V = logits_rows.shape[1]
    ids = np.full(N, t if t is not None else 0, np.int32)
    off = np.arange(N + 1, dtype=np.int32)
    rows = np.tile(logits_rows, (N, 1))
    return V, ids, off, np.full(N, q, np.float32), rows


@pytest.mark.parametrize("with_lse", [False, True])
@pytest.mark.parametrize("temp", [1.0, 0.7])
def test_emitted_token_follows_the_tempered_softmax(orc, temp, with_lse):
    """q = 1 at the proposal: accept with probability p(t), else the residual (p without t,
    renormalised), so the emitted token's law is p = softmax(logit / T)."""
    rng = np.random.default_rng(80)
    V, N, t = 6, 200_000, 2
    bits = bf16_bits(rng.normal(0, 1.5, (2, V)).astype(np.float32))
    it = np.float32(1.0 / temp)
    V, ids, off, q, rows = one_position_batch(rng, bits, 1.0, N, t)
    lse = row_lse(rows, np.full(len(rows), it)) if with_lse else None
    nacc, tok, _ = orc.verify_logits(V, ids, off, q, rows, np.full(N, it, np.float32), u24(rng, N), u24(rng, N),
                                     lse=lse)
    first = np.where(nacc > 0, t, tok)
    p = softmax64(bf16_value(bits[0]) * it)
    assert chi2_pvalue(np.bincount(first, minlength=V), p) > ALPHA
    assert abs(np.mean(nacc) - p[t]) < 5 * math.sqrt(p[t] * (1 - p[t]) / N)


@pytest.mark.parametrize("with_lse", [False, True])
def test_rejection_law_closed_form(orc, with_lse):
    """One-hot proposal of mass a at t: P(out = t) = min(1, p(t)/a), any other x in proportion
    to p(x) -- the transferred-proposal law, here with p = softmax(logit)."""
    rng = np.random.default_rng(81)
    V, N, t, a = 5, 200_000, 1, 0.6
    bits = bf16_bits(np.array([[0.2, 0.9, -0.4, 0.0, 0.5], [0.0] * 5], np.float32))
    V, ids, off, q, rows = one_position_batch(rng, bits, a, N, t)
    lse = row_lse(rows, np.ones(len(rows))) if with_lse else None
    nacc, tok, _ = orc.verify_logits(V, ids, off, q, rows, np.ones(N, np.float32), u24(rng, N), u24(rng, N),
                                     lse=lse)
    out = np.where(nacc > 0, t, tok)
    p = softmax64(bf16_value(bits[0]))
    keep = min(1.0, p[t] / a)
    law = np.array([(1 - keep) * p[x] / (1 - p[t]) for x in range(V)])
    law[t] = keep
    assert chi2_pvalue(np.bincount(out, minlength=V), law) > ALPHA


def test_exact_softmax_fixes_the_accept_boundary(orc):
    """Eight logits 0: every z = 31 exactly, e31 = 2^31, S = 8, p(t) = 1/8; with q = 1/4 the
    ratio is 1/2, so u = 1/2 - 2^-24 accepts and u = 1/2 rejects."""
    V = 8
    bits = bf16_bits(np.full((2, V), 0.0, np.float32))
    for u, want in ((0.5 - 2.0 ** -24, 1), (0.5, 0)):
        nacc, tok, z = orc.verify_logits(V, np.array([3], np.int32), np.array([0, 1], np.int32),
                                         np.array([0.25], np.float32), bits, np.ones(1, np.float32),
                                         np.array([u], np.float32), np.array([0.0], np.float32))
        assert nacc[0] == want
        if want == 0:  # residual: p(t) - q < 0, so t has no mass; Z = 7 * 2^31; u_sample = 0 -> first token
            assert int(z[0]) == 7 * 2 ** 31 and tok[0] == 0


def test_exact_normaliser_fixes_the_accept_boundary(orc):
    """The normaliser is taken as given: logit 0 with L = 0 gives P = 2^0 = 1 whatever the
    other logits are, so with q = 1/2 every u accepts; with L = ln 2 (fp32) and q = 1,
    P = 2^(-L log2 e) is within an ulp of 1/2 and u just below P accepts, u = P rejects."""
    V = 4
    bits = bf16_bits(np.array([[0.0, -5.0, -5.0, -5.0], [0.0] * 4], np.float32))
    one = lambda lse0, qv, u: orc.verify_logits(V, np.array([0], np.int32), np.array([0, 1], np.int32),
                                                np.array([qv], np.float32), bits, np.ones(1, np.float32),
                                                np.array([u], np.float32), np.array([0.0], np.float32),
                                                lse=np.array([lse0, 0.0], np.float32))
    assert one(0.0, 0.5, 1.0 - 2.0 ** -24)[0][0] == 1
    L = np.float32(math.log(2.0))
    P = float(orc.logit_prob(0.0, 1.0, L))
    assert abs(P - 0.5) <= 2.0 ** -24
    below = np.nextafter(np.float32(P), np.float32(0))
    assert one(L, 1.0, below)[0][0] == 1 and one(L, 1.0, np.float32(P))[0][0] == 0
    # rejected: the residual row 0 has mass only off the proposal; u_sample = 0 -> index 1
    nacc, tok, z = one(L, 1.0, np.float32(P))
    assert tok[0] == 1 and int(z[0]) > 0


def test_sentinels_nan_and_empty_rows(orc):
    V = 4
    bits = bf16_bits(np.zeros((7, V), np.float32))
    bits[5] = 0x7FC0                      # NaN logits: no mass
    bits[5, 2] = bf16_bits(np.float32(1.0))
    bits[6] = 0xFF80                      # -inf everywhere: Z = 0, token 0
    ids = np.array([1, 9, 0, 0], np.int32)  # stream 1 has an id outside [0, V)
    off = np.array([0, 1, 2, 3, 3], np.int32)
    # stream b's rows start at off[b] + b: stream 0 rows 0-1, stream 1 rows 2-3, stream 2 rows 4-5, stream 3 row 6
    q = np.ones(3, np.float32)
    it = np.array([1, 1, 1, 1], np.float32)
    ua = np.array([0.99, 0.99, 0.0], np.float32)  # stream 2 accepts its proposal
    nacc, tok, z = orc.verify_logits(V, ids, off, q, bits, it, ua, np.array([0.3, 0.3, 0.3, 0.7], np.float32))
    assert nacc[1] == -1 and tok[1] == -1
    assert nacc[2] == 1 and tok[2] == 2     # the bonus row's only finite logit (the rest are NaN)
    assert nacc[3] == 0 and tok[3] == 0 and int(z[3]) == 0
    bad_t = orc.verify_logits(V, ids[:1], off[:2], q[:1], bits, np.array([0.0], np.float32), ua[:1], ua[:1])
    assert bad_t[0][0] == -1
