"""The seeded input generator: string consistency, ranges, determinism, prefix property."""
import numpy as np
import pytest

from paper_2510_15545_amd import synth


@pytest.mark.parametrize("c,n", [(1, None), (2, 32), (3, 6), (4, 6), (5, 6)])
def test_generated_streams(c, n):
    wl = synth.make(c, n_streams=n)
    spec = synth.SPECS[c]
    vd, vt = wl.vocab_d, wl.vocab_t
    assert vd.n == spec.vd and vt.n == spec.vt
    for sym in spec.alphabet:  # every single symbol is a token on both sides
        assert bytes([sym]) in vd.index and bytes([sym]) in vt.index
    assert vd.max_len <= spec.max_len and vt.max_len <= spec.max_len
    for b in range(wl.n):
        d = wl.draft_ids[wl.draft_off[b]:wl.draft_off[b + 1]]
        t = wl.target_ids[wl.target_off[b]:wl.target_off[b + 1]]
        assert vd.decode(d) == vt.decode(t)  # App. A.1: identical byte strings
        if spec.k:
            assert len(d) == spec.k
        if spec.m_range:
            assert spec.m_range[0] <= len(t) <= spec.m_range[1]
    sub = wl.prob if c == 4 else wl
    rows_t = int(sub.target_off[-1]) + sub.n
    assert sub.target_probs.shape == (rows_t, sub.v_t)
    assert sub.draft_probs.shape == (int(sub.draft_off[-1]), sub.v_d)
    sums = sub.target_probs.sum(axis=1, dtype=np.float64)
    assert np.all(np.abs(sums - 1) < 1e-4) and np.all(sub.target_probs >= 0)
    assert np.all(sub.verify_ids < sub.v_t)
    # uniforms lie on the 2^-24 grid in [0, 1)
    k = sub.u_accept.astype(np.float64) * 2**24
    assert np.all(k == np.floor(k)) and np.all(sub.u_accept < 1) and np.all(sub.u_sample >= 0)


def test_deterministic_and_prefix_stable():
    a = synth.make(2, n_streams=8)
    b = synth.make(2, n_streams=4)
    assert np.array_equal(a.draft_ids[:a.draft_off[4]], b.draft_ids)
    assert np.array_equal(a.target_ids[:a.target_off[4]], b.target_ids)
    rows = int(b.target_off[-1]) + 4
    assert np.array_equal(a.target_probs[:rows], b.target_probs)
    assert np.array_equal(a.u_accept[:b.target_off[-1]], b.u_accept)
    assert np.array_equal(a.u_sample[:4], b.u_sample)
    c = synth.make(2, n_streams=4)
    assert np.array_equal(c.target_probs, b.target_probs) and np.array_equal(c.u_sample, b.u_sample)


def test_forcing_raises_proposal_mass():
    wl = synth.make(3, n_streams=24)
    rows = wl.target_off[:-1]
    f = wl.forced.astype(bool)
    assert 0.1 < f.mean() < 0.5
    p = np.array([wl.target_probs[wl.target_off[b] + b + j, wl.target_ids[wl.target_off[b] + j]]
                  for b in range(wl.n) for j in range(wl.target_off[b + 1] - wl.target_off[b])])
    assert np.median(p[f]) > 100 * np.median(p[~f])
    assert len(rows) == wl.n


def test_greedy_longest_match():
    v = synth.make_vocab(12, b"ab", 3, 0)
    t = synth.greedy_encode(b"abababba", v)
    assert v.decode(t) == b"abababba"
    # longest match: the first token is the longest vocabulary prefix
    first = v.tokens[t[0]]
    for ln in range(len(first) + 1, 4):
        assert b"abababba"[:ln] not in v.index
