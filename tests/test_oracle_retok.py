"""Pins for the oracle's re-tokenisation (Sec. 4.2.1, Alg. 2, App. A.1) with a greedy
longest-match target tokenizer: the string-consistency lemma, the longest-match property
checked by brute force over the whole vocabulary, agreement with the input generator's
own encoder (written separately), lowest id among equal strings, and the failure cases."""
import numpy as np

from paper_2510_15545_amd import synth


def table(tokens):
    off = np.zeros(len(tokens) + 1, np.int64)
    off[1:] = np.cumsum([len(t) for t in tokens])
    return np.frombuffer(b"".join(tokens), np.uint8), off


def test_string_consistency_and_longest_match(orc):
    for index, n in ((1, 1), (2, 6), (5, 4)):
        wl = synth.make(index, n_streams=n, probs=False)
        vd, vt = wl.vocab_d, wl.vocab_t
        ids, off = orc.retokenize(vd.data, vd.offsets, vt.data, vt.offsets, wl.draft_ids, wl.draft_off)
        toks_t = vt.tokens
        for b in range(wl.n):
            S = b"".join(vd.tokens[i] for i in wl.draft_ids[wl.draft_off[b]:wl.draft_off[b + 1]])
            T = [toks_t[i] for i in ids[off[b]:off[b + 1]]]
            assert b"".join(T) == S  # App. A.1: identical in the string space
            p = 0
            for t in T:  # no vocabulary token longer than t also prefixes the rest (brute force)
                longer = [u for u in toks_t if len(u) > len(t) and S.startswith(u, p)]
                assert not longer, (b, p, t, longer[:3])
                p += len(t)
        # the generator's encoder is an independent implementation of the same tokenizer
        assert np.array_equal(ids, wl.target_ids) and np.array_equal(off, wl.target_off)
    for index in (2, 3, 4, 5):  # every workload's batch (long pairs included)
        wl = synth.make(index, n_streams=64, probs=False)
        ids, off = orc.retokenize(wl.vocab_d.data, wl.vocab_d.offsets, wl.vocab_t.data, wl.vocab_t.offsets,
                                  wl.draft_ids, wl.draft_off)
        assert np.array_equal(ids, wl.target_ids) and np.array_equal(off, wl.target_off)


def test_lowest_id_among_equal_strings_and_failures(orc):
    vd_tokens = [b"ab", b"c", b"abc", b"z", b"q"]
    vt_tokens = [b"a", b"bc", b"b", b"c", b"abc", b"bc", b"ab"]  # "bc" twice: ids 1 and 5
    vd, vdo = table(vd_tokens)
    vt, vto = table(vt_tokens)
    streams = [[0, 1], [2], [1, 0], [3], [], [0, 1, 1], [4 + 5]]
    ids = np.array([x for s in streams for x in s], np.int32)
    off = np.array([0] + list(np.cumsum([len(s) for s in streams])), np.int32)
    got, goff = orc.retokenize(vd, vdo, vt, vto, ids, off, max_m=2)
    rows = [got[goff[b]:goff[b + 1]].tolist() for b in range(len(streams))]
    assert rows[0] == [4]        # "abc" -> the whole string
    assert rows[1] == [4]
    assert rows[2] == [3, 6]     # "cab" -> c, ab
    assert rows[3] == []         # "z": no target token starts with it
    assert rows[4] == []         # empty draft
    assert rows[5] == [4, 3]     # "abcc" -> abc, c
    assert rows[6] == []         # draft id outside the table
    got, goff = orc.retokenize(vd, vdo, vt, vto, ids, off, max_m=1)
    assert goff[6] - goff[5] == 0 and goff[3] - goff[2] == 0  # more than max_m tokens
    assert got[goff[0]:goff[1]].tolist() == [4]
    # "bc" resolves to the lower of its two ids
    got, goff = orc.retokenize(vt, vto, vt, vto, np.array([1, 5], np.int32), np.array([0, 2], np.int32))
    assert got.tolist() == [1, 1]
    # a string longer than max_bytes gets no tokens
    got, goff = orc.retokenize(vd, vdo, vt, vto, ids, off, max_bytes=3)
    assert goff[6] - goff[5] == 0 and goff[1] - goff[0] == 1
