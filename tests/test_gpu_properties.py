"""Property-based GPU parity (hypothesis): generated batches of short and long pairs, band
widths and probability seeds through tt_align, tt_transfer and tt_verify, every output compared
with the oracle (bit-exact; residual rows within 1e-6 relative)."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from gpu_util import compare_align, compare_verify, gpu_run, oracle_run
from test_gpu_edges import random_tokens, vocab_of, workload

pytestmark = pytest.mark.gpu

_rng = np.random.default_rng(2024)
TOKS = random_tokens(_rng, 90, 1, 7, alphabet=b"abcdef\x00\x80")
V = vocab_of(TOKS)


def pair_lists(max_len):
    ids = st.integers(0, len(TOKS) - 1)
    return st.lists(st.tuples(st.lists(ids, min_size=1, max_size=max_len), st.lists(ids, min_size=1, max_size=max_len)),
                    min_size=1, max_size=12)


@settings(max_examples=25, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(pairs=pair_lists(20), w=st.sampled_from([-1, 0, 2, 8]), seed=st.integers(0, 2**16))
def test_short_batches_match_the_oracle(pairs, w, seed):
    wl = workload(V, V, pairs, len(TOKS), len(TOKS), w=w, seed=seed)
    g, o = gpu_run(wl, w=w, residual=True), oracle_run(wl, w=w, residual=True)
    compare_align(wl, g, o)
    compare_verify(g, o, residual=True)


@settings(max_examples=10, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(pairs=pair_lists(150), w=st.sampled_from([-1, 3, 8]))
def test_long_batches_match_the_oracle(pairs, w):
    wl = workload(V, V, pairs, len(TOKS), len(TOKS), w=w, probs=False)
    compare_align(wl, gpu_run(wl, w=w), oracle_run(wl, w=w))
