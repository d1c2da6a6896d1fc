"""tt_delta_histogram (Sec. 5 Fig. CDF, App. K) against the oracle's histogram of the
oracle's own alignment: exact counts for short and long pairs, with and without a band,
sentinel and oversize pairs, one-bin and overflow cases, and replays of a captured HIP graph;
tt_delta_quantile (App. K's 0.9 rule) against the oracle's quantile of the same counts."""
import numpy as np
import pytest

import oracle
from gpu_util import gpu_align, oracle_run, to_dev, upload
from paper_2510_15545_amd import synth

pytestmark = pytest.mark.gpu


def gpu_hist(wl, d, plen, path, n_bins):
    import torch

    import paper_2510_15545_amd as tt

    h = tt.delta_histogram(d["draft_off"], d["target_off"], plen, path, n_bins)
    torch.cuda.synchronize()
    return h.cpu().numpy().astype(np.int64)


@pytest.mark.parametrize("index,w,n_bins", [(2, -1, 16), (2, 8, 4), (3, -1, 64), (5, 8, 1), (5, 8, 40)])
def test_histogram_matches_oracle(index, w, n_bins):
    print(f"[case] delta histogram workload {index} w={w} bins={n_bins}", flush=True)
    wl = synth.make(index, n_streams=64, probs=False, w=w)
    d = upload(wl)
    cost, plen, path, mp = gpu_align(wl, d, w)
    g = gpu_hist(wl, d, plen, path, n_bins)
    o = oracle_run(wl, w)
    want = oracle.delta_histogram(wl.draft_off, wl.target_off, o["path_len"], o["path"], n_bins)
    assert np.array_equal(g, want), (g, want)
    assert g.sum() == o["path_len"].sum()


def test_histogram_long_pairs():
    print("[case] delta histogram long pairs", flush=True)
    wl = synth.make(4, n_streams=48, probs=False, w=-1)
    d = upload(wl)
    cost, plen, path, mp = gpu_align(wl, d, -1)
    g = gpu_hist(wl, d, plen, path, 600)
    o = oracle_run(wl, -1)
    assert np.array_equal(g, oracle.delta_histogram(wl.draft_off, wl.target_off, o["path_len"], o["path"], 600))


def test_histogram_skips_sentinel_pairs_and_replays_in_a_graph():
    import torch

    import paper_2510_15545_amd as tt

    print("[case] delta histogram sentinels + graph", flush=True)
    wl = synth.make(2, probs=False, w=8)
    d = upload(wl)
    cost, plen, path, mp = gpu_align(wl, d, 8)
    plen_h = plen.cpu().numpy()
    plen_h[::3] = 0  # sentinel pairs
    plen_h[1] = 10_000  # longer than the pair's path area: contributes nothing
    k2, m2 = int(np.diff(wl.draft_off)[2]), int(np.diff(wl.target_off)[2])
    real = int(plen_h[2])
    plen_h[2] = k2 + m2  # the whole path area, past the path's own cells: counted
    pl = to_dev(plen_h)
    path_h = path.cpu().numpy()
    base2 = 2 * (int(wl.draft_off[2]) + int(wl.target_off[2]))
    path_h[base2 + 2 * real:base2 + 2 * (k2 + m2)] = np.tile([0, 5], k2 + m2 - real)  # known values there
    path = to_dev(path_h)
    want = oracle.delta_histogram(wl.draft_off, wl.target_off, plen_h, path_h, 8)
    hist = torch.full((8,), 77, dtype=torch.int32, device="cuda")
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            tt.delta_histogram(d["draft_off"], d["target_off"], pl, path, 8, out=hist)
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(3):
        hist.fill_(1000 + rep)  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(hist.cpu().numpy().astype(np.int64), want), rep


@pytest.mark.parametrize("index,w,n_bins", [(3, -1, 64), (4, -1, 600), (2, 8, 4)])
def test_quantile_matches_oracle(index, w, n_bins):
    """App. K: the deviation where the CDF reaches 9/10 (and other fractions), from the GPU
    histogram on the GPU, equals the oracle's rule on the oracle's histogram."""
    import paper_2510_15545_amd as tt

    print(f"[case] delta quantile workload {index} w={w} bins={n_bins}", flush=True)
    wl = synth.make(index, n_streams=48, probs=False, w=w)
    d = upload(wl)
    cost, plen, path, mp = gpu_align(wl, d, w)
    h = tt.delta_histogram(d["draft_off"], d["target_off"], plen, path, n_bins)
    o = oracle_run(wl, w)
    want_h = oracle.delta_histogram(wl.draft_off, wl.target_off, o["path_len"], o["path"], n_bins)
    for num, den in ((9, 10), (1, 2), (0, 1), (1, 1), (65535, 65536), (1, 65536)):
        got = tt.w_at_quantile(h, num, den)
        assert got == oracle.delta_quantile(want_h, num, den), (num, den)


def test_quantile_hand_cases_on_device():
    """Exact boundaries and empty counts on the device: CDF(0) = 9/10 exactly gives 0, an empty
    histogram 0, q = 1 the last bin holding any count, and 8,192 bins over every thread."""
    import paper_2510_15545_amd as tt

    print("[case] delta quantile hand cases", flush=True)
    cases = [([9, 1], 9, 10, 0), ([89, 10, 1], 9, 10, 1), ([0, 0, 0], 9, 10, 0), ([1] * 10, 1, 1, 9),
             ([0, 0, 5], 1, 2, 2), ([2, 3], 2, 5, 0), ([2, 3], 41, 100, 1)]
    for h, num, den, want in cases:
        assert tt.w_at_quantile(to_dev(np.array(h, np.int32)), num, den) == want, (h, num, den)
        assert oracle.delta_quantile(h, num, den) == want
    rng = np.random.default_rng(3)
    big = rng.integers(0, 1 << 20, 8192).astype(np.int32)
    for num, den in ((9, 10), (1, 3), (1, 65536), (65535, 65536)):
        assert tt.w_at_quantile(to_dev(big), num, den) == oracle.delta_quantile(big, num, den)
