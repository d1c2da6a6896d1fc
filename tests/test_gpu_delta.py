"""tt_delta_histogram (Sec. 5 Fig. CDF, App. K) against the oracle's histogram of the
oracle's own alignment: exact counts for short and long pairs, with and without a band,
sentinel pairs, one-bin and overflow cases, and replays of a captured HIP graph."""
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
    plen_h[1] = 10_000  # longer than the pair's path area: ignored
    pl = to_dev(plen_h)
    path_h = path.cpu().numpy()
    keep = plen_h.copy()
    keep[1] = 0
    want = oracle.delta_histogram(wl.draft_off, wl.target_off, keep, path_h, 8)
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
