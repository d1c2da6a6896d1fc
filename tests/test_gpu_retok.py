"""tt_token_index_build + tt_retokenize (Sec. 4.2.1, Alg. 2, App. A.1) against the oracle's
greedy longest-match re-tokenisation: every workload's batch (long pairs included),
tokens up to 64 bytes with any byte value, equal strings under several ids, the failure
cases that yield empty streams, an empty batch, and replays of a captured HIP graph."""
import numpy as np
import pytest

import oracle
from gpu_util import to_dev
from paper_2510_15545_amd import synth

pytestmark = pytest.mark.gpu


def vocab(tokens, max_len=None):
    import paper_2510_15545_amd as tt

    off = np.zeros(len(tokens) + 1, np.int32)
    off[1:] = np.cumsum([len(t) for t in tokens])
    data = np.frombuffer(b"".join(tokens), np.uint8).copy()
    return data, off, tt.Vocab.from_host(data, off, max_len or max(len(t) for t in tokens))


def run(vd, vt, idx, draft_ids, draft_off, max_bytes, max_m):
    import torch

    import paper_2510_15545_amd as tt

    ids, off = tt.retokenize(vd, vt, idx, to_dev(np.asarray(draft_ids, np.int32)),
                             to_dev(np.asarray(draft_off, np.int32)), max_bytes, max_m)
    torch.cuda.synchronize()
    off = off.cpu().numpy()
    return ids.cpu().numpy()[:off[-1]], off


@pytest.mark.parametrize("index,n", [(1, None), (2, None), (3, None), (5, 128), (4, 96), (2, 2300)])
def test_workload_batches(index, n):
    import paper_2510_15545_amd as tt

    print(f"[case] retokenize workload {index}", flush=True)
    wl = synth.make(index, n_streams=n, probs=False)
    vd = tt.Vocab.from_host(wl.vocab_d.data, wl.vocab_d.offsets, wl.vocab_d.max_len)
    vt = tt.Vocab.from_host(wl.vocab_t.data, wl.vocab_t.offsets, wl.vocab_t.max_len)
    idx = tt.token_index(vt)
    max_bytes = 4096
    max_m = int(np.max(np.diff(wl.target_off)))
    got, goff = run(vd, vt, idx, wl.draft_ids, wl.draft_off, max_bytes, max_m)
    want, woff = oracle.retokenize(wl.vocab_d.data, wl.vocab_d.offsets, wl.vocab_t.data, wl.vocab_t.offsets,
                                   wl.draft_ids, wl.draft_off, max_m=max_m, max_bytes=max_bytes)
    assert np.array_equal(goff, woff), np.nonzero(goff != woff)[0][:5]
    assert np.array_equal(got, want)
    assert np.array_equal(got, wl.target_ids) and np.array_equal(goff, wl.target_off)


def test_long_tokens_any_bytes_duplicates_and_failures():
    print("[case] retokenize edge vocabularies", flush=True)
    rng = np.random.default_rng(3)
    alpha = bytes(range(0, 6)) + b"\x80\xff"
    singles = [bytes([c]) for c in alpha[:-1]]  # 0xff has no single-byte token
    longs = set()
    while len(longs) < 300:
        ln = int(rng.integers(2, 65))
        longs.add(bytes(rng.choice(np.frombuffer(alpha[:-1], np.uint8), ln)))  # no target token holds 0xff
    vt_tokens = singles + sorted(longs)
    vt_tokens += [vt_tokens[7], vt_tokens[40], vt_tokens[2]]  # equal strings under higher ids
    vd_tokens = [vt_tokens[i] for i in rng.permutation(len(vt_tokens))[:120]] + [b"\xff", b"\x01\xff"]
    vd_tokens += [bytes(rng.choice(np.frombuffer(alpha[:-1], np.uint8), int(rng.integers(1, 40)))) for _ in range(80)]
    dd, do_, vd = vocab(vd_tokens)
    td, to_, vt = vocab(vt_tokens)
    import paper_2510_15545_amd as tt
    idx = tt.token_index(vt)
    streams = [list(rng.integers(0, len(vd_tokens) - 82, int(rng.integers(1, 30)))) for _ in range(40)]
    streams += [list(rng.integers(len(vd_tokens) - 80, len(vd_tokens), int(rng.integers(1, 60)))) for _ in range(40)]
    streams += [[], [len(vd_tokens) - 82], [len(vd_tokens) - 81, 0], [len(vd_tokens)], [-1, 2]]  # empty, 0xff, bad ids
    ids = np.array([x for s in streams for x in s], np.int32)
    off = np.zeros(len(streams) + 1, np.int32)
    off[1:] = np.cumsum([len(s) for s in streams])
    for max_bytes, max_m in ((4096, 4096), (300, 40), (64, 8)):
        got, goff = run(vd, vt, idx, ids, off, max_bytes, max_m)
        want, woff = oracle.retokenize(dd, do_, td, to_, ids, off, max_m=max_m, max_bytes=max_bytes)
        assert np.array_equal(goff, woff), (max_bytes, max_m, np.nonzero(goff != woff)[0][:5])
        assert np.array_equal(got, want), (max_bytes, max_m)
        counts = np.diff(goff)
        assert counts[-5:].tolist() == [0, 0, 0, 0, 0]
        assert 0 < (counts > 0).sum()
    # the duplicated strings resolve to their lowest ids
    got, goff = run(vt, vt, idx, np.array([len(vt_tokens) - 3, len(vt_tokens) - 2, len(vt_tokens) - 1], np.int32),
                    np.array([0, 1, 2, 3], np.int32), 4096, 64)
    assert got.tolist() == [7, 40, 2]


def test_empty_batch_and_graph_replays():
    import torch

    import paper_2510_15545_amd as tt

    print("[case] retokenize empty batch + graph", flush=True)
    wl = synth.make(2, probs=False)
    vd = tt.Vocab.from_host(wl.vocab_d.data, wl.vocab_d.offsets, wl.vocab_d.max_len)
    vt = tt.Vocab.from_host(wl.vocab_t.data, wl.vocab_t.offsets, wl.vocab_t.max_len)
    idx = tt.token_index(vt)
    got, goff = run(vd, vt, idx, np.zeros(0, np.int32), np.zeros(1, np.int32), 64, 8)
    assert goff.tolist() == [0]
    di, do_ = to_dev(wl.draft_ids), to_dev(wl.draft_off)
    out = (torch.full((wl.n * 16,), -7, dtype=torch.int32, device="cuda"),
           torch.full((wl.n + 1,), -7, dtype=torch.int32, device="cuda"))
    ws = torch.empty(1 << 16, dtype=torch.uint8, device="cuda")
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            tt.retokenize(vd, vt, idx, di, do_, 256, 16, out=out, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(3):
        out[0].fill_(-1 - rep)
        out[1].fill_(-1 - rep)
        ws.fill_(0xA5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        off = out[1].cpu().numpy()
        assert np.array_equal(off, wl.target_off), rep
        assert np.array_equal(out[0].cpu().numpy()[:off[-1]], wl.target_ids), rep
