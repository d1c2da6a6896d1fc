"""tt_step (align + transfer + verify in one call) against the three calls and the oracle.

With at least 256 streams and K, M <= 64 the call runs as one fused kernel; smaller
batches take the three calls' kernels.  Every output must equal the three-call path's
bit for bit and the oracle's.
"""
import numpy as np
import pytest

import paper_2510_15545_amd as tt
from gpu_util import compare_align, compare_verify, gpu_run, oracle_run, upload
from paper_2510_15545_amd import synth
from test_gpu_edges import random_tokens, vocab_of, workload

pytestmark = pytest.mark.gpu


def step_run(wl, d=None, w=None, residual=False, bounds=None):
    import torch

    d = upload(wl) if d is None else d
    w = wl.w if w is None else w
    mk, mm = (max(1, wl.max_k), max(1, wl.max_m)) if bounds is None else bounds
    out = tt.step(d["vd"], d["vt"], wl.v_d, wl.v_t, d["draft_ids"], d["draft_off"], d["target_ids"],
                  d["target_off"], w, mk, mm, d["draft_probs"], d["target_probs"], d["u_accept"],
                  d["u_sample"], n_path=tt.path_capacity(wl.draft_off[-1], wl.target_off[-1]),
                  residual=residual)
    torch.cuda.synchronize()
    names = ("cost", "path_len", "path", "map", "q", "n_accepted", "out_token", "residual")
    m_total = int(wl.target_off[-1])
    host = {}
    for k, v in zip(names, out):
        if v is None:
            host[k] = None
            continue
        a = v.cpu().numpy()
        host[k] = a[:m_total] if k in ("map", "q") else a
    return host


def same_as_three_calls(wl, s, g):
    for k in ("cost", "path_len", "map", "n_accepted", "out_token"):
        assert np.array_equal(s[k], g[k]), (k, np.nonzero(s[k] != g[k]))
    assert np.array_equal(s["q"].view(np.uint32), g["q"].view(np.uint32))  # NaNs included
    for b in range(wl.n):
        base = 2 * (int(wl.draft_off[b]) + int(wl.target_off[b]))
        n = 2 * int(g["path_len"][b])
        assert np.array_equal(s["path"][base:base + n], g["path"][base:base + n]), b
    if g.get("residual") is not None:
        assert np.array_equal(s["residual"].view(np.uint32), g["residual"].view(np.uint32))


@pytest.mark.parametrize("c,n", [(1, 300), (2, 256), (3, None), (2, 32), (5, 256), (5, None), (1, None), (1, 7)])
def test_step_matches_three_calls_and_oracle(c, n):
    print(f"[case] tt_step workload {c} streams={n}", flush=True)
    wl = synth.make(c, n_streams=n)
    d = upload(wl)
    res = c in (1, 2)
    s = step_run(wl, d, residual=res)
    g = gpu_run(wl, d=d, residual=res)
    same_as_three_calls(wl, s, g)
    o = oracle_run(wl, residual=res)
    compare_align(wl, s, o)
    compare_verify(s, o, residual=res)
    for w in (-1, 0):
        print(f"[case] tt_step workload {c} w={w}", flush=True)
        same_as_three_calls(wl, step_run(wl, d, w=w), gpu_run(wl, w=w, d=d))


@pytest.mark.parametrize("n,v_t", [(280, None), (40, 20_000)])
def test_step_sentinels_in_a_fused_batch(n, v_t):
    """Invalid pairs and streams inside a batch large enough for the fused kernel, and inside a
    small batch of long rows (the fused front up to gamma, then the split verification)."""
    rng = np.random.default_rng(21)
    toks = random_tokens(rng, 300, 1, 6)
    v = vocab_of(toks)
    pairs = []
    for _ in range(280):
        pairs.append((list(rng.integers(0, len(toks), int(rng.integers(1, 9)))),
                      list(rng.integers(0, len(toks), int(rng.integers(1, 20))))))
    pairs[3] = ([1, 999, 2], [4, 5])        # draft id outside the vocabulary: align sentinel
    pairs[10] = ([2, 3], [4, 5, -1])        # target id outside: align and verify sentinel
    pairs[11] = ([], [7, 8])                # K = 0: align sentinel, verify runs on q = NaN
    pairs[12] = ([5, 6], [])                # M = 0: align sentinel, verify samples the bonus row
    pairs[13] = (list(range(1, 12)), [9])   # K above the bound below
    pairs[14] = ([1], list(range(1, 22)))   # M above the bound below
    pairs = pairs[:n]
    wl = workload(v, v, pairs, len(toks), v_t or len(toks), seed=3)
    d = upload(wl)
    for bounds in ((10, 20), (64, 64)):
        print(f"[case] tt_step sentinels n={n} v_t={v_t} bounds={bounds}", flush=True)
        s = step_run(wl, d, bounds=bounds, residual=True)
        import copy
        wl2 = copy.copy(wl)
        g = {}
        cost, plen, path, mp = tt.align(d["vd"], d["vt"], d["draft_ids"], d["draft_off"], d["target_ids"],
                                        d["target_off"], wl.w, *bounds,
                                        n_path=tt.path_capacity(wl.draft_off[-1], wl.target_off[-1]))
        q = tt.transfer(wl.v_d, d["draft_ids"], d["draft_off"], d["target_off"], mp, d["draft_probs"])
        nacc, tok, res = tt.verify(wl.v_t, d["target_ids"], d["target_off"], q, d["target_probs"],
                                   d["u_accept"], d["u_sample"], bounds[1], residual=True)
        m_total = int(wl.target_off[-1])
        g = {"cost": cost.cpu().numpy(), "path_len": plen.cpu().numpy(), "path": path.cpu().numpy(),
             "map": mp.cpu().numpy()[:m_total], "q": q.cpu().numpy()[:m_total],
             "n_accepted": nacc.cpu().numpy(), "out_token": tok.cpu().numpy(), "residual": res.cpu().numpy()}
        same_as_three_calls(wl2, s, g)
        assert s["cost"][3] == -1 and s["cost"][10] == -1 and s["n_accepted"][10] == -1
        assert s["n_accepted"][12] == 0 and s["out_token"][12] >= 0


def test_step_workspace_reuse():
    import torch

    wl = synth.make(1, n_streams=300)
    d = upload(wl)
    ws = tt.step_workspace(wl.n, wl.v_t, wl.max_k, wl.max_m, wl.w, max(wl.vocab_d.max_len, wl.vocab_t.max_len))
    outs = []
    for fill in (0x00, 0xA5, 0xFF):
        ws.fill_(fill)
        o = tt.step(d["vd"], d["vt"], wl.v_d, wl.v_t, d["draft_ids"], d["draft_off"], d["target_ids"],
                    d["target_off"], wl.w, wl.max_k, wl.max_m, d["draft_probs"], d["target_probs"],
                    d["u_accept"], d["u_sample"], workspace=ws)
        torch.cuda.synchronize()
        host = [t.cpu().numpy() for t in o if t is not None]
        plen = host[1]
        keep = np.zeros(host[2].shape, bool)  # the path buffer is written up to each path_len
        for b in range(wl.n):
            base = 2 * (int(wl.draft_off[b]) + int(wl.target_off[b]))
            keep[base:base + 2 * int(plen[b])] = True
        host[2] = np.where(keep, host[2], -7)
        outs.append(host)
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


@pytest.mark.parametrize("v_t", [2_097_152, 2_097_153])
def test_row_width_at_the_row_path_limit(v_t):
    """256 streams over rows of 2,048 chunks (the widest rows the one-workgroup-per-stream kernels
    take: tt_verify's row path and the fused tt_step) and one float more (the split path and the
    fused front): tt_step equals the three calls and the oracle.  Most streams propose nothing
    (M = 0: the bonus row is sampled), 16 propose one token."""
    import copy

    print(f"[case] wide rows v_t={v_t}", flush=True)
    rng = np.random.default_rng(7)
    toks = random_tokens(rng, 64, 1, 4)
    v = vocab_of(toks)
    pairs = [([int(rng.integers(0, len(toks)))], [int(rng.integers(0, len(toks)))] if b % 16 == 0 else [])
             for b in range(256)]
    wl = workload(v, v, pairs, len(toks), len(toks), probs=True)
    wl = copy.copy(wl)
    n_rows = int(wl.target_off[-1]) + wl.n
    rows = rng.random((n_rows, v_t), dtype=np.float32)
    rows /= rows.sum(axis=1, keepdims=True, dtype=np.float32)
    wl.v_t = v_t
    wl.target_probs = rows
    d = upload(wl)
    s = step_run(wl, d, bounds=(64, 64))
    g = gpu_run(wl, d=d, bounds=(64, 64))
    same_as_three_calls(wl, s, g)
    o = oracle_run(wl)
    compare_verify(s, o)
