"""GPU edge cases, each compared with the oracle (or with the documented sentinel)."""
import numpy as np
import pytest

from gpu_util import compare_align, compare_verify, gpu_run, oracle_run, to_dev
from paper_2510_15545_amd import synth

pytestmark = pytest.mark.gpu


def vocab_of(tokens):
    tokens = list(tokens)
    off = np.zeros(len(tokens) + 1, np.int32)
    off[1:] = np.cumsum([len(t) for t in tokens])
    data = np.frombuffer(b"".join(tokens), np.uint8).copy()
    return synth.Vocab(tokens, {t: i for i, t in enumerate(tokens)}, data, off,
                       max([len(t) for t in tokens]))


def workload(vd, vt, pairs, v_d, v_t, w=8, seed=0, probs=True):
    def csr(lists):
        off = np.zeros(len(lists) + 1, np.int32)
        off[1:] = np.cumsum([len(l) for l in lists])
        return np.array([x for l in lists for x in l], np.int32), off

    di, do = csr([p[0] for p in pairs])
    ti, to = csr([p[1] for p in pairs])
    spec = synth.Spec(0, "edge", len(pairs), 0, v_d, v_t, b"", 64, None, w)
    wl = synth.Workload(spec, vd, vt, di, do, ti, to, w, v_d=v_d, v_t=v_t, verify_ids=ti)
    if probs:
        rng = np.random.default_rng(seed)
        n = len(pairs)

        def rows(k, width):
            x = rng.standard_normal((k, width)).astype(np.float32) * np.float32(2)
            e = np.exp(x - x.max(axis=1, keepdims=True)).astype(np.float32)
            return (e / e.sum(axis=1, keepdims=True, dtype=np.float32)).astype(np.float32)

        wl.draft_probs = rows(int(do[-1]), v_d)
        wl.target_probs = rows(int(to[-1]) + n, v_t)
        wl.u_accept = (rng.integers(0, 1 << 24, int(to[-1])) * 2.0**-24).astype(np.float32)
        wl.u_sample = (rng.integers(0, 1 << 24, n) * 2.0**-24).astype(np.float32)
    return wl


def random_tokens(rng, n, lo, hi, alphabet=b"abcdefgh"):
    out = set()
    alpha = np.frombuffer(alphabet, np.uint8)
    while len(out) < n:
        ln = int(rng.integers(lo, hi + 1))
        out.add(alpha[rng.integers(0, len(alpha), ln)].tobytes())
    return sorted(out)


@pytest.mark.parametrize("maxlen", [8, 16, 32, 64])
def test_token_slot_widths(maxlen):
    """Every token-width instantiation (8/16/32/64-byte slots) against the oracle."""
    print(f"[case] token slots maxlen={maxlen}", flush=True)
    rng = np.random.default_rng(maxlen)
    toks_d = random_tokens(rng, 300, 1, maxlen, bytes(range(0x20, 0x7F)) + b"\x00\xc3\xa9")
    toks_t = random_tokens(rng, 400, 1, maxlen, bytes(range(0x20, 0x7F)) + b"\x00\xc3\xa9")
    vd, vt = vocab_of(toks_d), vocab_of(toks_t)
    pairs = [(list(rng.integers(0, len(toks_d), rng.integers(1, 40))),
              list(rng.integers(0, len(toks_t), rng.integers(1, 40)))) for _ in range(40)]
    wl = workload(vd, vt, pairs, len(toks_d), len(toks_t))
    for w in (8, -1, 3):
        o = oracle_run(wl, w=w)
        g = gpu_run(wl, w=w)  # row-scan kernel
        compare_align(wl, g, o)
        compare_verify(g, o)
        compare_align(wl, gpu_run(wl, w=w, bounds=(65, 65)), o)  # strip kernel


def test_strips_longer_than_a_wave():
    """K and M well above 64 rows, every w in the paper's sweep (strip boundaries, band widening)."""
    rng = np.random.default_rng(5)
    toks = random_tokens(rng, 200, 1, 4)
    v = vocab_of(toks)
    pairs = []
    # band widths up to and past the widest precomputed band (512 cells per row): 64-row
    # strips whose band shifts one column per row span up to W + 126 sweep steps
    for k, m in ((65, 64), (64, 65), (130, 129), (200, 60), (60, 200), (128, 128), (1, 300), (300, 1),
                 (150, 100), (100, 150), (200, 210), (300, 520), (260, 520), (520, 300)):
        pairs.append((list(rng.integers(0, len(toks), k)), list(rng.integers(0, len(toks), m))))
    wl = workload(v, v, pairs, len(toks), len(toks), probs=False)
    for w in (4, 8, 16, -1, 0, 40, 70):
        print(f"[case] strips w={w}", flush=True)
        compare_align(wl, gpu_run(wl, w=w), oracle_run(wl, w=w))


def test_band_rows_wider_than_a_wave_of_code_words():
    """Band rows of more than 64 code words (W > 1008 cells): the backtrack reads code words
    from the workspace instead of staging strips in LDS, and a run may cross many words."""
    rng = np.random.default_rng(11)
    toks = random_tokens(rng, 120, 1, 4)
    v = vocab_of(toks)
    pairs = []
    for k, m in ((100, 1100), (1100, 100), (1030, 1050), (700, 1100), (1, 1100), (1100, 1)):
        pairs.append((list(rng.integers(0, len(toks), k)), list(rng.integers(0, len(toks), m))))
    # long runs of one repeated draft token make the path cross whole code words in one row
    pairs.append(([3] * 40, list(rng.integers(0, len(toks), 1100))))
    wl = workload(v, v, pairs, len(toks), len(toks), probs=False)
    for w in (8, -1):
        print(f"[case] wide rows w={w}", flush=True)
        compare_align(wl, gpu_run(wl, w=w), oracle_run(wl, w=w))


@pytest.mark.parametrize("kernel", ["rows", "strips"])
def test_short_pair_extremes(kernel):
    """Pairs at the row-scan kernel's limits (K, M in {1, 63, 64}), through both alignment
    kernels: bounds of 64 select the row-scan kernel, a bound of 65 the strip kernel."""
    rng = np.random.default_rng(11)
    toks = random_tokens(rng, 120, 1, 6)
    v = vocab_of(toks)
    shapes = ((64, 64), (1, 64), (64, 1), (1, 1), (63, 64), (64, 63), (64, 30), (30, 64), (2, 64), (64, 2))
    pairs = [(list(rng.integers(0, len(toks), k)), list(rng.integers(0, len(toks), m))) for k, m in shapes]
    wl = workload(v, v, pairs, len(toks), len(toks), probs=False)
    bounds = (64, 64) if kernel == "rows" else (65, 64)
    for w in (0, 1, 4, 8, -1, 70):
        print(f"[case] short pair extremes kernel={kernel} w={w}", flush=True)
        compare_align(wl, gpu_run(wl, w=w, bounds=bounds), oracle_run(wl, w=w))


@pytest.mark.parametrize("c", [2, 3, 5])
def test_strip_kernel_on_benchmark_shapes(c):
    """The strip kernel stays bit-exact on the short pairs the row-scan kernel normally takes."""
    from paper_2510_15545_amd import synth

    print(f"[case] strip kernel on workload {c}", flush=True)
    wl = synth.make(c, n_streams=16)
    for w in (8, -1):
        g = gpu_run(wl, w=w, bounds=(max(65, wl.max_k), max(65, wl.max_m)))
        compare_align(wl, g, oracle_run(wl, w=w))


def test_sentinel_pairs_and_streams():
    rng = np.random.default_rng(6)
    toks = random_tokens(rng, 50, 1, 5)
    v = vocab_of(toks)
    pairs = [([1, 2, 3], [4, 5]), ([1, 999], [3]), ([2, 3], [4, -1]), ([5], [6, 7, 8])]
    wl = workload(v, v, pairs, len(toks), len(toks))
    wl.verify_ids = wl.target_ids.copy()
    wl.verify_ids[wl.target_off[2] + 1] = 10**6  # out of range for verify as well
    g, o = gpu_run(wl), oracle_run(wl)
    compare_align(wl, g, o)
    assert list(g["cost"][1:3]) == [-1, -1] and list(g["map"][wl.target_off[1]:wl.target_off[3]]) == [-1] * 3
    compare_verify(g, o)
    assert int(g["n_accepted"][2]) == -1 and int(g["out_token"][2]) == -1


def test_bounds_smaller_than_pairs_give_sentinels():
    import paper_2510_15545_amd as tt

    rng = np.random.default_rng(7)
    toks = random_tokens(rng, 50, 1, 5)
    v = vocab_of(toks)
    pairs = [([1, 2, 3], [4, 5]), ([1, 2, 3, 4, 5, 6], [3]), ([2], [4, 5, 6, 7, 8, 9])]
    wl = workload(v, v, pairs, len(toks), len(toks), probs=False)
    from gpu_util import upload

    d = upload(wl)
    cost, plen, path, mp = tt.align(d["vd"], d["vt"], d["draft_ids"], d["draft_off"], d["target_ids"],
                                    d["target_off"], 8, 4, 4)
    cost = cost.cpu().numpy()
    assert cost[0] >= 0 and cost[1] == -1 and cost[2] == -1
    assert list(mp.cpu().numpy()[wl.target_off[2]:]) == [-1] * 6


def test_verify_edge_values():
    """M = 0 streams, q = 0 / NaN, u at the ends of [0,1), a zero-mass residual, rows not 16-B aligned."""
    import torch
    import oracle
    import paper_2510_15545_amd as tt

    V, ld = 3001, 3003  # ragged tail, ld % 4 != 0 -> scalar loads
    rng = np.random.default_rng(8)
    n = 7
    Ms = [0, 1, 2, 3, 1, 2, 1]
    off = np.zeros(n + 1, np.int32)
    off[1:] = np.cumsum(Ms)
    ids = rng.integers(0, V, int(off[-1])).astype(np.int32)
    rows = rng.random((int(off[-1]) + n, ld)).astype(np.float32)
    rows /= rows[:, :V].sum(axis=1, keepdims=True, dtype=np.float32)
    q = rng.random(int(off[-1])).astype(np.float32)
    ua = (rng.integers(0, 1 << 24, int(off[-1])) * 2.0**-24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, n) * 2.0**-24).astype(np.float32)
    q[off[1]] = 0.0             # stream 1: q = 0 -> accepted
    q[off[2]] = np.nan          # stream 2: NaN proposal -> rejected
    us[3] = 0.0
    us[4] = np.float32(1 - 2**-24)
    # stream 5: the residual is empty (all mass on the rejected proposal, q > 1)
    r5 = off[5] + 5
    rows[r5, :] = 0.0
    rows[r5, ids[off[5]]] = 1.0
    q[off[5]] = 2.0
    ua[off[5]] = 0.9
    # stream 6: NaN and negative entries in the bonus row, q tiny -> accepted
    q[off[6]] = 1e-30
    rows[off[6] + 6 + 1, 5] = np.nan
    rows[off[6] + 6 + 1, 6] = -0.5
    rows_c = np.ascontiguousarray(rows)
    o_nacc, o_tok, o_res, _ = oracle.verify(V, ids, off, q, rows_c, ua, us, residual=True)
    dev = {k: to_dev(v) for k, v in dict(ids=ids, off=off, q=q, ua=ua, us=us).items()}
    P = to_dev(rows_c)
    nacc, tok, res = tt.verify(V, dev["ids"], dev["off"], dev["q"], P, dev["ua"], dev["us"], 3, residual=True)
    torch.cuda.synchronize()
    assert np.array_equal(nacc.cpu().numpy(), o_nacc)
    assert np.array_equal(tok.cpu().numpy(), o_tok)
    r = res.cpu().numpy()[:, :V]
    ro = o_res[:, :V]
    assert np.all(np.abs(r.astype(np.float64) - ro) <= 1e-6 * np.abs(ro))
    assert int(o_tok[5]) == int(ids[off[5]])  # zero-mass fallback = first argmax


def test_empty_batch_and_argument_errors():
    import torch
    import paper_2510_15545_amd as tt

    e = torch.zeros(1, dtype=torch.int32, device="cuda")
    off = torch.zeros(1, dtype=torch.int32, device="cuda")
    P = torch.zeros((1, 8), dtype=torch.float32, device="cuda")
    f = torch.zeros(1, dtype=torch.float32, device="cuda")
    nacc, tok, _ = tt.verify(8, e, off, f, P, f, f, 0)
    assert nacc.numel() == 0 and tok.numel() == 0
    with pytest.raises(tt.TTError):
        tt.verify(8, e, torch.zeros(2, dtype=torch.int32, device="cuda"), f, P, f, f, -1)


@pytest.mark.parametrize("w", [-1, 0, 3, 8])
def test_strip_walk_segment_and_group_boundaries(w):
    """Pairs whose row counts sit on and around the 32-row segments and 64-row strips of the
    strip kernel's backtrack (segments walked in parallel from guessed columns, then corrected),
    with several band widths, some pairs far off the diagonal: bit-exact against the oracle."""
    print(f"[case] strip walk boundaries w={w}", flush=True)
    rng = np.random.default_rng(100 + w)
    toks = random_tokens(rng, 120, 1, 6, alphabet=b"abcdefgh")
    v = vocab_of(toks)
    ks = [31, 32, 33, 63, 64, 65, 95, 96, 97, 128, 200, 257, 300]
    pairs = []
    for k in ks:
        for m in (max(1, k // 3), k, k + 37, 2 * k):
            d = list(rng.integers(0, len(toks), k))
            # targets that share long stretches with the drafts (paths near the diagonal) or not
            t = (d[:m] + list(rng.integers(0, len(toks), max(0, m - k)))) if rng.random() < 0.5 else \
                list(rng.integers(0, len(toks), m))
            pairs.append((d, t))
    wl = workload(v, v, pairs, len(toks), len(toks), w=w, probs=False)
    g = gpu_run(wl, w=w)
    compare_align(wl, g, oracle_run(wl, w=w))


@pytest.mark.parametrize("n,V,dense", [(256, 300_000, False), (3, 9_000_000, False), (256, 300_000, True)])
def test_large_vocabularies(n, V, dense):
    """Rows past 256 chunks (the sampler's chunk sums no longer fit four per lane) on the
    one-workgroup-per-stream path, and rows past 8M floats (over the row path's LDS) on the
    split path; one-hot and dense proposals, bit-exact against the oracle."""
    print(f"[case] large vocabulary n={n} V={V} dense={dense}", flush=True)
    verify_case(n, V, dense)


@pytest.mark.parametrize("V", [640, 12_000, 30_000, 50_000, 100_000])
@pytest.mark.parametrize("dense", [False, True])
def test_row_path_workgroup_sizes(V, dense):
    """The one-workgroup-per-stream path sizes its workgroup from the row (about eight 1024-float
    chunks per wave): 64, 128, 256, 512 and 1024 threads for these widths."""
    print(f"[case] row path n=256 V={V} dense={dense}", flush=True)
    verify_case(256, V, dense)


def verify_case(n, V, dense):
    """Random rows of width V for n streams with 0-2 proposals each; GPU outputs against the
    oracle, bit for bit (one-hot proposals through tt_verify, dense through tt_verify_dense)."""
    import torch

    import oracle
    import paper_2510_15545_amd as tt

    rng = np.random.default_rng(V + n)
    Ms = rng.integers(0, 3, n)
    off = np.zeros(n + 1, np.int32)
    off[1:] = np.cumsum(Ms)
    nt = int(off[-1])
    ids = rng.integers(0, V, nt).astype(np.int32)
    rows = rng.random((nt + n, V), dtype=np.float32)
    rows /= rows.sum(axis=1, keepdims=True, dtype=np.float32)
    ids[::3] = np.argmax(rows[(off[:-1] + np.arange(n))[np.repeat(np.arange(n), Ms)][::3]], axis=1)  # likely accepts
    ua = (rng.integers(0, 1 << 24, nt) * 2.0**-24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, n) * 2.0**-24).astype(np.float32)
    us[0] = np.float32(1 - 2**-24)
    P = to_dev(rows)
    if dense:
        qrows = rng.random((max(1, nt), V), dtype=np.float32)
        qrows /= qrows.sum(axis=1, keepdims=True, dtype=np.float32)
        o_nacc, o_tok, _, _ = oracle.sd_verify(V, ids, off, qrows[:nt], rows, ua, us)
        nacc, tok, _ = tt.verify_dense(V, to_dev(ids), to_dev(off), to_dev(qrows), P, to_dev(ua), to_dev(us), 2)
    else:
        q = rng.random(nt).astype(np.float32) * np.float32(1e-5)
        o_nacc, o_tok, _, _ = oracle.verify(V, ids, off, q, rows, ua, us)
        nacc, tok, _ = tt.verify(V, to_dev(ids), to_dev(off), to_dev(q), P, to_dev(ua), to_dev(us), 2)
    torch.cuda.synchronize()
    assert np.array_equal(nacc.cpu().numpy(), o_nacc)
    assert np.array_equal(tok.cpu().numpy(), o_tok)
    assert 0 < (o_nacc < Ms).sum() or n < 8
