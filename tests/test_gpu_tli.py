"""tt_vocab_intersection + tt_tli_proposal (App. D Alg. 3, Token-Level Intersection) against
the oracle: the intersection of the benchmark's vocabularies and of edge vocabularies
(duplicate strings, empty and over-long tokens, any byte values, tokens up to 64 bytes), q'
rows bit for bit on ragged row lengths, padded and unaligned strides, subnormal, NaN,
negative and above-one inputs and rows without intersected mass, q' at the benchmark's
vocabulary sizes, and standard speculative sampling (tt_verify_dense) run on q'."""
import numpy as np
import pytest

import oracle
from gpu_util import to_dev
from paper_2510_15545_amd import synth

pytestmark = pytest.mark.gpu


def dev_vocab(data, off, max_len):
    import paper_2510_15545_amd as tt

    return tt.Vocab.from_host(np.asarray(data, np.uint8), np.asarray(off, np.int32), max_len)


def gpu_intersection(vd, vt):
    import torch

    import paper_2510_15545_amd as tt

    d2t, t2d = tt.vocab_intersection(vd, tt.token_index(vd), vt, tt.token_index(vt))
    torch.cuda.synchronize()
    return d2t, t2d


def table(strings):
    off = np.zeros(len(strings) + 1, np.int32)
    off[1:] = np.cumsum([len(s) for s in strings])
    data = np.frombuffer(b"".join(strings), np.uint8).copy() if off[-1] else np.zeros(1, np.uint8)
    return data, off


def test_intersection_of_the_benchmark_vocabularies():
    print("[case] intersection workload 3 vocabularies", flush=True)
    wl = synth.make(3, n_streams=4, probs=False)
    a, b = wl.vocab_d, wl.vocab_t
    d2t, t2d = gpu_intersection(dev_vocab(a.data, a.offsets, a.max_len), dev_vocab(b.data, b.offsets, b.max_len))
    want_d, want_t = oracle.vocab_intersection(a.data, a.offsets, b.data, b.offsets, a.max_len, b.max_len)
    assert np.array_equal(d2t.cpu().numpy(), want_d)
    assert np.array_equal(t2d.cpu().numpy(), want_t)
    assert 0 < np.count_nonzero(want_d >= 0) < len(want_d)


def test_intersection_of_edge_vocabularies():
    print("[case] intersection edge vocabularies", flush=True)
    rng = np.random.default_rng(41)
    alpha = bytes([0, 1, 2, 0x80, 0xff])

    def vocab(n):
        toks = [bytes(rng.choice(list(alpha), size=int(rng.integers(0, 4)))) for _ in range(n)]
        toks += [bytes(rng.choice(list(alpha), size=int(rng.integers(9, 65)))) for _ in range(n // 4)]
        return toks

    D, T = vocab(400), vocab(300)
    common = [bytes(rng.choice(list(alpha), size=int(rng.integers(5, 65)))) for _ in range(60)]
    D += common + common[:10]  # long shared strings, some held twice by the draft
    T += common[::-1]
    for max_d, max_t in ((64, 64), (40, 64), (64, 12)):  # tokens past the declared length are left out
        dd, do = table(D)
        td, to = table(T)
        d2t, t2d = gpu_intersection(dev_vocab(dd, do, max_d), dev_vocab(td, to, max_t))
        want_d, want_t = oracle.vocab_intersection(dd, do, td, to, max_d, max_t)
        assert np.array_equal(d2t.cpu().numpy(), want_d), (max_d, max_t)
        assert np.array_equal(t2d.cpu().numpy(), want_t), (max_d, max_t)


def random_maps(rng, v_d, v_t, frac):
    d2t = np.full(v_d, -1, np.int32)
    t2d = np.full(v_t, -1, np.int32)
    k = int(min(v_d, v_t) * frac)
    xs = rng.choice(v_d, k, replace=False)
    ys = rng.choice(v_t, k, replace=False)
    d2t[xs], t2d[ys] = ys, xs
    return d2t, t2d


def run_tli(d2t, t2d, q, ld_q=None, ld_out=None):
    import torch

    import paper_2510_15545_amd as tt

    n, v_d = q.shape
    ld_q = ld_q or v_d
    qp = np.zeros((n, ld_q), np.float32)
    qp[:, :v_d] = q
    out = torch.full((n, ld_out or len(t2d)), 7.0, dtype=torch.float32, device="cuda")
    tt.tli_proposal(to_dev(d2t), to_dev(t2d), to_dev(qp), v_d=v_d, out=out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("v_d,v_t,ld_q,ld_out", [(5000, 6001, None, None), (4099, 2053, 4101, 2057),
                                                 (4096, 4100, 4100, 4104), (1, 3, None, None)])
def test_proposal_rows_match_the_oracle(v_d, v_t, ld_q, ld_out):
    print(f"[case] tli rows v_d={v_d} v_t={v_t} ld={ld_q},{ld_out}", flush=True)
    rng = np.random.default_rng(v_d + v_t)
    d2t, t2d = random_maps(rng, v_d, v_t, 0.7)
    n = 7
    q = (rng.random((n, v_d)) ** 4).astype(np.float32)
    q /= q.sum(axis=1, keepdims=True)
    q[1, : min(v_d, 40)] = np.float32(2.0 ** -140)  # subnormal inputs and quotients
    q[2, 0] = np.nan
    q[2, -1] = -0.25
    q[3, 0] = 1.75
    q[4] = np.where(d2t >= 0, 0.0, q[4])  # no mass on the intersection: a zero row
    out = run_tli(d2t, t2d, q, ld_q, ld_out)
    want = oracle.tli_proposal(d2t, t2d, q)
    got = out[:, :v_t]
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), np.argwhere(got != want)[:5]
    if ld_out:
        assert np.all(out[:, v_t:] == 7.0)  # padding untouched
    assert np.all(got[4] == 0)


def test_proposal_at_the_benchmark_vocabulary_sizes():
    print("[case] tli rows workload 3 vocabularies", flush=True)
    wl = synth.make(3, n_streams=4, probs=False)
    a, b = wl.vocab_d, wl.vocab_t
    d2t, t2d = oracle.vocab_intersection(a.data, a.offsets, b.data, b.offsets, a.max_len, b.max_len)
    rng = np.random.default_rng(43)
    logits = rng.standard_normal((12, len(d2t))) * 3.0
    q = np.exp(logits - logits.max(axis=1, keepdims=True))
    q = (q / q.sum(axis=1, keepdims=True)).astype(np.float32)
    got = run_tli(d2t, t2d, q)
    want = oracle.tli_proposal(d2t, t2d, q)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    assert np.allclose(got.sum(axis=1, dtype=np.float64), 1.0, atol=1e-5)


def test_standard_sd_on_the_tli_proposal():
    """Alg. 3 then Alg. 4 on the GPU: q' from tt_tli_proposal, drafts drawn from q', then
    tt_verify_dense; accept counts and tokens equal the oracle's on the oracle's q'."""
    import torch

    import paper_2510_15545_amd as tt

    print("[case] tli + dense verify", flush=True)
    rng = np.random.default_rng(44)
    v_d, v_t, N, M = 3000, 2500, 96, 4
    d2t, t2d = random_maps(rng, v_d, v_t, 0.5)
    q = (rng.random((N * M, v_d)) ** 6).astype(np.float32)
    q /= q.sum(axis=1, keepdims=True)
    qp_gpu = tt.tli_proposal(to_dev(d2t), to_dev(t2d), to_dev(q))
    qp = oracle.tli_proposal(d2t, t2d, q)
    assert np.array_equal(qp_gpu.cpu().numpy().view(np.uint32), qp.view(np.uint32))
    cdf = np.cumsum(qp.astype(np.float64), axis=1)
    xs = np.array([min(int(np.searchsorted(c, rng.random() * c[-1], side="right")), v_t - 1) for c in cdf], np.int32)
    off = (np.arange(N + 1) * M).astype(np.int32)
    p = rng.random((N * (M + 1), v_t)).astype(np.float32)
    p /= p.sum(axis=1, keepdims=True)
    ua = rng.random(N * M).astype(np.float32)
    us = rng.random(N).astype(np.float32)
    nacc, tok, _ = tt.verify_dense(v_t, to_dev(xs), to_dev(off), qp_gpu, to_dev(p), to_dev(ua), to_dev(us), M)
    torch.cuda.synchronize()
    wn, wt, _, _ = oracle.sd_verify(v_t, xs, off, qp, p, ua, us)
    assert np.array_equal(nacc.cpu().numpy(), wn) and np.array_equal(tok.cpu().numpy(), wt)


def tli_case(rng, v_d, v_t, N, M, frac=0.6, ld_d=None, ld_t=None):
    """N streams of M_b <= M drafted positions: draft rows q over V_d, proposals y_j drawn from
    q' (target ids), target rows p over V_t (rows off[b] + b + j), uniforms."""
    d2t, t2d = random_maps(rng, v_d, v_t, frac)
    Ms = rng.integers(0, M + 1, N)
    off = np.zeros(N + 1, np.int32)
    off[1:] = np.cumsum(Ms)
    nt = int(off[-1])
    q = (rng.random((nt, v_d)) ** 6).astype(np.float32)
    q /= q.sum(axis=1, keepdims=True)
    qp = oracle.tli_proposal(d2t, t2d, q)
    ys = np.zeros(nt, np.int32)
    for r in range(nt):
        c = np.cumsum(qp[r].astype(np.float64))
        ys[r] = min(int(np.searchsorted(c, rng.random() * c[-1], side="right")), v_t - 1) if c[-1] > 0 else 0
    p = rng.random((nt + N, v_t)).astype(np.float32) ** 3
    p /= p.sum(axis=1, keepdims=True)
    # the target puts the proposal's mass or more on it now and then: acceptances, several rows
    hit = rng.random(nt) < 0.5
    rows_of = (off[:-1] + np.arange(N))[np.repeat(np.arange(N), Ms)] + (np.arange(nt) - np.repeat(off[:-1], Ms))
    p[rows_of[hit], ys[hit]] += qp[hit, ys[hit]] * 2
    ua = rng.random(nt).astype(np.float32)
    us = rng.random(N).astype(np.float32)
    qd = np.zeros((nt, ld_d or v_d), np.float32)
    qd[:, :v_d] = q
    pt = np.zeros((nt + N, ld_t or v_t), np.float32)
    pt[:, :v_t] = p
    return dict(d2t=d2t, t2d=t2d, off=off, Ms=Ms, q=q, qd=qd, ys=ys, p=p, pt=pt, ua=ua, us=us, v_d=v_d, v_t=v_t)


def fused(c, max_m, mass=None):
    import torch

    import paper_2510_15545_amd as tt

    nacc, tok = tt.verify_tli(to_dev(c["d2t"]), to_dev(c["t2d"]), to_dev(c["ys"]), to_dev(c["off"]), to_dev(c["qd"]),
                              to_dev(c["pt"]), to_dev(c["ua"]), to_dev(c["us"]), max_m,
                              draft_mass=None if mass is None else to_dev(np.asarray(mass, np.float32)), v_d=c["v_d"])
    torch.cuda.synchronize()
    return nacc.cpu().numpy(), tok.cpu().numpy()


def two_calls(c, max_m):
    import torch

    import paper_2510_15545_amd as tt

    qp = tt.tli_proposal(to_dev(c["d2t"]), to_dev(c["t2d"]), to_dev(c["qd"]), v_d=c["v_d"])
    nacc, tok, _ = tt.verify_dense(c["v_t"], to_dev(c["ys"]), to_dev(c["off"]), qp, to_dev(c["pt"]), to_dev(c["ua"]),
                                   to_dev(c["us"]), max_m)
    torch.cuda.synchronize()
    return nacc.cpu().numpy(), tok.cpu().numpy()


def oracle_tli(c, max_m, mass=None):
    qp = oracle.tli_proposal(c["d2t"], c["t2d"], c["q"], mass=mass)
    n, t, _, _ = oracle.sd_verify(c["v_t"], c["ys"], c["off"], qp, c["p"], c["ua"], c["us"], max_m=max_m)
    return n, t


def intersected_mass(c):
    return np.array([oracle.round_to_f32(sum(int(v) for v in np.floor(
        np.clip(np.nan_to_num(r, nan=0.0), 0, 1)[c["d2t"] >= 0].astype(np.float64) * 2.0 ** 62)), 62)
        for r in c["q"]], np.float32)


@pytest.mark.parametrize("v_d,v_t,N,M,ld_d,ld_t", [(3000, 2500, 40, 4, None, None), (4099, 5123, 24, 6, 4101, 5127),
                                                   (777, 1024, 70, 3, None, None), (64, 3, 9, 2, None, None)])
def test_fused_tli_verification_matches_the_two_calls_and_the_oracle(v_d, v_t, N, M, ld_d, ld_t):
    """tt_verify_tli against tt_tli_proposal + tt_verify_dense and the oracle's Alg. 3 then
    Alg. 4, bit for bit, with S formed in the kernel and passed in as the drafter's: ragged
    rows, odd strides, streams that draft nothing, rows whose intersection holds no mass
    (q' = 0 keeps the proposal), NaN and above-one draft masses, proposals outside the
    intersection, and sentinel streams (an id outside V_t, M above max_m)."""
    print(f"[case] fused tli v_d={v_d} v_t={v_t} N={N} M={M} ld={ld_d},{ld_t}", flush=True)
    rng = np.random.default_rng(v_d + v_t + N)
    c = tli_case(rng, v_d, v_t, N, M, ld_d=ld_d, ld_t=ld_t)
    nt = int(c["off"][-1])
    if nt >= 3:
        c["q"][0] = np.where(c["d2t"] >= 0, 0.0, c["q"][0])  # no intersected mass
        c["q"][1, 0] = np.nan
        c["q"][2, -1] = 1.5
        c["ys"][min(3, nt - 1)] = int(np.nonzero(c["t2d"] < 0)[0][0]) if (c["t2d"] < 0).any() else 0
        c["qd"][:, :v_d] = c["q"]
    want = oracle_tli(c, M)
    for got in (fused(c, M), fused(c, M, intersected_mass(c)), two_calls(c, M)):
        assert np.array_equal(got[0], want[0]), np.nonzero(got[0] != want[0])[0][:5]
        assert np.array_equal(got[1], want[1]), np.nonzero(got[1] != want[1])[0][:5]
    assert (want[0] > 0).any() and (want[0] < c["Ms"]).any()
    # sentinels: an id outside V_t in stream 1, max_m below stream 2's M
    b1 = int(np.argmax(c["Ms"] > 0))
    bad = dict(c, ys=c["ys"].copy())
    bad["ys"][c["off"][b1]] = v_t
    n1, t1 = fused(bad, M)
    assert n1[b1] == -1 and t1[b1] == -1
    keep = np.arange(N) != b1
    assert np.array_equal(n1[keep], want[0][keep]) and np.array_equal(t1[keep], want[1][keep])
    if c["Ms"].max() > 0:
        small = int(c["Ms"].max()) - 1
        n2, t2 = fused(c, small)
        over = c["Ms"] > small
        assert np.all(n2[over] == -1) and np.all(t2[over] == -1)


@pytest.mark.parametrize("v_d,v_t,frac", [(128256, 60000, 0.9), (1200000, 5000, 0.5)])
def test_fused_tli_dense_and_wide_draft_vocabularies(v_d, v_t, frac):
    """A dense intersection (54,000 of V_d = 128,256 ids: most lanes gather) and a draft
    vocabulary of 1.2 M ids, bit for bit against the oracle, with S formed in the kernel and
    passed in."""
    print(f"[case] fused tli dense/wide v_d={v_d} v_t={v_t} frac={frac}", flush=True)
    rng = np.random.default_rng(v_d + v_t)
    c = tli_case(rng, v_d, v_t, 3, 2, frac=frac)
    want = oracle_tli(c, 2)
    for got in (fused(c, 2), fused(c, 2, intersected_mass(c))):
        assert np.array_equal(got[0], want[0]), np.nonzero(got[0] != want[0])[0][:5]
        assert np.array_equal(got[1], want[1]), np.nonzero(got[1] != want[1])[0][:5]
    assert (want[0] < c["Ms"]).any()  # a residual row is sampled


def test_fused_tli_with_the_drafters_mass():
    """S_j taken as given (App. D Alg. 3 normalises q' on the draft side): masses off the
    intersected sum by up to a factor of two either way, and zero or NaN masses (q' = 0)."""
    print("[case] fused tli with draft masses", flush=True)
    rng = np.random.default_rng(48)
    c = tli_case(rng, 2000, 3000, 48, 5)
    mass = intersected_mass(c) * rng.uniform(0.5, 2.0, len(c["q"])).astype(np.float32)
    mass[::7] = 0.0
    mass[3::11] = np.nan
    want = oracle_tli(c, 5, mass=mass)
    got = fused(c, 5, mass)
    assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])


def test_fused_tli_at_the_benchmark_vocabulary_sizes():
    print("[case] fused tli workload 3 vocabulary sizes", flush=True)
    wl = synth.make(3, n_streams=4, probs=False)
    rng = np.random.default_rng(49)
    c = tli_case(rng, len(wl.vocab_d.offsets) - 1, len(wl.vocab_t.offsets) - 1, 32, 4, frac=0.8)
    want = oracle_tli(c, 4)
    for got in (fused(c, 4), fused(c, 4, intersected_mass(c)), two_calls(c, 4)):
        assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])


@pytest.mark.parametrize("v_t", [1 << 21, (1 << 21) + 1])
def test_fused_tli_at_the_row_limit(v_t):
    """Target rows of 2^21 floats (2,048 chunks: the chunk sums fill the kernel's LDS) match the
    oracle; one float more is refused with TT_EUNSUPPORTED before anything runs."""
    import paper_2510_15545_amd as tt

    print(f"[case] fused tli v_t={v_t}", flush=True)
    rng = np.random.default_rng(51)
    if v_t > 1 << 21:
        c = tli_case(rng, 300, 50, 2, 1)
        d2t, t2d = random_maps(rng, 300, v_t, 0.001)
        c.update(d2t=d2t, t2d=t2d, v_t=v_t, pt=np.zeros((int(c["off"][-1]) + 2, v_t), np.float32))
        with pytest.raises(tt.TTError) as e:
            fused(c, 1)
        assert e.value.status == tt.TT_EUNSUPPORTED
        return
    c = tli_case(rng, 4000, v_t, 3, 2, frac=0.5)
    want = oracle_tli(c, 2)
    for got in (fused(c, 2), fused(c, 2, intersected_mass(c))):
        assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])
