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
