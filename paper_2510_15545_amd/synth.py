"""Seeded synthetic workloads for the verification hot path.

This module only manufactures inputs: byte-string vocabularies, draft token
sequences, their greedy re-encoding into the target vocabulary, probability
rows and uniforms.  It contains none of the method's arithmetic (no token
distance, no warping, no acceptance test, no sampling), so the oracle and the
GPU path can both consume what it produces without sharing any code.

The paper's models, tokenizers and Spec-Bench prompts are not available; the
five workloads below stand in for them with the shapes the method sees in a
decode step (Sec. 3 "Speculative Decoding", Sec. 4.2.1 re-tokenisation,
App. A.1 string consistency):

  1  1 stream,    K=4, V_d=512,     V_t=640,     lowercase tokens of 1-4 bytes, M <= 8
  2  32 streams,  K=5, V_d=32,000,  V_t=151,936, printable-ASCII tokens 1-8 B, M in [3,12]
  3  256 streams, K=8, V_d=128,256, V_t=151,936, bf16 logits / T=0.7, 30% forced matches
  4  1024 long pairs (64-512 tokens per side) for alignment; probability stage at
     width 32,000 on 8 draft positions per pair
  5  512 streams, K=6, V_d=201,088, V_t=262,144, Zipf(1.1) rows, M in [4,16]

Every random draw comes from a numpy PCG64 stream keyed by (seed, purpose,
stream, position), so any stream or row can be regenerated on its own and a
reduced workload (fewer streams) is a prefix of the full one.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

LOWER = bytes(range(ord("a"), ord("z") + 1))
PRINTABLE = bytes(range(0x20, 0x7F))

# seed bases; the workload index is added to each
SEED_VOCAB, SEED_SEQ, SEED_LOGITS, SEED_UNIF = 1000, 2000, 3000, 4000

_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


# --------------------------------------------------------------------------- vocabularies
@dataclasses.dataclass
class Vocab:
    """Token id -> byte string table in CSR form (bytes u8, offsets i32[n+1])."""

    tokens: list  # list[bytes]
    index: dict  # bytes -> id
    data: np.ndarray  # uint8
    offsets: np.ndarray  # int32, len n+1
    max_len: int

    @property
    def n(self) -> int:
        return len(self.tokens)

    def decode(self, ids) -> bytes:
        return b"".join(self.tokens[int(i)] for i in ids)


def make_vocab(n_tokens: int, alphabet: bytes, max_len: int, seed) -> Vocab:
    """All single symbols of `alphabet` plus distinct random strings.

    Lengths of the random strings are uniform in {2..max_len}; bytes are uniform
    over the alphabet; duplicates are rejected and redrawn.  The final id order
    is a random permutation so that ids carry no structure.
    """
    rng = np.random.default_rng(seed)
    toks = {bytes([c]) for c in alphabet}
    assert n_tokens >= len(toks)
    if n_tokens > sum(len(alphabet) ** ln for ln in range(1, max_len + 1)):
        raise ValueError("alphabet too small for the requested vocabulary")
    alpha = np.frombuffer(alphabet, dtype=np.uint8)
    while len(toks) < n_tokens:
        need = n_tokens - len(toks)
        batch = max(1024, int(need * 1.3))
        lens = rng.integers(2, max_len + 1, size=batch)
        body = alpha[rng.integers(0, len(alpha), size=(batch, max_len))]
        for row, ln in zip(body, lens):
            toks.add(row[:ln].tobytes())
            if len(toks) == n_tokens:
                break
    ordered = sorted(toks)  # canonical order before the seeded shuffle
    perm = rng.permutation(len(ordered))
    tokens = [ordered[p] for p in perm]
    lens = np.fromiter((len(t) for t in tokens), dtype=np.int64, count=len(tokens))
    offsets = np.zeros(len(tokens) + 1, dtype=np.int32)
    np.cumsum(lens, out=offsets[1:])
    data = np.frombuffer(b"".join(tokens), dtype=np.uint8).copy()
    return Vocab(tokens, {t: i for i, t in enumerate(tokens)}, data, offsets, int(lens.max()))


def greedy_encode(text: bytes, vocab: Vocab) -> list:
    """Greedy longest-match tokenisation (stand-in for a target tokenizer).

    At each position the longest vocabulary token that prefixes the remaining
    bytes is taken.  Every single symbol is in the vocabulary, so this always
    succeeds and the concatenated token bytes equal `text`.
    """
    out = []
    pos, n, idx, lmax = 0, len(text), vocab.index, vocab.max_len
    while pos < n:
        for ln in range(min(lmax, n - pos), 0, -1):
            tid = idx.get(text[pos:pos + ln])
            if tid is not None:
                out.append(tid)
                pos += ln
                break
        else:  # pragma: no cover - singles are always present
            raise ValueError("byte not covered by vocabulary")
    return out


# --------------------------------------------------------------------------- helpers
def _uniform24(rng, n) -> np.ndarray:
    """U(0,1) on the 2^-24 grid: k * 2^-24, k uniform in {0..2^24-1} (exact in fp32)."""
    k = rng.integers(0, 1 << 24, size=n, dtype=np.int64)
    return (k.astype(np.float64) * 2.0**-24).astype(np.float32)


def _bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even), returned as fp32."""
    b = x.astype(np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) & 0xFFFF0000
    return b.astype(np.uint32).view(np.float32)


def _softmax_f32(x: np.ndarray) -> np.ndarray:
    x = x.astype(np.float32, copy=False)
    e = np.exp(x - x.max(), dtype=np.float32)
    e /= e.sum(dtype=np.float32)
    return e


def _coprime_multiplier(rng, n: int) -> int:
    while True:
        a = int(rng.integers(1, n))
        if np.gcd(a, n) == 1:
            return a


def _csr(lists) -> tuple:
    off = np.zeros(len(lists) + 1, dtype=np.int32)
    off[1:] = np.cumsum([len(l) for l in lists])
    flat = np.fromiter((t for l in lists for t in l), dtype=np.int32, count=int(off[-1]))
    return flat, off


# --------------------------------------------------------------------------- workloads
@dataclasses.dataclass
class Spec:
    index: int
    name: str
    n_streams: int
    k: int  # draft tokens per stream (fixed) ; 0 for the long-pair workload
    vd: int
    vt: int
    alphabet: bytes
    max_len: int
    m_range: tuple  # inclusive (lo, hi) accepted re-encoded lengths, None = any
    w: int = 8  # Sakoe-Chiba half-width used by default (the paper's global w=8)


SPECS = {
    1: Spec(1, "1 stream K=4 Vd=512 Vt=640", 1, 4, 512, 640, LOWER, 4, (1, 8)),
    2: Spec(2, "32 streams K=5 Vd=32000 Vt=151936", 32, 5, 32000, 151936, PRINTABLE, 8, (3, 12)),
    3: Spec(3, "256 streams K=8 Vd=128256 Vt=151936 bf16/T0.7 30% forced", 256, 8, 128256, 151936,
            PRINTABLE, 8, None),
    4: Spec(4, "1024 long pairs 64-512 tokens, prob stage 8 positions at width 32000", 1024, 0,
            32000, 151936, PRINTABLE, 8, (64, 512)),
    5: Spec(5, "512 streams K=6 Vd=201088 Vt=262144 Zipf(1.1)", 512, 6, 201088, 262144, PRINTABLE, 8,
            (4, 16)),
}


@dataclasses.dataclass
class Workload:
    """One batch of inputs for align -> transfer -> verify.

    CSR conventions (shared with the library):
      draft tokens of stream b:   draft_ids[draft_off[b]:draft_off[b+1]]           (K_b)
      target tokens of stream b:  target_ids[target_off[b]:target_off[b+1]]        (M_b)
      draft row for (b, i):       draft_probs[draft_off[b] + i]                    (width v_d)
      target row for (b, j):      target_probs[target_off[b] + b + j], j in [0, M_b] (width v_t)
      accept uniform for (b, j):  u_accept[target_off[b] + j];  sample uniform: u_sample[b]
    `verify_ids` are the ids the target rows are indexed with (equal to
    target_ids except in workload 4, whose rows are narrower than V_t).
    """

    spec: Spec
    vocab_d: Vocab
    vocab_t: Vocab
    draft_ids: np.ndarray
    draft_off: np.ndarray
    target_ids: np.ndarray
    target_off: np.ndarray
    w: int
    v_d: int = 0  # width of draft rows
    v_t: int = 0  # width of target rows
    verify_ids: np.ndarray | None = None
    draft_probs: np.ndarray | None = None
    target_probs: np.ndarray | None = None
    u_accept: np.ndarray | None = None
    u_sample: np.ndarray | None = None
    prob: "Workload | None" = None  # workload 4: the probability-stage batch
    forced: np.ndarray | None = None  # workload 3: per target position, 1 if forced

    @property
    def n(self) -> int:
        return len(self.draft_off) - 1

    @property
    def max_k(self) -> int:
        return int(np.diff(self.draft_off).max()) if self.n else 0

    @property
    def max_m(self) -> int:
        return int(np.diff(self.target_off).max()) if self.n else 0


_VOCAB_CACHE: dict = {}


def vocabs(spec_index: int) -> tuple:
    spec = SPECS[spec_index]
    src = 2 if spec_index == 4 else spec_index  # workload 4 reuses workload 2's vocabularies
    key = src
    if key not in _VOCAB_CACHE:
        s = SPECS[src]
        vd = make_vocab(s.vd, s.alphabet, s.max_len, [SEED_VOCAB + src, 0])
        vt = make_vocab(s.vt, s.alphabet, s.max_len, [SEED_VOCAB + src, 1])
        _VOCAB_CACHE[key] = (vd, vt)
    return _VOCAB_CACHE[key]


def _draw_stream(spec: Spec, vd: Vocab, vt: Vocab, b: int, seed_shift: int):
    """Draft ids uniform in V_d, re-encoded with V_t; redrawn until M is in range."""
    rng = np.random.default_rng([SEED_SEQ + spec.index + seed_shift, b])
    while True:
        d = [int(x) for x in rng.integers(0, vd.n, size=spec.k)]
        text = vd.decode(d)
        t = greedy_encode(text, vt)
        if spec.m_range is None or spec.m_range[0] <= len(t) <= spec.m_range[1]:
            assert vt.decode(t) == text  # string-level consistency (App. A.1 lemma)
            return d, t


def _draw_long_pair(spec: Spec, vd: Vocab, vt: Vocab, b: int, seed_shift: int):
    """Random printable text encoded with V_d, cut to K ~ U[64,512] tokens, re-encoded with V_t."""
    rng = np.random.default_rng([SEED_SEQ + spec.index + seed_shift, b])
    alpha = np.frombuffer(spec.alphabet, dtype=np.uint8)
    lo, hi = spec.m_range
    while True:
        k = int(rng.integers(lo, hi + 1))
        text = alpha[rng.integers(0, len(alpha), size=k * vd.max_len)].tobytes()
        d = greedy_encode(text, vd)
        if len(d) < k:
            continue
        d = d[:k]
        s = vd.decode(d)
        t = greedy_encode(s, vt)
        if lo <= len(t) <= hi:
            assert vt.decode(t) == s
            return d, t


def _span_owner(vd: Vocab, vt: Vocab, d, t) -> list:
    """For each target token, the draft token whose byte span holds its last byte.

    Pure string bookkeeping from the byte offsets of the two tokenisations; used
    only to decide which draft row to force in workload 3.
    """
    dend = np.cumsum([len(vd.tokens[x]) for x in d])
    tend = np.cumsum([len(vt.tokens[x]) for x in t])
    return [int(np.searchsorted(dend, e - 1, side="right")) for e in tend]


def _fill_rows(out: np.ndarray, jobs, fn):
    """Run fn(row_index, *args) -> fp32 row for every job, writing into `out`, threaded."""

    def run(job):
        r = job[0]
        out[r] = fn(*job)

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(run, jobs, chunksize=max(1, len(jobs) // (_THREADS * 8) or 1)))


def _normal_row(width: int, sigma: float, seed) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.standard_normal(width, dtype=np.float32) * np.float32(sigma)


def make(index: int, n_streams: int | None = None, seed_shift: int = 0, probs: bool = True,
         w: int | None = None, force_runs: float | None = None) -> Workload:
    """Build workload `index` (1-5), optionally only its first `n_streams` streams.

    force_runs (workload 3 only): instead of forcing each target position independently with
    probability 0.3, force a leading run of positions per stream whose length is the number
    of leading successes of Bernoulli(force_runs) trials, so that streams accept long
    prefixes as a well-matched draft model would (force_runs = 0.9: mean run about 9)."""
    spec = SPECS[index]
    vd, vt = vocabs(index)
    n = spec.n_streams if n_streams is None else int(n_streams)
    draw = _draw_long_pair if index == 4 else _draw_stream
    pairs = [draw(spec, vd, vt, b, seed_shift) for b in range(n)]
    draft_ids, draft_off = _csr([p[0] for p in pairs])
    target_ids, target_off = _csr([p[1] for p in pairs])
    wl = Workload(spec, vd, vt, draft_ids, draft_off, target_ids, target_off,
                  spec.w if w is None else w, v_d=spec.vd, v_t=spec.vt, verify_ids=target_ids)
    if index == 4:
        wl.v_d = wl.v_t = 0
        wl.prob = _long_pair_prob_stage(spec, vd, vt, pairs, seed_shift, probs, wl.w)
        return wl
    if probs:
        _make_probs(wl, seed_shift, force_runs)
    return wl


def _make_probs(wl: Workload, seed_shift: int, force_runs: float | None = None) -> None:
    spec, n = wl.spec, wl.n
    c = spec.index
    seed_l = SEED_LOGITS + c + seed_shift
    kd = np.diff(wl.draft_off)
    mt = np.diff(wl.target_off)
    n_draft_rows = int(wl.draft_off[-1])
    n_target_rows = int(wl.target_off[-1]) + n
    wl.draft_probs = np.empty((n_draft_rows, wl.v_d), dtype=np.float32)
    wl.target_probs = np.empty((n_target_rows, wl.v_t), dtype=np.float32)

    if c in (1, 2, 4):
        sigma = {1: 2.0, 2: 3.0, 4: 2.0}[c]
        djobs = [(int(wl.draft_off[b]) + i, b, i) for b in range(n) for i in range(kd[b])]
        tjobs = [(int(wl.target_off[b]) + b + j, b, j) for b in range(n) for j in range(mt[b] + 1)]
        _fill_rows(wl.draft_probs, djobs,
                   lambda r, b, i: _softmax_f32(_normal_row(wl.v_d, sigma, [seed_l, 0, b, i])))
        _fill_rows(wl.target_probs, tjobs,
                   lambda r, b, j: _softmax_f32(_normal_row(wl.v_t, sigma, [seed_l, 1, b, j])))
    elif c == 3:
        # bf16(3*N(0,1)) logits, softmax(logit / 0.7) in fp32.  Each target position
        # is forced with probability 0.3: the target logit of t_j and the draft logit
        # of the draft token owning t_j's last byte are raised to (row max + 1)
        # before the bf16 cast, so both models put their argmax on the proposal.
        inv_t = np.float32(1.0 / 0.7)
        forced = np.zeros(int(wl.target_off[-1]), dtype=np.int8)
        d_force = [dict() for _ in range(n)]  # per stream: draft position -> token to force
        t_force = [dict() for _ in range(n)]
        for b in range(n):
            rng = np.random.default_rng([SEED_SEQ + c + seed_shift, b, 7])
            d = wl.draft_ids[wl.draft_off[b]:wl.draft_off[b + 1]]
            t = wl.target_ids[wl.target_off[b]:wl.target_off[b + 1]]
            owner = _span_owner(wl.vocab_d, wl.vocab_t, d, t)
            if force_runs is None:
                hit = rng.random(len(t)) < 0.3
            else:  # a leading run: positions before the first failed Bernoulli(force_runs) trial
                trials = rng.random(len(t)) < force_runs
                hit = np.cumprod(trials).astype(bool)
            for j in np.nonzero(hit)[0]:
                forced[wl.target_off[b] + j] = 1
                t_force[b][int(j)] = int(t[j])
                d_force[b][owner[j]] = int(d[owner[j]])
        wl.forced = forced

        def row(width, seed, force_tok):
            x = _normal_row(width, 3.0, seed)
            if force_tok is not None:
                x[force_tok] = x.max() + np.float32(1.0)
            return _softmax_f32(_bf16_round(x) * inv_t)

        djobs = [(int(wl.draft_off[b]) + i, b, i) for b in range(n) for i in range(kd[b])]
        tjobs = [(int(wl.target_off[b]) + b + j, b, j) for b in range(n) for j in range(mt[b] + 1)]
        _fill_rows(wl.draft_probs, djobs,
                   lambda r, b, i: row(wl.v_d, [seed_l, 0, b, i], d_force[b].get(i)))
        _fill_rows(wl.target_probs, tjobs,
                   lambda r, b, j: row(wl.v_t, [seed_l, 1, b, j], t_force[b].get(j)))
    elif c == 5:
        # Zipf(1.1) mass over a random rank per token: rank(x) = (a*x + s) mod V with a
        # coprime to V (a seeded bijection), logit = bf16(log mass), fp32 softmax.
        def zipf_table(width):
            r = np.arange(width, dtype=np.float64)
            logit = _bf16_round((-1.1 * np.log1p(r)).astype(np.float32))
            return _softmax_f32(logit)

        pd, pt = zipf_table(wl.v_d), zipf_table(wl.v_t)

        def row(width, table, seed):
            rng = np.random.default_rng(seed)
            a, s = _coprime_multiplier(rng, width), int(rng.integers(0, width))
            rank = (np.arange(width, dtype=np.int64) * a + s) % width
            return table[rank]

        djobs = [(int(wl.draft_off[b]) + i, b, i) for b in range(n) for i in range(kd[b])]
        tjobs = [(int(wl.target_off[b]) + b + j, b, j) for b in range(n) for j in range(mt[b] + 1)]
        _fill_rows(wl.draft_probs, djobs, lambda r, b, i: row(wl.v_d, pd, [seed_l, 0, b, i]))
        _fill_rows(wl.target_probs, tjobs, lambda r, b, j: row(wl.v_t, pt, [seed_l, 1, b, j]))
    else:  # pragma: no cover
        raise ValueError(c)

    # accept uniforms in CSR order from one stream, sample uniforms from another, so a
    # reduced workload's uniforms are a prefix of the full workload's
    wl.u_accept = _uniform24(np.random.default_rng([SEED_UNIF + c + seed_shift, 0]), int(wl.target_off[-1]))
    wl.u_sample = _uniform24(np.random.default_rng([SEED_UNIF + c + seed_shift, 1]), n)


def _long_pair_prob_stage(spec, vd, vt, pairs, seed_shift, probs, w) -> Workload:
    """Probability stage of the long-pair workload.

    Each pair contributes a short stream made of its first 8 draft tokens and their
    greedy re-encoding; rows are 32,000 wide on both sides, so target ids are taken
    modulo 32,000 when indexing target rows (`verify_ids`).
    """
    width = 32000
    short = []
    for d, _t in pairs:
        dd = d[:8]
        s = vd.decode(dd)
        tt = greedy_encode(s, vt)
        assert vt.decode(tt) == s
        short.append((dd, tt))
    draft_ids, draft_off = _csr([p[0] for p in short])
    target_ids, target_off = _csr([p[1] for p in short])
    sub = Workload(spec, vd, vt, draft_ids, draft_off, target_ids, target_off, w,
                   v_d=width, v_t=width, verify_ids=(target_ids % width).astype(np.int32))
    if probs:
        _make_probs(sub, seed_shift)
    return sub



# --------------------------------------------------------------------------- dense proposals
@dataclasses.dataclass
class DenseWorkload:
    """Standard speculative decoding over one vocabulary (homogeneous draft and target).

    Stream b drafted M_b tokens draft_ids[off[b]:off[b+1]], token j drawn from the dense
    draft row draft_probs[off[b] + j]; the target scored M_b + 1 prefixes, rows
    target_probs[off[b] + b + j], j = 0..M_b."""
    name: str
    v: int
    draft_ids: np.ndarray
    off: np.ndarray
    draft_probs: np.ndarray
    target_probs: np.ndarray
    u_accept: np.ndarray
    u_sample: np.ndarray

    @property
    def n(self) -> int:
        return len(self.off) - 1

    @property
    def max_m(self) -> int:
        return int(np.max(np.diff(self.off))) if self.n else 0


DENSE_INDEX = 6  # seed offset of the dense-proposal workload


def make_dense(n_streams: int = 256, m: int = 8, v: int = 151_936, m_range: tuple | None = None,
               noise: float = 0.5, temperature: float = 0.7, seed_shift: int = 0) -> DenseWorkload:
    """Dense-proposal workload shaped like workload 3 on one vocabulary: target logits
    bf16(3 N(0,1)), draft logits bf16(target + noise N(0,1)) (a draft that mostly agrees with
    the target), fp32 softmax of logit / temperature.  Each drafted token is drawn from its
    draft row with a seeded uniform (the drafter's own sampling, an input here).  M_b = m, or
    uniform in m_range = (lo, hi) inclusive."""
    c = DENSE_INDEX + seed_shift
    rng_m = np.random.default_rng([SEED_SEQ + c, 0])
    ms = (np.full(n_streams, m, np.int64) if m_range is None
          else rng_m.integers(m_range[0], m_range[1] + 1, n_streams))
    off = np.zeros(n_streams + 1, np.int32)
    off[1:] = np.cumsum(ms)
    total = int(off[-1])
    inv_t = np.float32(1.0 / temperature)
    draft_probs = np.empty((total, v), np.float32)
    target_probs = np.empty((total + n_streams, v), np.float32)
    draft_ids = np.empty(total, np.int32)

    def logits(b, j):
        x = _normal_row(v, 3.0, [SEED_LOGITS + c, 1, b, j])
        return x

    def target_row(r, b, j):
        return _softmax_f32(_bf16_round(logits(b, j)) * inv_t)

    def draft_row(r, b, j):
        x = logits(b, j) + _normal_row(v, noise, [SEED_LOGITS + c, 0, b, j])
        q = _softmax_f32(_bf16_round(x) * inv_t)
        u = np.random.default_rng([SEED_SEQ + c, 1, b, j]).random()
        cdf = np.cumsum(q, dtype=np.float64)
        draft_ids[r] = min(int(np.searchsorted(cdf, u * cdf[-1], side="right")), v - 1)
        return q

    _fill_rows(target_probs, [(int(off[b]) + b + j, b, j) for b in range(n_streams) for j in range(ms[b] + 1)],
               target_row)
    _fill_rows(draft_probs, [(int(off[b]) + j, b, j) for b in range(n_streams) for j in range(ms[b])], draft_row)
    u_accept = _uniform24(np.random.default_rng([SEED_UNIF + c, 0]), total)
    u_sample = _uniform24(np.random.default_rng([SEED_UNIF + c, 1]), n_streams)
    return DenseWorkload(f"{n_streams} streams M={m if m_range is None else m_range} V={v} dense proposals",
                         v, draft_ids, off, draft_probs, target_probs, u_accept, u_sample)
