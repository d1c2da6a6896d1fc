"""CPU oracle for the TokenTiming verification hot path -- TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The GPU library never calls it and shares no code with it.

`tt_oracle.c` holds the arithmetic (plain C, fp32 where the inputs are fp32,
exact integers elsewhere); this module builds it with gcc and wraps it with
ctypes over numpy arrays.  The re-tokenisation, the vocabulary intersection and
the Token-Level Intersection proposal are written here in plain Python / numpy.  See the header of `tt_oracle.c` for the paper
passages each function follows and the readings taken where the paper is silent.

Parity status: every function here is pinned by tests under `tests/`
(test_oracle_*.py) against the paper's worked examples, closed forms,
brute force on tiny inputs and distributional properties.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tt_oracle.c")
_LIB = os.path.join(_HERE, "libtt_oracle.so")
CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-std=c11",
          "-Wall", "-Wextra", "-pthread"]

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into oracle/libtt_oracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f32, u64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_uint64
        L.orc_levenshtein.argtypes = [P, ctypes.c_int, P, ctypes.c_int]
        L.orc_levenshtein.restype = ctypes.c_int
        L.orc_align.argtypes = [P, P, i32, i32, P, P, i32, i32, i32, P, P, P, P, i32, i32, i32,
                                P, P, P, P, ctypes.c_int]
        L.orc_align.restype = None
        L.orc_transfer.argtypes = [i32, i32, P, P, P, P, P, i64, P]
        L.orc_transfer.restype = None
        L.orc_verify.argtypes = [i32, i32, P, P, P, P, i64, P, P, i32, P, P, P, P, P, i32,
                                 ctypes.c_int]
        L.orc_verify.restype = None
        L.orc_verify_dense.argtypes = [i32, P, P, i32, f32, f32, P]
        L.orc_verify_dense.restype = i32
        L.orc_sd_verify.argtypes = [i32, i32, P, P, P, i64, P, i64, P, P, i32, P, P, P, P, ctypes.c_int]
        L.orc_sd_verify.restype = None
        L.orc_delta_histogram.argtypes = [i32, P, P, P, P, i32, P]
        L.orc_delta_histogram.restype = None
        L.orc_delta_quantile.argtypes = [P, i32, i32, i32]
        L.orc_delta_quantile.restype = i32
        L.orc_exp2.argtypes = [f32]
        L.orc_exp2.restype = f32
        L.orc_logit_prob.argtypes = [f32, f32, f32]
        L.orc_logit_prob.restype = f32
        L.orc_verify_logits.argtypes = [i32, i32, P, P, P, P, i64, P, P, P, P, i32, P, P, P, ctypes.c_int]
        L.orc_verify_logits.restype = None
        L.orc_threshold.argtypes = [f32, u64]
        L.orc_threshold.restype = u64
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def threads_default() -> int:
    return max(1, len(os.sched_getaffinity(0)))


# ------------------------------------------------------------------------------------
def levenshtein(s: bytes, t: bytes) -> int:
    """App. H edit distance over bytes."""
    a = np.frombuffer(s, dtype=np.uint8) if s else np.zeros(1, np.uint8)
    b = np.frombuffer(t, dtype=np.uint8) if t else np.zeros(1, np.uint8)
    return int(lib().orc_levenshtein(_p(a), len(s), _p(b), len(t)))


def align(vd_bytes, vd_off, vd_maxlen, vt_bytes, vt_off, vt_maxlen, draft_ids, draft_off,
          target_ids, target_off, w, max_k=None, max_m=None, n_threads=None):
    """Alg. 1 over every pair.  Returns (cost, path_len, path, map) as numpy arrays.

    path is int32 [2*(sum K + sum M)]; pair b's (i, j) pairs start at
    2*(draft_off[b] + target_off[b]).
    """
    vd_bytes, vt_bytes = _c(vd_bytes, np.uint8), _c(vt_bytes, np.uint8)
    vd_off, vt_off = _c(vd_off, np.int32), _c(vt_off, np.int32)
    draft_ids, draft_off = _c(draft_ids, np.int32), _c(draft_off, np.int32)
    target_ids, target_off = _c(target_ids, np.int32), _c(target_off, np.int32)
    n = len(draft_off) - 1
    if max_k is None:
        max_k = int(np.diff(draft_off).max()) if n else 0
    if max_m is None:
        max_m = int(np.diff(target_off).max()) if n else 0
    cost = np.zeros(n, np.int32)
    plen = np.zeros(n, np.int32)
    path = np.full(2 * (int(draft_off[-1]) + int(target_off[-1])) + 2, -7, np.int32)
    mp = np.full(max(1, int(target_off[-1])), -7, np.int32)
    lib().orc_align(_p(vd_bytes), _p(vd_off), len(vd_off) - 1, vd_maxlen,
                    _p(vt_bytes), _p(vt_off), len(vt_off) - 1, vt_maxlen,
                    n, _p(draft_ids), _p(draft_off), _p(target_ids), _p(target_off),
                    max_k, max_m, w, _p(cost), _p(plen), _p(path), _p(mp),
                    n_threads or threads_default())
    return cost, plen, path[:-2], mp[:int(target_off[-1])]


def transfer(v_d, draft_ids, draft_off, target_off, mp, draft_probs):
    draft_ids, draft_off = _c(draft_ids, np.int32), _c(draft_off, np.int32)
    target_off, mp = _c(target_off, np.int32), _c(mp, np.int32)
    assert draft_probs.dtype == np.float32 and draft_probs.flags.c_contiguous
    q = np.zeros(max(1, int(target_off[-1])), np.float32)
    lib().orc_transfer(len(draft_off) - 1, v_d, _p(draft_ids), _p(draft_off), _p(target_off),
                       _p(mp), _p(draft_probs), draft_probs.shape[1], _p(q))
    return q[:int(target_off[-1])]


def verify(v_t, target_ids, target_off, q, target_probs, u_accept, u_sample, max_m=None,
           residual=False, select=None, n_threads=None):
    """Returns (n_accepted, out_token, residual or None, Z per stream as uint64)."""
    target_ids, target_off = _c(target_ids, np.int32), _c(target_off, np.int32)
    q, u_accept, u_sample = _c(q, np.float32), _c(u_accept, np.float32), _c(u_sample, np.float32)
    assert target_probs.dtype == np.float32 and target_probs.flags.c_contiguous
    n = len(target_off) - 1
    if max_m is None:
        max_m = int(np.diff(target_off).max()) if n else 0
    nacc = np.full(n, -7, np.int32)
    tok = np.full(n, -7, np.int32)
    z = np.zeros(n, np.uint64)
    res = np.zeros((n, target_probs.shape[1]), np.float32) if residual else None
    sel = None if select is None else _c(select, np.int32)
    # keep non-empty buffers alive for ctypes when arrays are empty
    q_ = q if q.size else np.zeros(1, np.float32)
    ua = u_accept if u_accept.size else np.zeros(1, np.float32)
    ti = target_ids if target_ids.size else np.zeros(1, np.int32)
    lib().orc_verify(n, v_t, _p(ti), _p(target_off), _p(q_), _p(target_probs),
                     target_probs.shape[1], _p(ua), _p(u_sample), max_m, _p(nacc), _p(tok),
                     _p(res), _p(z), _p(sel), 0 if sel is None else len(sel),
                     n_threads or threads_default())
    return nacc, tok, res, z


def verify_dense(p, qd, x, u_accept, u_sample):
    """Test-only: App. D Alg. 4 for one drafted position with a dense proposal."""
    p, qd = _c(p, np.float32), _c(qd, np.float32)
    acc = ctypes.c_int32(0)
    tok = lib().orc_verify_dense(len(p), _p(p), _p(qd), int(x), float(u_accept), float(u_sample),
                                 ctypes.byref(acc))
    return int(tok), int(acc.value)


def sd_verify(v, draft_ids, off, draft_probs, target_probs, u_accept, u_sample, max_m=None,
              residual=False, n_threads=None):
    """App. D Alg. 4 with dense proposals over one vocabulary, for a batch of streams.

    draft_ids/off: CSR drafted tokens; draft_probs row off[b]+j is the dense proposal of
    drafted position j; target_probs row off[b]+b+j (j = 0..M_b) the target distribution.
    Returns (n_accepted, out_token, residual or None, Z)."""
    draft_ids = _c(draft_ids, np.int32)
    off = _c(off, np.int32)
    draft_probs = _c(draft_probs, np.float32)
    target_probs = _c(target_probs, np.float32)
    u_accept = _c(u_accept, np.float32)
    u_sample = _c(u_sample, np.float32)
    n = len(off) - 1
    if max_m is None:
        max_m = int(np.max(np.diff(off))) if n > 0 else 0
    nacc = np.zeros(n, np.int32)
    tok = np.zeros(n, np.int32)
    z = np.zeros(n, np.uint64)
    res = np.zeros((n, target_probs.shape[1]), np.float32) if residual else None
    ids = draft_ids if draft_ids.size else np.zeros(1, np.int32)
    dp = draft_probs if draft_probs.size else np.zeros((1, 1), np.float32)
    ua = u_accept if u_accept.size else np.zeros(1, np.float32)
    lib().orc_sd_verify(n, int(v), _p(ids), _p(off), _p(dp), dp.shape[1], _p(target_probs),
                        target_probs.shape[1], _p(ua), _p(u_sample), int(max_m), _p(nacc), _p(tok),
                        _p(res), _p(z), n_threads or threads_default())
    return nacc, tok, res, z


def exp2(z: float) -> np.float32:
    """The logits path's specified 2^z (z held in [-1, 31])."""
    return np.float32(lib().orc_exp2(float(np.float32(z))))


def logit_prob(x: float, inv_temp: float, lse: float) -> np.float32:
    """P_t of one logit (the fp32 value of its bf16) under a caller's log-sum-exp."""
    return np.float32(lib().orc_logit_prob(float(np.float32(x)), float(np.float32(inv_temp)), float(np.float32(lse))))


def verify_logits(v, target_ids, target_off, q, logits_bf16, inv_temp, u_accept, u_sample, max_m=None,
                  lse=None, n_threads=None):
    """Verification from bf16 target logits (uint16 bit patterns, rows off[b]+b+j) and a per-stream
    inverse temperature: the target softmax formed with the specified exponential, then the
    one-hot acceptance and the residual sample.  With per-row log-sum-exp values `lse` the rows'
    normalisers are taken from them instead.  Returns (n_accepted, out_token, Z)."""
    target_ids, target_off = _c(target_ids, np.int32), _c(target_off, np.int32)
    q, inv_temp = _c(q, np.float32), _c(inv_temp, np.float32)
    u_accept, u_sample = _c(u_accept, np.float32), _c(u_sample, np.float32)
    logits_bf16 = _c(logits_bf16, np.uint16)
    n = len(target_off) - 1
    if max_m is None:
        max_m = int(np.diff(target_off).max()) if n else 0
    nacc = np.full(n, -7, np.int32)
    tok = np.full(n, -7, np.int32)
    z = np.zeros(n, np.uint64)
    ti = target_ids if target_ids.size else np.zeros(1, np.int32)
    q_ = q if q.size else np.zeros(1, np.float32)
    ua = u_accept if u_accept.size else np.zeros(1, np.float32)
    lse = None if lse is None else _c(lse, np.float32)
    lib().orc_verify_logits(n, int(v), _p(ti), _p(target_off), _p(q_), _p(logits_bf16), logits_bf16.shape[1],
                            _p(inv_temp), _p(lse), _p(ua), _p(u_sample), int(max_m), _p(nacc), _p(tok), _p(z),
                            n_threads or threads_default())
    return nacc, tok, z


def delta_histogram(draft_off, target_off, path_len, path, n_bins):
    """Fig. CDF / App. K: counts of |i - j| over every optimal path cell (last bin: >= n_bins-1)."""
    draft_off, target_off = _c(draft_off, np.int32), _c(target_off, np.int32)
    path_len = _c(path_len, np.int32)
    path = _c(path, np.int32) if np.size(path) else np.zeros(2, np.int32)
    hist = np.zeros(int(n_bins), np.int64)
    lib().orc_delta_histogram(len(draft_off) - 1, _p(draft_off), _p(target_off), _p(path_len), _p(path),
                              int(n_bins), _p(hist))
    return hist


def delta_quantile(hist, num=9, den=10):
    """App. K: the smallest deviation d whose CDF over the histogram reaches num/den (exact
    integer comparison); 0 for an empty histogram."""
    h = _c(hist, np.int64) if np.size(hist) else np.zeros(1, np.int64)
    return int(lib().orc_delta_quantile(_p(h), int(np.size(hist)), int(num), int(den)))


def retokenize(vd_bytes, vd_off, vt_bytes, vt_off, draft_ids, draft_off, max_m=None, max_bytes=None):
    """Sec. 4.2.1 / Alg. 2 (S = Tokenizer_d.encode(D), T = Tokenizer_t.decode(S)) and App. A.1
    with a greedy longest-match target tokenizer over byte strings: the draft tokens' bytes are
    concatenated into S; from the start of S, the longest target token that is a prefix of the
    rest is emitted (the lowest id if several tokens share those bytes), until S is consumed.

    Plain Python.  A stream whose string is longer than max_bytes, that encodes to more than
    max_m tokens, that holds a draft id outside the table, or that meets a byte no target token
    starts with, gets no tokens (an empty CSR row).  Returns (target_ids, target_off) int32."""
    vd_bytes = bytes(np.asarray(vd_bytes, np.uint8))
    vt_bytes = bytes(np.asarray(vt_bytes, np.uint8))
    vd_off = np.asarray(vd_off, np.int64)
    vt_off = np.asarray(vt_off, np.int64)
    table = {}
    longest = 0
    for t in range(len(vt_off) - 1):
        s = vt_bytes[vt_off[t]:vt_off[t + 1]]
        longest = max(longest, len(s))
        if s not in table:  # ids ascend: the first holder of a string is the lowest id
            table[s] = t
    out, off = [], [0]
    n_d = len(vd_off) - 1
    for b in range(len(draft_off) - 1):
        ids = [int(x) for x in draft_ids[draft_off[b]:draft_off[b + 1]]]
        toks = []
        if all(0 <= i < n_d for i in ids):
            S = b"".join(vd_bytes[vd_off[i]:vd_off[i + 1]] for i in ids)
            if max_bytes is None or len(S) <= max_bytes:
                p = 0
                while p < len(S):
                    for ln in range(min(longest, len(S) - p), 0, -1):
                        t = table.get(S[p:p + ln])
                        if t is not None:
                            toks.append(t)
                            p += ln
                            break
                    else:
                        toks = []
                        break
                if max_m is not None and len(toks) > max_m:
                    toks = []
        out.extend(toks)
        off.append(off[-1] + len(toks))
    return np.array(out, np.int32), np.array(off, np.int32)


def vocab_intersection(vd_bytes, vd_off, vt_bytes, vt_off, vd_max_bytes=None, vt_max_bytes=None):
    """App. D Alg. 3 (TLI): the intersection of the draft and target vocabularies, each taken as
    a set of byte strings.  Where several ids of one vocabulary share a string, the lowest id
    stands for it and the others are outside the intersection; tokens of length 0 or longer
    than the table's declared maximum are outside too.

    Plain Python.  Returns (d2t int32[V_d], t2d int32[V_t]): d2t[x] is the target id of draft
    id x's string when both sides have it, else -1; t2d is the converse."""
    def table(data, off, max_bytes):
        data = bytes(np.asarray(data, np.uint8))
        off = np.asarray(off, np.int64)
        first, strings = {}, []
        for t in range(len(off) - 1):
            s = data[off[t]:off[t + 1]]
            ok = 0 < len(s) and (max_bytes is None or len(s) <= max_bytes)
            strings.append(s if ok else None)
            if ok and s not in first:  # ids ascend: the first holder is the lowest id
                first[s] = t
        return first, strings

    fd, sd = table(vd_bytes, vd_off, vd_max_bytes)
    ft, st = table(vt_bytes, vt_off, vt_max_bytes)
    d2t = np.full(len(sd), -1, np.int32)
    t2d = np.full(len(st), -1, np.int32)
    for x, s in enumerate(sd):
        if s is not None and fd[s] == x and s in ft:
            d2t[x] = ft[s]
            t2d[ft[s]] = x
    return d2t, t2d


def round_to_f32(num: int, scale_bits: int) -> np.float32:
    """num * 2^-scale_bits (num >= 0 an exact integer) rounded once to the nearest fp32, ties
    to even (normal results only, which is all tli_proposal produces)."""
    if num == 0:
        return np.float32(0.0)
    shift = num.bit_length() - 24
    if shift <= 0:
        return np.float32(np.ldexp(float(num), -scale_bits))
    mant, rem = num >> shift, num & ((1 << shift) - 1)
    half = 1 << (shift - 1)
    if rem > half or (rem == half and (mant & 1)):
        mant += 1
    return np.float32(np.ldexp(float(mant), shift - scale_bits))


def tli_proposal(d2t, t2d, draft_probs, mass=None):
    """App. D Alg. 3 (TLI): q' over the target vocabulary from draft rows q over V_d,
    q'(y) = q(x) / S for y = d2t[x] in the intersection and 0 elsewhere, S the mass q puts on
    the intersection.  Readings: q is clamped to [0, 1] (NaN -> 0); S is the sum of the
    intersected masses, each truncated to a multiple of 2^-62 and summed exactly, then rounded
    once to the nearest fp32; q'(y) is the fp32 quotient; a row with S = 0 gives a zero row.
    mass (optional, one fp32 per row): S as the drafter formed it when it normalised q', used
    instead of the sum; a row whose S is not positive (or NaN) is a zero row.

    Rows of draft_probs are [n, V_d] float32; returns [n, V_t] float32."""
    q = np.asarray(draft_probs, np.float32)
    d2t = np.asarray(d2t, np.int64)
    t2d = np.asarray(t2d, np.int64)
    n = q.shape[0]
    out = np.zeros((n, len(t2d)), np.float32)
    inter = np.nonzero(d2t >= 0)[0]
    for r in range(n):
        qc = np.nan_to_num(q[r], nan=0.0)
        qc = np.minimum(np.maximum(qc, np.float32(0.0)), np.float32(1.0)).astype(np.float32)
        # floor(q * 2^62) is an exact integer below 2^63 (q has a 24-bit significand)
        if mass is None:
            fixed = np.floor(qc[inter].astype(np.float64) * 2.0 ** 62)
            S = round_to_f32(sum(int(v) for v in fixed), 62)
        else:
            S = np.float32(mass[r])
        if not S > 0:
            continue
        out[r, d2t[inter]] = qc[inter] / S  # fp32 quotients
    return out


def threshold(u: float, Z: int) -> int:
    return int(lib().orc_threshold(float(np.float32(u)), int(Z)))


# ------------------------------------------------------------------------------------
def run_workload(wl, n_threads=None, residual=False, select=None):
    """align -> transfer -> verify on a synth.Workload (probability stage included)."""
    vd, vt = wl.vocab_d, wl.vocab_t
    cost, plen, path, mp = align(vd.data, vd.offsets, vd.max_len, vt.data, vt.offsets, vt.max_len,
                                 wl.draft_ids, wl.draft_off, wl.target_ids, wl.target_off, wl.w,
                                 n_threads=n_threads)
    out = {"cost": cost, "path_len": plen, "path": path, "map": mp}
    if wl.draft_probs is not None:
        q = transfer(wl.v_d, wl.draft_ids, wl.draft_off, wl.target_off, mp, wl.draft_probs)
        nacc, tok, res, z = verify(wl.v_t, wl.verify_ids, wl.target_off, q, wl.target_probs,
                                   wl.u_accept, wl.u_sample, residual=residual, select=select,
                                   n_threads=n_threads)
        out.update(q=q, n_accepted=nacc, out_token=tok, residual=res, z=z)
    return out
