"""tt_verify_logits (verification from bf16 logits and a temperature) against the oracle, bit for
bit: ragged and aligned rows, padded and odd strides, temperatures, NaN and -inf logits, forced
acceptances (several rows per stream), sentinel streams, and the benchmark's row width; each with
and without caller-supplied per-row log-sum-exp values (exact ones, and shifted ones that push
P above 1 or below the true softmax)."""
import numpy as np
import pytest

import oracle
from gpu_util import to_dev
from test_oracle_logits import bf16_bits, row_lse

pytestmark = pytest.mark.gpu


def logits_case(n, V, ld=None, seed=0, max_m=8):
    rng = np.random.default_rng(seed + V)
    ld = ld or V
    Ms = rng.integers(0, max_m + 1, n)
    off = np.zeros(n + 1, np.int32)
    off[1:] = np.cumsum(Ms)
    nt = int(off[-1])
    x = rng.normal(0, 3, (nt + n, V)).astype(np.float32)
    ids = rng.integers(0, V, nt).astype(np.int32)
    rows_of = (off[:-1] + np.arange(n))[np.repeat(np.arange(n), Ms)] + (np.arange(nt) - np.repeat(off[:-1], Ms))
    force = rng.random(nt) < 0.6  # the target's argmax on the proposal: acceptances, several rows per stream
    x[rows_of[force], ids[force]] = x[rows_of[force]].max(axis=1) + 3.0
    x[rng.random(x.shape) < 0.001] = np.nan
    bits = np.zeros((nt + n, ld), np.uint16)
    bits[:, :V] = bf16_bits(x)
    q = (rng.random(nt) * 0.5 + 0.05).astype(np.float32)
    it = (1.0 / rng.uniform(0.5, 1.5, n)).astype(np.float32)
    ua = (rng.integers(0, 1 << 24, nt) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, n) * 2.0 ** -24).astype(np.float32)
    return ids, off, q, bits, it, ua, us, Ms


def case_lse(V, case, shift=0.0):
    """fp32 log-sum-exp of each row's logit * inv_temp (its stream's), plus shift."""
    ids, off, q, bits, it, ua, us, Ms = case
    row_it = np.repeat(it, Ms + 1)
    return (row_lse(bits[:, :V], row_it) + np.float32(shift)).astype(np.float32)


def run_both(V, case, max_m, lse=None):
    import torch

    import paper_2510_15545_amd as tt

    ids, off, q, bits, it, ua, us, Ms = case
    nacc, tok = tt.verify_logits(V, to_dev(ids), to_dev(off), to_dev(q), to_dev(bits.view(np.int16)),
                                 to_dev(it), to_dev(ua), to_dev(us), max_m,
                                 lse=None if lse is None else to_dev(lse))
    torch.cuda.synchronize()
    o_nacc, o_tok, _ = oracle.verify_logits(V, ids, off, q, bits, it, ua, us, max_m=max_m, lse=lse)
    assert np.array_equal(nacc.cpu().numpy(), o_nacc), np.nonzero(nacc.cpu().numpy() != o_nacc)[0][:5]
    assert np.array_equal(tok.cpu().numpy(), o_tok), np.nonzero(tok.cpu().numpy() != o_tok)[0][:5]
    return o_nacc, Ms


@pytest.mark.parametrize("n,V,ld", [(37, 1000, None), (20, 4099, 4101), (64, 16384, 16392), (300, 640, None)])
def test_logits_parity(n, V, ld):
    print(f"[case] logits n={n} V={V} ld={ld}", flush=True)
    nacc, Ms = run_both(V, logits_case(n, V, ld), 8)
    assert (nacc > 0).sum() > 0 and (nacc < Ms).sum() > 0  # both acceptances and rejections occur


@pytest.mark.parametrize("shift", [0.0, -0.7, 0.4])
@pytest.mark.parametrize("n,V,ld", [(37, 1000, None), (20, 4099, 4101), (300, 640, None)])
def test_logits_parity_with_lse(n, V, ld, shift):
    print(f"[case] logits+lse n={n} V={V} ld={ld} shift={shift}", flush=True)
    case = logits_case(n, V, ld, seed=3)
    nacc, Ms = run_both(V, case, 8, lse=case_lse(V, case, shift))
    assert (nacc > 0).sum() > 0 and (nacc < Ms).sum() > 0


@pytest.mark.parametrize("shift", [-100.0, -3e9])
def test_logits_lse_far_below_the_logits(shift):
    """A caller's log-sum-exp far below the row's logits: the scaled exponent z runs past 31 (up
    to about 4e9, where converting k to an int would overflow without the clamp at 31); every P
    clamps to 1 and each Q31 weight saturates at 2^31, on both sides alike."""
    print(f"[case] logits+lse shift={shift}", flush=True)
    case = logits_case(37, 1000, None, seed=4)
    nacc, Ms = run_both(V=1000, case=case, max_m=8, lse=case_lse(1000, case, shift))
    assert np.array_equal(nacc, Ms)  # P = 1 >= q: every proposal is accepted


@pytest.mark.parametrize("with_lse", [False, True])
def test_logits_wide_range(with_lse):
    """Logits spread over [-130, 5]: scaled exponents far below the clamp at -1, at it, and up
    to 31, so Q31 weights from 0 to 2^31 are compared."""
    print(f"[case] logits wide range lse={with_lse}", flush=True)
    V = 3000
    ids, off, q, bits, it, ua, us, Ms = logits_case(40, V, seed=11, max_m=4)
    rng = np.random.default_rng(12)
    x = rng.uniform(-130.0, 5.0, bits.shape).astype(np.float32)
    x[rng.random(x.shape) < 0.01] = -88.0  # exact bf16 values just past the cut-off
    bits = bf16_bits(x)
    it[:] = 1.0
    case = (ids, off, q, bits, it, ua, us, Ms)
    run_both(V, case, 4, lse=case_lse(V, case) if with_lse else None)


def test_logits_sentinels_and_degenerate_rows():
    print("[case] logits sentinels", flush=True)
    V = 2000
    ids, off, q, bits, it, ua, us, Ms = logits_case(12, V, seed=5, max_m=4)
    it[1] = 0.0                                   # no temperature: sentinel
    if Ms[2] > 0:
        ids[off[2]] = V + 3                       # an id outside the vocabulary: sentinel
    bits[off[3] + 3 + Ms[3]] = 0xFF80             # stream 3's last row all -inf: Z = 0 if reached
    bits[off[4] + 4] = 0x7FC0                     # stream 4's first row all NaN
    q[off[5]:off[6]] = 0.0                        # q = 0 keeps every proposal of stream 5
    case = (ids, off, q, bits, it, ua, us, Ms)
    run_both(V, case, 4)
    lse = case_lse(V, case)
    lse[off[6] + 6] = np.nan                      # stream 6's first row: a NaN normaliser, no mass
    run_both(V, case, 4, lse=lse)


def test_logits_at_the_benchmark_width():
    print("[case] logits 256 streams V=151936", flush=True)
    V = 151_936
    case = logits_case(256, V, seed=9, max_m=3)
    run_both(V, case, 3)
    run_both(V, case, 3, lse=case_lse(V, case))


@pytest.mark.parametrize("with_lse", [False, True])
def test_logits_every_bf16_pattern(with_lse):
    """Rows that are permutations of bf16 bit patterns, so every slot of the kernel's per-row
    weight table and every pattern outside its domain (magnitudes below 2^-20 or from 256 up,
    infinities, NaNs) meets the formula the oracle evaluates.  With a log-sum-exp: all 65,536
    patterns, normalisers that put the clamp at 31 inside the finite range.  Without: every
    pattern below 8 in magnitude, so the row's largest logit is finite and every value down to
    the subnormals carries weight."""
    print(f"[case] logits every bf16 pattern lse={with_lse}", flush=True)
    rng = np.random.default_rng(77)
    pats = np.arange(1 << 16, dtype=np.uint32)
    if not with_lse:
        mag = pats & 0x7FFF
        pats = pats[mag < 0x4100]
    V = len(pats)
    n = 12
    Ms = rng.integers(0, 3, n)
    off = np.zeros(n + 1, np.int32)
    off[1:] = np.cumsum(Ms)
    nt = int(off[-1])
    bits = np.stack([rng.permutation(pats) for _ in range(nt + n)]).astype(np.uint16)
    ids = rng.integers(0, V, nt).astype(np.int32)
    q = (rng.random(nt) * 0.5 + 0.05).astype(np.float32)
    it = (1.0 / rng.uniform(0.5, 1.5, n)).astype(np.float32)
    ua = (rng.integers(0, 1 << 24, nt) * 2.0 ** -24).astype(np.float32)
    us = (rng.integers(0, 1 << 24, n) * 2.0 ** -24).astype(np.float32)
    case = (ids, off, q, bits, it, ua, us, Ms)
    lse = None
    if with_lse:
        lse = rng.uniform(-5.0, 60.0, nt + n).astype(np.float32)
    run_both(V, case, 2, lse=lse)


def test_logits_lse_residual_at_a_scaled_exponent_just_below_zero():
    """A rejected proposal whose scaled exponent z lies in (-2^-25, 0): its probability E is 0
    (z < 0) while its Q31 weight floor(2^z) is 1 (the polynomial rounds to 1.0).  The residual's
    mass must drop the weight the row's sums counted (1), not the probability's 0: the row is
    ten unit weights and that entry, so the sampled unit is the (floor(10 u) + 1)-th; counting
    the entry's old weight would move the threshold past every entry."""
    print("[case] logits+lse residual at z just below 0", flush=True)
    V = 64
    it = np.float32(1.0 / 0.7)
    x_t = np.float32(1.265625)      # fma(x_t, c, 31 - L log2 e) = -2^-28 for this L
    L = np.float32(23.295599)
    y_unit = np.float32(x_t + 0.25)  # z about 0.5: weight 1
    z_t = np.float32(float(x_t) * float(np.float32(it * np.float32(1.4426950408889634))) +
                     float(np.float32(31.0) - np.float32(L * np.float32(1.4426950408889634))))
    assert -2.0 ** -25 < z_t < 0 and oracle.exp2(z_t) == 1.0 and oracle.logit_prob(x_t, it, L) == 0.0
    n = 4
    Ms = np.ones(n, np.int64)
    off = np.arange(n + 1, dtype=np.int32)
    rows = np.full((2 * n, V), -100.0, np.float32)
    ids = np.full(n, 5, np.int32)
    for b in range(n):
        r = b + b  # row of position 0 is off[b] + b
        rows[r, 5] = x_t
        rows[r, 20:30] = y_unit
        rows[r + 1, :] = 0.0
    bits = bf16_bits(rows)
    q = np.full(n, 0.5, np.float32)
    ua = np.full(n, 0.99, np.float32)
    us = np.float32([0.95, 0.05, 0.5, 0.999])
    lse = np.full(2 * n, L, np.float32)
    case = (ids, off, q, bits, np.full(n, it, np.float32), ua, us, Ms)
    o_nacc, _ = run_both(V, case, 1, lse=lse)
    assert np.array_equal(o_nacc, np.zeros(n))
    _, tok, z = oracle.verify_logits(V, ids, off, q, bits, np.full(n, it, np.float32), ua, us, max_m=1, lse=lse)
    assert np.array_equal(z, np.full(n, 10)) and np.array_equal(tok, 20 + np.floor(us.astype(np.float64) * 10))


@pytest.mark.parametrize("with_lse", [False, True])
def test_logits_at_the_row_limit(with_lse):
    """Rows of 2^23 bf16 logits (8,192 chunks: 64 KiB of chunk sums beside the 64 KiB weight
    table in LDS), with and without normalisers, against the oracle."""
    print(f"[case] logits V=2^23 lse={with_lse}", flush=True)
    V = 1 << 23
    rng = np.random.default_rng(52)
    n = 2
    Ms = np.array([1, 0])
    off = np.array([0, 1, 1], np.int32)
    x = rng.standard_normal((3, V), dtype=np.float32) * np.float32(3)
    ids = np.array([int(rng.integers(0, V))], np.int32)
    x[0, ids[0]] = x[0].max() + 1.0  # accepted often: the bonus row is reached as well
    bits = bf16_bits(x)
    q = np.float32([0.3])
    it = np.float32([1.0 / 0.7, 1.0])
    ua = np.float32([0.5])
    us = np.float32([0.25, 0.75])
    case = (ids, off, q, bits, it, ua, us, Ms)
    run_both(V, case, 1, lse=case_lse(V, case) if with_lse else None)
