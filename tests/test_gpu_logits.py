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
    """A caller's log-sum-exp far below the row's logits: x - L runs past 88 (up to about 3e9,
    where converting k to an int would overflow without the clamp at 88); every P clamps to 1
    and each e39 saturates, on both sides alike."""
    print(f"[case] logits+lse shift={shift}", flush=True)
    case = logits_case(37, 1000, None, seed=4)
    nacc, Ms = run_both(V=1000, case=case, max_m=8, lse=case_lse(1000, case, shift))
    assert np.array_equal(nacc, Ms)  # P = 1 >= q: every proposal is accepted


@pytest.mark.parametrize("with_lse", [False, True])
def test_logits_wide_range(with_lse):
    """Logits spread over [-130, 5]: every x - m in the exponential's cut-off band [-100, -87),
    below it, and near 0, so each e39 on both sides of the cut-off is compared."""
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
