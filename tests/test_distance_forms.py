"""Host emulations of the token-distance formulas the alignment kernels evaluate, checked
against the oracle's textbook Levenshtein (App. H).

The GPU parity tests check the kernels' outputs end to end; these tests check the formulas
themselves on inputs the workloads rarely reach (every pair of short strings, bytes 0x00 and
0x80-0xff, tokens up to 64 bytes), with the bit operations written as the device code performs
them in 32- or 64-bit words:

* the per-byte match mask by a SWAR zero-byte test of the packed token;
* the bit-parallel edit-distance recurrence (Myers 1999, Hyyro's global form) with the longer
  token as the pattern, read at the end from the vertical deltas;
* the closed form used when the draft token has at most two bytes (the draft token is the
  text, the target token the pattern).
"""
import itertools

import numpy as np
import pytest


def packed(s: bytes):
    """Little-endian 32-bit words of s, zero-padded."""
    b = s + b"\0" * (-len(s) % 4)
    return [int.from_bytes(b[k:k + 4], "little") for k in range(0, len(b), 4)]


def match_mask(words, c: int) -> int:
    """Bit k set where byte k of the packed pattern equals c (SWAR zero-byte test per word)."""
    bc = c * 0x01010101
    m = 0
    for w_i, w in enumerate(words):
        t = (w ^ bc) & 0xFFFFFFFF
        z = ~((((t & 0x7F7F7F7F) + 0x7F7F7F7F) & 0xFFFFFFFF) | t) & 0x80808080
        for k in range(4):
            if z & (0x80 << (8 * k)):
                m |= 1 << (4 * w_i + k)
    return m


def myers(a: bytes, b: bytes, width: int) -> int:
    """Edit distance by the bit-parallel recurrence over width-bit words, the longer token as
    the pattern and the shorter as the text."""
    p, t = (a, b) if len(a) >= len(b) else (b, a)
    full = (1 << width) - 1
    lim = full if len(p) >= width else (1 << len(p)) - 1
    words = packed(p)
    vp, vn = full, 0
    for c in t:
        eq = match_mask(words, c) & lim
        xv = eq | vn
        xh = ((((eq & vp) + vp) & full) ^ vp) | eq
        hp = (vn | (~(xh | vp) & full)) & full
        hn = vp & xh
        hp = ((hp << 1) | 1) & full
        hn = (hn << 1) & full
        vp = hn | (~(xv | hp) & full)
        vn = hp & xv
    return len(t) + bin(vp & lim).count("1") - bin(vn & lim).count("1")


def closed(draft: bytes, target: bytes) -> int:
    """The closed form for a draft token of at most two bytes (text) against a target token
    (pattern) of up to 32 bytes, as the strip kernel evaluates it."""
    xm, yn = len(draft), len(target)
    lim = 0xFFFFFFFF if yn >= 32 else (1 << yn) - 1
    words = packed(target)
    e1 = match_mask(words, draft[0] if xm > 0 else 0) & lim
    e2 = match_mask(words, draft[1] if xm > 1 else 0) & lim
    low1 = e1 & ((-e1) & 0xFFFFFFFF)
    in_order = (e2 & ~(((low1 << 1) - 1) & 0xFFFFFFFF)) != 0
    one = (e1 & (lim >> 1)) != 0 or (e2 & ~1 & 0xFFFFFFFF) != 0
    two = yn - 2 + (0 if in_order else (1 if one else 2))
    d2 = 2 - (1 if (e1 | e2) else 0) if yn == 1 else two
    d1 = yn - (1 if e1 else 0)
    return xm + yn if (xm == 0 or yn == 0) else (d1 if xm == 1 else d2)


def test_closed_form_every_short_pair(orc):
    """Every draft string of 0-2 bytes against every target string of 0-6 bytes over three
    symbols, one of them NUL (the padding byte of a packed slot)."""
    alphabet = [0x00, 0x61, 0xFF]
    n = 0
    for lx in range(3):
        for x in itertools.product(alphabet, repeat=lx):
            for ly in range(7):
                for y in itertools.product(alphabet, repeat=ly):
                    xb, yb = bytes(x), bytes(y)
                    assert closed(xb, yb) == orc.levenshtein(xb, yb), (xb, yb)
                    n += 1
    assert n == 13 * 1093


def test_closed_form_long_targets_any_bytes(orc):
    rng = np.random.default_rng(71)
    for _ in range(3000):
        xb = bytes(rng.integers(0, 256, int(rng.integers(0, 3))).astype(np.uint8))
        ly = int(rng.integers(0, 33))
        alpha = rng.integers(0, 256, int(rng.integers(1, 5)))  # few symbols: many matches
        yb = bytes(rng.choice(alpha, ly).astype(np.uint8))
        assert closed(xb, yb) == orc.levenshtein(xb, yb), (xb, yb)


@pytest.mark.parametrize("width,maxlen", [(32, 32), (64, 64)])
def test_bit_parallel_recurrence(orc, width, maxlen):
    rng = np.random.default_rng(72 + width)
    for _ in range(3000):
        k = int(rng.integers(1, 5))
        alpha = rng.integers(0, 256, k)
        a = bytes(rng.choice(alpha, int(rng.integers(0, maxlen + 1))).astype(np.uint8))
        b = bytes(rng.choice(alpha, int(rng.integers(0, maxlen + 1))).astype(np.uint8))
        assert myers(a, b, width) == orc.levenshtein(a, b), (a, b)


def test_match_mask_high_bytes_and_nul():
    """The SWAR test flags exactly the equal bytes, including 0x00, 0x7f, 0x80 and 0xff (a
    carry out of one byte must not flag its neighbour)."""
    for s in (b"\x00\x80\xff\x7f\x00\x01", b"\xff\xff\x00\x80", b"\x7f\x80\x81\x7e"):
        words = packed(s)
        for c in range(256):
            want = sum(1 << k for k, ch in enumerate(s) if ch == c)
            got = match_mask(words, c) & ((1 << len(s)) - 1)
            assert got == want, (s, c)
