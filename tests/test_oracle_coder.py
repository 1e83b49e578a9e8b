"""Pins of the oracle's integer parts: serialisation, table quantisation and
the arithmetic coder.  Each test checks the oracle against something other
than itself: closed forms, the paper's worked example, brute force, or
bounds from the paper."""
import json
import math
import os
import struct
from fractions import Fraction

import numpy as np
import pytest

from oracle import coder

HEX = [ord(c) for c in "0123456789abcdef"]
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _text(tok):
    return "".join(chr(t) for t in tok)


# ------------------------------------------------------------ serialisation --
@pytest.mark.parametrize("value,text", [
    (1.0, "3f800000 "),            # IEEE-754: sign 0, exponent 127, mantissa 0
    (-2.0, "c0000000 "),           # sign 1, exponent 128
    (0.5, "3f000000 "),
    (-0.0, "80000000 "),
    (float("inf"), "7f800000 "),
])
def test_hex_closed_forms(value, text):
    tok, sym = coder.serialize(np.array([value], np.float32), 4, 4, 1, HEX, 32)
    assert _text(tok) == text
    assert list(sym) == [int(c, 16) for c in text[:8]] + [16]


def test_hex_bit_patterns_and_lengths():
    bits = np.array([0x00000001, 0x7F7FFFFF, 0x00800000, 0xDEADBEEF], np.uint32)
    tok, _ = coder.serialize(bits.view(np.float32), 4, 4, 1, HEX, 32)
    assert _text(tok) == "00000001 7f7fffff 00800000 deadbeef "
    # little-endian memory order, high nibble of each byte first
    tok, _ = coder.serialize(bits.view(np.float32), 4, 4, 0, HEX, 32)
    assert _text(tok) == "01000000 ffff7f7f 00008000 efbeadde "
    for n in (0, 1, 7, 1000):
        assert coder.num_tokens(n, 4, 4) == 9 * n          # 8 digits + separator


@pytest.mark.parametrize("bpv,bpg", [(4, 0), (4, 1), (4, 2), (4, 3), (4, 4), (4, 8),
                                     (2, 2), (1, 1), (1, 4)])
def test_hex_grouping_structure(bpv, bpg):
    rng = np.random.default_rng(5)
    n = 37
    raw = rng.integers(0, 256, n * bpv, dtype=np.uint8)
    dt = {1: np.uint8, 2: np.uint16, 4: np.float32}[bpv]
    vals = raw.view(dt)
    tok, sym = coder.serialize(vals, bpv, bpg, 1, HEX, 32)
    nbytes = n * bpv
    ngroups = 0 if bpg == 0 else -(-nbytes // bpg)
    assert tok.size == 2 * nbytes + ngroups
    # brute force: rebuild the text from Python's own hex formatting
    stream = b"".join(v.tobytes()[::-1] for v in vals)      # most significant byte first
    want = []
    for i, byte in enumerate(stream):
        want.append(f"{byte:02x}")
        if bpg and ((i + 1) % bpg == 0 or i + 1 == nbytes):
            want.append(" ")
    assert _text(tok) == "".join(want)
    back = coder.deserialize(sym, n, bpv, bpg, 1, dt)
    assert back.tobytes() == vals.tobytes()


def test_deserialize_rejects_malformed():
    vals = np.array([1.0, 2.0], np.float32)
    _, sym = coder.serialize(vals, 4, 4, 1, HEX, 32)
    bad = sym.copy()
    bad[8], bad[7] = bad[7], bad[8]            # separator moved into a digit slot
    with pytest.raises(ValueError):
        coder.deserialize(bad, 2, 4, 4, 1, np.float32)
    with pytest.raises(ValueError):
        coder.deserialize(sym[:-1], 2, 4, 4, 1, np.float32)
    bad = sym.copy()
    bad[0] = 17                                # escape bin in the data
    with pytest.raises(ValueError):
        coder.deserialize(bad, 2, 4, 4, 1, np.float32)


# The paper's separator variants (Sec. 5.2, Table 1): H_s (space), H_c (comma),
# H_semi (semicolon), H_c+s (comma then space: two tokens, coder bins 16 and
# 17) and H_n (no separator: bytes per group 0).
@pytest.mark.parametrize("sep,sep2,text", [
    (ord(" "), -1, "3f800000 c0000000 "),
    (ord(","), -1, "3f800000,c0000000,"),
    (ord(";"), -1, "3f800000;c0000000;"),
    (ord(","), ord(" "), "3f800000, c0000000, "),
])
def test_separator_variants_closed_forms(sep, sep2, text):
    tok, sym = coder.serialize(np.array([1.0, -2.0], np.float32), 4, 4, 1, HEX, sep, sep2)
    assert _text(tok) == text
    digits = [int(c, 16) for c in "3f800000"], [int(c, 16) for c in "c0000000"]
    tail = [16, 17] if sep2 >= 0 else [16]
    assert list(sym) == digits[0] + tail + digits[1] + tail
    nsep = 2 if sep2 >= 0 else 1
    assert coder.num_tokens(2, 4, 4, nsep) == tok.size
    for n in (0, 1, 7, 1000):
        assert coder.num_tokens(n, 4, 4, nsep) == (8 + nsep) * n


def test_no_separator_variant():
    tok, sym = coder.serialize(np.array([1.0, -2.0], np.float32), 4, 0, 1, HEX, 32)
    assert _text(tok) == "3f800000c0000000"
    assert sym.max() < 16


@pytest.mark.parametrize("bpv,bpg", [(4, 1), (4, 2), (4, 3), (4, 4), (4, 8), (1, 1), (2, 3)])
@pytest.mark.parametrize("msb", [1, 0])
def test_two_token_separator_structure_and_roundtrip(bpv, bpg, msb):
    rng = np.random.default_rng(11 * bpg + bpv + msb)
    n = 29
    dt = {1: np.uint8, 2: np.uint16, 4: np.float32}[bpv]
    vals = rng.integers(0, 256, n * bpv, dtype=np.uint8).view(dt)
    tok, sym = coder.serialize(vals, bpv, bpg, msb, HEX, ord(","), ord(" "))
    nbytes = n * bpv
    assert tok.size == 2 * nbytes + 2 * -(-nbytes // bpg)
    # brute force from Python's hex formatting, ", " closing every group
    stream = b"".join(v.tobytes()[::-1] if msb else v.tobytes() for v in vals)
    want = []
    for i, byte in enumerate(stream):
        want.append(f"{byte:02x}")
        if (i + 1) % bpg == 0 or i + 1 == nbytes:
            want.append(", ")
    assert _text(tok) == "".join(want)
    back = coder.deserialize(sym, n, bpv, bpg, msb, dt, nsep=2)
    assert back.tobytes() == vals.tobytes()
    # the one-token reading of the same stream is malformed
    with pytest.raises(ValueError):
        coder.deserialize(sym, n, bpv, bpg, msb, dt, nsep=1)


def test_two_token_separator_rejects_malformed():
    vals = np.array([1.0, 2.0, 3.0], np.float32)
    _, sym = coder.serialize(vals, 4, 4, 1, HEX, ord(","), ord(" "))
    assert list(sym[8:10]) == [16, 17]
    for i, j in ((8, 9), (7, 8), (9, 10)):        # swapped separator tokens, digit/separator
        bad = sym.copy()
        bad[i], bad[j] = bad[j], bad[i]
        with pytest.raises(ValueError):
            coder.deserialize(bad, 3, 4, 4, 1, np.float32, nsep=2)
    bad = sym.copy()
    bad[19] = 16                                  # first separator token twice
    with pytest.raises(ValueError):
        coder.deserialize(bad, 3, 4, 4, 1, np.float32, nsep=2)
    bad = sym.copy()
    bad[3] = 18                                   # escape bin in the data
    with pytest.raises(ValueError):
        coder.deserialize(bad, 3, 4, 4, 1, np.float32, nsep=2)
    with pytest.raises(ValueError):
        coder.deserialize(sym[:-1], 3, 4, 4, 1, np.float32, nsep=2)


@pytest.mark.slow
def test_hex_roundtrip_all_float32_bit_patterns():
    """Every one of the 2^32 patterns (NaN payloads, +-0, subnormals, +-inf)
    comes back bit-exact."""
    assert coder.hex_roundtrip_all(msb_first=1) == 0


def test_hex_roundtrip_memory_order_sample():
    L = coder.lib()
    for lo in (0, 0x7F7F0000, 0x80000000, 0xFFFF0000):
        assert L.orc_hex_roundtrip_range(lo, lo + (1 << 16), 0) == 0


# -------------------------------------------------------- quantised tables --
@pytest.mark.parametrize("V,f_alpha,f_esc", [
    # uniform logits -> p = 1/V; f = 1 + floor((1/V) * 65518); esc = 65536 - 17 f
    (256, 256, 61184),
    (32000, 3, 65485),
    (50257, 2, 65502),
])
def test_quantize_uniform_closed_form(V, f_alpha, f_esc):
    lp = np.full((3, 17), -math.log(V), np.float32)
    cdf = coder.quantize(lp, 1 << 16)
    f = np.diff(cdf.astype(np.int64), axis=-1)
    assert (f[:, :17] == f_alpha).all()
    assert (f[:, 17] == f_esc).all()
    assert (cdf[:, 0] == 0).all() and (cdf[:, -1] == 65536).all()


@pytest.mark.parametrize("V,f_alpha,f_esc", [
    # 18-symbol alphabet (two-token separator): f = 1 + floor((1/V) * 65517),
    # esc = 65536 - 18 f
    (256, 256, 60928),
    (32000, 3, 65482),
    (50257, 2, 65500),
])
def test_quantize_uniform_closed_form_18_symbols(V, f_alpha, f_esc):
    lp = np.full((2, 18), -math.log(V), np.float32)
    cdf = coder.quantize(lp, 1 << 16)
    assert cdf.shape == (2, 20)
    f = np.diff(cdf.astype(np.int64), axis=-1)
    assert (f[:, :18] == f_alpha).all()
    assert (f[:, 18] == f_esc).all()
    assert (cdf[:, 0] == 0).all() and (cdf[:, -1] == 65536).all()


def test_quantize_invariants():
    rng = np.random.default_rng(0)
    for scale in (0.1, 1.0, 5.0, 30.0):
        z = rng.normal(0, scale, (2000, 40))                 # 40-entry vocabulary
        z[:, :17] += rng.normal(0, scale, (2000, 17))
        lse = np.log(np.exp(z - z.max(1, keepdims=True)).sum(1)) + z.max(1)
        lp = (z[:, :17] - lse[:, None]).astype(np.float32)
        cdf = coder.quantize(lp)
        f = np.diff(cdf.astype(np.int64), axis=-1)
        assert (f >= 1).all()
        assert (cdf[:, -1] == 65536).all()
        # monotone in p within a row
        p = np.exp(lp.astype(np.float64))
        for r in range(0, 2000, 97):
            o = np.argsort(p[r], kind="stable")
            assert (np.diff(f[r, :17][o]) >= 0).all()


def test_quantize_all_mass_on_one_symbol():
    lp = np.full((1, 17), -200.0, np.float32)
    lp[0, 5] = 0.0
    f = np.diff(coder.quantize(lp).astype(np.int64))[0]
    assert f[5] == 65536 - 17 and (np.delete(f, [5, 17]) == 1).all() and f[17] == 1


def test_quantize_all_mass_on_one_symbol_18_symbols():
    lp = np.full((1, 18), -200.0, np.float32)
    lp[0, 17] = 0.0
    f = np.diff(coder.quantize(lp).astype(np.int64))[0]
    assert f[17] == 65536 - 18 and (f[:17] == 1).all() and f[18] == 1


# Renormalised tables: the LM's distribution restricted to the alphabet and
# renormalised, no escape mass.  f_a = 1 + floor(p_a (T - A)); the largest
# takes T - sum; the escape bin is empty.
@pytest.mark.parametrize("A,f0,f_rest", [
    (17, 3856, 3855),      # 65519 / 17 = 3854.06 -> 3855; sum 65535, +1 to bin 0
    (18, 3656, 3640),      # 65518 / 18 = 3639.89 -> 3640; sum 65520, +16 to bin 0
])
def test_quantize_renorm_uniform_closed_form(A, f0, f_rest):
    lp = np.full((3, A), -math.log(A), np.float32)
    cdf = coder.quantize(lp, 1 << 16, renorm=True)
    f = np.diff(cdf.astype(np.int64), axis=-1)
    assert (f[:, 0] == f0).all() and (f[:, 1:A] == f_rest).all()
    assert (f[:, A] == 0).all()                                   # empty escape bin
    assert (cdf[:, -2] == 65536).all() and (cdf[:, -1] == 65536).all()


def test_quantize_renorm_all_mass_and_invariants():
    lp = np.full((1, 17), -200.0, np.float32)
    lp[0, 3] = 0.0
    f = np.diff(coder.quantize(lp, renorm=True).astype(np.int64))[0]
    assert f[3] == 65536 - 16 and (np.delete(f, [3, 17]) == 1).all() and f[17] == 0
    rng = np.random.default_rng(9)
    for T in (38, 1 << 16, 1 << 24):
        for A in (17, 18):
            z = rng.normal(0, 3.0, (500, A))
            lp = z - np.log(np.exp(z).sum(1, keepdims=True))      # normalised over the alphabet
            lp = lp.astype(np.float32)
            cdf = coder.quantize(lp, T, renorm=True)
            f = np.diff(cdf.astype(np.int64), axis=-1)
            assert (f[:, :A] >= 1).all() and (f[:, A] == 0).all() and (cdf[:, -1] == T).all()
            p = np.exp(lp.astype(np.float64))
            # each bin within p A + 1 of p T; the largest also absorbs T - sum <= A
            assert np.abs(f[:, :A] - p * T).max() <= 2 * A + 2


def test_renorm_tables_code_as_alphabet_only_tables():
    """An empty last bin codes exactly as the same table without it, and the
    stream stays within the Sec. 3 bound."""
    rng = np.random.default_rng(4)
    n = 400
    z = rng.normal(0, 2.0, (n, 17))
    lp = (z - np.log(np.exp(z).sum(1, keepdims=True))).astype(np.float32)
    cdf = coder.quantize(lp, renorm=True)
    sym = np.array([rng.choice(17, p=np.exp(r.astype(np.float64)) / np.exp(r.astype(np.float64)).sum())
                    for r in lp], np.uint8)
    pay, nbits = coder.ac_encode(cdf, sym)
    pay2, nbits2 = coder.ac_encode(np.ascontiguousarray(cdf[:, :18]), sym)   # 17 bins, no escape
    assert (pay, nbits) == (pay2, nbits2)
    f = cdf[np.arange(n), sym.astype(int) + 1].astype(np.int64) - cdf[np.arange(n), sym].astype(np.int64)
    H = float(-np.sum(np.log2(f / 65536.0)))
    assert H - 1e-6 <= nbits <= H + 2 + 1e-6
    dec = coder.StepDecoder(pay, nbits)
    assert [dec.decode(cdf[j]) for j in range(n)] == list(sym)


# -------------------------------------------------------- arithmetic coder --
def _bits_str(payload, nbits):
    return "".join(f"{b:08b}" for b in payload)[:nbits]


def test_paper_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "ac_worked_example.json")))
    freq = g["freq"]
    T = sum(freq)
    cdf_row = [0, freq[0], T]
    msg = [g["symbols"].index(c) for c in g["message"]]
    # the printed intervals follow from the probabilities (exact rationals)
    lo, hi = Fraction(0), Fraction(1)
    for s, (plo, phi) in zip(msg, g["intervals"][1:]):
        w = hi - lo
        lo, hi = lo + w * Fraction(cdf_row[s], T), lo + w * Fraction(cdf_row[s + 1], T)
        assert (lo, hi) == (Fraction(plo), Fraction(phi))
    cdf = np.array([cdf_row] * len(msg), np.uint32)
    payload, nbits = coder.ac_encode(cdf, np.array(msg, np.uint8))
    code = _bits_str(payload, nbits)
    # our code is a binary fraction inside the paper's final interval ...
    val = Fraction(int(code, 2), 2 ** nbits)
    assert lo <= val < hi
    # ... within the paper's bound H <= l <= H + 2 (H = -log2 of the width)
    H = -math.log2(float(hi - lo))
    assert H <= nbits <= H + 2
    assert code == "0111"
    # the paper's own code decodes to the message
    pbits = g["paper_code_bits"]
    out = coder.ac_decode(cdf, bytes([int(pbits, 2)]), len(pbits))
    assert "".join(g["symbols"][s] for s in out) == g["message"]


def test_uniform_16_table_costs_4_bits_per_digit():
    rng = np.random.default_rng(1)
    for T in (16, 1 << 16):
        for n in (1, 10, 4096):
            sym = rng.integers(0, 16, n).astype(np.uint8)
            row = np.arange(17, dtype=np.uint32) * (T // 16)
            cdf = np.tile(row, (n, 1))
            payload, nbits = coder.ac_encode(cdf, sym)
            assert nbits == 4 * n + 2
            assert (coder.ac_decode(cdf, payload, nbits) == sym).all()
            # with an MSB-first uniform code the bits are the digits themselves
            assert _bits_str(payload, 4 * n) == "".join(f"{s:04b}" for s in sym)


def _random_tables(rng, n, nsym, T, kind):
    if kind == "dirichlet":
        p = rng.dirichlet(np.full(nsym, 0.3), n)
    elif kind == "skew":
        p = np.full((n, nsym), 1e-9)
        p[np.arange(n), rng.integers(0, nsym, n)] = 1.0
    else:
        p = rng.random((n, nsym)) ** 8
    f = np.maximum(1, np.floor(p / p.sum(1, keepdims=True) * (T - nsym))).astype(np.int64)
    f[:, -1] += T - f.sum(1)
    assert (f >= 1).all()
    cdf = np.zeros((n, nsym + 1), np.uint32)
    cdf[:, 1:] = np.cumsum(f, 1)
    sym = np.array([rng.choice(nsym, p=fr / fr.sum()) for fr in f], np.uint8)
    return cdf, sym, f


@pytest.mark.parametrize("kind", ["dirichlet", "skew", "power"])
@pytest.mark.parametrize("T", [18, 1 << 10, 1 << 16, (1 << 24) + 3])
def test_roundtrip_and_length_bound(kind, T):
    rng = np.random.default_rng(hash((kind, T)) & 0xFFFF)
    for n in (0, 1, 2, 50, 3000):
        cdf, sym, f = _random_tables(rng, n, 18, T, kind)
        payload, nbits = coder.ac_encode(cdf, sym)
        assert (coder.ac_decode(cdf, payload, nbits) == sym).all()
        H = float(-np.sum(np.log2(f[np.arange(n), sym] / T))) if n else 0.0
        # Sec. 3: H <= l(c) <= H + 2 for one message
        assert H - 1e-6 <= nbits <= H + 2 + 1e-6


def test_roundtrip_hypothesis():
    hyp = pytest.importorskip("hypothesis")
    st = hyp.strategies

    @hyp.settings(max_examples=200, deadline=None)
    @hyp.given(st.lists(st.tuples(st.lists(st.integers(1, 5000), min_size=2, max_size=18),
                                  st.integers(0, 17)), min_size=0, max_size=60))
    def run(rows):
        nsym = 18
        cdf = np.zeros((len(rows), nsym + 1), np.uint32)
        sym = np.zeros(len(rows), np.uint8)
        for j, (fr, s) in enumerate(rows):
            f = np.ones(nsym, np.int64)
            f[:len(fr)] = fr
            cdf[j, 1:] = np.cumsum(f)
            sym[j] = s
        # each row may have its own total
        payload, nbits = coder.ac_encode(cdf, sym)
        assert (coder.ac_decode(cdf, payload, nbits) == sym).all()

    run()


def test_zero_frequency_symbol_is_rejected():
    cdf = np.array([[0, 5, 5, 10]], np.uint32)
    with pytest.raises(ValueError):
        coder.ac_encode(cdf, np.array([1], np.uint8))
