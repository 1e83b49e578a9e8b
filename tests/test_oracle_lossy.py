"""Pins of the oracle's lossy steps (Sec. 5.4, Eq. 4): top-k sparsification,
linear quantisation and SignSGD bit packing, each checked against closed
forms, brute force in plain Python, or an independent float32 emulation."""
import math
import struct

import numpy as np
import pytest

from oracle import lossy
from synth.configs import LOSSY_VARIANTS, lossy_bytes_per_value, parse_lossy
from synth.gen import gen_values


def _f32(x: float) -> float:
    """Round a Python float (double) to float32."""
    return struct.unpack("<f", struct.pack("<f", x))[0]


# ----------------------------------------------------------- sparsification --
def _brute_topk(vals, k):
    """Keep the k largest |v| (ties: lower index), in plain Python floats."""
    ranked = sorted(range(len(vals)), key=lambda i: (-abs(float(vals[i])), i))
    keep = set(ranked[:k])
    return [float(vals[i]) if i in keep else 0.0 for i in range(len(vals))]


@pytest.mark.parametrize("seed", range(6))
def test_sparsify_matches_brute_force_with_ties(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 60))
    # few distinct magnitudes, both signs, and signed zeros: many ties
    vals = (rng.integers(-4, 5, n) * 0.25).astype(np.float32)
    vals[rng.random(n) < 0.1] = -0.0
    for k in sorted({0, 1, n // 4, n // 2, n - 1, n}):
        got = lossy.sparsify_topk(vals, k)
        want = _brute_topk(vals, k)
        assert got.dtype == np.float32
        # bytewise: kept -0.0 stays -0.0, dropped entries are +0.0
        assert got.tobytes() == np.array(want, np.float32).tobytes(), (n, k)


def test_sparsify_keep_count_and_special_values():
    assert [lossy.keep_count(n, p) for n, p in ((8 << 20, 10), (500, 25), (7, 50), (3, 0))] == \
        [838860, 125, 3, 0]
    v = np.array([1.0, np.inf, -np.inf, np.nan, -2.0, 0.0], np.float32)
    got = lossy.sparsify_topk(v, 3)       # NaN, then +inf and -inf (tie: lower index)
    assert np.isnan(got[3]) and got[1] == np.inf and got[2] == -np.inf
    assert list(got[[0, 4, 5]]) == [0.0, 0.0, 0.0]
    out = lossy.sparsify_topk(v[:3], 10)  # k beyond n keeps everything
    assert out.tobytes() == v[:3].tobytes()


def test_sparsify_normal_vector_properties():
    v = gen_values("normal:1e-3", 100000, 4)
    for pct in (50, 25, 10):
        k = lossy.keep_count(v.size, pct)
        s = lossy.sparsify_topk(v, k)
        kept = s != 0
        assert kept.sum() == k                          # no exact zeros in a normal draw
        assert np.abs(v[kept]).min() >= np.abs(v[~kept]).max()
        assert np.array_equal(s[kept], v[kept])


# ------------------------------------------------------------- quantisation --
@pytest.mark.parametrize("bits,want", [
    (8, [0, 255, 128, 64]),              # 0.5 * 255 = 127.5 -> 128 (even); 0.25 * 255 = 63.75
    (16, [0, 65535, 32768, 16384]),      # 32767.5 -> 32768; 16383.75 -> 16384
    (1, [0, 1, 0, 0]),                   # 0.5 -> 0 (even), 0.25 -> 0
    (2, [0, 3, 2, 1]),                   # 1.5 -> 2, 0.75 -> 1
])
def test_quantize_closed_forms(bits, want):
    q, mn, mx = lossy.quantize_linear(np.array([0.0, 1.0, 0.5, 0.25], np.float32), bits)
    assert list(q) == want and (mn, mx) == (0.0, 1.0)
    assert q.dtype == (np.uint8 if bits <= 8 else np.uint16)


@pytest.mark.parametrize("bits", [1, 3, 8, 12, 16])
def test_quantize_matches_float32_emulation(bits):
    """Each float32 operation emulated as a double operation rounded to float32
    (exact for +, -, *, / of float32 operands); Python's round() is half-even."""
    v = gen_values("laplace:1e-3", 3000, bits)
    v[7] = 0.0
    q, mn, mx = lossy.quantize_linear(v, bits)
    lo, hi = min(map(float, v)), max(map(float, v))
    assert (mn, mx) == (lo, hi)
    span = _f32(hi - lo)
    levels = float((1 << bits) - 1)
    want = [round(_f32(_f32(_f32(float(x) - lo) / span) * levels)) for x in v]
    assert list(map(int, q)) == want
    assert q.max() == (1 << bits) - 1 and q.min() == 0
    order = np.argsort(v, kind="stable")
    assert (np.diff(q[order].astype(np.int64)) >= 0).all()     # monotone in v


def test_quantize_degenerate_and_rejected():
    q, mn, mx = lossy.quantize_linear(np.full(9, -3.5, np.float32), 8)
    assert not q.any() and mn == mx == -3.5
    assert lossy.quantize_linear(np.zeros(0, np.float32), 16)[0].dtype == np.uint16
    for bad in (np.nan, np.inf, -np.inf):
        with pytest.raises(ValueError):
            lossy.quantize_linear(np.array([1.0, bad, 2.0], np.float32), 8)
    for bits in (0, 17):
        with pytest.raises(ValueError):
            lossy.quantize_linear(np.ones(3, np.float32), bits)


# ------------------------------------------------------------- sign packing --
def test_sign_pack_closed_forms():
    v = np.array([-1.0, 2.0, -0.0, 0.0, -np.inf, np.nan, 3.0, -4.0, -5.0], np.float32)
    assert list(lossy.sign_pack(v)) == [0b10101001, 0b10000000]
    assert lossy.sign_pack(np.zeros(0, np.float32)).size == 0
    assert list(lossy.sign_pack(-np.ones(16, np.float32))) == [255, 255]


def test_sign_pack_brute_force():
    rng = np.random.default_rng(3)
    for n in (1, 7, 8, 9, 63, 64, 1000):
        v = rng.normal(size=n).astype(np.float32)
        got = lossy.sign_pack(v)
        want = []
        for j in range(0, n, 8):
            b = 0
            for t in range(8):
                b = (b << 1) | (1 if j + t < n and math.copysign(1.0, float(v[j + t])) < 0 else 0)
            want.append(b)
        assert list(got) == want


# ------------------------------------------------------------- composition --
def test_lossy_spec_grammar():
    assert parse_lossy("") == []
    assert parse_lossy("sparsify:10+quantize:8") == [("sparsify", 10), ("quantize", 8)]
    assert parse_lossy("sign") == [("sign", 0)]
    for bad in ("quantize:0", "quantize:17", "sparsify:101", "sign:1", "quantize:8+sparsify:10",
                "quantize:8+sign", "foo"):
        with pytest.raises(ValueError):
            parse_lossy(bad)
    assert {k: lossy_bytes_per_value(s) for k, s in LOSSY_VARIANTS.items()} == \
        dict(q16=2, q8=1, sign=1, s50=4, s25=4, s10=4, s10q8=1)


def test_sparsify_then_quantize():
    n = 100000
    v = gen_values("normal:1e-3", n, 0)
    q = lossy.prepare(v, "sparsify:10+quantize:8")
    assert q.dtype == np.uint8 and q.size == n
    assert q.min() == 0 and q.max() == 255                   # Eq. 4: min -> 0, max -> 2^n - 1
    zero_code = np.bincount(q, minlength=256).argmax()       # the 90% zeros share one code
    assert np.sum(q == zero_code) >= 0.9 * n
    s = lossy.sparsify_topk(v, n // 10)
    kept = s != 0
    order = np.argsort(v[kept], kind="stable")
    assert (np.diff(q[kept][order].astype(int)) >= 0).all()
    assert lossy.prepare(v, "sign").size == n // 8
    assert lossy.prepare(v, "quantize:16").dtype == np.uint16
    assert lossy.prepare(v, "").tobytes() == v.tobytes()
