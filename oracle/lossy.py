"""Reference lossy steps LM-GC is composed with -- TEST INFRASTRUCTURE ONLY.

Sec. 5.4 ("Compatibility") compresses the output of lossy gradient
compression: linear quantisation to n-bit indices (Eq. 4; n = 16, 8, and
1 bit read as SignSGD) and sparsification that keeps 50, 25 or 10 percent of
the values as float32.  Readings where the paper is silent:

* Sparsification keeps the k = floor(N * percent / 100) values of largest
  magnitude; ties go to the lower index; every other value becomes +0.0 and
  stays in the stream (the serialised vector keeps its length N).  Magnitude
  is compared on the IEEE bit pattern with the sign bit cleared, read as an
  unsigned integer: for numbers this is the order of |v| (+0.0 and -0.0 tie),
  and NaNs rank above infinities.
* Eq. 4 is evaluated in float32, one rounding per operation and no fused
  multiply-add: t = (v - min) / (max - min), q = round-half-even(t * (2^n - 1)).
  min and max are over the whole vector (zeros of a sparsified vector
  included).  A constant vector gives all-zero indices.  A vector holding a
  NaN or an infinity is rejected.  Indices are uint8 for n <= 8, uint16 up to
  n = 16.
* SignSGD's one bit per value is the IEEE sign bit (1 for negative numbers
  and -0.0).  Eight bits make a byte, the first value in the most significant
  bit; a partial last byte is padded with zero bits.  The byte stream is what
  LM-GC serialises.

This module is only for tests, the smoke check and the CPU baseline.
"""
from typing import Tuple

import numpy as np

from synth.configs import parse_lossy


def keep_count(n: int, percent: int) -> int:
    """Number of values sparsification keeps."""
    return n * percent // 100


def magnitude_key(v: np.ndarray) -> np.ndarray:
    """IEEE bits with the sign cleared, as unsigned integers."""
    return np.ascontiguousarray(v, np.float32).view(np.uint32) & np.uint32(0x7FFFFFFF)


def sparsify_topk(v: np.ndarray, k: int) -> np.ndarray:
    """Keep the k largest-magnitude values (ties: lower index first), zero the rest."""
    v = np.ascontiguousarray(v, np.float32)
    n = v.size
    k = max(0, min(int(k), n))
    key = magnitude_key(v).astype(np.int64)
    order = np.lexsort((np.arange(n), -key))       # by key descending, then index
    out = np.zeros(n, np.float32)
    keep = order[:k]
    out[keep] = v[keep]
    return out


def quantize_linear(v: np.ndarray, bits: int) -> Tuple[np.ndarray, float, float]:
    """Eq. 4: indices of n-bit linear quantisation, and the (min, max) it used."""
    if not 1 <= bits <= 16:
        raise ValueError("bits must be in [1, 16]")
    v = np.ascontiguousarray(v, np.float32)
    dtype = np.uint8 if bits <= 8 else np.uint16
    if v.size == 0:
        return np.zeros(0, dtype), 0.0, 0.0
    mn = np.float32(v.min())
    mx = np.float32(v.max())
    if not (np.isfinite(mn) and np.isfinite(mx)):
        raise ValueError("vector holds a NaN or an infinity")
    if mx == mn:
        return np.zeros(v.size, dtype), float(mn), float(mx)
    levels = np.float32((1 << bits) - 1)
    t = (v - mn) / np.float32(mx - mn)        # float32 arrays: one rounding per op
    q = np.rint(t * levels)                   # round half to even
    return q.astype(dtype), float(mn), float(mx)


def sign_pack(v: np.ndarray) -> np.ndarray:
    """SignSGD bits, eight per byte, first value in the most significant bit."""
    bits = (np.ascontiguousarray(v, np.float32).view(np.uint32) >> np.uint32(31)).astype(np.uint8)
    return np.packbits(bits, bitorder="big")


def prepare(values: np.ndarray, spec: str) -> np.ndarray:
    """Apply a lossy spec ('sparsify:10+quantize:8', 'sign', ...) left to right."""
    x = np.ascontiguousarray(values, np.float32)
    for kind, arg in parse_lossy(spec):
        if kind == "sparsify":
            x = sparsify_topk(x, keep_count(x.size, arg))
        elif kind == "quantize":
            x = quantize_linear(x, arg)[0]
        else:
            x = sign_pack(x)
    return x
