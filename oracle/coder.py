"""ctypes wrapper of the reference coder in coder.c -- TEST INFRASTRUCTURE ONLY.

Serialisation (Sec. 4, "Serialization"), probability-table quantisation
(Sec. 4, "Compression": P_AC = P_LM) and the arithmetic coder (Sec. 3,
"Arithmetic coding").  See coder.c for the readings taken where the paper is
silent.
"""
import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "coder.c")
_LIB_PATH = os.path.join(_HERE, "_coder.so")

NALPHA = 17  # alphabet with a one-token separator (18 with two)
NSYM = 18

_lib = None


def build(force: bool = False) -> str:
    """Compile coder.c with gcc (plain -O2, no FP contraction)."""
    if force or not os.path.exists(_LIB_PATH) or \
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-ffp-contract=off",
                               "-fPIC", "-shared", _SRC, "-lm", "-o", tmp])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB_PATH)
        i64, i32, u32, u64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64
        vp = ctypes.c_void_p
        L.orc_num_tokens.restype = i64
        L.orc_num_tokens.argtypes = [i64, i32, i32, i32]
        L.orc_serialize.restype = i64
        L.orc_serialize.argtypes = [vp, i64, i32, i32, i32, vp, i32, i32, vp, vp]
        L.orc_deserialize.restype = ctypes.c_int
        L.orc_deserialize.argtypes = [vp, i64, i64, i32, i32, i32, i32, vp]
        L.orc_hex_roundtrip_range.restype = i64
        L.orc_hex_roundtrip_range.argtypes = [u64, u64, i32]
        L.orc_quantize_rows.restype = None
        L.orc_quantize_rows.argtypes = [vp, i64, i32, i32, u32, vp]
        L.orc_ac_encode.restype = i64
        L.orc_ac_encode.argtypes = [vp, i32, vp, i64, vp, u64]
        L.orc_decoder_size.restype = ctypes.c_size_t
        L.orc_ac_decode_init.restype = None
        L.orc_ac_decode_init.argtypes = [vp, vp, u64]
        L.orc_ac_decode_symbol.restype = ctypes.c_int
        L.orc_ac_decode_symbol.argtypes = [vp, vp, i32]
        L.orc_ac_decode.restype = None
        L.orc_ac_decode.argtypes = [vp, i32, i64, vp, u64, vp]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ------------------------------------------------------------ serialisation --
def num_tokens(n_values: int, bytes_per_value: int, bytes_per_group: int, nsep: int = 1) -> int:
    return int(lib().orc_num_tokens(n_values, bytes_per_value, bytes_per_group, nsep))


def serialize(values: np.ndarray, bytes_per_value: int, bytes_per_group: int,
              msb_first: int, hex_ids, sep_id: int, sep2_id: int = -1):
    """values: float32 (bpv=4) or uint8 (bpv=1) vector -> (tokens int32, bins uint8).
    sep2_id >= 0 adds a second separator token (bin 17) after each group."""
    v = np.ascontiguousarray(values)
    assert v.dtype.itemsize == bytes_per_value
    n = v.size
    nt = num_tokens(n, bytes_per_value, bytes_per_group, 2 if sep2_id >= 0 else 1)
    tok = np.empty(nt, np.int32)
    sym = np.empty(nt, np.uint8)
    ids = np.ascontiguousarray(hex_ids, dtype=np.int32)
    assert ids.size == 16
    got = lib().orc_serialize(_p(v), n, bytes_per_value, bytes_per_group,
                              msb_first, _p(ids), sep_id, sep2_id, _p(tok), _p(sym))
    assert got == nt
    return tok, sym


def deserialize(sym: np.ndarray, n_values: int, bytes_per_value: int,
                bytes_per_group: int, msb_first: int, dtype, nsep: int = 1) -> np.ndarray:
    """Inverse on coder bins; raises ValueError on a malformed stream."""
    s = np.ascontiguousarray(sym, dtype=np.uint8)
    out = np.empty(n_values * bytes_per_value, np.uint8)
    rc = lib().orc_deserialize(_p(s), s.size, n_values, bytes_per_value,
                               bytes_per_group, msb_first, nsep, _p(out))
    if rc != 0:
        raise ValueError("malformed token stream")
    return out.view(dtype)


def hex_roundtrip_all(msb_first: int = 1, threads: int = None) -> int:
    """Round-trip all 2^32 float32 bit patterns; returns the mismatch count."""
    L = lib()
    threads = threads or max(1, min(16, os.cpu_count() or 1))
    parts = 64
    step = (1 << 32) // parts

    def run(i):
        return int(L.orc_hex_roundtrip_range(i * step, (i + 1) * step, msb_first))

    with ThreadPoolExecutor(threads) as ex:
        return sum(ex.map(run, range(parts)))


# -------------------------------------------------------------- quantiser --
def quantize(lp: np.ndarray, total: int = 1 << 16, renorm: bool = False) -> np.ndarray:
    """lp [..., A] float32 log-probs of the A alphabet symbols (17, or 18 with
    a two-token separator) -> cdf [..., A + 2] uint32.  renorm: lp is
    normalised over the alphabet and the escape bin is empty."""
    a = np.ascontiguousarray(lp, dtype=np.float32)
    na = a.shape[-1]
    assert na in (17, 18)
    rows = a.size // na
    out = np.empty(a.shape[:-1] + (na + 2,), np.uint32)
    lib().orc_quantize_rows(_p(a), rows, na, 1 if renorm else 0, total, _p(out))
    return out


# ----------------------------------------------------------------- coder --
def ac_encode(cdf: np.ndarray, sym: np.ndarray):
    """cdf [n, nsym+1] uint32, sym [n] uint8 -> (payload bytes, nbits)."""
    c = np.ascontiguousarray(cdf, dtype=np.uint32)
    s = np.ascontiguousarray(sym, dtype=np.uint8)
    n = s.size
    nsym = c.shape[-1] - 1
    assert c.shape[0] == n
    cap = 64 + n * 8
    out = np.zeros(cap, np.uint8)
    nbits = lib().orc_ac_encode(_p(c), nsym, _p(s), n, _p(out), cap)
    if nbits == -2:
        raise ValueError("symbol with zero frequency or out of range")
    if nbits < 0:
        raise RuntimeError("encoder buffer too small")
    return out[: (nbits + 7) // 8].tobytes(), int(nbits)


def ac_decode(cdf: np.ndarray, payload: bytes, nbits: int) -> np.ndarray:
    c = np.ascontiguousarray(cdf, dtype=np.uint32)
    n = c.shape[0]
    nsym = c.shape[-1] - 1
    buf = np.frombuffer(payload, np.uint8).copy() if len(payload) else np.zeros(1, np.uint8)
    out = np.empty(n, np.uint8)
    lib().orc_ac_decode(_p(c), nsym, n, _p(buf), nbits, _p(out))
    return out


class StepDecoder:
    """Symbol-at-a-time decoder (the model row for the next symbol is only
    known after the previous symbols are decoded)."""

    def __init__(self, payload: bytes, nbits: int):
        L = lib()
        self._buf = np.frombuffer(payload, np.uint8).copy() if len(payload) else np.zeros(1, np.uint8)
        self._st = ctypes.create_string_buffer(L.orc_decoder_size())
        L.orc_ac_decode_init(self._st, _p(self._buf), nbits)

    def decode(self, cdf_row: np.ndarray) -> int:
        c = np.ascontiguousarray(cdf_row, dtype=np.uint32)
        return int(lib().orc_ac_decode_symbol(self._st, _p(c), c.size - 1))
