"""Reference LM-GC codec -- TEST INFRASTRUCTURE ONLY.

Serialise -> cut into windows -> per window: BOS-shifted model input,
per-position log-probabilities of the alphabet symbols, integer tables,
arithmetic coding -> container.  Decompression mirrors it token by token
(Sec. 4, "Compression").

Windowing reading: the serialised stream is cut into consecutive windows of
W tokens (the last one shorter); window w's model input is BOS followed by
its first W-1 tokens, so position j predicts token j from BOS and tokens
0..j-1 (Eq. 2); BOS itself is never coded.  Positions restart at 0 in every
window.
"""
import struct
from typing import List, Tuple

import numpy as np

from . import coder
from .forward import IncrementalLM, Model

MAGIC = b"LMGC"
VERSION = 1
HEADER_BYTES = 128
DEFAULT_TOTAL = 1 << 16


def _sep2(serial) -> int:
    return int(getattr(serial, "sep2_id", -1))


def _renorm(serial) -> bool:
    """Tables of the LM's distribution renormalised over the alphabet (no
    escape mass) instead of the full-vocabulary distribution."""
    return bool(getattr(serial, "renorm", 0))


def alphabet_ids(serial) -> List[int]:
    """Token ids of the coder bins before the escape: the 16 hex digits, the
    separator, and the second separator token if there is one (H_c+s)."""
    ids = list(serial.hex_ids) + [serial.sep_id]
    if _sep2(serial) >= 0:
        ids.append(_sep2(serial))
    return ids


def serialize(values: np.ndarray, serial):
    return coder.serialize(values, serial.bytes_per_value, serial.bytes_per_group,
                           serial.msb_first, serial.hex_ids, serial.sep_id, _sep2(serial))


def windows(n_tokens: int, W: int) -> List[Tuple[int, int]]:
    """(start, length) of each window of the stream."""
    return [(s, min(W, n_tokens - s)) for s in range(0, n_tokens, W)]


def model_input(tok_window: np.ndarray, serial, length: int = None) -> np.ndarray:
    """BOS followed by the window's tokens, shifted by one (Eq. 2)."""
    n = tok_window.size if length is None else length
    x = np.full(n, serial.pad_id, np.int64)
    if n:
        x[0] = serial.bos_id
        k = min(n - 1, tok_window.size)
        x[1:1 + k] = tok_window[:k]
    return x


def window_logprobs(model: Model, tok_window: np.ndarray, serial, n_pos: int = None) -> np.ndarray:
    """[n_pos, A] log-probs of the alphabet at positions 0..n_pos-1."""
    n = tok_window.size if n_pos is None else n_pos
    return model.alphabet_logprobs(model_input(tok_window, serial, n), alphabet_ids(serial),
                                   _renorm(serial))


# ---------------------------------------------------------------- container --
def pack_container(serial, n_values: int, model_tag: int, total: int,
                   bits: List[int], payloads: List[bytes]) -> bytes:
    nsym = len(alphabet_ids(serial)) + 1
    hdr = struct.pack("<4sHHQQBBBBIII", MAGIC, VERSION, HEADER_BYTES, model_tag,
                      n_values, serial.bytes_per_value, serial.bytes_per_group,
                      serial.msb_first, nsym, serial.window, total, len(bits))
    hdr += struct.pack("<iii16iII", serial.bos_id, serial.pad_id, serial.sep_id,
                       *serial.hex_ids, _sep2(serial) + 1, int(_renorm(serial)))
    hdr += b"\0" * (HEADER_BYTES - len(hdr))
    assert len(hdr) == HEADER_BYTES
    return hdr + struct.pack(f"<{len(bits)}I", *bits) + b"".join(payloads)


def unpack_container(buf: bytes):
    if len(buf) < HEADER_BYTES or buf[:4] != MAGIC:
        raise ValueError("not an LM-GC container")
    (magic, ver, hbytes, tag, n_values, bpv, bpg, msb, nsym, W, total,
     nwin) = struct.unpack_from("<4sHHQQBBBBIII", buf, 0)
    ids = struct.unpack_from("<iii16iII", buf, 40)
    sep2 = ids[19] - 1
    if ids[20] > 1:
        raise ValueError("unsupported container")
    if ver != VERSION or hbytes != HEADER_BYTES or nsym != (19 if sep2 >= 0 else 18):
        raise ValueError("unsupported container")
    off = HEADER_BYTES
    if len(buf) < off + 4 * nwin:
        raise ValueError("truncated container")
    bits = list(struct.unpack_from(f"<{nwin}I", buf, off))
    off += 4 * nwin
    payloads = []
    for b in bits:
        nb = (b + 7) // 8
        if off + nb > len(buf):
            raise ValueError("truncated container")
        payloads.append(buf[off:off + nb])
        off += nb
    meta = dict(model_tag=tag, n_values=n_values, bytes_per_value=bpv,
                bytes_per_group=bpg, msb_first=msb, window=W, total=total,
                bos_id=ids[0], pad_id=ids[1], sep_id=ids[2], hex_ids=ids[3:19], sep2_id=sep2,
                renorm=bool(ids[20]))
    return meta, bits, payloads


# -------------------------------------------------------------------- codec --
def compress(values: np.ndarray, serial, model: Model, model_tag: int = 0,
             total: int = DEFAULT_TOTAL, incremental: bool = False) -> bytes:
    """Compress a vector.  incremental=True evaluates the model token by token
    (the same path decompress() takes); otherwise one full pass per window."""
    tok, sym = serialize(values, serial)
    wins = windows(tok.size, serial.window)
    if incremental:
        lp_rows = _incremental_logprobs(model, tok, wins, serial)
    elif wins:
        # all windows in one batched pass; positions past a window's end hold
        # pad tokens and, by causality, do not change the positions before it
        nmax = max(n for _, n in wins)
        X = np.stack([model_input(tok[s:s + n], serial, nmax) for s, n in wins])
        lp = model.alphabet_logprobs(X, alphabet_ids(serial), _renorm(serial))
        lp_rows = [lp[w, :n] for w, (_, n) in enumerate(wins)]
    else:
        lp_rows = []
    bits, payloads = [], []
    for (s, n), lp in zip(wins, lp_rows):
        cdf = coder.quantize(lp.astype(np.float32), total, _renorm(serial))
        pay, nb = coder.ac_encode(cdf, sym[s:s + n])
        bits.append(nb)
        payloads.append(pay)
    return pack_container(serial, values.size, model_tag, total, bits, payloads)


def _incremental_logprobs(model, tok, wins, serial):
    ids = alphabet_ids(serial)
    nb = len(wins)
    nmax = max(n for _, n in wins)
    lm = IncrementalLM(model, nb, nmax)
    toks = np.full((nb, nmax), serial.pad_id, np.int64)
    for w, (s, n) in enumerate(wins):
        toks[w, :n] = tok[s:s + n]
    out = np.empty((nb, nmax, len(ids)))
    x = np.full(nb, serial.bos_id, np.int64)
    from .forward import logprobs_from_logits
    for j in range(nmax):
        out[:, j] = logprobs_from_logits(lm.step(x), ids, _renorm(serial))
        x = toks[:, j]
    return [out[w, :n] for w, (_, n) in enumerate(wins)]


def decompress(buf: bytes, serial, model: Model, dtype) -> np.ndarray:
    """Token-by-token decoding from BOS, all windows in lockstep."""
    from .forward import logprobs_from_logits
    meta, bits, payloads = unpack_container(buf)
    total = meta["total"]
    W = meta["window"]
    n_values = meta["n_values"]
    nsep = 2 if meta["sep2_id"] >= 0 else 1
    n_tokens = coder.num_tokens(n_values, meta["bytes_per_value"], meta["bytes_per_group"], nsep)
    wins = windows(n_tokens, W)
    if len(wins) != len(bits):
        raise ValueError("window count mismatch")
    ids = alphabet_ids(serial)
    nb = len(wins)
    nmax = max((n for _, n in wins), default=0)
    decs = [coder.StepDecoder(p, b) for p, b in zip(payloads, bits)]
    lm = IncrementalLM(model, nb, nmax)
    sym = np.zeros(n_tokens, np.uint8)
    x = np.full(nb, serial.bos_id, np.int64)
    id_of = np.array(ids, np.int64)
    for j in range(nmax):
        lp = logprobs_from_logits(lm.step(x), ids, meta["renorm"]).astype(np.float32)
        cdf = coder.quantize(lp, total, meta["renorm"])
        nxt = np.full(nb, serial.pad_id, np.int64)
        for w, (s, n) in enumerate(wins):
            if j < n:
                b = decs[w].decode(cdf[w])
                if b >= len(ids):
                    raise ValueError("escape symbol decoded: corrupt stream")
                sym[s + j] = b
                nxt[w] = id_of[b]
        x = nxt
    return coder.deserialize(sym, n_values, meta["bytes_per_value"],
                             meta["bytes_per_group"], meta["msb_first"], dtype, nsep)
