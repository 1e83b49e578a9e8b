"""Host-side checks of liblmgc that need no GPU: the library loads and exports
every entry point of include/lmgc.h; its manifest, token counts, arithmetic
coder, deserialiser and container parser agree with the oracle."""
import dataclasses
import os
import re

import numpy as np
import pytest

from oracle import coder as ocoder
from oracle import pipeline as opipe
from paper_2409_17836_amd import binding as B
from synth import WORKLOADS, weight_manifest
from synth.configs import hex_serial

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "lmgc.h")


def test_library_exports_every_declared_symbol():
    text = open(HEADER).read()
    declared = set(re.findall(r"\b(lmgc_[a-z0-9_]+)\s*\(", text))
    assert len(declared) >= 20
    L = B.lib()
    missing = [s for s in sorted(declared) if not hasattr(L, s)]
    assert not missing, missing


def test_timing_kinds_mask():
    """lmgc_timing_kinds takes a mask of kernel kinds; an empty one is an error."""
    B.timing_kinds(["gemm_up"])
    B.timing_kinds(None)
    assert B.lib().lmgc_timing_kinds(0) == -1  # LMGC_EINVAL
    assert B.lib().lmgc_timing_kinds(1 << 31) == -1  # no valid kind
    assert b"no valid kind" in B.lib().lmgc_last_error()


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_manifest_matches_generator(name):
    w = WORKLOADS[name]
    got = B.manifest(B.model_config(w.model))
    want = [(n, tuple(s)) for n, s in weight_manifest(w.model)]
    assert got == want


@pytest.mark.parametrize("bpv,bpg", [(4, 4), (4, 0), (4, 1), (4, 3), (1, 1), (2, 2)])
@pytest.mark.parametrize("n", [0, 1, 7, 1000, 2 * (1 << 20)])
def test_token_and_window_counts(bpv, bpg, n):
    sp = B.serial_params(hex_serial(window=4096, bos_id=1, bytes_per_value=bpv, bytes_per_group=bpg))
    nt = ocoder.num_tokens(n, bpv, bpg)
    assert B.num_tokens(n, sp) == nt
    assert B.num_windows(n, sp) == -(-nt // 4096)


def _tables(rng, n, T, skew):
    p = rng.dirichlet(np.full(18, skew), n)
    f = np.maximum(1, np.floor(p * (T - 18))).astype(np.int64)
    f[:, 17] += T - f.sum(1)
    cdf = np.zeros((n, 19), np.uint32)
    cdf[:, 1:] = np.cumsum(f, 1)
    sym = np.array([rng.choice(17, p=fr[:17] / fr[:17].sum()) for fr in f], np.uint8)
    return cdf, sym


@pytest.mark.parametrize("T", [1 << 16, 1 << 24])
@pytest.mark.parametrize("skew", [0.05, 1.0])
def test_library_coder_is_byte_identical_to_oracle(T, skew):
    rng = np.random.default_rng(int(T) % 997 + int(skew * 10))
    W = 300
    n_win = 9
    cdf = np.zeros((n_win, W, 19), np.uint32)
    sym = np.zeros((n_win, W), np.uint8)
    lens = np.array([W, W, 1, 0, 17, W, 250, W, 2], np.int32)
    for w in range(n_win):
        cdf[w], sym[w] = _tables(rng, W, T, skew)
    payload, bits = B.encode(cdf, sym, lens)
    off = 0
    for w in range(n_win):
        ref, nb = ocoder.ac_encode(cdf[w, :lens[w]], sym[w, :lens[w]])
        assert bits[w] == nb
        assert payload[off:off + len(ref)] == ref
        off += len(ref)
        # the library's step decoder reads the oracle's stream back
        dec = B.StepDecoder(ref, nb)
        got = [dec.decode(cdf[w, j]) for j in range(lens[w])]
        assert got == list(sym[w, :lens[w]])
    assert off == len(payload)


def test_library_coder_paper_example_and_uniform():
    cdf = np.array([[[0, 4, 5]] * 4], np.uint32)
    payload, bits = B.encode(cdf, np.array([[0, 0, 0, 1]], np.uint8), np.array([4], np.int32))
    assert bits[0] == 4 and payload == bytes([0b01110000])
    row = np.arange(17, dtype=np.uint32) * 4096
    sym = np.random.default_rng(0).integers(0, 16, (1, 1000)).astype(np.uint8)
    _, bits = B.encode(np.tile(row, (1, 1000, 1)), sym, np.array([1000], np.int32))
    assert bits[0] == 4 * 1000 + 2


def test_library_coder_rejects_zero_frequency():
    cdf = np.array([[[0, 5, 5, 10]]], np.uint32)
    with pytest.raises(B.LMGCError) as e:
        B.encode(cdf, np.array([[1]], np.uint8), np.array([1], np.int32))
    assert e.value.code == -5


@pytest.mark.parametrize("bpv,bpg,msb", [(4, 4, 1), (4, 4, 0), (4, 0, 1), (4, 3, 1), (1, 1, 1)])
def test_library_deserialize_matches_oracle(bpv, bpg, msb):
    rng = np.random.default_rng(bpv * 10 + bpg + msb)
    dt = {1: np.uint8, 4: np.float32}[bpv]
    vals = rng.integers(0, 256, 501 * bpv, dtype=np.uint8).view(dt)
    _, sym = ocoder.serialize(vals, bpv, bpg, msb, list(range(48, 64)), 32)
    sp = B.serial_params(hex_serial(window=64, bos_id=1, bytes_per_value=bpv, bytes_per_group=bpg,
                                    msb_first=msb))
    back = B.deserialize(sym, vals.size, sp, dt)
    assert back.tobytes() == vals.tobytes()
    if bpg:
        bad = sym.copy()
        bad[2 * bpg] = 3                 # digit where a separator belongs
        with pytest.raises(B.LMGCError) as e:
            B.deserialize(bad, vals.size, sp, dt)
        assert e.value.code == -5


@pytest.mark.parametrize("bpv,bpg,msb", [(4, 4, 1), (4, 4, 0), (4, 3, 1), (1, 1, 1), (2, 8, 1)])
def test_library_two_token_separator_matches_oracle(bpv, bpg, msb):
    """H_c+s (Sec. 5.2): token counts, alphabet size and deserialisation."""
    rng = np.random.default_rng(7 * bpv + bpg + msb)
    dt = {1: np.uint8, 2: np.uint16, 4: np.float32}[bpv]
    vals = rng.integers(0, 256, 333 * bpv, dtype=np.uint8).view(dt)
    hex_ids = list(range(48, 64))
    _, sym = ocoder.serialize(vals, bpv, bpg, msb, hex_ids, 44, 32)
    sp = B.serial_params(hex_serial(window=64, bos_id=1, bytes_per_value=bpv, bytes_per_group=bpg,
                                    msb_first=msb, sep_id=44, sep2_id=32))
    assert B.alphabet_size(sp) == 18
    for n in (0, 1, 5, vals.size):
        assert B.num_tokens(n, sp) == ocoder.num_tokens(n, bpv, bpg, 2)
    assert B.deserialize(sym, vals.size, sp, dt).tobytes() == vals.tobytes()
    bad = sym.copy()
    bad[2 * bpg], bad[2 * bpg + 1] = bad[2 * bpg + 1], bad[2 * bpg]     # ", " -> " ,"
    with pytest.raises(B.LMGCError) as e:
        B.deserialize(bad, vals.size, sp, dt)
    assert e.value.code == -5


def test_library_serial_params_validation():
    assert B.alphabet_size(B.serial_params(hex_serial(window=8, bos_id=1))) == 17
    for sep, sep2 in ((44, 44), (44, 48), (44, -2), (48, -1)):   # repeats, digit ids, bad id
        sp = B.serial_params(hex_serial(window=8, bos_id=1, sep_id=sep, sep2_id=sep2))
        with pytest.raises(B.LMGCError) as e:
            B.alphabet_size(sp)
        assert e.value.code == -1


def test_library_reads_two_token_separator_container():
    ser = hex_serial(window=8, bos_id=1, sep_id=44, sep2_id=32)
    buf = opipe.pack_container(ser, 3, 5, 1 << 16, [7, 9, 1, 2], [b"\x01", b"\x02\x03", b"\x04", b"\x05"])
    assert buf[27] == 19 and int.from_bytes(buf[116:120], "little") == 33
    assert B.container_info(buf) == dict(n_values=3, bytes_per_value=4, n_windows=4, model_tag=5)
    bad = bytearray(buf)
    bad[27] = 18                     # bin count of a one-token alphabet with a second id
    with pytest.raises(B.LMGCError):
        B.container_info(bytes(bad))


def test_library_renorm_flag():
    """Table mode: validated in the parameters, stored at header offset 120."""
    sp = B.serial_params(hex_serial(window=8, bos_id=1))
    sp.renorm = 2
    with pytest.raises(B.LMGCError) as e:
        B.alphabet_size(sp)
    assert e.value.code == -1
    ser = dataclasses.replace(hex_serial(window=8, bos_id=1), renorm=1)
    buf = opipe.pack_container(ser, 2, 1, 1 << 16, [3, 4, 5], [b"\x01", b"\x02", b"\x03"])
    assert int.from_bytes(buf[120:124], "little") == 1
    assert B.container_info(buf)["n_windows"] == 3
    bad = bytearray(buf)
    bad[120] = 2
    with pytest.raises(B.LMGCError) as e:
        B.container_info(bytes(bad))
    assert e.value.code == -5


def test_container_info_and_corruption():
    ser = hex_serial(window=8, bos_id=1)
    bits = [13, 20, 5]
    buf = opipe.pack_container(ser, 2, 99, 1 << 16, bits, [b"\x01\x02", b"\x03\x04\x05", b"\x06"])
    info = B.container_info(buf)
    assert info == dict(n_values=2, bytes_per_value=4, n_windows=3, model_tag=99)
    with pytest.raises(B.LMGCError):
        B.container_info(b"XXXX" + buf[4:])
    with pytest.raises(B.LMGCError):
        B.container_info(buf[:100])
