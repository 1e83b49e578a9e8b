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


_C_SCALARS = {  # C type -> (size, signed, is_float)
    "int": (4, True, False), "int32_t": (4, True, False), "int64_t": (8, True, False),
    "uint32_t": (4, False, False), "uint64_t": (8, False, False), "size_t": (8, False, False),
    "float": (4, True, True), "double": (8, True, True), "uint8_t": (1, False, False),
    "uint16_t": (2, False, False), "char": (1, True, False), "void": (0, False, False),
}
_C_STRUCTS = {"lmgc_serial_params": "SerialParams", "lmgc_model_config": "ModelConfig",
              "lmgc_decoder": "DecoderState"}


def _prototypes(text):
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    text = re.sub(r"(?m)^\s*#.*$", " ", text)
    out = {}
    for m in re.finditer(r"([A-Za-z_][\w \t\*]*?)\b(lmgc_[a-z0-9_]+)\s*\(([^;{]*?)\)\s*;", text):
        ret, name, args = m.group(1), m.group(2), m.group(3).strip()
        params = [] if args in ("", "void") else [a.strip() for a in args.split(",")]
        out[name] = (ret.strip(), params)
    return out


def _ctype_of(decl):
    """(pointer depth, base type name) of a C parameter or return type."""
    decl = decl.replace("const", " ")
    depth = decl.count("*")
    words = decl.replace("*", " ").split()
    base = words[0]
    return depth, base


def _check_type(decl, ct, where):
    import ctypes
    depth, base = _ctype_of(decl)
    if depth == 0:
        size, signed, is_float = _C_SCALARS[base]
        if base == "void":
            assert ct is None, where
            return
        assert ct is not None and ctypes.sizeof(ct) == size, (where, decl, ct)
        if is_float:
            assert ct in (ctypes.c_float, ctypes.c_double), (where, decl, ct)
        else:
            assert ct not in (ctypes.c_float, ctypes.c_double), (where, decl, ct)
            signed_types = (ctypes.c_byte, ctypes.c_short, ctypes.c_int, ctypes.c_long,
                            ctypes.c_longlong)
            assert (ct in signed_types) == signed, (where, decl, ct)
        return
    # pointers: void* / char* / POINTER(T) with T matching the pointee
    if ct in (ctypes.c_void_p, ctypes.c_char_p):
        assert ct is ctypes.c_void_p or (base == "char" and depth == 1), (where, decl, ct)
        return
    assert hasattr(ct, "_type_") and issubclass(ct, ctypes._Pointer), (where, decl, ct)
    inner = ct._type_
    if depth == 1 and base in _C_STRUCTS:
        assert inner.__name__ == _C_STRUCTS[base], (where, decl, ct)
    elif depth == 1:
        _check_type(base, inner, where)
    else:  # T** (or T* const*): a pointer to pointers
        assert inner is ctypes.c_void_p, (where, decl, ct)


def test_binding_signatures_match_header():
    """Every entry point of include/lmgc.h is bound with the declared number of
    arguments, and each argument and result has the declared size, signedness
    and pointer-ness (a mismatch would pass garbage without any error)."""
    protos = _prototypes(open(HEADER).read())
    assert len(protos) >= 30
    L = B.lib()
    for name, (ret, params) in protos.items():
        f = getattr(L, name)
        assert f.argtypes is not None, name
        assert len(f.argtypes) == len(params), (name, params, f.argtypes)
        for i, (p, ct) in enumerate(zip(params, f.argtypes)):
            # drop the parameter name (the last word unless the type ends in '*');
            # an array parameter ("int64_t shape[2]") is a pointer
            if "[" in p:
                p = p[:p.index("[")].rsplit(None, 1)[0] + "*"
            decl = p if p.rstrip().endswith("*") else p.rsplit(None, 1)[0]
            if "*" in p and not decl.endswith("*"):
                decl = p[:p.rfind("*") + 1]
            _check_type(decl, ct, f"{name} arg {i}")
        _check_type(ret, f.restype, f"{name} result")


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


def test_size_limits_and_hostile_headers():
    """Vector sizes above LMGC_MAX_VALUES (2^56) are errors rather than int64
    overflow, and header fields that would overflow (a huge value count, a
    second-separator field of 2^31) are rejected as corrupt."""
    import struct
    sp = B.serial_params(hex_serial(window=4096, bos_id=1))
    L = B.lib()
    assert L.lmgc_num_tokens(1 << 56, sp) == 9 * (1 << 56)  # 8 digits + 1 separator
    assert L.lmgc_num_tokens((1 << 56) + 1, sp) < 0
    assert L.lmgc_num_tokens(-1, sp) < 0
    assert L.lmgc_num_windows((1 << 62), sp) < 0
    ser = hex_serial(window=8, bos_id=1)
    buf = bytearray(opipe.pack_container(ser, 2, 99, 1 << 16, [13, 20, 5],
                                         [b"\x01\x02", b"\x03\x04\x05", b"\x06"]))
    for off, val in [(16, 1 << 62), (16, (1 << 56) + 1), (16, (1 << 64) - 1)]:
        bad = bytearray(buf)
        struct.pack_into("<Q", bad, off, val)
        with pytest.raises(B.LMGCError) as e:
            B.container_info(bytes(bad))
        assert e.value.code == -5
    bad = bytearray(buf)
    struct.pack_into("<I", bad, 116, 1 << 31)  # sep2_id + 1 = 2^31
    with pytest.raises(B.LMGCError) as e:
        B.container_info(bytes(bad))
    assert e.value.code == -5


def test_host_allocation_failure_is_an_error_code():
    """A host allocation that cannot succeed (the encoder's scratch for 2^31
    windows of 2^20 tokens, about a petabyte, beyond the address space)
    comes back as LMGC_ENOMEM, not as an exception through the C ABI."""
    import ctypes
    cdf = np.zeros(19, np.uint32)
    sym = np.zeros(1, np.uint8)
    lens = np.zeros(1, np.int32)
    out = np.zeros(16, np.uint8)
    bits = np.zeros(1, np.uint32)
    used = ctypes.c_size_t()
    rc = B.lib().lmgc_encode(cdf.ctypes.data, 18, sym.ctypes.data, lens.ctypes.data, (1 << 31) - 1,
                             1 << 20, out.ctypes.data, out.size, bits.ctypes.data,
                             ctypes.byref(used), 1)
    assert rc == -2, rc  # LMGC_ENOMEM
    assert b"allocation" in B.lib().lmgc_last_error()


def test_keep_count_matches_oracle():
    """The Sec. 5.4 keep count is the library's arithmetic (the binding only
    forwards it); it equals the oracle's floor(n * percent / 100)."""
    from oracle import lossy as olossy
    for n in (0, 1, 7, 99, 100, 101, 1 << 23, (1 << 31) - 1):
        for pct in (0, 1, 10, 25, 33, 50, 99, 100):
            assert B.keep_count(n, pct) == olossy.keep_count(n, pct)
    for n, pct in ((-1, 10), (1 << 31, 10), (10, -1), (10, 101)):
        with pytest.raises(B.LMGCError):
            B.keep_count(n, pct)
