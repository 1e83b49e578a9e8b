"""End-to-end pins of the oracle codec and of the seeded input generators."""
import dataclasses
import math

import numpy as np
import pytest

from oracle import coder, lossy, pipeline
from oracle.forward import Model
from synth import get_workload
from synth.configs import LOSSY_VARIANTS, SEPARATORS, hex_serial, lossy_bytes_per_value
from synth.gen import gen_values, gen_weights, workload_values


@pytest.fixture(scope="module")
def tiny():
    w = get_workload("tiny")
    return w, Model(w.model, gen_weights(w.model, w.weight_seed)), workload_values(w)


def test_tiny_roundtrip_is_lossless(tiny):
    """The whole tiny workload: 4096 values, 36864 tokens, 144 windows."""
    w, model, vals = tiny
    buf = pipeline.compress(vals, w.serial, model, model_tag=7, incremental=True)
    meta, bits, payloads = pipeline.unpack_container(buf)
    assert meta["n_values"] == 4096 and len(bits) == 144 and meta["model_tag"] == 7
    back = pipeline.decompress(buf, w.serial, model, np.float32)
    assert back.tobytes() == vals.tobytes()
    # full-window evaluation gives (up to float64 rounding) the same tables
    buf2 = pipeline.compress(vals, w.serial, model, model_tag=7)
    assert abs(len(buf2) - len(buf)) <= 0.0005 * len(buf)


def test_code_length_matches_model_information(tiny):
    """Per window: H <= bits <= H + 2 where H = sum of -log2 f/T (Sec. 3)."""
    w, model, vals = tiny
    tok, sym = pipeline.serialize(vals[:300], w.serial)
    for s, n in pipeline.windows(tok.size, w.serial.window):
        lp = pipeline.window_logprobs(model, tok[s:s + n], w.serial).astype(np.float32)
        cdf = coder.quantize(lp)
        f = (cdf[np.arange(n), sym[s:s + n].astype(int) + 1].astype(np.int64)
             - cdf[np.arange(n), sym[s:s + n]].astype(np.int64))
        H = float(-np.sum(np.log2(f / 65536.0)))
        _, nbits = coder.ac_encode(cdf, sym[s:s + n])
        assert H - 1e-6 <= nbits <= H + 2 + 1e-6


def test_bos_shift_and_windows():
    ser = hex_serial(window=4, bos_id=1)
    tok = np.array([10, 11, 12, 13, 14, 15], np.int32)
    wins = pipeline.windows(tok.size, 4)
    assert wins == [(0, 4), (4, 2)]
    assert list(pipeline.model_input(tok[0:4], ser)) == [1, 10, 11, 12]
    assert list(pipeline.model_input(tok[4:6], ser)) == [1, 14]          # 2 positions
    assert list(pipeline.model_input(tok[4:6], ser, length=4)) == [1, 14, 15, 1]  # pad = BOS


def test_corrupt_container_is_rejected(tiny):
    w, model, vals = tiny
    v = vals[:40]
    buf = pipeline.compress(v, w.serial, model, incremental=True)
    with pytest.raises(ValueError):
        pipeline.unpack_container(buf[:-3])
    with pytest.raises(ValueError):
        pipeline.unpack_container(b"XXXX" + buf[4:])
    # flipping payload bits either raises or gives different values
    bad = bytearray(buf)
    bad[-5] ^= 0xFF
    try:
        out = pipeline.decompress(bytes(bad), w.serial, model, np.float32)
        assert out.tobytes() != v.tobytes()
    except ValueError:
        pass


@pytest.mark.parametrize("variant", sorted(LOSSY_VARIANTS))
def test_lossy_variant_roundtrip_small(variant):
    """Sec. 5.4 streams: 8-bit indices (2 digits + separator), 16-bit indices
    (4 digits + separator), packed sign bytes, sparsified float32."""
    w = get_workload("tiny")
    spec = LOSSY_VARIANTS[variant]
    bpv = lossy_bytes_per_value(spec)
    ser = hex_serial(window=64, bos_id=1, bytes_per_value=bpv)
    vals = lossy.prepare(gen_values("normal:1e-3", 160, seed=3), spec)
    model = Model(w.model, gen_weights(w.model, 1))
    buf = pipeline.compress(vals, ser, model, incremental=True)
    back = pipeline.decompress(buf, ser, model, vals.dtype)
    assert back.dtype == vals.dtype and back.tobytes() == vals.tobytes()


@pytest.mark.parametrize("variant", ["H_c", "H_semi", "H_c+s"])
def test_separator_variant_roundtrip(tiny, variant):
    """Sec. 5.2 serialisations: H_c+s codes two separator tokens per group with
    an 18-symbol alphabet (19 bins with the escape) and stores the second id in
    the container."""
    w, model, vals = tiny
    sep, sep2 = SEPARATORS[variant]
    ser = dataclasses.replace(w.serial, sep_id=sep, sep2_id=sep2)
    v = vals[:60]
    buf = pipeline.compress(v, ser, model, model_tag=3, incremental=True)
    meta, bits, _ = pipeline.unpack_container(buf)
    assert meta["sep_id"] == sep and meta["sep2_id"] == sep2
    nsep = 2 if sep2 >= 0 else 1
    assert buf[27] == 17 + nsep                            # coder bins incl. escape
    assert len(bits) == -(-(60 * (8 + nsep)) // ser.window)
    assert pipeline.decompress(buf, ser, model, np.float32).tobytes() == v.tobytes()
    # full-window tables give the same stream up to float64 rounding
    buf2 = pipeline.compress(v, ser, model, model_tag=3)
    assert abs(len(buf2) - len(buf)) <= max(2, 0.0005 * len(buf))


def test_renormalised_tables_roundtrip_and_gain(tiny):
    """Tables renormalised over the alphabet: lossless, recorded in the
    container, and shorter than the full-vocabulary tables (the tiny model
    puts about 239/256 of its mass outside the alphabet)."""
    w, model, vals = tiny
    v = vals[:60]
    ser = dataclasses.replace(w.serial, renorm=1)
    buf = pipeline.compress(v, ser, model, incremental=True)
    meta, _, _ = pipeline.unpack_container(buf)
    assert meta["renorm"] is True
    assert pipeline.decompress(buf, ser, model, np.float32).tobytes() == v.tobytes()
    full = pipeline.compress(v, w.serial, model, incremental=True)
    assert len(buf) < 0.7 * len(full)
    buf2 = pipeline.compress(v, ser, model)
    assert abs(len(buf2) - len(buf)) <= max(2, 0.0005 * len(buf))


# ------------------------------------------------------- input generators --
def test_value_distributions():
    x = gen_values("normal:1e-3", 200000, 0)
    assert x.dtype == np.float32 and abs(x.std() - 1e-3) < 2e-5
    x = gen_values("laplace:1e-3", 200000, 0)
    assert abs(np.mean(np.abs(x)) - 1e-3) < 2e-5           # E|x| = b
    x = gen_values("mixture:1e-4:0.01:1e-2", 400000, 0)
    frac_big = np.mean(np.abs(x) > 1e-3)                     # ~ 0.01 * P(|N(0,1e-2)| > 1e-3)
    assert abs(frac_big - 0.01 * math.erfc(0.1 / math.sqrt(2))) < 2e-3
    np.testing.assert_array_equal(gen_values("laplace:1e-3", 100, 5),
                                  gen_values("laplace:1e-3", 100, 5))
