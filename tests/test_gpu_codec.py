"""The full codec through the C ABI: lmgc_compress (serialise -> LM tables ->
arithmetic coding, host coding overlapped with the GPU) and lmgc_decode
(token-by-token decoding from BOS), against the oracle's container size and
the original bytes."""
import numpy as np
import pytest

from gpu_util import build_model, log
from oracle import lossy as olossy
from oracle import pipeline as opipe
from oracle.forward import Model as OModel
from paper_2409_17836_amd import binding as B
from synth import get_workload
from synth import parse_lossy
from synth.configs import LOSSY_VARIANTS, SEPARATORS, hex_serial, lossy_bytes_per_value
from synth.gen import gen_values, workload_values

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]


def _roundtrip(model, om, vals, spec, batch, tag=5, dtype=np.float32):
    import torch
    sp = B.serial_params(spec)
    dv = torch.from_numpy(vals.view(np.int16) if vals.dtype == np.uint16 else vals).cuda()
    buf = B.compress(model, dv, sp, batch=batch, model_tag=tag)
    ref = opipe.compress(vals, spec, om, model_tag=tag)
    log(f"compressed {vals.nbytes} B -> {len(buf)} B (oracle {len(ref)} B)")
    assert abs(len(buf) - len(ref)) <= 0.005 * len(ref)
    back = B.decode(model, buf, batch=batch, model_tag=tag, dtype=dtype)
    assert back.tobytes() == vals.tobytes(), "not lossless"
    with pytest.raises(B.LMGCError):
        B.decode(model, buf, batch=batch, model_tag=tag + 1, dtype=dtype)
    return buf


def test_tiny_whole_workload_roundtrip():
    w = get_workload("tiny")
    model, host = build_model(w.model, w.weight_seed)
    vals = workload_values(w)
    _roundtrip(model, OModel(w.model, host), vals, w.serial, batch=48)
    model.close()


def test_tiny_empty_and_single_value():
    """Degenerate inputs: no values give a header-only container (no window,
    no model call) and one value gives one ragged window of 9 tokens. Both
    decode back; the headers equal the oracle's byte for byte and the sizes
    match it (one byte of slack for the float32 against float64 tables)."""
    import torch
    w = get_workload("tiny")
    model, host = build_model(w.model, w.weight_seed)
    om = OModel(w.model, host)
    spec = hex_serial(window=256, bos_id=1)
    sp = B.serial_params(spec)
    for n in (0, 1):
        vals = gen_values("laplace:1e-3", n, 3) if n else np.zeros(0, np.float32)
        log(f"{n} values")
        buf = B.compress(model, torch.from_numpy(vals).cuda(), sp, batch=4, model_tag=5)
        ref = opipe.compress(vals, spec, om, model_tag=5)
        assert buf[:B.HEADER_BYTES] == ref[:B.HEADER_BYTES]
        assert abs(len(buf) - len(ref)) <= (0 if n == 0 else 1), (len(buf), len(ref))
        assert B.container_info(buf)["n_windows"] == n
        back = B.decode(model, buf, batch=4, model_tag=5)
        assert back.size == n and back.tobytes() == vals.tobytes()
    model.close()


def _split_container(buf, n_windows):
    """(bit counts, payloads) of a container body holding n_windows windows."""
    bits = [int(b) for b in np.frombuffer(buf, np.uint32, n_windows, B.HEADER_BYTES)]
    off = B.HEADER_BYTES + 4 * n_windows
    pays = []
    for b in bits:
        pays.append(buf[off:off + (b + 7) // 8])
        off += (b + 7) // 8
    assert off == len(buf)
    return bits, pays


def test_window_ranges_code_like_the_whole_vector():
    """Coding a range of windows (the benchmark codes one batch of windows per
    step) gives each window the bits and payload it gets when the whole
    vector is coded, with another batch size; a range is not a whole-vector
    container, so decoding rejects it, and a range past the end is an error."""
    import torch
    w = get_workload("tiny")
    model, _ = build_model(w.model, w.weight_seed, keep_host=False)
    sp = B.serial_params(hex_serial(window=256, bos_id=1))
    vals = gen_values("laplace:1e-3", 200, 21)  # 1800 tokens: 7 full windows + 8 tokens
    dv = torch.from_numpy(vals).cuda()
    full = B.compress(model, dv, sp, batch=3, model_tag=5)
    nw = B.container_info(full)["n_windows"]
    assert nw == 8
    fbits, fpays = _split_container(full, nw)
    for a, n in [(0, 1), (1, 2), (3, nw - 3), (nw - 1, 1)]:
        log(f"windows [{a}, {a + n})")
        part = B.compress(model, dv, sp, batch=2, model_tag=5, first_window=a, n_windows=n)
        pbits, ppays = _split_container(part, n)
        assert pbits == fbits[a:a + n] and ppays == fpays[a:a + n]
        with pytest.raises(B.LMGCError):
            B.decode(model, part, batch=2, model_tag=5)
    with pytest.raises(B.LMGCError):
        B.compress(model, dv, sp, batch=2, first_window=nw - 1, n_windows=2)
    model.close()


def test_tiny_bytes_per_group_variants():
    w = get_workload("tiny")
    model, host = build_model(w.model, w.weight_seed)
    om = OModel(w.model, host)
    vals = gen_values("laplace:1e-3", 150, 8)
    for bpg in (0, 1, 2, 3, 8):
        _roundtrip(model, om, vals, hex_serial(window=256, bos_id=1, bytes_per_group=bpg), batch=4)
    model.close()


def test_tiny_separator_variants():
    """H_c, H_semi and H_c+s (Sec. 5.2); H_c+s codes 18 alphabet symbols."""
    w = get_workload("tiny")
    model, host = build_model(w.model, w.weight_seed)
    om = OModel(w.model, host)
    vals = gen_values("laplace:1e-3", 150, 9)
    for variant, (sep, sep2) in sorted(SEPARATORS.items()):
        log(f"separator variant {variant}")
        spec = hex_serial(window=256, bos_id=1, sep_id=sep, sep2_id=sep2)
        buf = _roundtrip(model, om, vals, spec, batch=4)
        assert buf[27] == (19 if sep2 >= 0 else 18)
    model.close()


@pytest.mark.parametrize("variant", ["q16", "sign", "s50", "s25"])
def test_tiny_lossy_variants(variant):
    """Sec. 5.4 streams prepared on the GPU: 16-bit indices (4 digits +
    separator), packed sign bytes, sparsified float32 at 50 and 25 percent."""
    import torch
    w = get_workload("tiny")
    model, host = build_model(w.model, w.weight_seed)
    om = OModel(w.model, host)
    lossy = LOSSY_VARIANTS[variant]
    raw = gen_values("laplace:1e-3", 400, 12)
    dv = B.lossy_prepare(torch.from_numpy(raw).cuda(), parse_lossy(lossy))
    vals = olossy.prepare(raw, lossy)
    got = dv.cpu().numpy()
    assert got.tobytes() == vals.tobytes()
    bpv = lossy_bytes_per_value(lossy)
    spec = hex_serial(window=256, bos_id=1, bytes_per_value=bpv)
    log(f"lossy variant {variant}: {vals.size} values of {bpv} bytes")
    _roundtrip(model, om, vals, spec, batch=8, dtype=vals.dtype)
    model.close()


def test_renormalised_tables_roundtrip():
    """Renormalised tables (no escape mass): tiny float32 and GPT-2 bf16."""
    import dataclasses
    w = get_workload("tiny")
    model, host = build_model(w.model, w.weight_seed)
    vals = gen_values("laplace:1e-3", 300, 13)
    spec = dataclasses.replace(w.serial, renorm=1)
    buf = _roundtrip(model, OModel(w.model, host), vals, spec, batch=8)
    assert int.from_bytes(buf[120:124], "little") == 1
    model.close()
    w = get_workload("gpt2")
    model, host = build_model(w.model, w.weight_seed, "perturbed")
    spec = dataclasses.replace(w.serial, renorm=1)
    _roundtrip(model, OModel(w.model, host), workload_values(w)[:250], spec, batch=2)
    model.close()


def test_gpt2_short_roundtrip():
    w = get_workload("gpt2")
    model, host = build_model(w.model, w.weight_seed, "perturbed")
    vals = workload_values(w)[:250]                          # 2250 tokens -> 3 windows
    _roundtrip(model, OModel(w.model, host), vals, w.serial, batch=2)
    model.close()


def test_tinyllama_short_roundtrip():
    w = get_workload("tinyllama")
    model, host = build_model(w.model, w.weight_seed)
    spec = hex_serial(window=128, bos_id=1)
    vals = workload_values(w)[:60]                           # 540 tokens -> 5 windows
    _roundtrip(model, OModel(w.model, host), vals, spec, batch=4)
    model.close()


def test_tinyllama_decode_groups_up_to_32():
    """lmgc_decode with groups of more than 16 windows per step (two 16-row
    MFMA blocks in the one-row kernels) on a bf16 model: 43 windows of 64
    tokens, decoded in groups of 32 + 11 and of 20 + 20 + 3, lossless."""
    import torch
    w = get_workload("tinyllama")
    model, _ = build_model(w.model, w.weight_seed, keep_host=False)
    spec = hex_serial(window=64, bos_id=1)
    vals = workload_values(w)[:300]                          # 2700 tokens -> 43 windows
    sp = B.serial_params(spec)
    assert B.num_windows(vals.size, sp) == 43
    buf = B.compress(model, torch.from_numpy(vals).cuda(), sp, batch=8, model_tag=9)
    for batch in (32, 20):
        log(f"tinyllama decode, batch {batch}")
        back = B.decode(model, buf, batch=batch, model_tag=9)
        assert back.tobytes() == vals.tobytes(), f"not lossless with batch {batch}"
    model.close()
