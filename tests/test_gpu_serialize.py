"""lmgc_serialize on the GPU vs the oracle's serialiser: bit-exact tokens and
coder bins, including window ranges, the padded last window, byte orders,
separator groupings and variants, 8-bit values and the full-size 7B-shape vector."""
import numpy as np
import pytest

from gpu_util import log
from oracle import coder as ocoder
from oracle import lossy as olossy
from paper_2409_17836_amd import binding as B
from synth import get_workload, parse_lossy
from synth.configs import SEPARATORS, hex_serial
from synth.gen import gen_values, workload_values

pytestmark = pytest.mark.gpu


def _check(vals, spec, first=0, count=None):
    import torch
    sp = B.serial_params(spec)
    dv = torch.from_numpy(vals).to("cuda")
    tok, sym = B.serialize(dv, sp, first, count)
    torch.cuda.synchronize()
    otok, osym = ocoder.serialize(vals, spec.bytes_per_value, spec.bytes_per_group, spec.msb_first,
                                  spec.hex_ids, spec.sep_id, spec.sep2_id)
    W = spec.window
    nw = tok.shape[0]
    ftok = np.full((first + nw) * W, spec.pad_id, np.int32)
    fsym = np.full((first + nw) * W, 255, np.uint8)
    n = min(otok.size, ftok.size)
    ftok[:n] = otok[:n]
    fsym[:n] = osym[:n]
    assert np.array_equal(tok.cpu().numpy().reshape(-1), ftok[first * W:])
    assert np.array_equal(sym.cpu().numpy().reshape(-1), fsym[first * W:])


@pytest.mark.parametrize("name", ["tiny", "gpt2", "7b"])
def test_serialize_workloads(name):
    w = get_workload(name)
    log(f"serialize {name}: {w.n_values} values")
    _check(workload_values(w), w.serial)


def test_serialize_lossy_workload():
    w = get_workload("lossy7b")
    vals = gen_values(w.dist, 1 << 20, w.value_seed)       # a 1M-value slice of the 8M vector
    import torch
    prepped = B.lossy_prepare(torch.from_numpy(vals).cuda(), parse_lossy(w.lossy))
    want = olossy.prepare(vals, w.lossy)
    got = prepped.cpu().numpy()
    assert got.tobytes() == want.tobytes()
    _check(want, w.serial)


@pytest.mark.parametrize("bpg", [0, 1, 2, 3, 4, 8])
@pytest.mark.parametrize("msb", [1, 0])
def test_serialize_groupings(bpg, msb):
    vals = gen_values("laplace:1e-3", 999, 4)
    spec = hex_serial(window=100, bos_id=1, bytes_per_group=bpg, msb_first=msb)
    _check(vals, spec)


def test_serialize_window_ranges_and_edges():
    vals = gen_values("normal:1e-3", 1000, 5)
    spec = hex_serial(window=64, bos_id=7)
    nw = -(-9000 // 64)
    _check(vals, spec, first=3, count=5)
    _check(vals, spec, first=nw - 1, count=1)              # ragged last window
    _check(vals[:1], spec)                                 # one value
    special = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, -3.4e38], np.float32)
    _check(special, spec)


@pytest.mark.parametrize("variant", sorted(SEPARATORS))
@pytest.mark.parametrize("bpv,bpg", [(4, 4), (4, 3), (1, 1), (2, 8)])
def test_serialize_separator_variants(variant, bpv, bpg):
    """Sec. 5.2 separators, H_c+s with two tokens per group (bins 16, 17)."""
    sep, sep2 = SEPARATORS[variant]
    n = 777
    raw = np.random.default_rng(bpg + 10 * bpv).integers(0, 256, n * bpv, dtype=np.uint8)
    vals = raw.view({1: np.uint8, 2: np.int16, 4: np.float32}[bpv])
    spec = hex_serial(window=96, bos_id=1, bytes_per_value=bpv, bytes_per_group=bpg,
                      sep_id=sep, sep2_id=sep2)
    _check(vals, spec)
    _check(vals, spec, first=2, count=3)
