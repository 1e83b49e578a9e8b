"""lmgc_probs at the TinyLlama-1.1B and Llama-2-7B shapes (bf16, random
init): the benchmark launch configuration on the GPU, checked against the
oracle on sampled positions (window prefixes, which causality makes exact
sub-problems), plus determinism / prefix invariance at full size and a
lossless round trip of a short vector through the 7B-shape model.

Tolerance for these deep bf16 models: two correct evaluations of the same
bf16 model that differ only in accumulation precision (the oracle in float64
and in float32, identical bf16 rounding points) already disagree by more
than 2e-2 at 22-32 layers, because a one-ulp difference in where a value
rounds to bf16 is amplified with depth.  The test measures that floor on the
very positions it checks and requires the GPU to stay within twice it (and
within 2e-2 where the floor is lower), and the code length of the checked
positions to stay within 0.5% of the oracle's."""
import numpy as np
import pytest

from gpu_util import build_model, log
from oracle import coder as ocoder
from oracle import lossy as olossy
from oracle import pipeline as opipe
from oracle.forward import Model as OModel
from paper_2409_17836_amd import binding as B
from synth import get_workload, parse_lossy
from synth.configs import hex_serial
from synth.gen import gen_values, workload_values

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _parity(w, model, om, om32, n_win, check_windows, P):
    import torch
    vals = workload_values(w)
    sp = B.serial_params(w.serial)
    tok, _ = B.serialize(torch.from_numpy(vals).cuda(), sp, 0, n_win)
    log(f"{w.name}: probs B={n_win} W={w.serial.window}")
    cdf, logp = B.probs(model, tok, sp)
    torch.cuda.synchronize()
    lp = logp.cpu().numpy()
    otok, _ = opipe.serialize(vals, w.serial)
    W = w.serial.window
    X = np.stack([opipe.model_input(otok[c * W:(c + 1) * W], w.serial, P) for c in check_windows])
    ids = opipe.alphabet_ids(w.serial)
    log(f"{w.name}: oracle on windows {check_windows} x {P} positions")
    ref = om.alphabet_logprobs(X, ids)
    log(f"{w.name}: oracle (float32 accumulation) on the same positions")
    ref32 = om32.alphabet_logprobs(X, ids)
    floor = np.abs(ref32 - ref)
    d = np.abs(lp[check_windows, :P] - ref)
    log(f"{w.name}: max |lp - oracle| = {d.max():.3g}, mean {d.mean():.3g}; oracle f32-vs-f64 "
        f"floor max {floor.max():.3g}, mean {floor.mean():.3g}")
    assert d.max() <= max(2e-2, 2 * floor.max())
    assert d.mean() <= max(5e-3, 2 * floor.mean())
    gcdf = cdf.cpu().numpy().view(np.uint32)
    assert np.array_equal(gcdf, ocoder.quantize(lp))
    # code length of the checked positions with the GPU's and the oracle's tables
    _, osym = opipe.serialize(vals, w.serial)
    sym = np.stack([osym[c * W:c * W + P] for c in check_windows]).astype(np.int64)
    ocdf = ocoder.quantize(ref.astype(np.float32)).astype(np.int64)
    g = gcdf[check_windows, :P].astype(np.int64)
    take = lambda c, k: np.take_along_axis(c, k[..., None], -1)[..., 0]
    bits_gpu = -np.log2((take(g, sym + 1) - take(g, sym)) / 65536.0).sum()
    bits_ref = -np.log2((take(ocdf, sym + 1) - take(ocdf, sym)) / 65536.0).sum()
    log(f"{w.name}: code length of checked positions {bits_gpu:.1f} bits vs oracle {bits_ref:.1f}")
    assert abs(bits_gpu - bits_ref) <= 0.005 * bits_ref
    return sp, tok, cdf, logp


def test_tinyllama_launch_config():
    w = get_workload("tinyllama")
    log("tinyllama: building model")
    model, host = build_model(w.model, w.weight_seed, "perturbed")
    _parity(w, model, OModel(w.model, host), OModel(w.model, host, acc="f32"), 16, [0, 9], 96)
    model.close()


@pytest.fixture(scope="module")
def llama7b():
    w = get_workload("7b")
    log("7b: building model (6.7e9 parameters)")
    model, host = build_model(w.model, w.weight_seed, "paper")
    yield w, model, OModel(w.model, host), OModel(w.model, host, acc="f32")
    model.close()


def test_7b_launch_config_parity_and_invariance(llama7b):
    import torch
    w, model, om, om32 = llama7b
    sp, tok, cdf, logp = _parity(w, model, om, om32, w.batch, [0, 7], 12)
    # the same launch again is bitwise identical; a changed suffix leaves the
    # prefix bitwise identical
    j = 3000
    t2 = tok.clone()
    t2[:, j:] = 48
    c2, l2 = B.probs(model, t2, sp)
    c3, l3 = B.probs(model, tok, sp)
    torch.cuda.synchronize()
    assert torch.equal(c3, cdf) and torch.equal(l3, logp)
    assert torch.equal(c2[:, :j + 1], cdf[:, :j + 1]) and torch.equal(l2[:, :j + 1], logp[:, :j + 1])
    # probabilities of the 17 symbols can never exceed 1 in total
    tot = torch.exp(logp.double()).sum(-1)
    assert float(tot.max()) <= 1.0 + 1e-5


def test_7b_lossy_roundtrip_short(llama7b):
    """8-bit indices (2 hex digits + separator), short windows: compress with
    the library, decode token by token with the library, compare bytes."""
    import torch
    w, model, om, _ = llama7b
    spec = hex_serial(window=64, bos_id=1, bytes_per_value=1)
    raw = gen_values("normal:1e-3", 100, 3)                    # 300 tokens -> 5 windows
    dv = B.lossy_prepare(torch.from_numpy(raw).cuda(), parse_lossy("sparsify:10+quantize:8"))
    vals = olossy.prepare(raw, "sparsify:10+quantize:8")
    assert dv.cpu().numpy().tobytes() == vals.tobytes()
    sp = B.serial_params(spec)
    buf = B.compress(model, dv, sp, batch=4, model_tag=77)
    back = B.decode(model, buf, batch=4, model_tag=77, dtype=np.uint8)
    assert back.tobytes() == vals.tobytes()
    ref = opipe.compress(vals, spec, om, model_tag=77)
    log(f"7b lossy: {len(buf)} bytes vs oracle {len(ref)}")
    assert abs(len(buf) - len(ref)) <= 0.005 * len(ref)
