"""lmgc_probs vs the oracle on the tiny float32 decoder (the whole workload)
and the GPT-2-small-shape bf16 decoder (its 32-window launch, two windows
checked at every position), plus the determinism and invariance properties
lossless decoding depends on."""
import numpy as np
import pytest

from gpu_util import build_model, log
from oracle import coder as ocoder
from oracle import pipeline as opipe
from oracle.forward import Model as OModel
from paper_2409_17836_amd import binding as B
from synth import get_workload
from synth.gen import workload_values

pytestmark = pytest.mark.gpu


def _tokens_for(w, vals, n_win):
    """GPU-serialised windows [n_win, W] (product path) and the oracle's own
    serialised stream for the same values."""
    import torch
    sp = B.serial_params(w.serial)
    tok, _ = B.serialize(torch.from_numpy(vals).cuda(), sp, 0, n_win)
    otok, _ = opipe.serialize(vals, w.serial)
    return sp, tok, otok


@pytest.fixture(scope="module")
def tiny():
    w = get_workload("tiny")
    model, host = build_model(w.model, w.weight_seed, "paper")
    return w, model, OModel(w.model, host)


@pytest.fixture(scope="module")
def tiny_perturbed():
    w = get_workload("tiny")
    model, host = build_model(w.model, 5, "perturbed")
    return w, model, OModel(w.model, host)


@pytest.mark.parametrize("which", ["paper", "perturbed"])
def test_tiny_whole_workload_logprobs(which, tiny, tiny_perturbed):
    """All 144 windows x 256 positions, float32 path: |lp - oracle| <= 1e-4."""
    import torch
    w, model, om = tiny if which == "paper" else tiny_perturbed
    vals = workload_values(w)
    sp, tok, otok = _tokens_for(w, vals, 144)
    cdf, logp = B.probs(model, tok, sp)
    torch.cuda.synchronize()
    lp = logp.cpu().numpy()
    W = w.serial.window
    X = np.stack([opipe.model_input(otok[s:s + n], w.serial) for s, n in opipe.windows(otok.size, W)])
    ref = om.alphabet_logprobs(X, opipe.alphabet_ids(w.serial))
    err = np.abs(lp - ref).max()
    log(f"tiny {which}: max |lp - oracle| = {err:.3g}")
    assert err <= 1e-4
    # tables: the oracle's quantiser applied to the GPU log-probs, bit for bit
    assert np.array_equal(cdf.cpu().numpy().view(np.uint32), ocoder.quantize(lp))


def test_tiny_two_token_separator_tables(tiny_perturbed):
    """H_c+s: 18 alphabet log-probs and 20-entry tables per position."""
    import dataclasses
    import torch
    w, model, om = tiny_perturbed
    ser = dataclasses.replace(w.serial, sep_id=44, sep2_id=32)
    vals = workload_values(w)[:400]                 # 15 windows (stepwise: B <= 32)
    sp = B.serial_params(ser)
    nw = B.num_windows(vals.size, sp)
    tok, _ = B.serialize(torch.from_numpy(vals).cuda(), sp, 0, nw)
    cdf, logp = B.probs(model, tok, sp)
    torch.cuda.synchronize()
    assert tuple(cdf.shape) == (nw, ser.window, 20) and tuple(logp.shape) == (nw, ser.window, 18)
    lp = logp.cpu().numpy()
    otok, _ = opipe.serialize(vals, ser)
    X = np.stack([opipe.model_input(otok[s:s + n], ser, ser.window)
                  for s, n in opipe.windows(otok.size, ser.window)])
    ref = om.alphabet_logprobs(X, opipe.alphabet_ids(ser))
    err = np.abs(lp - ref).max()
    log(f"tiny H_c+s: max |lp - oracle| = {err:.3g}")
    assert err <= 1e-4
    assert np.array_equal(cdf.cpu().numpy().view(np.uint32), ocoder.quantize(lp))
    cdf2, logp2 = B.probs_stepwise(model, tok, sp)
    assert np.array_equal(cdf2.cpu().numpy(), cdf.cpu().numpy())
    assert np.array_equal(logp2.cpu().numpy().view(np.uint32), lp.view(np.uint32))


@pytest.fixture(scope="module")
def gpt2():
    w = get_workload("gpt2")
    model, host = build_model(w.model, w.weight_seed, "perturbed")
    return w, model, OModel(w.model, host)


def test_gpt2_launch_config_logprobs(gpt2):
    """The benchmark launch (32 windows x 1024 tokens); windows 0 and 17
    compared with the oracle at every position (bf16: |lp - oracle| <= 2e-2)."""
    import torch
    w, model, om = gpt2
    vals = workload_values(w)
    sp, tok, otok = _tokens_for(w, vals, 32)
    cdf, logp = B.probs(model, tok, sp)
    torch.cuda.synchronize()
    lp = logp.cpu().numpy()
    W = w.serial.window
    X = np.stack([opipe.model_input(otok[s * W:(s + 1) * W], w.serial) for s in (0, 17)])
    ref = om.alphabet_logprobs(X, opipe.alphabet_ids(w.serial))
    err = np.abs(lp[[0, 17]] - ref).max()
    log(f"gpt2: max |lp - oracle| = {err:.3g}, mean {np.abs(lp[[0, 17]] - ref).mean():.3g}")
    assert err <= 2e-2
    assert np.array_equal(cdf.cpu().numpy().view(np.uint32), ocoder.quantize(lp))


@pytest.mark.parametrize("which", ["tiny", "gpt2"])
def test_renormalised_tables(which, tiny_perturbed, gpt2):
    """Tables renormalised over the alphabet (only the A alphabet columns of
    the LM head): log-probs vs the oracle (1e-4 float32, 2e-2 bf16), tables
    equal to the oracle's quantiser bit for bit, escape bin empty, and the
    decoder's stepwise tables equal to the encoder's."""
    import dataclasses
    import torch
    w, model, om = tiny_perturbed if which == "tiny" else gpt2
    ser = dataclasses.replace(w.serial, renorm=1)
    n_val = 400 if which == "tiny" else 230               # 15 windows / 3 windows
    vals = workload_values(w)[:n_val]
    sp = B.serial_params(ser)
    nw = B.num_windows(vals.size, sp)
    tok, _ = B.serialize(torch.from_numpy(vals).cuda(), sp, 0, nw)
    cdf, logp = B.probs(model, tok, sp)
    torch.cuda.synchronize()
    lp = logp.cpu().numpy()
    otok, _ = opipe.serialize(vals, ser)
    X = np.stack([opipe.model_input(otok[s:s + n], ser, ser.window)
                  for s, n in opipe.windows(otok.size, ser.window)])
    ref = om.alphabet_logprobs(X, opipe.alphabet_ids(ser), renorm=True)
    err = np.abs(lp - ref).max()
    log(f"{which} renormalised: max |lp - oracle| = {err:.3g}")
    assert err <= (1e-4 if which == "tiny" else 2e-2)
    c = cdf.cpu().numpy().view(np.uint32)
    assert np.array_equal(c, ocoder.quantize(lp, renorm=True))
    assert (c[..., -2] == 65536).all() and (c[..., -1] == 65536).all()
    cdf2, logp2 = B.probs_stepwise(model, tok, sp)
    assert np.array_equal(cdf2.cpu().numpy(), cdf.cpu().numpy())
    assert np.array_equal(logp2.cpu().numpy().view(np.uint32), lp.view(np.uint32))


def _invariance(model, sp, tok, W):
    """Bitwise: repeat, suffix change, batch composition, shorter window."""
    import torch
    c0, l0 = B.probs(model, tok, sp)
    c1, l1 = B.probs(model, tok, sp)
    torch.cuda.synchronize()
    assert torch.equal(c0, c1) and torch.equal(l0, l1), "not deterministic"
    # suffix: change every token after position j of every window
    j = W // 2 + 3
    t2 = tok.clone()
    g = torch.Generator(device="cpu").manual_seed(0)
    t2[:, j:] = torch.randint(48, 58, t2[:, j:].shape, generator=g).to(torch.int32).cuda()
    c2, l2 = B.probs(model, t2, sp)
    torch.cuda.synchronize()
    assert torch.equal(c2[:, :j + 1], c0[:, :j + 1]) and torch.equal(l2[:, :j + 1], l0[:, :j + 1])
    # batch: windows [2, 0] as a batch of two
    idx = torch.tensor([2, 0], device="cuda")
    c3, l3 = B.probs(model, tok[idx].contiguous(), sp)
    torch.cuda.synchronize()
    assert torch.equal(c3, c0[idx]) and torch.equal(l3, l0[idx]), "depends on batch composition"
    # window length: the first W/2 tokens as a window of W/2
    Wh = W // 2
    c4, l4 = B.probs(model, tok[:, :Wh].contiguous(), sp)
    torch.cuda.synchronize()
    assert torch.equal(c4, c0[:, :Wh]) and torch.equal(l4, l0[:, :Wh]), "depends on W"


def test_tiny_invariances(tiny_perturbed):
    w, model, _ = tiny_perturbed
    vals = workload_values(w)
    sp, tok, _ = _tokens_for(w, vals, 6)
    _invariance(model, sp, tok, w.serial.window)


def test_gpt2_invariances(gpt2):
    w, model, _ = gpt2
    vals = workload_values(w)
    sp, tok, _ = _tokens_for(w, vals, 5)
    _invariance(model, sp, tok, w.serial.window)
