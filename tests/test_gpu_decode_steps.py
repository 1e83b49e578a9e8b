"""The decoder's path: lmgc_probs_stepwise computes the tables one position at
a time through the per-layer K/V cache, exactly as lmgc_decode does.  Lossless
decoding needs these tables to equal the encoder's (lmgc_probs on whole
windows) bit for bit, so that is what is checked here, for every decoder
shape and a ragged window; the full round trips through lmgc_decode are in
test_gpu_codec.py and test_gpu_probs_large.py."""
import dataclasses

import numpy as np
import pytest

from gpu_util import build_model, log
from paper_2409_17836_amd import binding as B
from synth import get_workload
from synth.gen import gen_values, workload_values

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _compare(w, model, n_win, W=None, values=None):
    import torch
    serial = w.serial if W is None else dataclasses.replace(w.serial, window=W)
    sp = B.serial_params(serial)
    vals = workload_values(w) if values is None else values
    tok, _ = B.serialize(torch.from_numpy(vals).cuda(), sp, 0, n_win)
    log(f"{w.name}: lmgc_probs B={n_win} W={serial.window}")
    cdf, logp = B.probs(model, tok, sp)
    log(f"{w.name}: lmgc_probs_stepwise ({serial.window} steps)")
    cdf2, logp2 = B.probs_stepwise(model, tok, sp)
    torch.cuda.synchronize()
    a, b = cdf.cpu().numpy(), cdf2.cpu().numpy()
    la, lb = logp.cpu().numpy(), logp2.cpu().numpy()
    bad = np.argwhere(np.any(a != b, axis=-1))
    assert bad.size == 0, f"tables differ at (window, position) {bad[:5].tolist()}"
    assert np.array_equal(la.view(np.uint32), lb.view(np.uint32))


def test_tiny_float32_whole_windows():
    w = get_workload("tiny")
    model, _ = build_model(w.model, 5, "perturbed", keep_host=False)
    _compare(w, model, 16)
    model.close()


def test_gpt2_layernorm_bias_gelu_and_ragged_window():
    w = get_workload("gpt2")
    model, _ = build_model(w.model, w.weight_seed, "perturbed", keep_host=False)
    _compare(w, model, 3, W=1024)
    # W = 200: the last key tile of each query block is ragged
    _compare(w, model, 5, W=200, values=gen_values(w.dist, 1000, 7))
    model.close()


def test_tinyllama_gqa():
    w = get_workload("tinyllama")
    model, _ = build_model(w.model, w.weight_seed, "paper", keep_host=False)
    _compare(w, model, 4, W=320)
    # 21 windows: the decoding step's one-row kernels take two 16-row blocks,
    # the second partly filled
    _compare(w, model, 21, W=64)
    model.close()


def test_7b_shape_several_key_tiles():
    w = get_workload("7b")
    model, _ = build_model(w.model, w.weight_seed, "paper", keep_host=False)
    _compare(w, model, 2, W=256)
    # the largest decoding group: 32 windows, two full 16-row blocks
    _compare(w, model, 32, W=128)
    model.close()


def test_gpt2_group_of_17():
    """GELU and the bias epilogues with a second row block of one window."""
    w = get_workload("gpt2")
    model, _ = build_model(w.model, w.weight_seed, "perturbed", keep_host=False)
    _compare(w, model, 17, W=136, values=gen_values(w.dist, 700, 9))
    model.close()


def test_stepwise_group_limit():
    """At most 32 windows per decoding step: the workspace helper gives 0
    above that and lmgc_probs_stepwise rejects the call before any GPU work."""
    import torch
    w = get_workload("tiny")
    model, _ = build_model(w.model, 5, "perturbed", keep_host=False)
    assert model.step_workspace(32, 64) > 0
    assert model.step_workspace(33, 64) == 0
    sp = B.serial_params(w.serial)
    tok = torch.ones((33, 64), dtype=torch.int32, device="cuda")
    with pytest.raises(B.LMGCError):
        B.probs_stepwise(model, tok, sp, ws=B.workspace(1 << 20, tok.device))
    model.close()
