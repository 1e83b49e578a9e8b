"""Pins of the oracle's decoder forward pass: a scalar brute-force evaluation
written independently (plain Python floats, math.fsum, complex rotations),
library cross-checks (torch float64), closed-form special cases and
invariants."""
import cmath
import math

import numpy as np
import pytest
import torch

from oracle import forward as F
from synth import ModelShape, f32_to_bf16_bits
from synth.gen import gen_weights

MINI_LLAMA = ModelShape(arch="llama", dtype="f32", n_layers=2, d_model=16, n_heads=4,
                        n_kv_heads=2, d_ff=24, vocab=40, max_pos=16)
MINI_GPT2 = ModelShape(arch="gpt2", dtype="f32", n_layers=2, d_model=16, n_heads=2,
                       n_kv_heads=2, d_ff=32, vocab=40, max_pos=16)


def _bf16(x):
    """Library rounding: float32 -> torch.bfloat16 (round to nearest even)."""
    return float(torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64))


# ------------------------------------------------------------ brute force --
class Brute:
    """Scalar evaluation of the decoder equations, one position at a time."""

    def __init__(self, shape, weights):
        self.m = shape
        self.W = {k: F.storage_to_f64(v, shape.dtype).tolist() for k, v in weights.items()}
        self.rnd = (_bf16 if shape.dtype == "bf16" else (lambda x: x))

    def mv(self, name, a, bias=None):
        Wt = self.W[name]
        out = [math.fsum(Wt[o][i] * a[i] for i in range(len(a))) for o in range(len(Wt))]
        if bias is not None:
            out = [o + b for o, b in zip(out, self.W[bias])]
        return out

    def rms(self, h, g):
        r = 1.0 / math.sqrt(math.fsum(x * x for x in h) / len(h) + self.m.norm_eps)
        return [self.rnd(x * r * gi) for x, gi in zip(h, self.W[g])]

    def ln(self, h, g, b):
        mu = math.fsum(h) / len(h)
        var = math.fsum((x - mu) ** 2 for x in h) / len(h)
        r = 1.0 / math.sqrt(var + self.m.norm_eps)
        return [self.rnd((x - mu) * r * gi + bi) for x, gi, bi in zip(h, self.W[g], self.W[b])]

    def rot(self, vec, pos):
        hd = len(vec)
        half = hd // 2
        out = [0.0] * hd
        for i in range(half):
            z = complex(vec[i], vec[i + half]) * cmath.exp(
                1j * pos * self.m.rope_theta ** (-2.0 * i / hd))
            out[i], out[i + half] = z.real, z.imag
        return out

    def logprobs(self, x):
        m = self.m
        n, d, hd = len(x), m.d_model, m.head_dim
        H, Hkv = m.n_heads, m.n_kv_heads
        llama = m.arch == "llama"
        hs = []
        for j in range(n):
            if llama:
                hs.append(list(self.W["tok_emb"][x[j]]))
            else:
                hs.append([a + b for a, b in zip(self.W["wte"][x[j]], self.W["wpe"][j])])
        for l in range(m.n_layers):
            p = f"l{l}."
            Q, K, V = [], [], []
            for j in range(n):
                if llama:
                    a = self.rms(hs[j], p + "attn_norm")
                    q, k, v = self.mv(p + "wq", a), self.mv(p + "wk", a), self.mv(p + "wv", a)
                    q = sum((self.rot(q[h * hd:(h + 1) * hd], j) for h in range(H)), [])
                    k = sum((self.rot(k[h * hd:(h + 1) * hd], j) for h in range(Hkv)), [])
                else:
                    a = self.ln(hs[j], p + "ln1_g", p + "ln1_b")
                    qkv = self.mv(p + "w_qkv", a, p + "b_qkv")
                    q, k, v = qkv[:d], qkv[d:2 * d], qkv[2 * d:]
                Q.append([self.rnd(t) for t in q])
                K.append([self.rnd(t) for t in k])
                V.append([self.rnd(t) for t in v])
            for j in range(n):
                o = []
                for h in range(H):
                    g = h * Hkv // H
                    qs = Q[j][h * hd:(h + 1) * hd]
                    s = [math.fsum(qs[i] * K[t][g * hd + i] for i in range(hd)) / math.sqrt(hd)
                         for t in range(j + 1)]
                    mx = max(s)
                    e = [math.exp(si - mx) for si in s]
                    z = math.fsum(e)
                    o += [self.rnd(math.fsum(e[t] * V[t][g * hd + i] for t in range(j + 1)) / z)
                          for i in range(hd)]
                if llama:
                    hs[j] = [a + b for a, b in zip(hs[j], self.mv(p + "wo", o))]
                    b = self.rms(hs[j], p + "ffn_norm")
                    gt, up = self.mv(p + "w_gate", b), self.mv(p + "w_up", b)
                    # silu(g) = g * sigmoid(g), sigmoid written through tanh
                    act = [self.rnd(gi * 0.5 * (1.0 + math.tanh(gi / 2.0)) * ui)
                           for gi, ui in zip(gt, up)]
                    hs[j] = [a + b for a, b in zip(hs[j], self.mv(p + "w_down", act))]
                else:
                    hs[j] = [a + b for a, b in zip(hs[j], self.mv(p + "w_o", o, p + "b_o"))]
                    c = self.ln(hs[j], p + "ln2_g", p + "ln2_b")
                    f = self.mv(p + "w_fc", c, p + "b_fc")
                    k0 = math.sqrt(2.0 / math.pi)
                    f = [self.rnd(0.5 * u * (1.0 + math.tanh(k0 * (u + 0.044715 * u * u * u))))
                         for u in f]
                    hs[j] = [a + b for a, b in zip(hs[j], self.mv(p + "w_proj", f, p + "b_proj"))]
        out = []
        for j in range(n):
            if llama:
                hf = self.rms(hs[j], "final_norm")
                z = self.mv("lm_head", hf)
            else:
                hf = self.ln(hs[j], "lnf_g", "lnf_b")
                z = self.mv("wte", hf)
            mx = max(z)
            lse = mx + math.log(math.fsum(math.exp(t - mx) for t in z))
            out.append([t - lse for t in z])
        return np.array(out)


@pytest.mark.parametrize("shape", [MINI_LLAMA, MINI_GPT2,
                                   MINI_LLAMA.__class__(**{**MINI_LLAMA.__dict__, "dtype": "bf16"}),
                                   MINI_GPT2.__class__(**{**MINI_GPT2.__dict__, "dtype": "bf16"})],
                         ids=["llama-f32", "gpt2-f32", "llama-bf16", "gpt2-bf16"])
def test_forward_matches_brute_force(shape):
    w = gen_weights(shape, seed=3, init="perturbed")
    x = np.random.default_rng(4).integers(0, shape.vocab, 7)
    model = F.Model(shape, w)
    lp = F.logprobs_from_logits(model.logits(x), np.arange(shape.vocab))
    ref = Brute(shape, w).logprobs(list(x))
    np.testing.assert_allclose(lp, ref, rtol=0, atol=1e-9)


# ------------------------------------------------------- library routines --
def test_round_bf16_matches_library_and_bit_rounding():
    rng = np.random.default_rng(0)
    x = (rng.normal(0, 1, 20000) * np.exp(np.clip(rng.normal(0, 8, 20000), -60, 60))).astype(np.float32)
    # exact ties: low 16 bits = 0x8000, both parities of the kept bit
    ties = (rng.integers(0, 1 << 6, 2000, dtype=np.uint32) << 17 | 0x3F000000 | 0x8000
            | (rng.integers(0, 2, 2000, dtype=np.uint32) << 16)).view(np.float32)
    x = np.concatenate([x, ties])
    ours = F.round_bf16(x.astype(np.float64))
    lib = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    bits = (f32_to_bf16_bits(x).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert (ours == lib).all()
    assert (ours == bits).all()


def test_norms_and_activations_match_torch():
    rng = np.random.default_rng(1)
    h = rng.normal(0, 3, (5, 64))
    g = rng.normal(1, 0.1, 64)
    b = rng.normal(0, 0.1, 64)
    th = torch.from_numpy(h)
    np.testing.assert_allclose(F.layer_norm(h, g, b, 1e-5),
                               torch.nn.functional.layer_norm(th, (64,), torch.from_numpy(g),
                                                              torch.from_numpy(b), 1e-5).numpy(),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(F.rms_norm(h, g, 1e-5),
                               torch.nn.functional.rms_norm(th, (64,), torch.from_numpy(g),
                                                            1e-5).numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(F.silu(h), torch.nn.functional.silu(th).numpy(), rtol=1e-12,
                               atol=1e-14)
    np.testing.assert_allclose(F.gelu_tanh(h),
                               torch.nn.functional.gelu(th, approximate="tanh").numpy(),
                               rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("hq,hkv", [(4, 4), (8, 2), (6, 1)])
def test_causal_attention_matches_sdpa(hq, hkv):
    rng = np.random.default_rng(2)
    n, hd = 33, 16
    q, k, v = rng.normal(size=(n, hq, hd)), rng.normal(size=(n, hkv, hd)), rng.normal(size=(n, hkv, hd))
    ours = F.causal_attention(q, k, v).reshape(n, hq, hd)
    rep = hq // hkv
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(rep, 0)
    tv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(rep, 0)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    np.testing.assert_allclose(ours, ref.permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-12)


# ----------------------------------------------------- closed-form cases --
def test_rope_identity_at_zero_and_relative_position():
    rng = np.random.default_rng(3)
    q, k = rng.normal(size=(1, 1, 64)), rng.normal(size=(1, 1, 64))
    np.testing.assert_array_equal(F.rope(q, np.array([0]), 1e4), q)
    dots = []
    for m, n in ((5, 2), (13, 10), (103, 100)):           # same m - n
        a = F.rope(q, np.array([m]), 1e4)[0, 0]
        b = F.rope(k, np.array([n]), 1e4)[0, 0]
        dots.append(a @ b)
    np.testing.assert_allclose(dots, dots[0], rtol=1e-10)
    # rotation keeps the norm of every pair
    r = F.rope(q, np.array([77]), 1e4)[0, 0]
    np.testing.assert_allclose(r[:32] ** 2 + r[32:] ** 2, q[0, 0, :32] ** 2 + q[0, 0, 32:] ** 2)


def test_first_position_attends_only_to_itself():
    rng = np.random.default_rng(4)
    q, k, v = rng.normal(size=(3, 2, 8)), rng.normal(size=(3, 2, 8)), rng.normal(size=(3, 2, 8))
    o = F.causal_attention(q, k, v).reshape(3, 2, 8)
    np.testing.assert_allclose(o[0], v[0], rtol=0, atol=1e-15)


@pytest.mark.parametrize("shape", [MINI_LLAMA, MINI_GPT2])
def test_zero_head_gives_uniform_distribution(shape):
    w = gen_weights(shape, seed=5, init="perturbed")
    if shape.arch == "llama":
        w["lm_head"] = np.zeros_like(w["lm_head"])
    else:                                  # tied head: zero the final LayerNorm instead
        w["lnf_g"] = np.zeros_like(w["lnf_g"])
        w["lnf_b"] = np.zeros_like(w["lnf_b"])
    x = np.arange(9) % shape.vocab
    lp = F.Model(shape, w).alphabet_logprobs(x, [0, 5, 39])
    np.testing.assert_allclose(lp, -math.log(shape.vocab), rtol=0, atol=1e-13)


def test_probabilities_sum_to_one_and_prefix_invariance():
    w = gen_weights(MINI_LLAMA, seed=6, init="perturbed")
    model = F.Model(MINI_LLAMA, w)
    x = np.random.default_rng(6).integers(0, 40, 15)
    lp = F.logprobs_from_logits(model.logits(x), np.arange(40))
    np.testing.assert_allclose(np.exp(lp).sum(-1), 1.0, atol=1e-13)
    lp5 = F.logprobs_from_logits(model.logits(x[:5]), np.arange(40))
    np.testing.assert_allclose(lp5, lp[:5], rtol=0, atol=1e-12)


@pytest.mark.parametrize("shape", [MINI_LLAMA, MINI_GPT2])
def test_incremental_equals_full(shape):
    w = gen_weights(shape, seed=7, init="perturbed")
    model = F.Model(shape, w)
    rng = np.random.default_rng(7)
    x = rng.integers(0, shape.vocab, (3, 11))
    lm = F.IncrementalLM(model, 3, 11)
    inc = np.stack([lm.step(x[:, j]) for j in range(11)], 1)
    full = np.stack([model.logits(x[b]) for b in range(3)])
    np.testing.assert_allclose(inc, full, rtol=0, atol=1e-11)


@pytest.mark.parametrize("shape", [MINI_LLAMA, MINI_GPT2])
def test_batched_windows_equal_single_windows(shape):
    w = gen_weights(shape, seed=8, init="perturbed")
    model = F.Model(shape, w)
    x = np.random.default_rng(8).integers(0, shape.vocab, (3, 9))
    batched = model.logits(x)
    for b in range(3):
        np.testing.assert_allclose(batched[b], model.logits(x[b]), rtol=0, atol=1e-12)


def test_renormalised_logprobs_identities():
    """Restricting to the alphabet and renormalising: lp_renorm = lp_full -
    log sum_alphabet exp(lp_full); the renormalised probabilities sum to one;
    with every vocabulary id as the alphabet the two modes agree."""
    from oracle.forward import logprobs_from_logits
    rng = np.random.default_rng(2)
    z = rng.normal(0, 2.0, (5, 7, 40))
    ids = [3, 0, 39, 17, 8, 21]
    full = logprobs_from_logits(z, ids)
    ren = logprobs_from_logits(z, ids, renorm=True)
    np.testing.assert_allclose(ren, full - np.log(np.exp(full).sum(-1, keepdims=True)), atol=1e-12)
    np.testing.assert_allclose(np.exp(ren).sum(-1), 1.0, atol=1e-12)
    every = list(range(40))
    np.testing.assert_allclose(logprobs_from_logits(z, every, renorm=True), logprobs_from_logits(z, every),
                               atol=1e-12)
