"""Reference decoder forward pass -- TEST INFRASTRUCTURE ONLY.

Plain NumPy float64 evaluation of p(t_k | BOS, t_<k) (Eq. 2) for the decoder
shapes LM-GC uses as priors.  Matrix products use np.matmul; everything else
is written out.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may use this module.

Model definition (the paper only names the LLMs, Sec. 5.1; these are the
standard LLaMA and GPT-2 block equations):

  LLaMA:  h = E[x]
          per layer:  a = RMSNorm(h) * g1
                      q, k, v = a Wq^T, a Wk^T, a Wv^T; RoPE on q, k
                      h = h + Attn(q, k, v) Wo^T
                      b = RMSNorm(h) * g2
                      h = h + (silu(b Wg^T) * (b Wu^T)) Wd^T
          z = (RMSNorm(h) * gf) Wlm^T
  GPT-2:  h = wte[x] + wpe[pos]
          per layer:  a = LN(h; g1, b1)
                      q, k, v = split(a Wqkv^T + bqkv)
                      h = h + Attn(q, k, v) Wo^T + bo
                      c = LN(h; g2, b2)
                      h = h + gelu_tanh(c Wfc^T + bfc) Wproj^T + bproj
          z = LN(h; gf, bf) wte^T                      (tied head)
  Attn:   per query head, kv head = floor(head * Hkv / Hq); causal softmax of
          q.k / sqrt(head_dim).
  RoPE:   rotate-half pairs (i, i + hd/2), angle pos * theta^(-2i/hd).

Precision reading for bf16 models: weights are bf16 values; the operands of
every matrix product (normed activations, q/k/v after RoPE, attention output,
FFN activation, final normed state) are rounded to bf16; everything else
(residual stream, norms, the attention probabilities and their softmax,
logits) is exact float64 here.  f32 models use no rounding.
"""
from typing import Callable, Dict, Optional

import numpy as np


# ---------------------------------------------------------------- numerics --
def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits, ties to even), in float64."""
    m, e = np.frexp(x)
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


def _decode_chunk(w: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        assert w.dtype == np.uint16
        return (w.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return np.asarray(w, dtype=np.float32).astype(np.float64)


def storage_to_f64(w: np.ndarray, dtype: str) -> np.ndarray:
    """Decode stored parameters: bf16 bit patterns (uint16) or float32.
    Large tensors are decoded in row chunks on several threads."""
    if w.size < (1 << 22) or w.ndim < 2:
        return _decode_chunk(w, dtype)
    from concurrent.futures import ThreadPoolExecutor
    import os
    out = np.empty(w.shape, np.float64)
    step = max(1, w.shape[0] // 32)

    def run(r0):
        out[r0:r0 + step] = _decode_chunk(w[r0:r0 + step], dtype)

    with ThreadPoolExecutor(max(1, min(16, os.cpu_count() or 1))) as ex:
        list(ex.map(run, range(0, w.shape[0], step)))
    return out


def rms_norm(h, g, eps):
    ms = np.mean(h * h, axis=-1, keepdims=True)
    return h / np.sqrt(ms + eps) * g


def layer_norm(h, g, b, eps):
    mu = np.mean(h, axis=-1, keepdims=True)
    var = np.mean((h - mu) ** 2, axis=-1, keepdims=True)
    return (h - mu) / np.sqrt(var + eps) * g + b


def silu(z):
    return z / (1.0 + np.exp(-z))


def gelu_tanh(z):
    return 0.5 * z * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (z + 0.044715 * z ** 3)))


def rope(x, pos, theta):
    """x: [..., n, H, hd]; pos: [n] positions."""
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * np.arange(half) / hd)
    ang = pos[:, None].astype(np.float64) * inv[None, :]          # [n, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def causal_attention(q, k, v):
    """q: [n, Hq, hd], k/v: [n, Hkv, hd] -> [n, Hq*hd]."""
    n, hq, hd = q.shape
    hkv = k.shape[1]
    out = np.empty((n, hq, hd))
    mask = np.triu(np.ones((n, n), bool), 1)
    for h in range(hq):
        kv = (h * hkv) // hq
        s = (q[:, h, :] @ k[:, kv, :].T) / np.sqrt(hd)
        s = np.where(mask, -np.inf, s)
        s = s - s.max(axis=-1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=-1, keepdims=True)
        out[:, h, :] = p @ v[:, kv, :]
    return out.reshape(n, hq * hd)


# ------------------------------------------------------------------- model --
class Model:
    """Holds a decoder shape and its parameters (name -> stored array, or a
    callable name -> stored array for lazily generated large models).

    acc="f64" (the reference) evaluates everything in float64.  acc="f32"
    evaluates the same equations with the same bf16 rounding points but in
    float32 (the precision of the GPU's accumulators and residual stream);
    the gap between the two measures how far two correct evaluations of the
    same bf16 model drift apart through the network's depth."""

    def __init__(self, shape, weights, cache: Optional[bool] = None, acc: str = "f64"):
        self.m = shape
        self._get: Callable[[str], np.ndarray] = (weights.__getitem__
                                                  if isinstance(weights, dict) else weights)
        n_params = shape.vocab * shape.d_model * 2 + shape.n_layers * (
            4 * shape.d_model ** 2 + 3 * shape.d_model * shape.d_ff)
        self._cache_on = (n_params < 80_000_000) if cache is None else cache
        self._cache: Dict[str, np.ndarray] = {}
        self.acc = np.float64 if acc == "f64" else np.float32
        if shape.dtype == "bf16":
            self.rnd = (round_bf16 if acc == "f64"
                        else (lambda x: round_bf16(x).astype(np.float32)))
        else:
            self.rnd = (lambda x: x)

    def w(self, name: str) -> np.ndarray:
        if name in self._cache:
            return self._cache[name]
        x = storage_to_f64(self._get(name), self.m.dtype)
        if self.acc is not np.float64:
            x = x.astype(self.acc)
        if self._cache_on:
            self._cache[name] = x
        return x

    # -- one sequence, all positions --------------------------------------
    def final_hidden(self, x: np.ndarray) -> np.ndarray:
        """x: [n] (or [nb, n] independent windows) model input ids, BOS
        first -> bf16-rounded normed final state [..., n, d] that feeds the
        LM head."""
        m, rnd, w = self.m, self.rnd, self.w
        n = x.shape[-1]
        lead = x.shape[:-1]
        hd = m.head_dim
        pos = np.arange(n)

        def attend(q, k, v):
            if not lead:
                return causal_attention(q, k, v)
            return np.stack([causal_attention(q[i], k[i], v[i]) for i in range(q.shape[0])])
        if m.arch == "llama":
            h = w("tok_emb")[x]
            for l in range(m.n_layers):
                p = f"l{l}."
                a = rnd(rms_norm(h, w(p + "attn_norm"), m.norm_eps))
                q = (a @ w(p + "wq").T).reshape(*lead, n, m.n_heads, hd)
                k = (a @ w(p + "wk").T).reshape(*lead, n, m.n_kv_heads, hd)
                v = (a @ w(p + "wv").T).reshape(*lead, n, m.n_kv_heads, hd)
                q = rnd(rope(q, pos, m.rope_theta))
                k = rnd(rope(k, pos, m.rope_theta))
                v = rnd(v)
                o = rnd(attend(q, k, v))
                h = h + o @ w(p + "wo").T
                b = rnd(rms_norm(h, w(p + "ffn_norm"), m.norm_eps))
                act = rnd(silu(b @ w(p + "w_gate").T) * (b @ w(p + "w_up").T))
                h = h + act @ w(p + "w_down").T
            return rnd(rms_norm(h, w("final_norm"), m.norm_eps))
        if m.arch == "gpt2":
            d = m.d_model
            h = w("wte")[x] + w("wpe")[pos]
            for l in range(m.n_layers):
                p = f"l{l}."
                a = rnd(layer_norm(h, w(p + "ln1_g"), w(p + "ln1_b"), m.norm_eps))
                qkv = a @ w(p + "w_qkv").T + w(p + "b_qkv")
                q = rnd(qkv[..., :d]).reshape(*lead, n, m.n_heads, hd)
                k = rnd(qkv[..., d:2 * d]).reshape(*lead, n, m.n_heads, hd)
                v = rnd(qkv[..., 2 * d:]).reshape(*lead, n, m.n_heads, hd)
                o = rnd(attend(q, k, v))
                h = h + (o @ w(p + "w_o").T + w(p + "b_o"))
                c = rnd(layer_norm(h, w(p + "ln2_g"), w(p + "ln2_b"), m.norm_eps))
                f = rnd(gelu_tanh(c @ w(p + "w_fc").T + w(p + "b_fc")))
                h = h + (f @ w(p + "w_proj").T + w(p + "b_proj"))
            return rnd(layer_norm(h, w("lnf_g"), w("lnf_b"), m.norm_eps))
        raise ValueError(m.arch)

    def head_matrix(self) -> np.ndarray:
        return self.w("lm_head") if self.m.arch == "llama" else self.w("wte")

    def logits(self, x: np.ndarray) -> np.ndarray:
        """x: [..., n] -> logits [..., n, V]."""
        return self.final_hidden(x) @ self.head_matrix().T

    def alphabet_logprobs(self, x: np.ndarray, ids, renorm: bool = False) -> np.ndarray:
        """x: [..., n] -> [..., n, len(ids)] natural-log probabilities of the
        given ids, normalised over the whole vocabulary (Eq. 2), or over the
        given ids only (renorm)."""
        return logprobs_from_logits(self.logits(x), ids, renorm)


def logprobs_from_logits(z: np.ndarray, ids, renorm: bool = False) -> np.ndarray:
    """log softmax of the logits at ids; over the whole vocabulary, or, with
    renorm, over the ids alone (the distribution restricted to them)."""
    za = z[..., np.asarray(ids)]
    zn = za if renorm else z
    mx = zn.max(axis=-1, keepdims=True)
    lse = mx + np.log(np.sum(np.exp(zn - mx), axis=-1, keepdims=True))
    return za - lse


# ---------------------------------------------------- incremental (decode) --
class IncrementalLM:
    """Token-at-a-time evaluation with cached keys/values, batched over
    independent windows.  Used for both directions of the reference codec's
    own round trip, so that encoder and decoder compute every table with the
    same sequence of operations (Sec. 4: decompression starts from BOS and
    feeds each decoded token back)."""

    def __init__(self, model: Model, nb: int, n_max: int):
        self.M = model
        m = model.m
        self.nb = nb
        self.j = 0
        hd = m.head_dim
        self.kc = [np.zeros((nb, n_max, m.n_kv_heads, hd)) for _ in range(m.n_layers)]
        self.vc = [np.zeros((nb, n_max, m.n_kv_heads, hd)) for _ in range(m.n_layers)]

    def _attend(self, l, q, k, v):
        m = self.M.m
        j = self.j
        self.kc[l][:, j] = k
        self.vc[l][:, j] = v
        hd = m.head_dim
        out = np.empty((self.nb, m.n_heads, hd))
        for h in range(m.n_heads):
            kv = (h * m.n_kv_heads) // m.n_heads
            K = self.kc[l][:, : j + 1, kv, :]                     # [nb, j+1, hd]
            V = self.vc[l][:, : j + 1, kv, :]
            s = np.einsum("bd,btd->bt", q[:, h, :], K) / np.sqrt(hd)
            s = s - s.max(axis=-1, keepdims=True)
            p = np.exp(s)
            p = p / p.sum(axis=-1, keepdims=True)
            out[:, h, :] = np.einsum("bt,btd->bd", p, V)
        return out.reshape(self.nb, m.n_heads * hd)

    def step(self, x: np.ndarray) -> np.ndarray:
        """x: [nb] ids at position j -> logits [nb, V] for position j."""
        M, m = self.M, self.M.m
        rnd, w = M.rnd, M.w
        nb, hd = self.nb, m.head_dim
        pos = np.array([self.j])
        if m.arch == "llama":
            h = w("tok_emb")[x]
            for l in range(m.n_layers):
                p = f"l{l}."
                a = rnd(rms_norm(h, w(p + "attn_norm"), m.norm_eps))
                q = (a @ w(p + "wq").T).reshape(nb, 1, m.n_heads, hd)
                k = (a @ w(p + "wk").T).reshape(nb, 1, m.n_kv_heads, hd)
                v = (a @ w(p + "wv").T).reshape(nb, m.n_kv_heads, hd)
                q = rnd(rope(q, pos, m.rope_theta))[:, 0]
                k = rnd(rope(k, pos, m.rope_theta))[:, 0]
                o = rnd(self._attend(l, q, k, rnd(v)))
                h = h + o @ w(p + "wo").T
                b = rnd(rms_norm(h, w(p + "ffn_norm"), m.norm_eps))
                act = rnd(silu(b @ w(p + "w_gate").T) * (b @ w(p + "w_up").T))
                h = h + act @ w(p + "w_down").T
            hf = rnd(rms_norm(h, w("final_norm"), m.norm_eps))
        else:
            d = m.d_model
            h = w("wte")[x] + w("wpe")[self.j]
            for l in range(m.n_layers):
                p = f"l{l}."
                a = rnd(layer_norm(h, w(p + "ln1_g"), w(p + "ln1_b"), m.norm_eps))
                qkv = a @ w(p + "w_qkv").T + w(p + "b_qkv")
                q = rnd(qkv[:, :d]).reshape(nb, m.n_heads, hd)
                k = rnd(qkv[:, d:2 * d]).reshape(nb, m.n_heads, hd)
                v = rnd(qkv[:, 2 * d:]).reshape(nb, m.n_heads, hd)
                o = rnd(self._attend(l, q, k, v))
                h = h + (o @ w(p + "w_o").T + w(p + "b_o"))
                c = rnd(layer_norm(h, w(p + "ln2_g"), w(p + "ln2_b"), m.norm_eps))
                f = rnd(gelu_tanh(c @ w(p + "w_fc").T + w(p + "b_fc")))
                h = h + (f @ w(p + "w_proj").T + w(p + "b_proj"))
            hf = rnd(layer_norm(h, w("lnf_g"), w("lnf_b"), m.norm_eps))
        self.j += 1
        return hf @ M.head_matrix().T
