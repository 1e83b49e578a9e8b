"""Seeded generators: gradient vectors and random-init decoder weights.

Everything here is deterministic in (workload, seed) and independent of the
number of threads used.  Normal samples come from NumPy's ziggurat
(`Generator.standard_normal`, float32), which is table/integer based and so
gives the same bits on every x86-64 host.
"""
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Iterator, List, Tuple

import numpy as np

from .configs import ModelShape, Workload

_CHUNK = 1 << 22


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


# ----------------------------------------------------------------- bfloat16 --
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bfloat16 (ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    t = u >> np.uint32(16)
    t &= np.uint32(1)
    t += np.uint32(0x7FFF)
    t += u
    t >>= np.uint32(16)
    return t.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# ------------------------------------------------------------ value vectors --
def gen_values(dist: str, n: int, seed: int = 0) -> np.ndarray:
    """Synthetic gradient vector.

    dist grammar:
      normal:<sigma>                 float32 N(0, sigma^2)
      laplace:<b>                    float32 Laplace(0, b)
      mixture:<s0>:<p>:<s1>          N(0,s0^2), replaced with prob p by N(0,s1^2)
    Samples are drawn in float64 from default_rng(seed) and cast to float32.
    Lossy workloads apply their sparsification/quantisation steps to this
    vector (Workload.lossy); those steps are not part of this module.
    """
    rng = np.random.default_rng(seed)
    kind, *args = dist.split(":")
    a = [float(x) for x in args]
    if kind == "normal":
        return rng.normal(0.0, a[0], n).astype(np.float32)
    if kind == "laplace":
        return rng.laplace(0.0, a[0], n).astype(np.float32)
    if kind == "mixture":
        base = rng.normal(0.0, a[0], n)
        mask = rng.random(n) < a[1]
        outl = rng.normal(0.0, a[2], n)
        return np.where(mask, outl, base).astype(np.float32)
    raise ValueError(f"unknown distribution {dist!r}")


def workload_values(w: Workload) -> np.ndarray:
    return gen_values(w.dist, w.n_values, w.value_seed)


# ------------------------------------------------------------------ weights --
def weight_manifest(m: ModelShape) -> List[Tuple[str, Tuple[int, ...]]]:
    """(name, shape) of every parameter in the order the C-ABI expects.
    Matrices are [out, in] (row n holds the weights of output feature n)."""
    d, hd, F, V = m.d_model, m.head_dim, m.d_ff, m.vocab
    out: List[Tuple[str, Tuple[int, ...]]] = []
    if m.arch == "llama":
        out.append(("tok_emb", (V, d)))
        for l in range(m.n_layers):
            p = f"l{l}."
            out += [(p + "attn_norm", (d,)),
                    (p + "wq", (m.n_heads * hd, d)),
                    (p + "wk", (m.n_kv_heads * hd, d)),
                    (p + "wv", (m.n_kv_heads * hd, d)),
                    (p + "wo", (d, m.n_heads * hd)),
                    (p + "ffn_norm", (d,)),
                    (p + "w_gate", (F, d)),
                    (p + "w_up", (F, d)),
                    (p + "w_down", (d, F))]
        out += [("final_norm", (d,)), ("lm_head", (V, d))]
    elif m.arch == "gpt2":
        out += [("wte", (V, d)), ("wpe", (m.max_pos, d))]
        for l in range(m.n_layers):
            p = f"l{l}."
            out += [(p + "ln1_g", (d,)), (p + "ln1_b", (d,)),
                    (p + "w_qkv", (3 * d, d)), (p + "b_qkv", (3 * d,)),
                    (p + "w_o", (d, d)), (p + "b_o", (d,)),
                    (p + "ln2_g", (d,)), (p + "ln2_b", (d,)),
                    (p + "w_fc", (F, d)), (p + "b_fc", (F,)),
                    (p + "w_proj", (d, F)), (p + "b_proj", (d,))]
        out += [("lnf_g", (d,)), ("lnf_b", (d,))]
    else:
        raise ValueError(m.arch)
    return out


def _role(name: str) -> str:
    base = name.split(".")[-1]
    if base.endswith("norm") or base.endswith("_g"):
        return "gain"
    if base.startswith("b_") or base.endswith("_b"):
        return "bias"
    return "matrix"


def _normal_f32(shape, seed: int, idx: int, pool: ThreadPoolExecutor,
                scale: float = 1.0) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, np.float32)
    ss = np.random.SeedSequence(entropy=seed, spawn_key=(idx,))
    kids = ss.spawn((n + _CHUNK - 1) // _CHUNK)

    def fill(c):
        lo = c * _CHUNK
        hi = min(n, lo + _CHUNK)
        np.random.default_rng(kids[c]).standard_normal(out=out[lo:hi], dtype=np.float32)
        if scale != 1.0:
            out[lo:hi] *= np.float32(scale)

    list(pool.map(fill, range(len(kids))))
    return out.reshape(shape)


def _finish(x: np.ndarray, dtype: str, pool: ThreadPoolExecutor) -> np.ndarray:
    if dtype == "f32":
        return x
    flat = x.reshape(-1)
    out = np.empty(flat.size, np.uint16)

    def conv(c):
        lo = c * _CHUNK
        hi = min(flat.size, lo + _CHUNK)
        out[lo:hi] = f32_to_bf16_bits(flat[lo:hi])

    list(pool.map(conv, range((flat.size + _CHUNK - 1) // _CHUNK)))
    return out.reshape(x.shape)


def gen_tensor(m: ModelShape, name: str, seed: int = 1, init: str = "paper",
               pool: ThreadPoolExecutor = None) -> np.ndarray:
    """One parameter tensor.  bf16 models get uint16 bfloat16 bit patterns,
    f32 models float32.

    init="paper":     matrices/embeddings N(0, 0.02), gains 1, biases 0.
    init="perturbed": same matrices; gains 1 + N(0, 0.1^2), biases N(0, 0.02^2)
                      (used by tests so that gain/bias paths are exercised).
    """
    man = weight_manifest(m)
    idx = [k for k, (nm, _) in enumerate(man) if nm == name]
    if not idx:
        raise KeyError(name)
    idx = idx[0]
    shape = man[idx][1]
    own = pool is None
    if own:
        pool = ThreadPoolExecutor(_threads())
    try:
        role = _role(name)
        if role == "matrix":
            x = _normal_f32(shape, seed, idx, pool, 0.02)
        elif init == "paper":
            x = np.full(shape, 1.0 if role == "gain" else 0.0, np.float32)
        elif init == "perturbed":
            z = _normal_f32(shape, seed, idx, pool)
            x = (np.float32(1.0) + np.float32(0.1) * z) if role == "gain" else np.float32(0.02) * z
            x = x.astype(np.float32)
        else:
            raise ValueError(init)
        return _finish(x, m.dtype, pool)
    finally:
        if own:
            pool.shutdown()


def iter_weights(m: ModelShape, seed: int = 1, init: str = "paper") -> Iterator[Tuple[str, np.ndarray]]:
    with ThreadPoolExecutor(_threads()) as pool:
        for name, _ in weight_manifest(m):
            yield name, gen_tensor(m, name, seed, init, pool)


def gen_weights(m: ModelShape, seed: int = 1, init: str = "paper") -> Dict[str, np.ndarray]:
    return dict(iter_weights(m, seed, init))


def gen_normal(shape, seed: int, scale: float = 1.0) -> np.ndarray:
    """float32 N(0, scale^2) array of any size, generated on several threads
    (deterministic in seed, independent of the thread count)."""
    with ThreadPoolExecutor(_threads()) as pool:
        return _normal_f32(tuple(shape), seed, 0, pool, scale)
