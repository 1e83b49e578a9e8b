"""Helpers shared by the GPU tests: build models on the device from the seeded
generators, and run the oracle on the same inputs."""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2409_17836_amd import binding as B  # noqa: E402
from synth.gen import iter_weights  # noqa: E402


def log(msg: str):
    print(msg, flush=True)


def to_device(arr: np.ndarray, dev="cuda"):
    import torch
    if arr.dtype == np.uint16:
        arr = arr.view(np.int16)
    return torch.from_numpy(np.ascontiguousarray(arr)).to(dev)


def build_model(shape, seed: int = 1, init: str = "paper", keep_host: bool = True):
    """Generate weights, upload them, create the library model.  Returns
    (model, host weight dict or None)."""
    import torch
    cfg = B.model_config(shape)
    host = {} if keep_host else None
    dev = []
    for name, arr in iter_weights(shape, seed, init):
        if keep_host:
            host[name] = arr
        dev.append(to_device(arr))
    model = B.Model(cfg, dev)
    del dev
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return model, host


def bf16_tensor(x: np.ndarray):
    """float array -> torch bfloat16 on the GPU (round to nearest even)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda").to(torch.bfloat16)


def bf16_values(x: np.ndarray) -> np.ndarray:
    """x rounded to bfloat16 (round to nearest even), returned as float32."""
    from synth.gen import f32_to_bf16_bits, bf16_bits_to_f32
    return bf16_bits_to_f32(f32_to_bf16_bits(x))
