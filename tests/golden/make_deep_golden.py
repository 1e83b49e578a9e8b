"""Writes the oracle's alphabet log-probabilities over whole windows of the
deep bf16 workloads, for the GPU parity tests of late positions.

Causal attention makes every position of a window depend on all earlier
ones (Sec. 4, Eq. 2), and the window ablation (Sec. 5.3, Fig. 2) runs the LM
over windows of up to 4096 tokens, so RoPE angles and attention over
thousands of keys have to be compared with the oracle at model level.  The
float64 oracle needs minutes per such window on the CPU, too long to run
inside a GPU test, so this script runs it once and stores the result.

It imports only the oracle (oracle/) and the seeded input generators
(synth/); nothing here comes from the GPU library.  For each case it writes
  deep_<case>.npy   float32 [n_pos, A]: log-probabilities of the A alphabet
                    tokens at positions 0 .. n_pos-1 of the window, from the
                    float64 oracle (float32 storage adds < 1e-6)
and one deep_golden.json with, per case, the inputs (workload, weight init,
window index, SHA-256 of the model input ids) and the floor: how far the
same equations evaluated with float32 accumulation (same bf16 rounding
points) land from the float64 oracle, max and mean over all values and per
position range.

    python tests/golden/make_deep_golden.py [case ...]      # default: all
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import lossy as olossy  # noqa: E402
from oracle import pipeline as opipe  # noqa: E402
from oracle.forward import Model  # noqa: E402
from synth import get_workload  # noqa: E402
from synth.gen import gen_weights, workload_values  # noqa: E402

# case -> (workload, weight init, window index, positions)
CASES = {
    "tinyllama": ("tinyllama", "perturbed", 0, 2048),
    "7b": ("7b", "paper", 0, 4096),
    "lossy7b": ("lossy7b", "paper", 0, 4096),
}
RANGES = ((0, 256), (256, 1024), (1024, 2048), (2048, 4096))


def model_input(case):
    """Model input ids of the case's window (BOS + its first n-1 tokens) and
    the window's coded symbols."""
    wname, _, win, n_pos = CASES[case]
    w = get_workload(wname)
    vals = workload_values(w)
    if w.lossy:
        vals = olossy.prepare(vals, w.lossy)
    tok, sym = opipe.serialize(vals, w.serial)
    W = w.serial.window
    x = opipe.model_input(tok[win * W:(win + 1) * W], w.serial, n_pos)
    return w, x, sym[win * W:win * W + n_pos]


def input_sha(x: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(x, dtype=np.int64).tobytes()).hexdigest()


def run_case(case, weights_cache):
    wname, init, win, n_pos = CASES[case]
    w, x, _ = model_input(case)
    key = (w.model, w.weight_seed, init)
    if key not in weights_cache:
        weights_cache.clear()
        t0 = time.time()
        weights_cache[key] = gen_weights(w.model, w.weight_seed, init)
        print(f"[{case}] weights generated in {time.time() - t0:.0f} s", flush=True)
    host = weights_cache[key]
    ids = opipe.alphabet_ids(w.serial)
    t0 = time.time()
    lp = Model(w.model, host).alphabet_logprobs(x, ids)
    t64 = time.time() - t0
    print(f"[{case}] float64 oracle: {n_pos} positions in {t64:.0f} s", flush=True)
    t0 = time.time()
    lp32 = Model(w.model, host, acc="f32").alphabet_logprobs(x, ids)
    print(f"[{case}] float32-accumulation variant in {time.time() - t0:.0f} s", flush=True)
    floor = np.abs(lp32.astype(np.float64) - lp)
    per_range = {}
    for a, b in RANGES:
        if a < n_pos:
            f = floor[a:min(b, n_pos)]
            per_range[f"{a}-{min(b, n_pos) - 1}"] = {"max": float(f.max()), "mean": float(f.mean())}
    np.save(os.path.join(HERE, f"deep_{case}.npy"), lp.astype(np.float32), allow_pickle=False)
    return {
        "workload": wname,
        "weight_init": init,
        "weight_seed": w.weight_seed,
        "window": win,
        "positions": n_pos,
        "alphabet_ids": [int(i) for i in ids],
        "input_sha256": input_sha(x),
        "floor_f32_vs_f64": {"max": float(floor.max()), "mean": float(floor.mean()),
                             "by_position": per_range},
        "oracle_seconds": round(t64, 1),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("cases", nargs="*", default=list(CASES))
    args = ap.parse_args()
    path = os.path.join(HERE, "deep_golden.json")
    meta = json.load(open(path)) if os.path.exists(path) else {}
    cache = {}
    for case in args.cases:
        meta[case] = run_case(case, cache)
        with open(path, "w") as f:
            json.dump(meta, f, indent=1, sort_keys=True)
            f.write("\n")
        print(f"[{case}] written: {json.dumps(meta[case]['floor_f32_vs_f64'])}", flush=True)


if __name__ == "__main__":
    main()
