"""LM-GC compression throughput on one MI355X.

Workload: the Llama-2-7B-shape decoder (32 layers, d=4096, 32 heads, SwiGLU
11008, vocab 32000, RoPE) in bf16 with random-init weights, compressing
float32 gradients ~ Laplace(0, 1e-3) serialised as 8 hex digits + separator,
4096-token windows, 8 windows per LM call.

One step = one batch of 8 windows through the whole hot path: serialise the
batch's tokens on the GPU, run the LM to per-position integer tables,
copy tables and coder bins to the host, arithmetic-code the 8 windows (host
coding of a batch overlaps the GPU work of the next).  The value is the
whole job's float32 gradient bytes per second (inputs resident in HBM).

Prints one JSON line.  Extra fields: the dominant kernel's roofline (HIP
events around each of its launches in the timed region) and the CPU oracle's
throughput on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 matrix peak
DOMINANT = "gemm_up"               # gate/up projection + SwiGLU: 44% of the FLOPs


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def cpu_baseline(w, host_weights, values, n_values_sample):
    """Time the oracle (as it stands) compressing the first values of the
    vector: one window prefix of the same workload."""
    import numpy as np

    from oracle import pipeline as opipe
    from oracle.forward import Model as OModel

    om = OModel(w.model, host_weights)
    sample = values[:n_values_sample]
    t0 = time.perf_counter()
    buf = opipe.compress(sample, w.serial, om)
    dt = time.perf_counter() - t0
    threads = min(16, os.cpu_count() or 1)  # weight-decoding pool of the oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([threads] + [i.get("num_threads", 1) for i in threadpool_info()])
    except ImportError:
        pass
    return {
        "value": sample.nbytes / dt / 1e6,
        "unit": "MB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{n_values_sample} values = {9 * n_values_sample} tokens (a prefix of window 0) "
                  f"through the float64 NumPy forward + quantiser + coder; {dt:.1f} s, "
                  f"{len(buf)} bytes",
        "seconds": dt,
    }


# Sources of the dominant kernel: a stored traffic figure is used only while
# they are unchanged since its counters were taken.
KERNEL_SOURCES = ("paper_2409_17836_amd/csrc/gemm_bf16.hip", "paper_2409_17836_amd/csrc/epilogue.h",
                  "paper_2409_17836_amd/csrc/common.h")


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def load_traffic(path):
    """HBM bytes per launch of the dominant kernel from the stored counter
    summary, or None when it is missing or the kernel changed since."""
    if not os.path.exists(path):
        return None
    try:
        tj = json.load(open(path))
    except (OSError, ValueError):
        return None
    if tj.get("source_sha256") != kernel_source_hash():
        log("[bench] stored traffic figure is for other kernel sources; reporting null")
        return None
    return tj.get("bytes_per_launch")


def describe_model(m):
    if m.arch == "gpt2":
        return f"GPT-2-shape decoder ({m.n_layers} layers, d={m.d_model}, vocab {m.vocab}, {m.dtype})"
    size = "Llama-2-7B-shape" if m.d_model == 4096 else "Llama-style"
    return (f"{size} decoder ({m.n_layers} layers, d={m.d_model}, {m.n_heads}/{m.n_kv_heads} heads, "
            f"SwiGLU {m.d_ff}, vocab {m.vocab}, {m.dtype})")


def describe_serial(s, tok_per_value):
    sep = "".join(chr(c) for c in (s.sep_id, s.sep2_id) if c >= 0)
    group = "no separator" if s.bytes_per_group == 0 else \
        f"separator {sep!r} after every {s.bytes_per_group} bytes"
    tables = "tables renormalised over the alphabet" if getattr(s, "renorm", 0) else \
        "full-vocabulary tables"
    return f"{s.bytes_per_value}-byte values as hex digits, {group} ({tok_per_value:g} tokens per value), {tables}"


def copy_calibration(mib):
    """Plain device-to-device copies of a known size, for scaling the HBM
    byte counters (run under the profiler's counter collection)."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.empty(n, dtype=torch.float32, device="cuda:0").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "copies": 3}), flush=True)


def decode_bench(B, model, dv, sp, Bw, W, name):
    """The decoder's path: lmgc_probs_stepwise computes the tables one
    position at a time through the K/V cache, all Bw windows of the batch per
    token step, as lmgc_decode does between its host decoding steps.  Timed
    over whole windows of W positions; the tables are checked bit for bit
    against lmgc_probs (the encoder's), which lossless decoding needs."""
    import torch
    tok, _ = B.serialize(dv, sp, 0, Bw)
    B.probs_stepwise(model, tok[:, :64].contiguous(), sp)  # warm-up
    ws = B.workspace(model.step_workspace(Bw, W), tok.device)
    torch.cuda.synchronize()
    log(f"[bench] decoding path: {W} token steps of {Bw} windows")
    t0 = time.perf_counter()
    cdf1, lp1 = B.probs_stepwise(model, tok, sp, ws=ws)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    cdf0, lp0 = B.probs(model, tok, sp)
    same = bool(torch.equal(cdf0, cdf1)) and bool(torch.equal(lp0.view(torch.int32), lp1.view(torch.int32)))
    print(json.dumps({"metric": "decoding path, ms per token step (all windows of the batch)",
                      "value": round(dt * 1e3 / W, 4), "unit": "ms", "higher_is_better": False,
                      "workload": name, "windows": Bw, "window_tokens": W, "token_steps": W,
                      "tables_bit_identical_to_encoder": same}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=12)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="7b")
    ap.add_argument("--separator", default=None,
                    help="serialisation variant of Sec. 5.2: H_s (default), H_c, H_semi, H_c+s")
    ap.add_argument("--bpg", type=int, default=None, help="bytes per separator group (0 = H_n)")
    ap.add_argument("--renorm", action="store_true",
                    help="tables renormalised over the alphabet (LM head cut to the alphabet)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-values", type=int, default=2)
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic_gemm_up_7b.json"))
    ap.add_argument("--decode", action="store_true",
                    help="time the decoding path (per-position tables through the K/V cache) instead")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run plain copies of this size (counter calibration)")
    args = ap.parse_args()
    if args.copy_calibration_mib:
        copy_calibration(args.copy_calibration_mib)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); windows are independent, "
              "so more GPUs would each compress their own window range", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import dataclasses

    from paper_2409_17836_amd import binding as B
    from synth import get_workload, parse_lossy
    from synth.configs import SEPARATORS
    from synth.gen import iter_weights, workload_values

    w = get_workload(args.workload)
    serial = w.serial
    if args.separator:
        sep, sep2 = SEPARATORS[args.separator]
        serial = dataclasses.replace(serial, sep_id=sep, sep2_id=sep2)
    if args.bpg is not None:
        serial = dataclasses.replace(serial, bytes_per_group=args.bpg)
    if args.renorm:
        serial = dataclasses.replace(serial, renorm=1)
    w = w.with_(serial=serial)
    Bw, W = w.batch, w.serial.window
    dev = torch.device("cuda:0")
    log(f"[bench] workload {w.name}: generating {w.n_values} values and weights")
    values = workload_values(w)
    host = {}
    dweights = []
    for name, arr in iter_weights(w.model, w.weight_seed):
        host[name] = arr
        a = arr.view(np.int16) if arr.dtype == np.uint16 else arr
        dweights.append(torch.from_numpy(a).to(dev))
    cfg = B.model_config(w.model)
    model = B.Model(cfg, dweights)
    del dweights
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    sp = B.serial_params(w.serial)
    dv = torch.from_numpy(values).to(dev)
    lossy_ms = None
    if w.lossy:
        # Sec. 5.4: the lossy steps run once over the whole vector on the GPU;
        # the timed steps compress their output, resident in HBM
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        dv = B.lossy_prepare(dv, parse_lossy(w.lossy))
        torch.cuda.synchronize()
        lossy_ms = (time.perf_counter() - t0) * 1e3
        log(f"[bench] lossy steps {w.lossy}: {lossy_ms:.2f} ms for {w.n_values} values")
    if args.decode:
        decode_bench(B, model, dv, sp, Bw, W, w.name)
        return
    n_vals = dv.numel()
    n_win = B.num_windows(n_vals, sp)
    need = (args.warmup + args.steps) * Bw
    assert need <= n_win, f"{need} windows needed, workload has {n_win}"
    ws = B.workspace(model.codec_workspace(n_vals, sp, Bw))
    stream = torch.cuda.current_stream()
    log(f"[bench] model ready; warmup {args.warmup} step(s)")

    if args.warmup:
        B.compress(model, dv, sp, batch=Bw, first_window=0, n_windows=args.warmup * Bw, ws=ws)
    torch.cuda.synchronize()

    log(f"[bench] timing {args.steps} step(s)")
    # inside the timed region events are recorded only around the dominant
    # kernel's launches (each event pair adds a little time between launches)
    B.timing_kinds([DOMINANT])
    B.timing_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    buf = B.compress(model, dv, sp, batch=Bw, first_window=args.warmup * Bw,
                     n_windows=args.steps * Bw, ws=ws)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    dom = B.timing_read(DOMINANT)
    B.timing_enable(False)
    # per-kernel breakdown from one more, untimed step with events on every kind
    B.timing_kinds(None)
    B.timing_enable(True)
    B.compress(model, dv, sp, batch=Bw, first_window=0, n_windows=Bw, ws=ws)
    torch.cuda.synchronize()
    kern = {k: B.timing_read(k) for k in B.KINDS}
    B.timing_enable(False)
    kern[DOMINANT] = dom

    n_tok = B.num_tokens(n_vals, sp)
    tok_done = min(n_tok, (args.warmup + args.steps) * Bw * W) - args.warmup * Bw * W
    tok_per_value = n_tok / max(n_vals, 1)
    grad_bytes = tok_done / tok_per_value * w.serial.bytes_per_value
    value = grad_bytes / dt / 1e6
    ms_step = dt * 1e3 / args.steps

    flops_step = {k: model.flops(Bw, W, k) for k in B.KINDS}
    total_flops = sum(flops_step.values())
    mfma_util = total_flops * args.steps / dt / (PEAK_BF16_TFLOPS * 1e12)
    ms_k, n_k = kern[DOMINANT]
    launches_per_step = w.model.n_layers
    flop_launch = flops_step[DOMINANT] / launches_per_step
    avg_ms = ms_k / max(n_k, 1)
    achieved = flop_launch / (avg_ms * 1e-3) / 1e12
    traffic = load_traffic(args.traffic_json)
    kernel_ms = {k: round(ms / (args.steps if k == DOMINANT else 1), 3) for k, (ms, n) in kern.items() if n}

    out = {
        "metric": "gradient MB/s compressed (LM probs + AC) at 7B-shape bf16; MFMA util",
        "value": round(value, 6),
        "unit": "MB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Laplace gradients, random-init weights)",
        "config": {
            "workload": f"{w.name}: {describe_model(w.model)}, gradients ~ {w.dist}"
                        + (f" then {w.lossy}" if w.lossy else "")
                        + f", {describe_serial(w.serial, tok_per_value)}",
            "windows_per_step": Bw,
            "window_tokens": W,
            "tokens_per_step": Bw * W,
            "values_per_step": round(Bw * W / tok_per_value, 1),
            "parallelism": "single GPU",
        },
        "tokens_per_s": round(tok_done / dt, 1),
        "mfma_util": round(mfma_util, 4),
        "container_bytes": len(buf),
        "compression_rate_pct": round(100.0 * len(buf) / grad_bytes, 2),
        "kernel_ms_per_step": kernel_ms,
        "roofline": {
            "kernel": f"{DOMINANT} (gate/up projection {Bw * W}x{2 * w.model.d_ff}x{w.model.d_model} "
                      "with fused SwiGLU)",
            "bound": "mfma",
            "achieved": round(achieved, 1),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "avg_launch_ms": round(avg_ms, 4),
            "flop_per_launch": flop_launch,
        },
    }
    if lossy_ms is not None:
        out["lossy_prep_ms"] = round(lossy_ms, 3)
    if not args.no_cpu_baseline and not w.lossy:
        log("[bench] timing the CPU oracle on a bounded sample")
        cb = cpu_baseline(w, host, values, args.cpu_sample_values)
        out["cpu_baseline"] = {k: v for k, v in cb.items() if k != "seconds"}
    print(json.dumps(out), flush=True)
    model.close()


if __name__ == "__main__":
    main()
