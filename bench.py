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
PEAK_F32_VECTOR_TFLOPS = 157.3     # MI355X float32 vector peak (the tiny model's FMA kernels)
HBM_PEAK_GBS = 8000.0              # MI355X HBM3E bandwidth (the decoding step is bound by it)
DOMINANT = "gemm_up"               # gate/up projection + SwiGLU: 44% of the FLOPs


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def cpu_info():
    """nproc and the CPU model name of this host."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return os.cpu_count() or 1, model


WHOLE_VECTOR_TOKENS = 1 << 16


def cpu_baseline(w, host_weights, raw_values, all_positions=256, one_positions=32):
    """The oracle as it stands, timed on this host's cores.  Its float64
    weights are decoded once, outside the timed region.  Two legs, each
    compressing a prefix of the workload's vector (window 0's first
    positions; the whole vector if it is smaller): all cores on at least
    `all_positions` tokens, one thread on at least `one_positions` tokens.
    Lossy workloads run the oracle's own lossy steps on the raw vector first
    (timed separately)."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import lossy as olossy
    from oracle import pipeline as opipe
    from oracle.forward import Model as OModel
    from synth.gen import weight_manifest

    nproc, cpu_model = cpu_info()
    om = OModel(w.model, host_weights, cache=True)
    t0 = time.perf_counter()
    for name, _ in weight_manifest(w.model):
        om.w(name)
    decode_s = time.perf_counter() - t0
    values, prep_s = raw_values, 0.0
    if w.lossy:
        t0 = time.perf_counter()
        values = olossy.prepare(raw_values, w.lossy)
        prep_s = time.perf_counter() - t0
    tok_per_value = opipe.serialize(values[:64], w.serial)[0].size / min(64, values.size)
    legs = {}
    # a vector of at most WHOLE_VECTOR_TOKENS tokens (the tiny workload) is
    # compressed whole on all cores
    whole = values.size * tok_per_value <= WHOLE_VECTOR_TOKENS
    for leg, positions, threads in (("all_cores", all_positions, None), ("one_thread", one_positions, 1)):
        n = values.size if (whole and threads is None) else \
            min(values.size, int(np.ceil(positions / tok_per_value)))
        sample = values[:n]
        with threadpool_limits(threads):
            used = max([1] + [i.get("num_threads", 1) for i in threadpool_info()])
            t0 = time.perf_counter()
            buf = opipe.compress(sample, w.serial, om)
            dt = time.perf_counter() - t0
        ntok = opipe.serialize(sample, w.serial)[0].size
        legs[leg] = {"threads": used, "values": int(n), "tokens": int(ntok), "seconds": round(dt, 2),
                     "tokens_per_s": round(ntok / dt, 2),
                     "grad_MB_per_s": sample.nbytes / dt / 1e6, "container_bytes": len(buf)}
    a = legs["all_cores"]
    return {
        "value": a["grad_MB_per_s"],
        "unit": "MB/s",
        "cores": a["threads"],
        "kind": "oracle",
        "sample": f"{a['values']} values = {a['tokens']} tokens "
                  f"({'the whole vector' if whole else 'window 0 prefix'}) through the float64 "
                  f"NumPy forward + quantiser + coder on {a['threads']} threads in {a['seconds']} s; "
                  f"weights decoded once beforehand ({decode_s:.1f} s, not timed)",
        "tokens_per_s": a["tokens_per_s"],
        "one_thread": legs["one_thread"],
        "nproc": nproc,
        "cpu_model": cpu_model,
        "lossy_prep_s": round(prep_s, 2) if w.lossy else None,
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


def decode_step_bytes(m, Bw, W, wbytes):
    """HBM bytes one decoding step must move, averaged over a window of W
    positions: every weight matrix once (the step's products read each
    layer's weights whatever the number of windows) and, in attention, the
    K and V of positions 0..p of every window at position p."""
    d, hd, F, V = m.d_model, m.head_dim, m.d_ff, m.vocab
    per_layer = (m.n_heads + 2 * m.n_kv_heads) * hd * d + d * d
    per_layer += (2 * F * d + F * d) if m.arch == "llama" else (F * d + d * F)
    weights = (m.n_layers * per_layer + V * d) * wbytes
    kv_mean = m.n_layers * 2 * m.n_kv_heads * hd * wbytes * Bw * (W + 1) / 2.0
    return weights + kv_mean


def decode_bench(B, model, dv, sp, Bw, W, name, mshape=None):
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
    line = {"metric": "decoding path, ms per token step (all windows of the batch)",
            "value": round(dt * 1e3 / W, 4), "unit": "ms", "higher_is_better": False,
            "tokens_per_s": round(Bw * W / dt, 1),
            "workload": name, "windows": Bw, "window_tokens": W, "token_steps": W,
            "tables_bit_identical_to_encoder": same}
    if mshape is not None:
        # the step is bound by HBM: weights once per step plus the K/V prefix
        nb = decode_step_bytes(mshape, Bw, W, 2 if mshape.dtype == "bf16" else 4)
        ach = nb / (dt / W) / 1e9
        line["roofline"] = {"bound": "hbm", "algorithmic_GB_per_step": round(nb / 1e9, 3),
                            "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                            "frac": round(ach / HBM_PEAK_GBS, 4)}
    print(json.dumps(line), flush=True)


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
    ap.add_argument("--repeats", type=int, default=3, help="timed repeats of --steps steps (median reported)")
    ap.add_argument("--cpu-positions", type=int, default=256,
                    help="tokens of the oracle's all-core timing sample")
    ap.add_argument("--cpu-positions-one", type=int, default=32,
                    help="tokens of the oracle's one-thread timing sample")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic_gemm_up_7b.json"))
    ap.add_argument("--decode", action="store_true",
                    help="time the decoding path (per-position tables through the K/V cache) instead")
    ap.add_argument("--decode-batch", type=int, default=0,
                    help="windows per decoding step with --decode (default: the workload's batch; at most 32)")
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
        decode_bench(B, model, dv, sp, args.decode_batch or Bw, W, w.name, w.model)
        return
    n_vals = dv.numel()
    n_win = B.num_windows(n_vals, sp)
    ws = B.workspace(model.codec_workspace(n_vals, sp, Bw))
    log(f"[bench] model ready; warmup {args.warmup} step(s)")
    # Window ranges: steps take consecutive batches of the vector's windows;
    # a workload with fewer windows than the run needs (the tiny one is one
    # batch) compresses the same batch in every step, one call per step.
    per_call = (args.warmup + args.repeats * args.steps) * Bw <= n_win
    reuse = not per_call

    def run_steps(first_step, n_steps):
        if per_call:
            return B.compress(model, dv, sp, batch=Bw, first_window=first_step * Bw,
                              n_windows=n_steps * Bw, ws=ws)
        out = None
        for _ in range(n_steps):
            out = B.compress(model, dv, sp, batch=Bw, first_window=0, n_windows=min(Bw, n_win), ws=ws)
        return out

    if args.warmup:
        run_steps(0, args.warmup)
    torch.cuda.synchronize()

    # inside the timed region events are recorded only around the dominant
    # kernel's launches (each event pair adds a little time between launches)
    B.timing_kinds([DOMINANT])
    B.timing_enable(True)
    times = []
    for r in range(args.repeats):
        log(f"[bench] repeat {r + 1}/{args.repeats}: timing {args.steps} step(s)")
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        buf = run_steps(args.warmup + r * args.steps, args.steps)
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t0)
    dom = B.timing_read(DOMINANT)
    B.timing_enable(False)
    # per-kernel breakdown from one more, untimed step with events on every kind
    B.timing_kinds(None)
    B.timing_enable(True)
    run_steps(0, 1)
    torch.cuda.synchronize()
    kern = {k: B.timing_read(k) for k in B.KINDS}
    B.timing_enable(False)
    kern[DOMINANT] = dom

    dt = float(np.median(times))
    n_tok = B.num_tokens(n_vals, sp)
    tok_per_value = n_tok / max(n_vals, 1)
    tok_step = min(Bw * W, n_tok) if reuse else Bw * W
    tok_done = tok_step * args.steps
    grad_bytes = tok_done / tok_per_value * w.serial.bytes_per_value
    value = grad_bytes / dt / 1e6
    ms_step = dt * 1e3 / args.steps

    f32 = w.model.dtype == "f32"
    peak = PEAK_F32_VECTOR_TFLOPS if f32 else PEAK_BF16_TFLOPS
    flops_step = {k: model.flops(Bw, W, k) for k in B.KINDS}
    total_flops = sum(flops_step.values())
    mfma_util = None if f32 else total_flops * args.steps / dt / (PEAK_BF16_TFLOPS * 1e12)
    ms_k, n_k = kern[DOMINANT]
    launches_per_step = w.model.n_layers
    flop_launch = flops_step[DOMINANT] / launches_per_step
    avg_ms = ms_k / max(n_k, 1)
    achieved = flop_launch / (avg_ms * 1e-3) / 1e12
    traffic = load_traffic(args.traffic_json) if w.name == "7b" and not f32 else None
    kernel_ms = {k: round(ms / (args.steps * args.repeats if k == DOMINANT else 1), 3)
                 for k, (ms, n) in kern.items() if n}
    ms_list = sorted(t * 1e3 / args.steps for t in times)

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
        "dtype": "f32" if f32 else "bf16",
        "data": "synthetic (seeded " + w.dist.split(":")[0] + " gradients, random-init weights)",
        "config": {
            "workload": f"{w.name}: {describe_model(w.model)}, gradients ~ {w.dist}"
                        + (f" then {w.lossy}" if w.lossy else "")
                        + f", {describe_serial(w.serial, tok_per_value)}",
            "windows_per_step": Bw,
            "window_tokens": W,
            "tokens_per_step": tok_step,
            "values_per_step": round(tok_step / tok_per_value, 1),
            "windows_reused_every_step": reuse,
            "parallelism": "single GPU",
        },
        "repeats": {"n": args.repeats, "steps_each": args.steps,
                    "ms_per_step": [round(x, 3) for x in ms_list],
                    "median_ms": round(ms_step, 3),
                    "spread_pct": round(100.0 * (ms_list[-1] - ms_list[0]) / ms_step, 2)},
        "tokens_per_s": round(tok_done / dt, 1),
        "mfma_util": None if mfma_util is None else round(mfma_util, 4),
        "container_bytes": len(buf),
        "compression_rate_pct": round(100.0 * len(buf) / (tok_step / tok_per_value * w.serial.bytes_per_value
                                                           * (args.steps if per_call else 1)), 2),
        "kernel_ms_per_step": kernel_ms,
        # GPU-only time of a step: the kernels of lmgc_probs from the events
        # (the serialiser, about 0.01 ms, is not among the timed kinds)
        "gpu_ms_per_step": round(sum(kernel_ms.values()), 3),
        "roofline": {
            "kernel": f"{DOMINANT} ({'fc' if w.model.arch == 'gpt2' else 'gate/up'} projection "
                      f"{Bw * W}x{(1 if w.model.arch == 'gpt2' else 2) * w.model.d_ff}x{w.model.d_model} "
                      f"with fused {'GELU' if w.model.arch == 'gpt2' else 'SwiGLU'}"
                      + (", float32 FMA kernel" if f32 else "") + ")",
            "bound": "alu" if f32 else "mfma",
            "achieved": round(achieved, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": traffic,
            "avg_launch_ms": round(avg_ms, 4),
            "flop_per_launch": flop_launch,
        },
    }
    if w.serial.bytes_per_value != 4:
        # the lossy stream's values stand for float32 gradients of 4 bytes each
        out["f32_equivalent_MB_per_s"] = round(tok_done / tok_per_value * 4 / dt / 1e6, 6)
    if lossy_ms is not None:
        out["lossy_prep_ms"] = round(lossy_ms, 3)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(w, host, values, args.cpu_positions, args.cpu_positions_one)
    print(json.dumps(out), flush=True)
    model.close()


if __name__ == "__main__":
    main()
