"""Throughput of attention forward + backward on one MI355X.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload 3]

One step is the whole hot path on one batch: mg_attn_fwd (O, LSE) followed
by mg_attn_bwd (D = rowsum(dO o O), the dK/dV kernel, the dQ kernel), with
every input resident in HBM before the timed region.  The timed region is
exactly `steps` steps, bracketed by device synchronization.  FLOPs are
credited only for what exact attention must compute on unmasked (i, j)
pairs: 4d per pair forward (Q K^T and P V) and 10d per pair backward (the
score recompute, dP, dV, dK and dQ products).

Rank 0 prints one JSON line.  Besides the contract fields it carries
`roofline` for the dominant kernel (its algorithmic FLOPs per launch over its
average duration, timed with HIP events on the launch stream inside the timed
region), `cpu_baseline` (the f64 oracle on the host's cores, same workload),
and `parity` (the timed run's outputs against the oracle).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "attention fwd+bwd TFLOP/s (strict f32) at B8 H8 L1024 d64; % MFMA peak"
F32_MFMA_PEAK, LOWP_MFMA_PEAK = 157.3, 2516.6   # MI355X dense MFMA, f32 and bf16/f16
# Whole-step peak: the accelerated contract runs its forward (4d flop per
# pair) on f16 and its backward (10d) on f32 matrix cores, so its ideal step
# time is the sum of the two at their own peaks.
PEAK_TFLOPS = {"strict_f32": F32_MFMA_PEAK, "fast_bf16": LOWP_MFMA_PEAK,
               "accelerated": 14.0 / (4.0 / LOWP_MFMA_PEAK + 10.0 / F32_MFMA_PEAK)}
TOLERANCE = {"strict_f32": 1e-4, "fast_bf16": 2e-2, "accelerated": 5e-3}
DTYPE = {"strict_f32": "f32", "fast_bf16": "bf16", "accelerated": "f16 fwd / f32 bwd"}
HBM_PEAK_GBS = 8000.0
KERNEL_SOURCE_DIR = "paper_2608_01563_amd/csrc"
COUNTER_FILE = "profiles/hbm_traffic_{workload}.json"


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3,
                    help="workload id (3 = causal B8 H8 L1024 d64 strict f32)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="repeat the oracle sample until this much CPU wall time (>= 3 runs)")
    ap.add_argument("--no-kernel-events", action="store_true",
                    help="do not bracket kernels with events (no roofline)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the run, copy one buffer of this many MiB (a plain copy "
                         "kernel of known size, to scale HBM byte counters)")
    return ap.parse_args()


def kernel_source_digest():
    """sha256 over the names and contents of every file the library is built
    from (kernels, headers, host code): a counter record taken on any other
    source is stale."""
    h = hashlib.sha256()
    base = os.path.join(ROOT, KERNEL_SOURCE_DIR)
    for name in sorted(os.listdir(base)):
        path = os.path.join(base, name)
        if os.path.isfile(path):
            h.update(name.encode() + b"\0")
            with open(path, "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def kernel_work(name, w, pairs, rows, key_len=None):
    """Algorithmic work of one launch of kernel `name`: (amount, unit, bound)."""
    d, es = w.d, (4 if w.contract == "strict_f32" else 2)
    if name.startswith("attn_fwd"):
        return 4.0 * d * pairs, "flop", "mfma"
    if name.startswith("attn_dkdvreduce"):
        # reads S dK and S dV partials, writes dK and dV (all f32)
        n = w.B * w.H * w.key_length * d
        return 4.0 * 2 * n * (query_splits(w) + 1), "byte", "hbm"
    if name.startswith("attn_dkdvq"):
        return 10.0 * d * pairs, "flop", "mfma"       # S recompute, dV, dP, dK, dQ
    if name.startswith("attn_dkdv"):
        return 8.0 * d * pairs, "flop", "mfma"        # S recompute, dV, dP, dK
    if name.startswith("attn_dqreduce"):
        # reads one d-vector partial per (key tile, query row) pair that
        # holds an allowed key, writes dQ
        return 4.0 * d * partial_rows(w, key_len) + 4.0 * w.B * w.H * w.L * d, "byte", "hbm"
    if name.startswith("attn_dq"):
        return 2.0 * d * pairs, "flop", "mfma"        # the dQ product itself
    if name.startswith("attn_rowdot"):
        n = w.B * w.H * w.L * d
        return 2.0 * n * es + 4.0 * rows, "byte", "hbm"
    raise KeyError(name)


def kernel_peak(name):
    """Dense MFMA peak of the matrix type a kernel multiplies in."""
    return LOWP_MFMA_PEAK if ("_bf16_" in name or "_accel_" in name) else F32_MFMA_PEAK


def fused_key_rows(w):
    return 128 if (w.causal and -(-w.key_length // 128) * w.B * w.H >= 512) else 64


def query_splits(w):
    """Workgroups over which the fused backward splits each key tile's query
    tiles (the rule the library's workspace query documents)."""
    grid = -(-w.key_length // fused_key_rows(w)) * w.B * w.H
    if grid >= 512:
        return 1
    return max(1, min(-(-1024 // grid), -(-w.L // 32) // 4))


def partial_rows(w, key_len):
    """(key tile, query row) pairs the fused dQ reduction reads (key tiles of
    128 keys when causal with >= 512 such tiles, else 64)."""
    Lk = w.key_length
    key_rows = fused_key_rows(w)
    total = 0
    kls = [Lk] * w.B if key_len is None else [int(n) for n in key_len]
    for n in kls:
        nk = -(-max(0, min(n, Lk)) // key_rows)
        for i in range(w.L):
            last = i + Lk - w.L          # causal: last key row i sees
            total += (0 if last < 0 else min(nk, last // key_rows + 1)) if w.causal else nk
    return total * w.H


def traffic_for(kernel, w):
    """HBM bytes per launch of `kernel` on workload `w` from the committed
    FETCH_SIZE / WRITE_SIZE counter runs (scaled by a plain copy of known
    size), or None if absent or taken on a different kernel source."""
    path = os.path.join(ROOT, COUNTER_FILE.format(workload=w.name))
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256") != kernel_source_digest():
        return None
    return rec.get("kernels", {}).get(kernel, {}).get("bytes_per_launch")


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only; --gpus %d is not supported "
              "(B*H heads shard across GPUs with no exchange, see the design notes)"
              % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2608_01563_amd as mg
    from workloads import WORKLOADS, workload_inputs, unmasked_pairs

    w = WORKLOADS[args.workload]
    x = workload_inputs(args.workload)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def dev_tensor(name):
        if w.contract == "fast_bf16":
            return torch.from_numpy(x.bits[name].view(np.int16).copy()).to(dev).view(
                torch.bfloat16)
        return torch.from_numpy(getattr(x, name).copy()).to(dev)

    Q, K, V, dO = (dev_tensor(n) for n in ("Q", "K", "V", "dO"))
    kl = None if x.key_len is None else torch.from_numpy(x.key_len.copy()).to(dev)
    O = torch.empty_like(Q)
    LSE = torch.empty(Q.shape[:3], dtype=torch.float32, device=dev)
    dQ, dK, dV = torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V)
    ws = torch.empty(mg.mg_attn_bwd_cross_workspace_bytes(w.B, w.H, w.L, w.key_length, w.d,
                                                          w.causal, w.contract),
                     dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        mg.mg_attn_fwd_cross(Q, K, V, O, LSE, kl, causal=w.causal, scale=w.scale,
                             contract=w.contract, stream=stream)
        mg.mg_attn_bwd_cross(Q, K, V, O, LSE, dO, dQ, dK, dV, kl, causal=w.causal,
                             scale=w.scale, contract=w.contract, workspace=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # Timed region: exactly `steps` steps between device synchronizations.
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    stops = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        starts[k].record(stream)
        step()
        stops[k].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    samples = sorted(a.elapsed_time(b) for a, b in zip(starts, stops))

    # Per-kernel durations: the same `steps` steps again, with the library
    # bracketing every kernel launch by HIP events on the launch stream.
    kernels = {}
    events_ms_per_step = None
    if not args.no_kernel_events:
        mg.mg_profile_reset()
        mg.mg_profile_enable(True)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        events_ms_per_step = (time.perf_counter() - t1) * 1e3 / args.steps
        mg.mg_profile_enable(False)
        kernels = mg.mg_profile_collect()

    pairs = unmasked_pairs(w.B, w.H, w.L, w.causal, x.key_len, Lk=w.key_length)
    rows = w.B * w.H * w.L
    flops = 14.0 * w.d * pairs
    ms_per_step = elapsed * 1e3 / args.steps
    value = flops / (ms_per_step * 1e-3) / 1e12

    out = {
        "metric": METRIC if args.workload == 3 else
        "attention fwd+bwd TFLOP/s (%s) at %s" % (w.contract, w.name),
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE[w.contract],
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "L": w.L, "Lk": w.key_length,
                   "d": w.d,
                   "causal": w.causal, "key_padding": w.padded, "contract": w.contract,
                   "unmasked_pairs": pairs, "credited_gflop_per_step": flops / 1e9},
        "step_ms": {"median": round(float(np.median(samples)), 4),
                    "q1": round(float(np.percentile(samples, 25)), 4),
                    "q3": round(float(np.percentile(samples, 75)), 4),
                    "min": round(samples[0], 4), "max": round(samples[-1], 4)},
        "pct_of_mfma_peak": round(100.0 * value / PEAK_TFLOPS[w.contract], 2),
    }
    if events_ms_per_step is not None:
        out["ms_per_step_with_kernel_events"] = round(events_ms_per_step, 4)

    if kernels:
        per = {}
        for name, (n, total) in kernels.items():
            avg = total / n
            amount, unit, bound = kernel_work(name, w, pairs, rows, x.key_len)
            rate = amount / (avg * 1e-3) / (1e12 if unit == "flop" else 1e9)
            per[name] = {"launches": n, "avg_ms": round(avg, 5), "bound": bound,
                         "achieved": round(rate, 3),
                         "unit": "TFLOP/s" if unit == "flop" else "GB/s"}
        out["kernels"] = per
        dom = max(kernels, key=lambda k: kernels[k][1])
        n, total = kernels[dom]
        amount, unit, bound = kernel_work(dom, w, pairs, rows, x.key_len)
        avg_s = total / n * 1e-3
        if unit == "flop":
            ach, peak, u = amount / avg_s / 1e12, kernel_peak(dom), "TFLOP/s"
        else:
            ach, peak, u = amount / avg_s / 1e9, HBM_PEAK_GBS, "GB/s"
        out["roofline"] = {"kernel": dom, "bound": bound, "achieved": round(ach, 3),
                           "peak": peak, "unit": u, "frac": round(ach / peak, 4),
                           "traffic": traffic_for(dom, w),
                           "algorithmic_per_launch": amount}
        out["bwd_credited_tflops"] = round(
            10.0 * w.d * pairs / (sum(kernels[k][1] / kernels[k][0] for k in kernels
                                      if not k.startswith("attn_fwd")) * 1e-3) / 1e12, 3)

    if not args.no_cpu_baseline:
        out["cpu_baseline"], out["parity"] = cpu_baseline(args, w, x, pairs,
                                                          (O, LSE, dQ, dK, dV))
    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = n * 4
    print(json.dumps(out), flush=True)


def cpu_baseline(args, w, x, pairs, gpu_outputs):
    """Time the f64 oracle on this host over the whole workload (or a head
    sample for the largest one), and compare the timed run's outputs to it."""
    import numpy as np
    from oracle import oracle_forward, oracle_backward, oracle_num_threads
    B, H = w.B, w.H
    heads = None
    if B * H * w.L * w.key_length * w.d > 2 ** 33:   # keep the CPU leg to seconds
        heads = [(b, h) for b in range(B) for h in range(H)][:: max(1, (B * H) // 4)][:4]
    # repeat the sample until about --cpu-seconds of oracle work (at least 3
    # runs, at most 100), so the figure is a bounded, stable CPU measurement
    times = []
    while len(times) < 3 or (sum(times) < args.cpu_seconds and len(times) < 100):
        t0 = time.perf_counter()
        O, LSE = oracle_forward(x.Q, x.K, x.V, w.causal, w.scale, key_len=x.key_len, heads=heads)
        dQ, dK, dV, _ = oracle_backward(x.Q, x.K, x.V, x.dO, w.causal, w.scale,
                                        key_len=x.key_len, heads=heads)
        times.append(time.perf_counter() - t0)
    total = float(sum(times))
    frac = 1.0 if heads is None else len(heads) / float(B * H)
    value = 14.0 * w.d * pairs * frac * len(times) / total / 1e12
    what = ("the whole workload (%d heads)" % (B * H)) if heads is None else (
        "%d of %d heads" % (len(heads), B * H))
    sample = ("%s, fwd+bwd, run %d times back to back (%.1f s of CPU wall time, "
              "%.2f s per run)" % (what, len(times), total, total / len(times)))
    base = {"value": round(value, 6), "unit": "TFLOP/s", "cores": oracle_num_threads(),
            "kind": "oracle", "sample": sample}
    ref = {"O": O, "LSE": LSE, "dQ": dQ, "dK": dK, "dV": dV}
    parity = {}
    for name, tens in zip(("O", "LSE", "dQ", "dK", "dV"), gpu_outputs):
        g = tens.detach().float().cpu().numpy().astype(np.float64)
        r = ref[name]
        if heads is not None:
            g = np.stack([g[b, h] for b, h in heads])
            r = np.stack([r[b, h] for b, h in heads])
        fin = np.isfinite(r)
        den = np.max(np.abs(r[fin])) if fin.any() else 1.0
        parity[name] = float(np.max(np.abs(g[fin] - r[fin])) / den) if fin.any() else 0.0
    parity["tolerance"] = TOLERANCE[w.contract]
    parity["pass"] = all(v <= parity["tolerance"] for k, v in parity.items()
                         if k in ("O", "LSE", "dQ", "dK", "dV"))
    return base, parity


if __name__ == "__main__":
    main()
