"""Throughput of attention forward + backward on one MI355X.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload 3]

One step is the whole hot path on one batch: mg_attn_fwd (O, LSE) followed
by mg_attn_bwd (D = rowsum(dO o O), the dK/dV kernel, the dQ kernel), with
every input resident in HBM before the timed region.  The timed region is
exactly `steps` steps, bracketed by device synchronization.  FLOPs are
credited only for what exact attention must compute on unmasked (i, j)
pairs: 4d per pair forward (Q K^T and P V) and 10d per pair backward (the
score recompute, dP, dV, dK and dQ products).

The timed region enqueues nothing but the steps (one event pair around it);
per-step samples, the forward-only and backward-only series and the
per-kernel durations come from further regions of `steps` steps each, timed
with HIP events on the launch stream (the library brackets each of its
launches while mg_profile_enable is on).

Rank 0 prints one JSON line.  Besides the contract fields it carries
`roofline` for the dominant kernel (its algorithmic FLOPs per launch over its
average duration in the per-kernel region, against the published peak and
against the sustained rate of the library's MFMA probe), `cpu_baseline` (the
f64 oracle on the host's cores, same workload), and `parity` (the timed
run's outputs against the oracle).
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

# The paper's own figures, reported beside every line as context only: they
# are whole training steps (forward, loss and backward) of its models on other
# GPUs under Vulkan or Metal, as ratios of its time to PyTorch's on the same
# device (below 1 is faster than PyTorch), from its strict-f32 results table
# (medians of 20 samples after 5 warmups); no kernel-level attention
# throughput is reported there, so nothing here is comparable to `value`.
# The attention-backward profile is its Sec. 7.3 measurement on Apple M3.
_PAPER_DEVICES = ("NVIDIA RTX 5070 (Vulkan vs CUDA, compiled)",
                  "AMD RX 7900 XT (Vulkan vs ROCm, compiled)",
                  "AMD Radeon 780M (Vulkan vs ROCm, compiled)",
                  "Intel RPL-U iGPU (Vulkan vs PyTorch CPU fallback)",
                  "Apple M3 (Metal vs MPS, eager)")
PAPER_CONTEXT_ATTENTION = {
    "kind": "paper's end-to-end training-step time / PyTorch's, other hardware (context only)",
    "source": "strict-f32 results table; Sec. 7.3 profile",
    "whisper_tiny_fwd_loss_bwd": dict(zip(_PAPER_DEVICES, (2.78, 0.90, 1.22, 1.39, 2.84))),
    "whisper_tiny_note": "the paper marks its Radeon 780M figure invalid (backward gate failed)",
    "smollm2_135m_fwd_loss_bwd": dict(zip(_PAPER_DEVICES, (2.87, 1.22, 0.95, 1.00, 2.00))),
    "apple_m3_whisper_step_profile": {"step_ms": 330, "dkdv_kernel_ms": 141.9, "dq_kernel_ms": 57.5,
                                      "backward_attention_share": 0.583},
}
PAPER_CONTEXT_CONV = {
    "kind": "paper's end-to-end training-step time / PyTorch's, other hardware (context only)",
    "source": "strict-f32 results table; Sec. 7.3 profile",
    "resnet50_fwd_loss_bwd": dict(zip(_PAPER_DEVICES, (2.24, 2.41, 1.60, 0.79, 2.34))),
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--warmup-ms", type=float, default=250.0,
                    help="after the W warmup steps, keep running untimed steps until this "
                         "much wall time has passed: the GPU raises its clocks over the "
                         "first ~30 ms of sustained load, and a timed region that starts "
                         "earlier measures the ramp, not the kernels")
    ap.add_argument("--workload", type=int, default=3,
                    help="workload id (3 = causal B8 H8 L1024 d64 strict f32)")
    ap.add_argument("--conv", action="store_true",
                    help="time the convolution derivatives of one ResNet-50 backward step "
                         "(batch 4, 224x224) instead of attention")
    ap.add_argument("--lds-probe", action="store_true",
                    help="print the LDS clocks per read of the kernels' access patterns for "
                         "the row strides they use and the alternatives, then exit")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="repeat the oracle sample until this much CPU wall time (>= 3 runs)")
    ap.add_argument("--no-mfma-probe", action="store_true",
                    help="do not measure the sustained MFMA throughput for the roofline")
    ap.add_argument("--no-kernel-events", action="store_true",
                    help="do not bracket kernels with events (no roofline)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the run, copy one buffer of this many MiB (a plain copy "
                         "kernel of known size, to scale HBM byte counters)")
    return ap.parse_args()


def kernel_source_digest(conv=False):
    """sha256 over the names and contents of the files a kernel family is
    built from (attention: every file directly under csrc/ except the MFMA
    and LDS probes; convolution:
    csrc/conv/ plus the shared device and host headers): a counter record
    taken on any other source is stale."""
    h = hashlib.sha256()
    base = os.path.join(ROOT, KERNEL_SOURCE_DIR)
    if conv:
        names = ["conv/" + n for n in sorted(os.listdir(os.path.join(base, "conv")))]
        names += ["device_common.h", "host_runtime.h", "host_runtime.cpp"]
    else:
        # the MFMA and LDS probes are measuring tools, not attention code
        names = sorted(n for n in os.listdir(base) if n not in ("mfma_probe.hip", "lds_probe.hip"))
    for name in names:
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
    if name.startswith("attn_bwdreduce"):
        # query-split fused backward: reads S dK and S dV partials and writes
        # dK and dV (all f32), and reduces the dQ partials as attn_dqreduce
        n = w.B * w.H * w.key_length * d
        dq = 4.0 * d * partial_rows(w, key_len) + 4.0 * w.B * w.H * w.L * d
        return 4.0 * 2 * n * (query_splits(w) + 1) + dq, "byte", "hbm"
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


MFMA_PROBE_ITERS = {"f32": 20000, "bf16": 40000, "f16": 40000}   # ~15-20 ms each


def mfma_kind(name):
    """Matrix type a kernel multiplies in (the probe kind)."""
    return "bf16" if "_bf16_" in name else ("f16" if "_accel_" in name else "f32")


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
    nqt = -(-w.L // 32)
    return max(1, min(-(-1024 // grid), nqt // (2 if nqt <= 8 else 4)))


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


def traffic_for(kernel, workload_name, conv=False):
    """HBM bytes per launch of `kernel` on a workload from the committed
    FETCH_SIZE / WRITE_SIZE counter runs (scaled by a plain copy of known
    size), or None if absent or taken on a different kernel source."""
    path = os.path.join(ROOT, COUNTER_FILE.format(workload=workload_name))
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256") != kernel_source_digest(conv):
        return None
    return rec.get("kernels", {}).get(kernel, {}).get("bytes_per_launch")


# The kernels' LDS read patterns (mg_lds_probe numbering) and the tiles that
# use them, with the row stride each tile uses (bytes).
LDS_PATTERNS = [
    (2, "32x32x16 operand rows: accelerated forward K", {32: 112, 64: 144, 128: 304}),
    (4, "32x32x16 transpose reads: accelerated forward V^T", {32: 64, 64: 192, 128: 320}),
    (1, "16x16x4 f32 operand groups: strict fused backward Q, dO tiles", {32: 144, 64: 272}),
    (6, "f32 products over rows: strict fused backward dO, Q (4-byte reads)", {32: 144, 64: 272}),
    (0, "16x16x32 operand rows on padded rows (reference for pattern 7)", {128: 288}),
    (3, "16x16x32 transpose reads on padded rows (reference for pattern 8)", {128: 288}),
]
# The bf16 kernels' swizzled column-block tiles (pattern, what), each beside
# the same reads on unswizzled blocks (pattern + 5).
LDS_BLOCK_PATTERNS = [
    (7, "bf16 dK/dV Q, dO rows (16x16x32 operands)"),
    (8, "bf16 dK/dV Q^T, dO^T (16x16x32 transpose reads)"),
    (9, "bf16 forward K, dQ K and V rows (32x32x16 operands)"),
    (10, "bf16 dQ K^T (32x32x16 transpose reads)"),
    (11, "bf16 forward V^T (32x32x16 transpose reads, 64-column blocks)"),
]
# The strict f32 forward's chunk-permuted d = 64 tiles (pattern, what, the
# same read shape on unpermuted 256-byte rows: (pattern, row bytes)).
LDS_F32_FWD_PATTERNS = [
    (17, "f32 forward K (16x16x4 operand groups)", (1, 256)),
    (18, "f32 forward V (4-byte reads over rows)", (6, 256)),
]


def lds_probe_main():
    """One JSON line: for each padded-row pattern and head dimension, the
    clocks per read at the stride the kernel uses and at every stride of the
    same row length padded by 0..240 bytes; for the bf16 kernels' column-block
    tiles, the clocks per read with and without their chunk swizzle."""
    import torch
    import paper_2608_01563_amd as mg
    torch.cuda.set_device(0)
    mg.load_library()
    out = {"metric": "LDS clocks per read instruction per CU (probe)",
           "contiguous_16B": mg.mg_lds_probe(5, 256), "patterns": []}
    for pattern, what, strides in LDS_PATTERNS:
        for d, used in strides.items():
            row = {"pattern": pattern, "tile": what, "d": d, "used": used, "by_stride": {}}
            base = {32: 64, 64: 128, 128: 256}[d] if pattern not in (1, 6) else {32: 128, 64: 256}[d]
            for pad in range(0, 256, 16):
                rb = base + pad
                if rb <= 480:
                    row["by_stride"][rb] = round(mg.mg_lds_probe(pattern, rb), 2)
            row["clocks_used"] = row["by_stride"].get(used, round(mg.mg_lds_probe(pattern, used), 2))
            out["patterns"].append(row)
    out["block_layouts"] = []
    for pattern, what in LDS_BLOCK_PATTERNS:
        rb = 128 if pattern == 11 else 64
        out["block_layouts"].append({
            "pattern": pattern, "tile": what, "row_bytes": rb,
            "clocks_swizzled": round(mg.mg_lds_probe(pattern, rb), 2),
            "clocks_unswizzled": round(mg.mg_lds_probe(pattern + 5, rb), 2)})
    for pattern, what, (plain, prb) in LDS_F32_FWD_PATTERNS:
        out["block_layouts"].append({
            "pattern": pattern, "tile": what, "row_bytes": 256,
            "clocks_swizzled": round(mg.mg_lds_probe(pattern, 256), 2),
            "clocks_unswizzled": round(mg.mg_lds_probe(plain, prb), 2)})
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.lds_probe:
        return lds_probe_main()
    if args.gpus != 1:
        print("bench.py: the library runs on one GPU only; --gpus %d is not supported "
              "(B*H heads shard across GPUs with no exchange, see the design notes)"
              % args.gpus, file=sys.stderr)
        sys.exit(2)
    if args.conv:
        return conv_main(args)

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

    warm = warm_up(step, args, torch)

    # Timed region: exactly `steps` steps between device synchronizations,
    # nothing else enqueued (no per-step events: each event record adds a
    # few microseconds between the steps), one event pair around the region.
    region = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    region[0].record(stream)
    for _ in range(args.steps):
        step()
    region[1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    region_ms = region[0].elapsed_time(region[1])

    # Per-step samples come from separate regions of `steps` steps each:
    # events around every fwd+bwd step, then around the forward call alone
    # and the backward call alone (events on the launch stream).
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    stops = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    for k in range(args.steps):
        starts[k].record(stream)
        step()
        stops[k].record(stream)
    torch.cuda.synchronize()
    samples_raw = [a.elapsed_time(b) for a, b in zip(starts, stops)]   # in timing order
    samples = sorted(samples_raw)
    series = {"fwd_bwd": samples_raw}
    for part in ("fwd", "bwd"):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
        for a, b in ev:
            if part == "bwd":
                mg.mg_attn_fwd_cross(Q, K, V, O, LSE, kl, causal=w.causal, scale=w.scale,
                                     contract=w.contract, stream=stream)
            a.record(stream)
            if part == "fwd":
                mg.mg_attn_fwd_cross(Q, K, V, O, LSE, kl, causal=w.causal, scale=w.scale,
                                     contract=w.contract, stream=stream)
            else:
                mg.mg_attn_bwd_cross(Q, K, V, O, LSE, dO, dQ, dK, dV, kl, causal=w.causal,
                                     scale=w.scale, contract=w.contract, workspace=ws,
                                     stream=stream)
            b.record(stream)
        torch.cuda.synchronize()
        series[part] = [a.elapsed_time(b) for a, b in ev]

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
        "warmup_steps_run": warm[0],
        "warmup_ms": round(warm[1], 1),
        "ms_per_step": round(ms_per_step, 4),
        "gpu_ms_per_step": round(region_ms / args.steps, 4),   # events around the timed region
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE[w.contract],
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "L": w.L, "Lk": w.key_length,
                   "d": w.d,
                   "causal": w.causal, "key_padding": w.padded, "contract": w.contract,
                   "unmasked_pairs": pairs, "credited_gflop_per_step": flops / 1e9},
        # per-step samples (events around each step, a separate region)
        "step_ms": {"median": round(float(np.median(samples)), 4),
                    "q1": round(float(np.percentile(samples, 25)), 4),
                    "q3": round(float(np.percentile(samples, 75)), 4),
                    "min": round(samples[0], 4), "max": round(samples[-1], 4)},
        "pct_of_mfma_peak": round(100.0 * value / PEAK_TFLOPS[w.contract], 2),
        "paper_context": PAPER_CONTEXT_ATTENTION,
        "series_ms": {k: summarize(v) for k, v in series.items()},
        "series_tflops": {
            "fwd": round(4.0 * w.d * pairs / (np.median(series["fwd"]) * 1e-3) / 1e12, 3),
            "bwd": round(10.0 * w.d * pairs / (np.median(series["bwd"]) * 1e-3) / 1e12, 3),
            # the conservative count: 8d per pair, no credit for the score recompute
            "bwd_8d": round(8.0 * w.d * pairs / (np.median(series["bwd"]) * 1e-3) / 1e12, 3)},
        "env": environment(),
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
                           "traffic": traffic_for(dom, w.name),
                           "algorithmic_per_launch": amount}
        if unit == "flop" and not args.no_mfma_probe:
            # the same fraction against what the matrix cores sustain at the
            # running clock (the library's MFMA probe, no memory traffic)
            kind = mfma_kind(dom)
            measured = mg.mg_mfma_peak(kind, MFMA_PROBE_ITERS[kind])
            out["roofline"]["measured_peak"] = round(measured, 2)
            out["roofline"]["measured_peak_kind"] = kind
            out["roofline"]["frac_of_measured"] = round(ach / measured, 4)
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


def summarize(samples):
    """Median, quartiles, extremes and the raw samples (ms) of one series."""
    import numpy as np
    a = np.asarray(samples, dtype=np.float64)
    return {"median": round(float(np.median(a)), 4),
            "q1": round(float(np.percentile(a, 25)), 4),
            "q3": round(float(np.percentile(a, 75)), 4),
            "min": round(float(a.min()), 4), "max": round(float(a.max()), 4),
            "samples": [round(float(v), 4) for v in samples]}


def warm_up(step, args, torch):
    """Run the W requested warmup steps, then more untimed steps until
    --warmup-ms of wall time has passed (the GPU's clock ramp under sustained
    load), synchronizing every few steps.  Returns (steps run, ms)."""
    t0 = time.perf_counter()
    n = 0
    for _ in range(args.warmup):
        step()
        n += 1
    torch.cuda.synchronize()
    while (time.perf_counter() - t0) * 1e3 < args.warmup_ms and n < 100000:
        for _ in range(8):
            step()
            n += 1
        torch.cuda.synchronize()
    return n, (time.perf_counter() - t0) * 1e3


def environment():
    """GPU name, HIP/torch versions, the source revision and the GPU clocks
    (each null when unavailable).  Nothing here starts a child process: the
    revision is read from .git when the tree has one, else it is the digest
    of the kernel sources, and the clocks come from the driver's sysfs
    files."""
    import torch
    return {"gpu": torch.cuda.get_device_name(0), "hip": torch.version.hip,
            "torch": torch.__version__, "git_revision": source_revision(),
            "clocks": gpu_clocks(torch)}


def source_revision():
    """'git:<commit>' from .git/HEAD (a loose or packed ref, or a detached
    commit), else 'src-sha256:<digest of the kernel sources>' for a copy of
    the tree without its history."""
    git = os.path.join(ROOT, ".git")
    try:
        with open(os.path.join(git, "HEAD")) as f:
            head = f.read().strip()
        if head.startswith("ref: "):
            ref = head[5:]
            path = os.path.join(git, ref)
            if os.path.isfile(path):
                with open(path) as f:
                    return "git:" + f.read().strip()[:12]
            with open(os.path.join(git, "packed-refs")) as f:
                for line in f:
                    parts = line.split()
                    if len(parts) == 2 and parts[1] == ref:
                        return "git:" + parts[0][:12]
        elif head:
            return "git:" + head[:12]
    except OSError:
        pass
    return "src-sha256:" + kernel_source_digest()[:16]


def gpu_clocks(torch):
    """The amdgpu driver's clock levels (pp_dpm_sclk, pp_dpm_mclk,
    pp_dpm_fclk: the active level ends in '*') for the card at device 0's
    PCI address when torch reports it, else for every card listed; keyed by
    PCI address.  None when no such file is readable."""
    import glob
    import re
    want = None
    try:
        pr = torch.cuda.get_device_properties(0)
        bus, dev = getattr(pr, "pci_bus_id", None), getattr(pr, "pci_device_id", None)
        if bus is not None and dev is not None:
            want = "%04x:%02x:%02x" % (getattr(pr, "pci_domain_id", 0) or 0, bus, dev)
    except (RuntimeError, AttributeError, TypeError):
        pass
    out = {}
    for card in sorted(glob.glob("/sys/class/drm/card*")):
        if not re.search(r"card\d+$", card):
            continue
        dev_dir = os.path.join(card, "device")
        addr = os.path.basename(os.path.realpath(dev_dir))
        if want is not None and not addr.startswith(want):
            continue
        ent = {}
        for name in ("sclk", "mclk", "fclk"):
            try:
                with open(os.path.join(dev_dir, "pp_dpm_" + name)) as f:
                    levels = [l.strip() for l in f if l.strip()]
            except OSError:
                continue
            active = [l for l in levels if l.endswith("*")]
            ent[name] = active[0] if active else None
            ent[name + "_levels"] = levels
        if ent:
            out[addr] = ent
    return out or None


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


# ------------------------------------------------- convolution derivatives --
CONV_WORKLOAD = "resnet50_conv_bwd_b4_224_f32"
CONV_METRIC = ("ResNet-50 convolution derivatives TFLOP/s (data + filter gradients of all "
               "53 layers, batch 4, 224x224, strict f32)")


def conv_main(args):
    """One step = the data gradient (every layer but the first) and the
    filter gradient of each of ResNet-50's 53 convolutions, in backward
    order, on resident inputs.  The step's launches are captured once into a
    HIP graph and replayed (105 host calls per step would otherwise leave
    the GPU waiting on the host); every replay's results are checked against
    the eager step's.  Credited work: 2*N*P*Q*K*R*S*C flop per derivative."""
    import numpy as np
    import torch
    import paper_2608_01563_amd as mg
    from workloads.conv import layer_inputs, resnet50_layers

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layers = resnet50_layers()
    bufs = []
    for i, L in enumerate(layers):
        x = layer_inputs(L, seed=i)
        X, W, dY = (torch.from_numpy(a.copy()).to(dev) for a in (x.X, x.W, x.dY))
        dX = torch.empty_like(X) if L.input_grad else None
        dW = torch.empty_like(W)
        need = mg.mg_conv2d_bwd_filter_workspace_bytes(X.shape, W.shape, x.stride, x.pad)
        need_x = mg.mg_conv2d_bwd_data_workspace_bytes(X.shape, W.shape, x.stride, x.pad)
        need_b = mg.mg_conv2d_bwd_workspace_bytes(X.shape, W.shape, x.stride, x.pad)
        ws = torch.empty(max(need, need_x, need_b, 256), dtype=torch.uint8, device=dev)
        bufs.append((L, x, X, W, dY, dX, dW, ws, need, need_x))

    def step():
        # both derivatives in one call per layer; the first layer's input
        # (the image) takes no gradient
        for L, x, X, W, dY, dX, dW, ws, _, _ in reversed(bufs):
            if dX is not None:
                mg.mg_conv2d_bwd(X, W, dY, dX, dW, stride=x.stride, pad=x.pad, workspace=ws)
            else:
                mg.mg_conv2d_bwd_filter(X, dY, dW, stride=x.stride, pad=x.pad, workspace=ws)

    def outputs():
        return [(b[5].clone() if b[5] is not None else None, b[6].clone()) for b in bufs]

    warm = warm_up(step, args, torch)
    eager = outputs()

    # eager step time (host launch bound) for reference
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    eager_ms = (time.perf_counter() - t0) * 1e3 / args.steps

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, capture_error_mode="relaxed"):
        step()
    torch.cuda.synchronize()
    for b in bufs:                      # clear, so replays must rewrite every output
        if b[5] is not None:
            b[5].fill_(float("nan"))
        b[6].fill_(float("nan"))
    mismatches = 0
    for _ in range(3):
        graph.replay()
        torch.cuda.synchronize()
        mismatches += sum(int(not torch.equal(a[1], b[6])) +
                          int(a[0] is not None and not torch.equal(a[0], b[5]))
                          for a, b in zip(eager, bufs))
    if mismatches:
        raise RuntimeError("graph replay differs from the eager step (%d tensors)" % mismatches)

    stream = torch.cuda.current_stream()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    stops = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        starts[k].record(stream)
        graph.replay()
        stops[k].record(stream)
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    samples_raw = [a.elapsed_time(b) for a, b in zip(starts, stops)]   # in timing order
    samples = sorted(samples_raw)

    flops = sum(L.flops() * (2 if L.input_grad else 1) for L in layers)
    value = flops / (ms_per_step * 1e-3) / 1e12

    # per-kernel durations: eager steps with the library's per-launch events
    kernels = {}
    if not args.no_kernel_events:
        mg.mg_profile_reset()
        mg.mg_profile_enable(True)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        mg.mg_profile_enable(False)
        kernels = mg.mg_profile_collect()
    work = {"conv_bwd_f32": (sum(2 * L.flops() for L in layers if L.input_grad), "flop"),
            "conv_bwd_reduce_f32": (sum(b[8] + b[9] + 4.0 * b[0].K * b[0].R * b[0].S * b[0].C *
                                        (b[8] > 0) + 4.0 * b[0].N * b[0].H * b[0].W * b[0].C *
                                        (b[9] > 0) for b in bufs if b[0].input_grad and
                                        b[8] + b[9] > 0), "byte"),
            "conv_dgrad_f32": (sum(L.flops() for L in layers if L.input_grad), "flop"),
            "conv_wgrad_f32": (sum(L.flops() for L in layers if not L.input_grad), "flop"),
            # each reads every split's partials and writes the output once
            "conv_wgrad_reduce_f32": (sum(b[8] + 4.0 * b[0].K * b[0].R * b[0].S * b[0].C
                                          for b in bufs if b[8] > 0 and not b[0].input_grad),
                                      "byte"),
            "conv_dgrad_reduce_f32": (sum(b[9] + 4.0 * b[0].N * b[0].H * b[0].W * b[0].C
                                          for b in bufs if b[9] > 0 and b[0].input_grad),
                                      "byte")}
    out = {
        "metric": CONV_METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": warm[0],
        "warmup_ms": round(warm[1], 1),
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": CONV_WORKLOAD, "layers": len(layers), "batch": 4,
                   "image": 224, "layout": "NHWC / KRSC", "credited_gflop_per_step": flops / 1e9,
                   "launch": "HIP graph of the whole step"},
        "step_ms": {"median": round(float(np.median(samples)), 4),
                    "min": round(samples[0], 4), "max": round(samples[-1], 4)},
        "eager_ms_per_step": round(eager_ms, 4),
        "paper_context": PAPER_CONTEXT_CONV,
        "pct_of_mfma_peak": round(100.0 * value / F32_MFMA_PEAK, 2),
        "series_ms": {"step": summarize(samples_raw)},
        "env": environment(),
    }
    if kernels:
        per = {}
        for name, (n, total) in kernels.items():
            amount, unit = work[name]
            per_step_ms = total / args.steps
            rate = amount / (per_step_ms * 1e-3) / (1e12 if unit == "flop" else 1e9)
            per[name] = {"launches_per_step": n // args.steps, "ms_per_step": round(per_step_ms, 4),
                         "achieved": round(rate, 3),
                         "unit": "TFLOP/s" if unit == "flop" else "GB/s"}
        out["kernels"] = per
        dom = max(kernels, key=lambda k: kernels[k][1])
        n, total = kernels[dom]
        amount, unit = work[dom]
        per_launch = amount * args.steps / n
        avg_s = total / n * 1e-3
        if unit == "flop":
            ach, peak, u, bound = per_launch / avg_s / 1e12, F32_MFMA_PEAK, "TFLOP/s", "mfma"
        else:
            ach, peak, u, bound = per_launch / avg_s / 1e9, HBM_PEAK_GBS, "GB/s", "hbm"
        out["roofline"] = {"kernel": dom, "bound": bound, "achieved": round(ach, 3),
                           "peak": peak, "unit": u, "frac": round(ach / peak, 4),
                           "traffic": traffic_for(dom, CONV_WORKLOAD, conv=True),
                           "algorithmic_per_launch": per_launch,
                           "note": "averages over the step's launches of this kernel "
                                   "(one per layer, shapes differ)"}
        if unit == "flop" and not args.no_mfma_probe:
            measured = mg.mg_mfma_peak("f32", MFMA_PROBE_ITERS["f32"])
            out["roofline"]["measured_peak"] = round(measured, 2)
            out["roofline"]["measured_peak_kind"] = "f32"
            out["roofline"]["frac_of_measured"] = round(ach / measured, 4)
        out["layers_ms"] = conv_layer_times(mg, bufs, torch)
    if not args.no_cpu_baseline:
        out["cpu_baseline"], out["parity"] = conv_cpu_baseline(args, layers, bufs)
    if args.copy_calibration_mib > 0:
        nf = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(nf, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = nf * 4
    print(json.dumps(out), flush=True)


def conv_layer_times(mg, bufs, torch, reps=5):
    """Per-layer kernel time (ms) of the data and filter gradients, from the
    library's per-launch events over `reps` eager runs of each layer."""
    res = {}
    for L, x, X, W, dY, dX, dW, ws, _, _ in bufs:
        mg.mg_profile_reset()
        mg.mg_profile_enable(True)
        for _ in range(reps):
            if dX is not None:
                mg.mg_conv2d_bwd(X, W, dY, dX, dW, stride=x.stride, pad=x.pad, workspace=ws)
            else:
                mg.mg_conv2d_bwd_filter(X, dY, dW, stride=x.stride, pad=x.pad, workspace=ws)
        torch.cuda.synchronize()
        mg.mg_profile_enable(False)
        ks = mg.mg_profile_collect()
        res[L.name] = {k.replace("conv_", "").replace("_f32", ""): round(v[1] / v[0], 4)
                       for k, v in ks.items()}
    return res


def conv_cpu_baseline(args, layers, bufs):
    """The f64 oracle on the host's cores over a bounded sample: the two
    derivatives of one mid-network layer (layer3.1.conv2, 3x3 256->256 at
    14x14), repeated until about --cpu-seconds; plus sampled parity of the
    timed run's outputs for that layer and for the first layer."""
    import numpy as np
    from oracle import oracle_num_threads
    from oracle.conv import (oracle_conv2d_bwd_data, oracle_conv2d_bwd_filter,
                             oracle_conv2d_bwd_filter_at)
    idx = [i for i, L in enumerate(layers) if L.name == "layer3.1.conv2"][0]
    L, x = bufs[idx][0], bufs[idx][1]
    times = []
    while len(times) < 3 or (sum(times) < args.cpu_seconds and len(times) < 100):
        t0 = time.perf_counter()
        rX = oracle_conv2d_bwd_data(x.dY, x.W, x.X.shape, x.stride, x.pad)
        rW = oracle_conv2d_bwd_filter(x.X, x.dY, x.W.shape, x.stride, x.pad)
        times.append(time.perf_counter() - t0)
    total = float(sum(times))
    value = 2 * L.flops() * len(times) / total / 1e12
    base = {"value": round(value, 6), "unit": "TFLOP/s", "cores": oracle_num_threads(),
            "kind": "oracle",
            "sample": "both derivatives of %s (3x3, 256->256, 14x14, batch 4), run %d times "
                      "back to back (%.1f s of CPU wall time)" % (L.name, len(times), total)}
    parity = {}
    gX = bufs[idx][5].cpu().numpy().astype(np.float64)
    gW = bufs[idx][6].cpu().numpy().astype(np.float64)
    parity[L.name + ".dX"] = float(np.max(np.abs(gX - rX)) / np.max(np.abs(rX)))
    parity[L.name + ".dW"] = float(np.max(np.abs(gW - rW)) / np.max(np.abs(rW)))
    L0, x0 = bufs[0][0], bufs[0][1]
    g0 = bufs[0][6].cpu().numpy().astype(np.float64).reshape(-1)
    iw = np.random.default_rng(0).integers(0, g0.size, 512)
    r0 = oracle_conv2d_bwd_filter_at(x0.X, x0.dY, x0.W.shape, iw, x0.stride, x0.pad)
    parity[L0.name + ".dW_sampled"] = float(np.max(np.abs(g0[iw] - r0)) / np.max(np.abs(g0)))
    parity["tolerance"] = 1e-4
    parity["pass"] = all(v <= 1e-4 for k, v in parity.items() if k not in ("tolerance",))
    return base, parity


if __name__ == "__main__":
    main()
