"""Benchmark of the routed-MoE layer on one MI355X.

One step = one layer forward over one batch: route -> permute -> grouped FP4
GEMM (activation quantisation, gate/up + SwiGLU, down) -> fixed-order combine,
all in the library's HIP kernels, inputs resident in HBM.

Default workload: the decode-shaped layer (T=64, H=4096, 256 routed experts
top-8 + 1 shared, I=2048), whose throughput is `value`. The 8K-token prefill
layer (same dims) is measured beside it and reported under "prefill".

Prints ONE JSON line: the decode throughput as `value`, its roofline, the
per-step breakdown, the prefill measurement and the CPU oracle baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
REPEATS = 5                    # timed regions per workload for the median and minimum
MFMA_PEAK_FP8_TFLOPS = 5000.0  # dense FP8 (the FP8 x FP4 scaled MFMA issue rate)
MFMA_PEAK_FP4_TFLOPS = 10100.0  # dense MXFP4


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# Source files each timed kernel is built from; a stored counter reading is
# only reused while these are unchanged.
KERNEL_SOURCES = {
    "s1_stream2_kernel": ["gemm_stream.hip", "gemm_common.h", "gemm_launch.h", "moe_dev.h"],
    "s1_tiled_kernel": ["gemm_tiled.hip", "gemm_tiled_body.h", "gemm_common.h", "gemm_launch.h",
                        "quant_dev.h", "moe_dev.h"],
}
PROFILES = os.path.join(ROOT, "profiles")


def sources_hash(kernel):
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2609_15627_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic(kernel, workload, fmt="e4m3"):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summaries (lines
    'traffic_bytes kernel=... workload=... bytes=... sources=...', taken with
    MXFP8 activations), or None when there is none, the activation format
    differs or the kernel's sources changed since it was taken."""
    if fmt != "e4m3":
        return None
    want = sources_hash(kernel)
    if not os.path.isdir(PROFILES):
        return None
    for name in sorted(os.listdir(PROFILES)):
        with open(os.path.join(PROFILES, name)) as fh:
            for line in fh:
                if not line.startswith("traffic_bytes "):
                    continue
                kv = dict(f.split("=", 1) for f in line.split()[1:])
                if kv.get("kernel") == kernel and kv.get("workload") == workload and \
                        kv.get("sources") == want:
                    return float(kv["bytes"])
    return None


def expert_bytes(H, I):
    """Packed FP4 codes + E8M0 scales of one expert: (W13, W2)."""
    return 2 * I * H // 2 + 2 * I * H // 32, H * I // 2 + H * I // 32


def measure(cfg, weights_np, steps, warmup, fmt, use_graph=True, fused=False):
    import torch

    import synth
    from paper_2609_15627_amd import moe

    dev = torch.device("cuda:0")
    x_np = synth.gen_x(cfg)
    x = torch.from_numpy(x_np.view(np.int16)).to(dev).view(torch.bfloat16)
    if cfg.routing == "router":  # the step starts from bf16 router weights (a1 included)
        logits = None
        wr = torch.from_numpy(synth.gen_router_weight(cfg).view(np.int16)).to(dev).view(
            torch.bfloat16)
    else:                        # the step starts from the workload's logits
        logits = torch.from_numpy(synth.gen_logits(cfg)).to(dev)
        wr = None
    # codes in the grouped GEMM's block layout, packed once at load time
    w = moe.pack_expert_weights(tuple(torch.from_numpy(a[: cfg.NE]).to(dev) for a in weights_np))
    layer = moe.MoELayer(cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.n_shared, fmt, device=dev,
                         fused=fused)
    stream = torch.cuda.current_stream()

    def fwd(events=None):
        return layer.forward(x, w, logits=logits, w_router=wr, events=events)

    for _ in range(warmup):
        fwd()
    torch.cuda.synchronize()
    variant = moe.moe_last_variant()

    def timed(step_fn, n):
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        t0.record(stream)
        for _ in range(n):
            step_fn()
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / n, time.perf_counter() - w0

    # timed region 1: K steps of the layer as one HIP graph launch each (the
    # graph holds the whole path: route, permute, grouped GEMM, combine)
    graph_ms = None
    if use_graph:
        layer.capture(x, w, logits=logits, w_router=wr)
        for _ in range(warmup):
            layer.replay()
        graph_ms, graph_wall = timed(layer.replay, steps)
    # timed region 2: K steps launched eagerly, kernel by kernel
    eager_ms, eager_wall = timed(fwd, steps)
    use_g = graph_ms is not None and graph_ms < eager_ms
    # spread of the step time in the faster launch mode: the timed region
    # (K steps, events only at its two ends) repeated; median and minimum of
    # the per-step times over the repeats (an event between single steps
    # costs more than a short step)
    one = layer.replay if use_g else fwd
    per_step = np.array([graph_ms if use_g else eager_ms] +
                        [timed(one, steps)[0] for _ in range(REPEATS - 1)])
    # per-step breakdown (separate pass: events between the steps of the layer)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(7)] for _ in range(steps)]
    for i in range(steps):
        fwd(events=ev[i])
    torch.cuda.synchronize()
    names = ["route", "permute", "quant_tiles", "gate_up", "down", "combine"]
    stage_ms = {n: float(np.mean([e[j].elapsed_time(e[j + 1]) for e in ev]))
                for j, n in enumerate(names)}

    counts = layer.perm[0].cpu().numpy()
    touched = int((counts > 0).sum())
    A = cfg.A
    w13b, w2b = expert_bytes(cfg.H, cfg.I)
    # bytes per activation element as the method moves them (e2m3: 6 bits; its
    # workspace slots hold 8, which the HBM counters see)
    eb = {"e4m3": 1 + 1 / 32, "e2m3": 0.75 + 1 / 32, "e2m1": 0.5 + 1 / 32, "bf16": 2.0}[fmt]
    xb = cfg.T * cfg.H * eb                                 # x codes + scales (bf16: x itself)
    hb = A * cfg.I * eb                                     # h codes + scales (bf16: h)
    gate_up_bytes = touched * w13b + xb + hb
    # down writes fp32 partial rows, or (fused with the combine) the bf16 output
    down_bytes = touched * w2b + hb + (cfg.T * cfg.H * 2 if layer.fused else A * cfg.H * 4)
    layer_bytes = touched * (w13b + w2b) + cfg.T * cfg.H * 2 * 2 + cfg.T * cfg.E * 4
    if wr is not None:  # router weights instead of logits read
        layer_bytes += cfg.E * cfg.H * 2
    gate_up_flops = 4.0 * cfg.H * cfg.I * A
    layer_flops = 6.0 * cfg.H * cfg.I * A
    # the reported step: the faster of the two launch modes (both run every kernel of the path)
    ms = graph_ms if use_g else eager_ms
    wall = graph_wall if use_g else eager_wall
    return dict(ms_per_step=ms, wall_s=wall, tokens_per_s=cfg.T / (ms * 1e-3), stage_ms=stage_ms,
                step_ms_median=float(np.median(per_step)), step_ms_min=float(per_step.min()),
                eager_ms_per_step=eager_ms, graph_ms_per_step=graph_ms, graph=use_g,
                touched=touched, variant=variant, fused=layer.fused, gate_up_bytes=gate_up_bytes,
                down_bytes=down_bytes, layer_bytes=layer_bytes, gate_up_flops=gate_up_flops,
                layer_flops=layer_flops)


def measure_workload(name, steps, fmt, use_graph, weights_np=None):
    """One of the other full-size workloads (the Zipf-skewed 32K prefill, the
    TP-shard shape at I=256): layer time, stage times and both rooflines of
    the whole layer (algorithmic bytes against HBM, flops against the matrix
    cores' FP8-rate and FP4 peaks)."""
    import synth
    cfg = synth.CONFIGS[name]
    log(f"measuring {name}")
    # expert e's weights depend only on (seed, e, H, I): same-dims workloads share them
    r = measure(cfg, weights_np if weights_np is not None else synth.gen_all_experts(cfg),
                steps, 2, fmt, use_graph)
    s = r["ms_per_step"] * 1e-3
    gb = r["layer_bytes"] / s / 1e9
    tf = r["layer_flops"] / s / 1e12
    return {"workload": f"{name}: T={cfg.T} H={cfg.H} E={cfg.E}+{cfg.n_shared} k={cfg.k} "
                        f"I={cfg.I}, {cfg.routing} routing",
            "tokens_per_s": r["tokens_per_s"], "ms_per_step": r["ms_per_step"],
            "step_ms_median": r["step_ms_median"], "step_ms_min": r["step_ms_min"],
            "eager_ms_per_step": r["eager_ms_per_step"],
            "graph_ms_per_step": r["graph_ms_per_step"],
            "launch": "hip_graph" if r["graph"] else "eager", "variant": r["variant"],
            "experts_touched": r["touched"], "stage_ms": r["stage_ms"],
            "down_fused_with_combine": r["fused"],
            "layer_GBps": gb, "layer_hbm_frac": gb / HBM_PEAK_GBS,
            "layer_TFLOPs": tf, "layer_frac_of_fp8_peak": tf / MFMA_PEAK_FP8_TFLOPS,
            "layer_frac_of_fp4_peak": tf / MFMA_PEAK_FP4_TFLOPS,
            "gate_up_traffic": stored_traffic("s1_tiled_kernel", name, fmt),
            "gate_up_algorithmic_bytes": r["gate_up_bytes"]}


MFMA_PEAK_BF16_TFLOPS = 2500.0  # dense bf16


def measure_bf16_contract(weights_np, steps, use_graph):
    """The BF16 contract (bf16 activations, FP4 weights expanded to bf16 in
    registers, bf16 intermediate) on the decode and 8K prefill workloads:
    layer time, and stage 1 against the HBM roofline (decode) and the dense
    bf16 matrix-core peak (prefill)."""
    import synth
    out = {}
    for name, n in (("decode", steps), ("prefill8k", max(3, steps // 10))):
        cfg = synth.CONFIGS[name]
        log(f"measuring the BF16 contract on {name}")
        r = measure(cfg, weights_np, n, 2, "bf16", use_graph)
        gu = r["stage_ms"]["gate_up"] * 1e-3
        out[name] = {"ms_per_step": r["ms_per_step"], "tokens_per_s": r["tokens_per_s"],
                     "stage_ms": r["stage_ms"], "variant": r["variant"],
                     "gate_up_GBps": r["gate_up_bytes"] / gu / 1e9,
                     "gate_up_hbm_frac": r["gate_up_bytes"] / gu / 1e9 / HBM_PEAK_GBS,
                     "gate_up_TFLOPs": r["gate_up_flops"] / gu / 1e12,
                     "gate_up_frac_of_bf16_peak": r["gate_up_flops"] / gu / 1e12
                     / MFMA_PEAK_BF16_TFLOPS}
    return out


def measure_router(cfg, steps):
    """The router front-end: fused projection + top-k (moe_router_topk) against
    the two-call path (moe_router_logits, then moe_route_topk), bf16 router
    weights N(0, 0.02) of the workload's dims."""
    import torch

    import synth
    from paper_2609_15627_amd import moe

    dev = torch.device("cuda:0")
    x = torch.from_numpy(synth.gen_x(cfg).view(np.int16)).to(dev).view(torch.bfloat16)
    rng = np.random.default_rng(7)
    wr32 = (0.02 * rng.standard_normal((cfg.E, cfg.H))).astype(np.float32)
    wr = torch.from_numpy((wr32.view(np.uint32) >> 16).astype(np.uint16).view(np.int16)).to(
        dev).view(torch.bfloat16)
    kt = cfg.k + cfg.n_shared
    ids = torch.empty((cfg.T, kt), dtype=torch.int32, device=dev)
    w = torch.empty((cfg.T, kt), dtype=torch.float32, device=dev)
    lg = torch.empty((cfg.T, cfg.E), dtype=torch.float32, device=dev)

    def fused():  # one call; with a logits buffer the library picks its path by T
        moe.moe_router_topk(x, wr, cfg.k, cfg.n_shared, logits=lg, topk_ids=ids, topk_w=w)

    def two_call():
        moe.moe_router_logits(x, wr, logits=lg)
        moe.moe_route_topk(lg, cfg.k, cfg.n_shared, ids, w)

    out = {}
    for name, fn, n in (("router_topk_ms", fused, steps),
                        ("two_call_ms", two_call, max(2, steps // 10))):
        fn()
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(n):
            fn()
        t1.record()
        torch.cuda.synchronize()
        out[name] = t0.elapsed_time(t1) / n
    nbytes = cfg.T * cfg.H * 2 + cfg.E * cfg.H * 2 + cfg.T * kt * 8
    out["path"] = "fused" if cfg.T >= 1024 else "logits kernel + routing kernel"
    out["router_topk_GBps"] = nbytes / (out["router_topk_ms"] * 1e-3) / 1e9
    out["router_topk_TFLOPs"] = 2.0 * cfg.T * cfg.H * cfg.E / (out["router_topk_ms"] * 1e-3) / 1e12
    return out


def host_cpu():
    """(threads to use, cores in this process's affinity mask, CPU model name).
    The thread count is the affinity mask's size, capped by OMP_NUM_THREADS
    when that is set (the process's share of a shared host)."""
    aff = len(os.sched_getaffinity(0))
    omp = os.environ.get("OMP_NUM_THREADS", "")
    cores = min(aff, int(omp)) if omp.isdigit() and int(omp) > 0 else aff
    model = None
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for ln in out.splitlines():
            if ln.startswith("Model name:"):
                model = ln.split(":", 1)[1].strip()
                break
    except Exception:  # lscpu missing: the model stays unknown
        pass
    return cores, aff, model


def gpu_processes():
    """Processes on the GPUs before this one starts (amd-smi process), so a
    measurement taken beside another owner of the GPU shows it: the number
    of listed processes, or None when amd-smi is missing or fails. Run
    before this process touches the GPU."""
    import shutil
    import subprocess
    # Under a profiler its preloaded library starts the GPU in every child, so
    # a child that replaces itself (a script's "#!/usr/bin/env python3") would
    # exec after GPU start-up: skip the check there, and run a Python script
    # through this interpreter rather than through its "#!" line.
    if any(k.startswith("ROCPROF") for k in os.environ):
        return None
    exe = shutil.which("amd-smi")
    if not exe:
        return None
    cmd = [exe, "process", "--json"]
    try:
        real = os.path.realpath(exe)
        with open(real, "rb") as fh:
            if fh.readline().startswith(b"#!") and real.endswith(".py"):
                cmd = [sys.executable, real, "process", "--json"]
    except OSError:
        return None
    try:
        r = subprocess.run(cmd, capture_output=True, text=True, timeout=30)
        data = json.loads(r.stdout)
    except Exception:  # no JSON or no answer: unknown
        return None
    n = 0
    for gpu in data if isinstance(data, list) else []:
        for proc in gpu.get("process_list", []):
            info = proc.get("process_info")
            if isinstance(info, dict):  # a process (the empty list is a message string)
                n += 1
    return n


def cpu_baseline(cfg, weights_np, fmt):
    """The fp64 oracle, as it is, on the whole layer of the workload (every
    token, routing included), on the whole tiny layer (router projection
    included) and on the whole TP-shard layer, BLAS threads set to the host
    cores this process may use. (The 8K and 32K prefill layers are left out:
    any token sample of them touches every expert, and the oracle expands
    each expert's weights to fp64 first, about a minute of CPU time.)"""
    import synth
    from oracle import moe as omoe
    from threadpoolctl import threadpool_limits
    cores, aff, model = host_cpu()
    x = synth.gen_x(cfg)
    logits = synth.gen_logits(cfg)
    tiny = synth.CONFIGS["tiny"]
    tin = synth.make_inputs(tiny)
    with threadpool_limits(limits=cores):
        t = time.perf_counter()
        omoe.layer(tin.x, *tin.weights, k=tiny.k, n_shared=tiny.n_shared, wr_bits=tin.wr, fmt=fmt)
        dt0 = time.perf_counter() - t
        t = time.perf_counter()
        omoe.layer(x, *weights_np, k=cfg.k, n_shared=cfg.n_shared, logits=logits, fmt=fmt)
        dt = time.perf_counter() - t
        # the TP-shard layer in full as well (I = 256: ~12 s on 8 threads)
        tp = synth.CONFIGS["tpshard"]
        tpi = synth.make_inputs(tp, lazy=True)
        t = time.perf_counter()
        omoe.layer(tpi.x, *tpi.weights, k=tp.k, n_shared=tp.n_shared, logits=tpi.logits, fmt=fmt)
        dt4 = time.perf_counter() - t
    return {"value": cfg.T / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"the whole {cfg.name} layer (all {cfg.T} tokens, {cfg.k}+{cfg.n_shared} "
                      f"experts each, routing included), {dt:.1f} s on {cores} threads",
            "seconds": dt, "cpu_model": model, "affinity_cores": aff,
            "tiny": {"tokens_per_s": tiny.T / dt0, "seconds": dt0,
                     "sample": f"the whole tiny layer (T={tiny.T}, router projection included)"},
            "tpshard": {"tokens_per_s": tp.T / dt4, "seconds": dt4,
                        "sample": f"the whole tpshard layer (all {tp.T} tokens)"}}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="decode")
    ap.add_argument("--fmt", default="e4m3", choices=["e4m3", "e2m3", "e2m1", "bf16"])
    ap.add_argument("--no-prefill", action="store_true", help="skip the 8K prefill measurement")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-router", action="store_true", help="skip the router front-end timing")
    ap.add_argument("--workloads", action=argparse.BooleanOptionalAction, default=True,
                    help="also time the skewed 32K prefill and the TP-shard workloads")
    ap.add_argument("--fp4-prefill", action=argparse.BooleanOptionalAction, default=True,
                    help="also time the 8K prefill with MXFP4 activations (the FP4-rate run)")
    ap.add_argument("--fused", action=argparse.BooleanOptionalAction, default=True,
                    help="also time the down projection fused with the combine")
    ap.add_argument("--bf16-contract", action=argparse.BooleanOptionalAction, default=True,
                    help="also time the BF16 contract (bf16 activations and intermediate)")
    ap.add_argument("--no-graph", action="store_true",
                    help="time eager launches only (default: one HIP graph launch per step)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB five times (the "
                         "reference for scaling HBM byte counters) and exit")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE {world}).", file=sys.stderr)
        sys.exit(2)

    foreign = gpu_processes()  # before this process touches the GPU
    import torch

    import synth
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
        for i in range(5):
            ev[i].record()
            dst.copy_(src)
        ev[5].record()
        torch.cuda.synchronize()
        ms = min(ev[i].elapsed_time(ev[i + 1]) for i in range(1, 5))
        print(json.dumps({"calibrate_copy_bytes": n, "copies": 5, "best_ms": ms,
                          "copy_GBps_read_plus_write": 2 * n / ms / 1e6}), flush=True)
        return
    cfg = synth.CONFIGS[args.config]
    log(f"generating weights for {cfg.name}")
    weights_np = synth.gen_all_experts(cfg.with_(E=cfg.E, n_shared=max(cfg.n_shared, 0)))
    log("measuring")
    r = measure(cfg, weights_np, args.steps, args.warmup, args.fmt, not args.no_graph)
    log(f"{cfg.name}: {r['ms_per_step']:.4f} ms/step, stages {r['stage_ms']}")
    gu_ms = r["stage_ms"]["gate_up"]
    achieved = r["gate_up_bytes"] / (gu_ms * 1e-3) / 1e9
    layer_gbs = r["layer_bytes"] / (r["ms_per_step"] * 1e-3) / 1e9
    line = {
        "metric": "MoE-layer tokens/s",
        "value": r["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"e4m3": "mxfp8 x mxfp4 (fp32 accumulate)", "e2m3": "mxfp6 x mxfp4 (fp32 accumulate)",
                  "e2m1": "mxfp4 x mxfp4 (fp32 accumulate)",
                  "bf16": "bf16 x fp4-expanded-to-bf16 (fp32 accumulate)"}[args.fmt],
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: T={cfg.T} H={cfg.H} E={cfg.E}+{cfg.n_shared} "
                               f"k={cfg.k} I={cfg.I}, FP4 e2m1 weights with E8M0 per-32 scales",
                   "global_batch": cfg.T, "act_format": args.fmt,
                   "experts_touched": r["touched"], "variant": r["variant"],
                   "down_fused_with_combine": r["fused"],
                   "launch": "hip_graph" if r["graph"] else "eager"},
        "eager_ms_per_step": r["eager_ms_per_step"],
        "graph_ms_per_step": r["graph_ms_per_step"],
        "roofline": {"kernel": "gate_up (stage 1)", "bound": "hbm", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": stored_traffic("s1_stream2_kernel", cfg.name, args.fmt),
                     "algorithmic_bytes": r["gate_up_bytes"]},
        "stage_ms": r["stage_ms"],
        "step_ms_median": r["step_ms_median"],
        "step_ms_min": r["step_ms_min"],
        "step_stats": f"median and minimum of the per-step time over {REPEATS} timed regions "
                      f"of {args.steps} steps (the first is the one `value` comes from)",
        # the whole layer against HBM: algorithmic bytes (weights of the touched
        # experts, x, out, logits) over the step time; the graded decode figure
        "layer_roofline": {"bound": "hbm", "achieved": layer_gbs, "peak": HBM_PEAK_GBS,
                           "unit": "GB/s", "frac": layer_gbs / HBM_PEAK_GBS,
                           "algorithmic_bytes": r["layer_bytes"]},
        "layer_hbm_frac": layer_gbs / HBM_PEAK_GBS,
        "gpu_processes_before": foreign,
    }
    if cfg.name == "decode":
        log("measuring the tiny layer")
        tcfg = synth.CONFIGS["tiny"]
        tr = measure(tcfg, synth.gen_all_experts(tcfg), args.steps, args.warmup, args.fmt,
                     not args.no_graph)
        line["tiny"] = {"workload": f"tiny: T={tcfg.T} H={tcfg.H} E={tcfg.E} k={tcfg.k} "
                                    f"I={tcfg.I}, bf16 router weights (router projection in the step)",
                        "us_per_step": tr["ms_per_step"] * 1e3,
                        "us_per_step_median": tr["step_ms_median"] * 1e3,
                        "us_per_step_min": tr["step_ms_min"] * 1e3,
                        "launch": "hip_graph" if tr["graph"] else "eager",
                        "eager_us_per_step": tr["eager_ms_per_step"] * 1e3,
                        "tokens_per_s": tr["tokens_per_s"], "stage_ms": tr["stage_ms"]}
    if not args.no_prefill and cfg.name == "decode":
        pcfg = synth.CONFIGS["prefill8k"]
        log("measuring prefill8k")
        p = measure(pcfg, weights_np, max(3, args.steps // 10), 2, args.fmt, not args.no_graph)
        gu = p["stage_ms"]["gate_up"]
        tf = p["gate_up_flops"] / (gu * 1e-3) / 1e12
        line["prefill"] = {
            "workload": f"prefill8k: T={pcfg.T}, same dims", "tokens_per_s": p["tokens_per_s"],
            "ms_per_step": p["ms_per_step"], "eager_ms_per_step": p["eager_ms_per_step"],
            "step_ms_median": p["step_ms_median"], "step_ms_min": p["step_ms_min"],
            "graph_ms_per_step": p["graph_ms_per_step"],
            "launch": "hip_graph" if p["graph"] else "eager",
            "stage_ms": p["stage_ms"], "variant": p["variant"],
            "down_fused_with_combine": p["fused"],
            "roofline": {"kernel": "gate_up (stage 1)", "bound": "mfma", "achieved": tf,
                         "peak": MFMA_PEAK_FP8_TFLOPS, "unit": "TFLOP/s",
                         "frac": tf / MFMA_PEAK_FP8_TFLOPS,
                         "frac_of_fp4_peak": tf / MFMA_PEAK_FP4_TFLOPS,
                         "traffic": stored_traffic("s1_tiled_kernel", pcfg.name, args.fmt),
                         "algorithmic_bytes": p["gate_up_bytes"]},
            "layer_mfma_frac_of_fp4_peak": p["layer_flops"] / (p["ms_per_step"] * 1e-3) / 1e12
            / MFMA_PEAK_FP4_TFLOPS,
        }
        if args.fmt == "e4m3" and args.fp4_prefill:
            # the FP4-peak run with MXFP4 activations (both operands at the FP4 rate;
            # parity-tested against the oracle with the same activation format)
            log("measuring prefill8k with MXFP4 activations")
            q = measure(pcfg, weights_np, max(3, args.steps // 10), 2, "e2m1", not args.no_graph)
            gq = q["stage_ms"]["gate_up"]
            tq = q["gate_up_flops"] / (gq * 1e-3) / 1e12
            line["prefill"]["mxfp4_activations"] = {
                "act_format": "e2m1", "ms_per_step": q["ms_per_step"],
                "tokens_per_s": q["tokens_per_s"], "stage_ms": q["stage_ms"],
                "gate_up_TFLOPs": tq, "gate_up_frac_of_fp4_peak": tq / MFMA_PEAK_FP4_TFLOPS,
                "layer_frac_of_fp4_peak": q["layer_flops"] / (q["ms_per_step"] * 1e-3) / 1e12
                / MFMA_PEAK_FP4_TFLOPS}
            # MXFP6 activations: also at the FP4 rate, with about the MXFP8
            # error against the unquantised reading (narrower than the paper's
            # 8-bit activations all the same)
            log("measuring prefill8k with MXFP6 activations")
            q6 = measure(pcfg, weights_np, max(3, args.steps // 10), 2, "e2m3", not args.no_graph)
            g6 = q6["stage_ms"]["gate_up"]
            t6 = q6["gate_up_flops"] / (g6 * 1e-3) / 1e12
            line["prefill"]["mxfp6_activations"] = {
                "act_format": "e2m3", "ms_per_step": q6["ms_per_step"],
                "tokens_per_s": q6["tokens_per_s"], "stage_ms": q6["stage_ms"],
                "gate_up_TFLOPs": t6, "gate_up_frac_of_fp4_peak": t6 / MFMA_PEAK_FP4_TFLOPS,
                "layer_frac_of_fp4_peak": q6["layer_flops"] / (q6["ms_per_step"] * 1e-3) / 1e12
                / MFMA_PEAK_FP4_TFLOPS}
    from paper_2609_15627_amd import moe as _moe
    if args.fused and _moe.moe_fp4_grouped_gemm_combine_supported(cfg.T, cfg.H, cfg.I, cfg.NE,
                                                                  cfg.k_total, args.fmt):
        log("measuring the down projection fused with the combine")
        u = measure(cfg, weights_np, args.steps, args.warmup, args.fmt, not args.no_graph,
                    fused=True)
        line["fused_down_combine"] = {
            "ms_per_step": u["ms_per_step"], "eager_ms_per_step": u["eager_ms_per_step"],
            "graph_ms_per_step": u["graph_ms_per_step"], "stage_ms": u["stage_ms"],
            "down_combine_GBps": u["down_bytes"] / (u["stage_ms"]["down"] * 1e-3) / 1e9}
    if args.bf16_contract and cfg.name == "decode":
        line["bf16_contract"] = measure_bf16_contract(weights_np, args.steps, not args.no_graph)
    if args.workloads and cfg.name == "decode":
        line["workloads"] = {
            "skew32k": measure_workload("skew32k", 5, args.fmt, not args.no_graph, weights_np),
            "tpshard": measure_workload("tpshard", 10, args.fmt, not args.no_graph)}
    if not args.no_router and cfg.name == "decode":
        log("measuring the router front-end")
        line["router"] = {"decode": measure_router(cfg, args.steps),
                          "prefill8k": measure_router(synth.CONFIGS["prefill8k"], 20)}
    if not args.no_cpu_baseline:
        log("timing the CPU oracle")
        line["cpu_baseline"] = cpu_baseline(cfg, weights_np, args.fmt)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
