#!/usr/bin/env python3
"""Throughput of one SMoES MoE layer forward on one MI355X.

One step = one smoes_moe_forward call over one synthetic batch: router GEMM,
softmax and top-k; Gaussian modality score (with the statistics update when
the workload re-estimates them); inter-bin MI loss and its logit gradient;
expert-contiguous permutation; grouped SwiGLU expert GEMMs with shared
experts; weighted combine. Inputs are resident in HBM before timing starts.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

Prints one JSON line (the last line on stdout). `value` is tokens/s; the
`roofline` object covers the stage that takes the most time, with its
algorithmic work divided by its mean duration measured with HIP events on the
launch stream inside the timed loop; `cpu_baseline` times the float64 CPU
oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tokens/sec through SMoES MoE layer fwd (+MI loss); % bf16 MFMA peak, % HBM BW"
PEAK_BF16_TFLOPS = 2500.0   # dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # fp32 vector
PEAK_HBM_GBS = 8000.0       # HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_traffic.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def stage_work(cfg, T, merged=False, fused=False):
    """Algorithmic flops and HBM bytes of every stage for T tokens. merged:
    the GEMM1 / GEMM2 stages cover the routed and the shared experts in one
    launch (the schedule with side streams); the *_shared stages are empty.
    fused (with merged: bf16 packed layers with shared experts): GEMM2 covers
    the routed experts only and GEMM2_SHARED is the shared down GEMM with the
    combine in its epilogue (no shared output to HBM); the combine is empty."""
    s = 2 if cfg.dtype == "bf16" else 4
    d, E, k, I, SI = cfg.d, cfg.E, cfg.k, cfg.inter, cfg.shared_inter
    R = T * k
    upd = 2 if cfg.update_stats else 1
    w = {
        "route": dict(flops=2 * T * d * E, bytes=T * d * s + E * d * 4 + T * E * 8 + T * k * 8),
        "modality": dict(flops=6 * T * d * upd, bytes=upd * T * d * s + T * 8 + T * (1 if upd > 1 else 0)),
        "mi": dict(flops=4 * T * E, bytes=T * (12 * E + 16)),
        "permute": dict(flops=0, bytes=2 * R * 4 + 2 * R * 4),
        "gemm1": dict(flops=4 * R * d * I, bytes=(E * 2 * I * d + R * d + R * I) * s),
        "gemm2": dict(flops=2 * R * I * d, bytes=(E * d * I + R * I + R * d) * s),
        "combine": dict(flops=2 * R * d, bytes=(R + (T if SI else 0) + T) * d * s + R * 8),
        "gemm1_shared": dict(flops=4 * T * d * SI, bytes=(2 * SI * d + T * d + T * SI) * s),
        "gemm2_shared": dict(flops=2 * T * SI * d, bytes=(d * SI + T * SI + T * d) * s),
    }
    if merged:
        for g in (("gemm1",) if fused else ("gemm1", "gemm2")):
            sh = w.pop(g + "_shared")
            w[g] = dict(flops=w[g]["flops"] + sh["flops"], bytes=w[g]["bytes"] + sh["bytes"])
            w[g + "_shared"] = dict(flops=0, bytes=0)
        if fused:
            w["gemm2_shared"] = dict(flops=2 * T * SI * d + 2 * R * d,
                                     bytes=(d * SI + T * SI + R * d + T * d) * s + R * 8)
            w["combine"] = dict(flops=0, bytes=0)
    return w


def source_digest(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(kernel_stage, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when it is missing, was taken on another workload, or the kernel
    source changed since it was taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("workload") != workload:
        return None
    ent = rec.get(kernel_stage)
    if not ent:
        return None
    src = os.path.join(ROOT, ent["source"])
    if not os.path.exists(src) or source_digest(src) != ent["source_sha256"]:
        return None
    return ent["bytes_per_launch"]


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, inp, n_samples, runs=3):
    """The float64 oracle, as it stands, on the first n_samples samples: one
    warm-up run, then the median of `runs` timed runs (runs=1: one run, no
    warm-up)."""
    import numpy as np
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    Ts = int(inp.sample_offsets[n_samples])
    off = inp.sample_offsets[:n_samples + 1]
    x = inp.x[:Ts]
    mid = inp.modality_id[:Ts]

    def once():
        t0 = time.perf_counter()
        st = O.GaussState.zeros(cfg.d)
        st = O.gauss_update(st, x, mid, cfg.beta)
        O.layer_forward(x, mid, off, inp.w_gate, inp.logit_bias, inp.expert_to_bin, cfg.n_bins, cfg.k,
                        inp.w13, inp.w2, inp.ws13, inp.ws2, st, update_stats=cfg.update_stats,
                        beta=cfg.beta, tau=cfg.tau)
        return time.perf_counter() - t0

    if runs > 1:
        once()  # warm-up
    dt = float(np.median([once() for _ in range(runs)]))
    affinity = len(os.sched_getaffinity(0))
    cores = min(threads, affinity)
    return {"value": Ts / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"first {n_samples} sample(s) ({Ts} tokens) of the workload: full layer forward "
                      f"(statistics, routing, MI + gradient, permutation, experts) in float64 NumPy; "
                      + (f"median of {runs} runs after one warm-up" if runs > 1 else "one run") +
                      f", {dt:.2f} s per run; "
                      f"{threads} BLAS threads, {affinity} CPUs in the affinity mask ({cpu_model()})"}


def memory_bound_rows(S, W, cfg, spec, dev_in, outs, ws, work, reps):
    """Per-call times of the memory-bound entry points with the MALL flushed
    before each call (a 1 GiB write), their algorithmic GB/s against the 8 TB/s
    peak and against a measured 1 GiB device-to-device copy; the combine is
    timed inside a single-stream layer call (its input, the routed rows, is
    written by the GEMM just before it)."""
    import numpy as np
    import torch
    dev = dev_in["x"].device
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)  # 1 GiB
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def timed(fn, flushed=True):
        fn()
        ts = []
        for _ in range(max(reps, 5)):
            if flushed:
                flush.fill_(1.0)
            ev[0].record()
            fn()
            ev[1].record()
            torch.cuda.synchronize()
            ts.append(ev[0].elapsed_time(ev[1]))
        return float(np.median(ts))

    src = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    src.fill_(2.0)
    dst = torch.empty_like(src)
    copy_ms = timed(lambda: dst.copy_(src))
    copy_gbs = 2 * (1 << 30) / (copy_ms * 1e-3) / 1e9
    del src, dst
    L = S.lib()
    T, d, E, k = cfg.T, cfg.d, cfg.E, cfg.k
    xdt = S.SMOES_BF16 if cfg.dtype == W.BF16 else S.SMOES_F32
    nr = int(L.smoes_route_workspace_size(T, d, E, xdt))
    wr = torch.empty(max(nr, 1), dtype=torch.uint8, device=dev)
    nm = int(L.smoes_modality_workspace_size(T, d))
    wm = torch.empty(nm, dtype=torch.uint8, device=dev)
    nmi = int(L.smoes_mi_workspace_size(T, E, cfg.n_batch, cfg.n_bins))
    wmi = torch.empty(nmi, dtype=torch.uint8, device=dev)
    npm = int(L.smoes_permute_workspace_size(T, E, k))
    wpm = torch.empty(npm, dtype=torch.uint8, device=dev)
    M = torch.empty((T, 2), dtype=torch.float32, device=dev)
    p = S._p
    calls = {
        "route": lambda: S._check(L.smoes_route(p(dev_in["x"]), xdt, T, d, p(dev_in["w_gate"]), p(dev_in["logit_bias"]),
                                                E, k, 0, p(outs["logits"]), p(outs["probs"]), p(outs["topk_idx"]),
                                                p(outs["topk_w"]), p(wr), nr, S._stream()), "smoes_route"),
        "modality": lambda: S._check(L.smoes_modality_score(p(dev_in["x"]), xdt, T, d, p(dev_in["modality_id"]),
                                                            p(dev_in["gauss_n"]), p(dev_in["gauss_smu"]),
                                                            p(dev_in["gauss_ssig"]), 0, cfg.beta, cfg.tau, 1e-6,
                                                            p(M), p(wm), nm, S._stream()), "smoes_modality_score"),
        "mi": lambda: S._check(L.smoes_mi_loss(p(outs["probs"]), p(M), T, E, p(dev_in["sample_offsets"]), cfg.n_batch,
                                               p(dev_in["expert_to_bin"]), cfg.n_bins, 1.0, p(outs["mi_per_sample"]),
                                               p(outs["loss"]), p(outs["dlogits"]), p(wmi), nmi, S._stream()),
                               "smoes_mi_loss"),
        "permute": lambda: S._check(L.smoes_permute(p(outs["topk_idx"]), T, E, k, p(outs["expert_offsets"]),
                                                    p(outs["perm_token"]), p(outs["perm_inv"]), None, xdt, d, None,
                                                    p(wpm), npm, S._stream()), "smoes_permute"),
    }
    rows = {"copy_ceiling": {"what": "device-to-device copy of 1 GiB (read + write), MALL flushed",
                             "ms": round(copy_ms, 5), "gbs": round(copy_gbs, 1),
                             "frac_hbm": round(copy_gbs / PEAK_HBM_GBS, 4)}}
    for name, fn in calls.items():
        ms_f = timed(fn)
        ms_w = timed(fn, flushed=False)
        # the modality score alone (update = 0) reads x once and writes M
        b = T * d * (2 if cfg.dtype == W.BF16 else 4) + 8 * T if name == "modality" else work[name]["bytes"]
        gbs = b / (ms_f * 1e-3) / 1e9
        rows[name] = {"ms": round(ms_f, 5), "ms_warm": round(ms_w, 5), "bytes": int(b), "gbs": round(gbs, 1),
                      "frac_hbm": round(gbs / PEAK_HBM_GBS, 4), "frac_copy": round(gbs / copy_gbs, 4)}
    # combine inside a single-stream layer call, MALL flushed before the call
    ci = S.STAGES.index("combine")
    cms = []
    for _ in range(max(reps, 5)):
        e = S.Events(only=ci)
        flush.fill_(1.0)
        S.moe_forward(spec, dev_in, outs, ws, events=e)
        torch.cuda.synchronize()
        cms.append(e.stage_ms(ci))
        e.close()
    c_ms = float(np.median(cms))
    gbs = work["combine"]["bytes"] / (c_ms * 1e-3) / 1e9
    rows["combine"] = {"ms": round(c_ms, 5), "bytes": int(work["combine"]["bytes"]), "gbs": round(gbs, 1),
                       "frac_hbm": round(gbs / PEAK_HBM_GBS, 4), "frac_copy": round(gbs / copy_gbs, 4),
                       "note": "inside the layer call, after the routed down GEMM wrote its input"}
    del flush
    return rows


def gemm_ceiling_rows(cfg, counts, reps):
    """The vendor GEMM (torch.matmul, hipBLASLt) at this layer's expert GEMM
    shapes, bf16 operands and float32 accumulation: a measured reference for
    the grouped expert kernels on this chip and clock. The routed rows are
    timed as one dense GEMM (an upper bound for the grouped work: no row
    gather, no ragged groups, no fused SwiGLU), and the largest expert's rows
    as one GEMM."""
    import numpy as np
    import torch
    dev = "cuda:0"
    R, d, I, SI = cfg.T * cfg.k, cfg.d, cfg.inter, cfg.shared_inter
    big = int(np.max(counts))
    shapes = {"routed_gate_up_dense": (R, 2 * I, d), "routed_down_dense": (R, d, I),
              "largest_expert_gate_up": (big, 2 * I, d), "largest_expert_down": (big, d, I)}
    if SI > 0:
        shapes["shared_gate_up"] = (cfg.T, 2 * SI, d)
        shapes["shared_down"] = (cfg.T, d, SI)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    rows = {}
    for name, (m, n, k) in shapes.items():
        if m == 0:
            continue
        a = torch.randn((m, k), device=dev, dtype=torch.bfloat16)
        b = torch.randn((k, n), device=dev, dtype=torch.bfloat16)  # contiguous right operand
        for _ in range(2):
            c = a @ b
        torch.cuda.synchronize()
        ts = []
        for _ in range(max(reps, 5)):
            ev[0].record()
            c = a @ b
            ev[1].record()
            torch.cuda.synchronize()
            ts.append(ev[0].elapsed_time(ev[1]))
        ms = float(np.median(ts))
        tf = 2.0 * m * n * k / (ms * 1e-3) / 1e12
        rows[name] = {"m": m, "n": n, "k": k, "ms": round(ms, 5), "tflops": round(tf, 1),
                      "frac_mfma": round(tf / PEAK_BF16_TFLOPS, 4)}
        del a, b, c
    torch.cuda.empty_cache()
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=None,
                    help="workload name (default: the largest single-GPU layer, large-skewed-vlm)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-samples", type=int, default=None,
                    help="samples the CPU oracle runs on (default: 1 at hidden size >= 4096, else 2)")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the rows timed beside the layer (memory-bound kernels, statistics update, "
                         "binning, GMM, attention score, training step)")
    ap.add_argument("--rowmajor-weights", action="store_true",
                    help="bf16 expert weights row-major instead of the packed fragment order")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="first run a plain device-to-device copy of this many MiB (untimed): "
                         "a known-size reference for hardware byte counters")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures the single-GPU layer only: the library runs one layer on one MI355X, "
              "with no expert parallelism or collectives; use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2604_23996_amd import smoes as S
    from paper_2604_23996_amd import workloads as W

    S.lib()  # fail loudly if the HIP library is missing
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = "cuda:0"
    cfg = W.workload(args.workload or W.BENCH_WORKLOAD)
    log(f"[bench] generating workload {cfg.name} (seed {cfg.seed})")
    inp = W.make_layer_inputs(cfg)

    def t(a):
        if a is None:
            return None
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(a).to(dev)

    act = torch.bfloat16 if cfg.dtype == W.BF16 else torch.float32
    spec = S.LayerSpec(T=cfg.T, d=cfg.d, E=cfg.E, k=cfg.k, inter=cfg.inter,
                       shared_inter=cfg.shared_inter, n_bins=cfg.n_bins, n_batch=cfg.n_batch,
                       act_dtype=S.SMOES_BF16 if cfg.dtype == W.BF16 else S.SMOES_F32,
                       tau=cfg.tau, beta=cfg.beta, update_stats=cfg.update_stats,
                       weights_packed=cfg.dtype == W.BF16 and not args.rowmajor_weights)
    dev_in = dict(x=t(inp.x), modality_id=t(inp.modality_id), sample_offsets=t(inp.sample_offsets),
                  w_gate=t(inp.w_gate), logit_bias=t(inp.logit_bias), expert_to_bin=t(inp.expert_to_bin),
                  w13=t(inp.w13), w2=t(inp.w2), ws13=t(inp.ws13), ws2=t(inp.ws2),
                  gauss_n=torch.zeros(2, device=dev), gauss_smu=torch.zeros((2, cfg.d), device=dev),
                  gauss_ssig=torch.zeros((2, cfg.d), device=dev))
    if spec.weights_packed:  # weights are stored packed (converted once, when they are loaded)
        S.pack_layer_inputs(spec, dev_in)
        torch.cuda.synchronize()
    if not cfg.update_stats:  # statistics estimated once from the batch, outside the timed call
        S.modality_score(dev_in["x"], dev_in["gauss_n"], dev_in["gauss_smu"], dev_in["gauss_ssig"],
                         dev_in["modality_id"], update=True, beta=cfg.beta, tau=cfg.tau)
    if args.copy_probe_mb > 0:
        n = args.copy_probe_mb * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    outs = S.alloc_outputs(spec, dev, act)
    ws = torch.empty(S.workspace_bytes(spec), dtype=torch.uint8, device=dev)
    streams = S.Streams()  # side streams: modality + MI, and the shared experts
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        S.moe_forward(spec, dev_in, outs, ws, streams=streams)
    torch.cuda.synchronize()
    # Stage breakdown: calls with an event pair around every stage (untimed:
    # 18 event records per call stretch the call); it names the longest stage.
    n_stage = max(args.steps // 2, 3)
    log(f"[bench] stage breakdown over {n_stage} calls")
    events = [S.Events() for _ in range(n_stage)]
    for i in range(n_stage):
        S.moe_forward(spec, dev_in, outs, ws, events=events[i], streams=streams)
    torch.cuda.synchronize()
    stage_ms = {}
    for si, name in enumerate(S.STAGES):
        stage_ms[name] = float(np.mean([ev.stage_ms(si) for ev in events]))
    for ev in events:
        ev.close()
    dom = max(S.STAGES, key=lambda n: stage_ms[n])
    # Timed region: K calls; the only events recorded are the longest stage's
    # pair, whose durations give the roofline figure of this very region.
    log(f"[bench] timing {args.steps} steps")
    dom_events = [S.Events(only=S.STAGES.index(dom)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        S.moe_forward(spec, dev_in, outs, ws, events=dom_events[i], streams=streams)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps
    value = cfg.T / (ms * 1e-3)
    dom_ms = float(np.mean([ev.stage_ms(S.STAGES.index(dom)) for ev in dom_events]))
    for ev in dom_events:
        ev.close()
    work = stage_work(cfg, cfg.T)  # one launch per GEMM part (the serial schedule)
    # the timed schedule: routed + shared per GEMM launch, or the shared down
    # GEMM with the combine in its epilogue (bf16 packed layers with shared experts)
    fused = spec.act_dtype == S.SMOES_BF16 and bool(spec.weights_packed) and cfg.shared_inter > 0
    work_m = stage_work(cfg, cfg.T, merged=True, fused=fused)
    stages = {}
    for name in S.STAGES:
        wk = work_m[name]
        if wk["flops"] == 0 and wk["bytes"] == 0:
            continue  # part of the merged GEMM launches (or of the fused combine)
        sec = stage_ms[name] * 1e-3
        stages[name] = {"ms": round(stage_ms[name], 5),
                        "tflops": round(wk["flops"] / sec / 1e12, 3) if wk["flops"] else 0.0,
                        "gbs": round(wk["bytes"] / sec / 1e9, 1)}
    sec = dom_ms * 1e-3
    work_dom = work_m[dom]
    if dom in ("gemm1", "gemm2", "route") and cfg.dtype == W.BF16:
        achieved = work_dom["flops"] / sec / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4)}
    elif dom in ("gemm1", "gemm2"):
        achieved = work_dom["flops"] / sec / 1e12
        roof = {"bound": "alu", "achieved": round(achieved, 3), "peak": PEAK_FP32_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP32_TFLOPS, 4)}
    else:
        achieved = work_dom["bytes"] / sec / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof["kernel"] = dom
    roof["kernel_ms"] = round(dom_ms, 5)  # mean over the timed calls (HIP events on its stream)
    roof["traffic"] = measured_traffic(dom, cfg.name)

    # The same stages with every stage on the caller's stream (no side
    # streams): each kernel owns the chip, so these are the kernels' own
    # rates (the layer step above overlaps the shared experts with the routed
    # path and is faster as a whole).
    log(f"[bench] serial stage breakdown over {n_stage} calls")
    ser_events = [S.Events() for _ in range(n_stage)]
    for i in range(n_stage):
        S.moe_forward(spec, dev_in, outs, ws, events=ser_events[i])
    torch.cuda.synchronize()
    stages_serial = {}
    for si, name in enumerate(S.STAGES):
        ms_i = float(np.median([ev.stage_ms(si) for ev in ser_events]))
        wk = work[name]
        stages_serial[name] = {"ms": round(ms_i, 5),
                               "tflops": round(wk["flops"] / (ms_i * 1e-3) / 1e12, 3) if wk["flops"] else 0.0,
                               "gbs": round(wk["bytes"] / (ms_i * 1e-3) / 1e9, 1)}
        if name in ("gemm1", "gemm2", "gemm1_shared", "gemm2_shared") and cfg.dtype == W.BF16:
            stages_serial[name]["frac_mfma"] = round(stages_serial[name]["tflops"] / PEAK_BF16_TFLOPS, 4)
    for ev in ser_events:
        ev.close()

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == W.BF16 else "f32", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: SMoES MoE layer, T={cfg.T} tokens "
                               f"({cfg.n_batch} samples of vision+text), d={cfg.d}, E={cfg.E} routed"
                               f" + {cfg.n_shared} shared experts, top-{cfg.k}, inter={cfg.inter}, "
                               f"{cfg.n_bins} bins",
                   "T": cfg.T, "d": cfg.d, "E": cfg.E, "k": cfg.k, "inter": cfg.inter,
                   "n_shared": cfg.n_shared, "n_bins": cfg.n_bins, "update_stats": cfg.update_stats,
                   "expert_weights": "packed" if spec.weights_packed else "row-major",
                   "parallelism": "none (1 GPU)"},
        "roofline": roof,
        "stages": stages,
        "stages_serial": stages_serial,
    }
    # Memory-bound kernels with the 256 MB MALL flushed: a 1 GiB write before
    # every timed call, each entry point called on its own (HIP events on the
    # stream it runs on), next to a plain device copy of 1 GiB (the measured
    # copy ceiling) and the 8 TB/s HBM peak.
    if not args.no_extras:
        log("[bench] memory-bound kernels, MALL flushed")
        line["memory_bound"] = memory_bound_rows(S, W, cfg, spec, dev_in, outs, ws, work, args.steps)
        # the vendor GEMM at the same shapes (reference for the expert kernels)
        log("[bench] vendor GEMM at the expert shapes")
        counts = np.diff(outs["expert_offsets"].cpu().numpy())
        line["gemm_ceiling"] = gemm_ceiling_rows(cfg, counts, args.steps)
    if not args.no_extras:
        # Gaussian statistics update (Eq. 5-7) followed by the score (Eq. 8-9) on
        # this workload's tokens: the modality stage of a layer that re-estimates
        # its statistics from the batch. Timed on its own, on copies of the state.
        T_, d_ = cfg.T, cfg.d
        g_n, g_mu, g_sig = dev_in["gauss_n"].clone(), dev_in["gauss_smu"].clone(), dev_in["gauss_ssig"].clone()
        M_u = torch.empty((T_, 2), dtype=torch.float32, device=dev)
        nws_u = int(S.lib().smoes_modality_workspace_size(T_, d_))
        ws_u = torch.empty(nws_u, dtype=torch.uint8, device=dev)
        xdt = 1 if cfg.dtype == W.BF16 else 0

        def update_call():
            S._check(S.lib().smoes_modality_score(S._p(dev_in["x"]), xdt, T_, d_, S._p(dev_in["modality_id"]),
                                                  S._p(g_n), S._p(g_mu), S._p(g_sig), 1, cfg.beta, cfg.tau, 1e-6,
                                                  S._p(M_u), S._p(ws_u), nws_u, S._stream()), "smoes_modality_score")
        for _ in range(3):
            update_call()
        ev_u = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        u_ms = []
        for _ in range(args.steps):
            ev_u[0].record()
            update_call()
            ev_u[1].record()
            torch.cuda.synchronize()
            u_ms.append(ev_u[0].elapsed_time(ev_u[1]))
        um = float(np.median(u_ms))
        u_bytes = 2 * T_ * d_ * (2 if cfg.dtype == W.BF16 else 4) + T_ + T_ * 8
        # Momentum-adaptive binning + bin-level balance loss (+ gradient, added onto
        # the MI gradient) + MSI on this step's routing: timed on its own, not part
        # of the layer step above.
        T, E = cfg.T, cfg.E
        e2b_next = torch.empty(E, dtype=torch.int32, device=dev)
        load_ema = torch.zeros((2, E), dtype=torch.float64, device=dev)
        nws = int(S.lib().smoes_binning_workspace_size(T, E, cfg.n_bins))
        bws = torch.empty(nws, dtype=torch.uint8, device=dev)
        bin_out = dict(counts=torch.empty((2, E), dtype=torch.int32, device=dev),
                       f_spec=torch.empty(E, dtype=torch.float64, device=dev),
                       loss=torch.empty(1, dtype=torch.float32, device=dev),
                       msi=torch.empty(1, dtype=torch.float32, device=dev))

        def binning_call():
            S._check(S.lib().smoes_binning(S._p(outs["probs"]), S._p(outs["topk_idx"]), S._p(dev_in["modality_id"]),
                                           T, E, cfg.k, S._p(dev_in["expert_to_bin"]), cfg.n_bins, cfg.beta,
                                           S._p(load_ema), S._p(bin_out["counts"]), S._p(bin_out["f_spec"]),
                                           S._p(e2b_next), 1e-3, S._p(bin_out["loss"]), S._p(outs["dlogits"]), 1,
                                           S._p(bin_out["msi"]), S._p(bws), bws.numel(), S._stream()), "smoes_binning")

        for _ in range(3):
            binning_call()
        b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        b0.record()
        for _ in range(args.steps):
            binning_call()
        b1.record()
        torch.cuda.synchronize()
        bin_ms = b0.elapsed_time(b1) / args.steps
        bin_bytes = T * (2 * 4 * E + 4 * cfg.k + 1)  # probs read, dlogits read+write, top-k, labels
        line["extra"] = {"gauss_update": {"what": "Gaussian statistics update from the batch (EMA-Welford, Eq. 5-7) then "
                                                  "the modality score (Eq. 8-9), one layer; x read twice",
                                          "ms": round(um, 5), "gbs": round(u_bytes / (um * 1e-3) / 1e9, 1),
                                          "frac_hbm": round(u_bytes / (um * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)},
                         "binning": {"what": "momentum-adaptive bins + bin-level load balance loss and gradient "
                                             "(added onto dlogits) + MSI, one layer, this step's routing",
                                     "ms": round(bin_ms, 5), "gbs": round(bin_bytes / (bin_ms * 1e-3) / 1e9, 1),
                                     "frac_hbm": round(bin_bytes / (bin_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}}
        # GMM estimator (K = 2 components per modality, the supplementary GMM
        # ablation's best setting): one stepwise-EM update on this batch, then the
        # score. Timed on its own, not part of the layer step above.
        K_gmm = 2
        rng_g = np.random.default_rng(cfg.seed + 200)
        gst = W.random_gmm_state(rng_g, cfg.d, K_gmm, count=1000.0, spread=0.05)
        g_n, g_smu, g_ssig = (torch.from_numpy(a).to(dev) for a in gst)
        g_M = torch.empty((cfg.T, 2), dtype=torch.float32, device=dev)
        g_nb = int(S.lib().smoes_gmm_workspace_size(cfg.T, cfg.d, K_gmm))
        g_ws = torch.empty(g_nb, dtype=torch.uint8, device=dev)
        x_code = S.SMOES_BF16 if cfg.dtype == W.BF16 else S.SMOES_F32

        def gmm_call():
            S._check(S.lib().smoes_gmm_modality_score(S._p(dev_in["x"]), x_code, cfg.T, cfg.d, K_gmm,
                                                      S._p(dev_in["modality_id"]), S._p(g_n), S._p(g_smu), S._p(g_ssig),
                                                      1, cfg.beta, cfg.tau, 1e-6, S._p(g_M), None, S._p(g_ws), g_nb,
                                                      S._stream()), "smoes_gmm_modality_score")

        for _ in range(3):
            gmm_call()
        g_times = []
        for _ in range(args.steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            gmm_call()
            e1.record()
            torch.cuda.synchronize()
            g_times.append(e0.elapsed_time(e1))
        g_ms = float(np.median(g_times))
        x_bytes = cfg.T * cfg.d * (2 if cfg.dtype == W.BF16 else 4)
        g_bytes = 3 * x_bytes + 2 * 3 * K_gmm * cfg.d * 4 * 2  # x read by the E-step, the statistics and the score; state
        line["extra"]["gmm_score"] = {
            "what": f"GMM estimator, K={K_gmm} diagonal components per modality: E-step, stepwise-EM update of the "
                    "state, mixture-likelihood score (one layer)",
            "ms": round(g_ms, 5), "tokens_per_s": round(cfg.T / (g_ms * 1e-3), 1),
            "gbs": round(g_bytes / (g_ms * 1e-3) / 1e9, 1),
            "frac_hbm": round(g_bytes / (g_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
        # Attention-accumulated score (Eq. 2-4) on the same token layout: causal
        # per-sample attention of a 16-head, d_head = 128 attention layer (the
        # backbone's hidden size 2048) with the scores as two extra value
        # channels, then the head mean and the norm-weighted update. Timed on its
        # own, not part of the layer step above.
        head_dim = 128
        n_heads = cfg.d // head_dim
        if head_dim in (64, 128):
            log("[bench] attention-accumulated score")
            ai = W.make_attention_inputs(cfg.samples, cfg.d, n_heads, n_heads, head_dim, seed=cfg.seed + 100)
            aq, ak, av, ax, axa = t(ai.q), t(ai.k), t(ai.v), t(ai.x), t(ai.x_attn)
            aoff, am = t(ai.sample_offsets), t(ai.m_in)
            ao = torch.empty((cfg.T, n_heads, head_dim), dtype=torch.bfloat16, device=dev)
            amh = torch.empty((cfg.T, n_heads, 2), dtype=torch.float32, device=dev)
            amo = torch.empty((cfg.T, 2), dtype=torch.float32, device=dev)

            def attn_call():
                S.attention_scores(aq, ak, av, aoff, am, o=ao, m_heads=amh)
                S.attn_score_update(ax, axa, amh, am, out=amo)

            for _ in range(3):
                attn_call()
            a_ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            a_att = []
            a_tot = []
            for _ in range(args.steps):
                a_ev[0].record()
                S.attention_scores(aq, ak, av, aoff, am, o=ao, m_heads=amh)
                a_ev[1].record()
                S.attn_score_update(ax, axa, amh, am, out=amo)
                a_ev[2].record()
                torch.cuda.synchronize()
                a_att.append(a_ev[0].elapsed_time(a_ev[1]))
                a_tot.append(a_ev[0].elapsed_time(a_ev[2]))
            att_ms = float(np.median(a_att))
            tot_ms = float(np.median(a_tot))
            lens = np.diff(ai.sample_offsets).astype(np.float64)
            att_flops = float(n_heads * 4 * head_dim * np.sum(lens * (lens + 1) / 2))  # causal half only
            upd_bytes = cfg.T * (2 * cfg.d * (2 if cfg.dtype == W.BF16 else 4) + n_heads * 8 + 16)
            line["extra"]["attention_score"] = {
                "what": f"causal per-sample attention ({n_heads} heads x {head_dim}) carrying the modality scores "
                        "as fp32 value channels + head mean + norm-weighted update (Eq. 2-4), one layer",
                "ms": round(tot_ms, 5), "attention_ms": round(att_ms, 5),
                "tokens_per_s": round(cfg.T / (tot_ms * 1e-3), 1),
                "attention_tflops": round(att_flops / (att_ms * 1e-3) / 1e12, 2),
                "attention_frac_mfma": round(att_flops / (att_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                "update_gbs": round(upd_bytes / ((tot_ms - att_ms) * 1e-3) / 1e9, 1) if tot_ms > att_ms else None}
        # Training step of the layer: the forward above, then the backward with a
        # synthetic upstream gradient and the MI gradient as the auxiliary logit
        # gradient (every gradient: combine weights, logits, router weight and
        # bias, routed and shared expert weights, input). Timed on its own.
        log("[bench] training step (forward + backward)")
        packed_t = None  # fp32 layers and row-major bf16 weights: the backward reads the row-major weights
        if spec.weights_packed:
            rm = {n: t(getattr(inp, n)) for n in ("w13", "w2", "ws13", "ws2")}
            packed_t = S.pack_transposed_weights(spec, rm)
            del rm
        rng_b = np.random.default_rng(cfg.seed + 300)
        g32 = rng_b.standard_normal((cfg.T, cfg.d)).astype(np.float32)
        dout = t(W.f32_to_bf16_bits(g32) if cfg.dtype == W.BF16 else g32)
        # the packed training forward keeps the experts' gate / up pre-activations for the backward
        spec_tr = dataclasses.replace(spec, save_preact=spec.weights_packed)
        ws_tr = torch.empty(S.workspace_bytes(spec_tr), dtype=torch.uint8, device=dev)
        bws_t = torch.empty(S.backward_workspace_bytes(spec_tr), dtype=torch.uint8, device=dev)
        S.moe_forward(spec_tr, dev_in, outs, ws_tr, streams=streams)
        grads = S.moe_backward(spec_tr, dev_in, outs, ws_tr, packed_t, dout, outs["dlogits"], workspace=bws_t,
                               streams=streams)
        for _ in range(3):
            S.moe_forward(spec_tr, dev_in, outs, ws_tr, streams=streams)
            S.moe_backward(spec_tr, dev_in, outs, ws_tr, packed_t, dout, outs["dlogits"], grads=grads,
                           workspace=bws_t, streams=streams)
        tr_ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        f_ms, b_ms = [], []
        for _ in range(args.steps):
            tr_ev[0].record()
            S.moe_forward(spec_tr, dev_in, outs, ws_tr, streams=streams)
            tr_ev[1].record()
            S.moe_backward(spec_tr, dev_in, outs, ws_tr, packed_t, dout, outs["dlogits"], grads=grads,
                           workspace=bws_t, streams=streams)
            tr_ev[2].record()
            torch.cuda.synchronize()
            f_ms.append(tr_ev[0].elapsed_time(tr_ev[1]))
            b_ms.append(tr_ev[1].elapsed_time(tr_ev[2]))
        fm, bm = float(np.median(f_ms)), float(np.median(b_ms))
        R = cfg.T * cfg.k
        # dgrad (dH, dX) and wgrad (dW2, dW13): 12 d inter flops per routed row and per token for the
        # shared block; the recompute of the gate / up pre-activations adds 4 more
        bwd_flops = 12.0 * cfg.d * (R * cfg.inter + cfg.T * cfg.shared_inter)
        bwd_peak = PEAK_BF16_TFLOPS if spec.weights_packed else PEAK_FP32_TFLOPS
        line["extra"]["training_step"] = {
            "what": ("forward keeping the experts' gate / up pre-activations" if spec.weights_packed
                     else "forward") + " + backward of the layer (all gradients; MI gradient added to the "
                    "logit gradient)",
            "ms": round(fm + bm, 5), "forward_ms": round(fm, 5), "backward_ms": round(bm, 5),
            "tokens_per_s": round(cfg.T / ((fm + bm) * 1e-3), 1),
            "backward_tflops": round(bwd_flops / (bm * 1e-3) / 1e12, 2),
            # the packed path's matrix cores against the dense bf16 peak; the float32
            # FMA path (fp32 layers, row-major bf16 weights) against the fp32 vector peak
            "backward_peak_tflops": bwd_peak,
            "backward_frac_peak": round(bwd_flops / (bm * 1e-3) / 1e12 / bwd_peak, 4)}
        del packed_t, grads, bws_t, ws_tr
    if not args.no_cpu_baseline:
        n_cpu = args.cpu_samples if args.cpu_samples is not None else (1 if cfg.d >= 4096 else 2)
        log(f"[bench] CPU oracle on {n_cpu} sample(s)")
        line["cpu_baseline"] = cpu_baseline(cfg, inp, min(n_cpu, cfg.n_batch), runs=1 if cfg.d >= 4096 else 3)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
