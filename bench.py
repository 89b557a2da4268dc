#!/usr/bin/env python3
"""Benchmark of the denoise loop on one MI355X.

A bench step is one whole pass of the hot path for one observation: the
prefix cross-K/V build plus the full solver loop (time conditioning, T Euler
steps of the expert, denormalisation) for the pi0-shaped bf16 expert at
batch 1 (18 layers, width 1024, 8 x 256 query heads, 1 K/V head, GeGLU 4096,
816 prefix tokens of width 2048, chunk 50 x 32, T = 10).  Inputs are seeded,
synthetic and resident in HBM before the timed region.

Prints one JSON line: chunks/s as `value`, the per-solver-step latency from
the linear fit chunk(T) = fixed + T * step over T in {1, 2, 5, 10}, the
roofline of the dominant kernel (algorithmic bytes per launch over its mean
launch time, both from a live per-launch HIP-event pass), and the CPU
oracle timed on a bounded sample on this host.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # dense bf16 MFMA
WORKLOAD = "pi0_bf16"
PROFILE_REPS = 20              # back-to-back repetitions per timed launch
LOOP_MODE = 2                  # persistent step kernel (the library's default driver)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def time_chunks_each(torch, pipe, tau, iters):
    """Per-chunk durations (ms) from a HIP event pair around every chunk on the
    stream that runs it."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
    torch.cuda.synchronize()
    for a, b in ev:
        a.record()
        pipe.build_cache()
        pipe.denoise(tau)
        b.record()
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ev]


def time_chunks(torch, pipe, tau, iters):
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(iters):
        pipe.build_cache()
        pipe.denoise(tau)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / iters


def time_build(torch, pipe, iters):
    """Mean prefix K/V build time (ms): a HIP event pair around `iters` builds."""
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(iters):
        pipe.build_cache()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / iters


def time_denoise(torch, pipe, tau, iters):
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(iters):
        pipe.denoise(tau)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / iters


def roofline_from_profile(ops, T):
    """Dominant kernel = the (kind, shape) group with the largest total time."""
    groups = {}
    for o in ops:
        key = (o["kind"], o["M"], o["N"], o["K"])
        g = groups.setdefault(key, {"n": 0, "ms": 0.0, "bytes": 0.0, "flops": 0.0})
        g["n"] += 1
        g["ms"] += o["ms"]
        g["bytes"] += o["bytes"]
        g["flops"] += o["flops"]
    breakdown = sorted(({"op": f"{k[0]} M={k[1]} N={k[2]} K={k[3]}", "launches": v["n"],
                         "mean_us": round(1000.0 * v["ms"] / v["n"], 2),
                         "GBps": round(v["bytes"] / (v["ms"] * 1e-3) / 1e9, 1),
                         "share": 0.0, "ms": v["ms"]} for k, v in groups.items()),
                       key=lambda r: -r["ms"])
    tot = sum(r["ms"] for r in breakdown)
    for r in breakdown:
        r["share"] = round(r.pop("ms") / tot, 3)
    (kind, M, N, K), g = max(groups.items(), key=lambda kv: kv[1]["ms"])
    bytes_per = g["bytes"] / g["n"]
    us_per = 1000.0 * g["ms"] / g["n"]
    achieved = bytes_per / (us_per * 1e-6) / 1e9
    total_ms = sum(o["ms"] for o in ops)
    step_bytes = sum(o["bytes"] for o in ops) / T
    return {
        "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(kind),
        "kernel": f"{kind} M={M} N={N} K={K}", "launches_per_chunk": g["n"],
        "bytes_per_launch": int(bytes_per), "launch_us": round(us_per, 3),
        "flops_per_launch": int(g["flops"] / g["n"]),
        "share_of_profiled_time": round(g["ms"] / total_ms, 3),
        "alg_bytes_per_solver_step": int(step_bytes),
        "breakdown": breakdown[:12],
    }


def measured_traffic(kernel_kind):
    """HBM-side bytes per launch of the dominant kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE record, scaled by a plain copy of known
    size; None when there is no record or the kernel source changed since."""
    if kernel_kind != "persist":
        return None
    import hashlib
    rec_path = os.path.join(ROOT, "profiles", "persist_kernel_pi0_bf16_traffic.json")
    try:
        with open(rec_path) as f:
            rec = json.load(f)
        with open(os.path.join(ROOT, rec["source"]), "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()
    except (OSError, KeyError, ValueError):
        return None
    return int(rec["traffic_bytes_per_launch"]) if sha == rec.get("source_sha256") else None


def hbm_copy_rate(torch, mib=1024, reps=10):
    """Measured HBM rate on this GPU: a device-to-device copy of `mib` MiB,
    counted as bytes read + bytes written per second (GB/s)."""
    n = mib << 18  # fp32 elements
    src = torch.empty(n, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(reps):
        dst.copy_(src)
    end.record()
    torch.cuda.synchronize()
    sec = start.elapsed_time(end) / 1000.0 / reps
    del src, dst
    torch.cuda.empty_cache()
    return round(2.0 * n * 4 / sec / 1e9, 1)


def cpu_env():
    """What the oracle runs on: logical CPUs, the affinity set, the CPU model
    and the BLAS thread pool numpy uses."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas = None
    return {"nproc": os.cpu_count(), "affinity": len(os.sched_getaffinity(0)), "cpu_model": model,
            "blas_threads": blas}


def oracle_fit(cfg, W, inp, threads=None):
    """The oracle as it stands on this host: the prefix K/V build, then the
    denoise loop at T = 1 and T = 2 (the paper's inference(T) = prefill +
    T * step fit).  Returns seconds for the build, the fixed part and one step.
    threads: limit numpy's BLAS pool (None = all)."""
    import contextlib
    import workloads as wl
    from oracle import vla_oracle as O
    ctx = contextlib.nullcontext()
    if threads is not None:
        from threadpoolctl import threadpool_limits
        ctx = threadpool_limits(limits=threads)
    with ctx:
        # untimed warm-up: starts the BLAS thread pool and touches the weights
        O.denoise(cfg, W, O.prefix_kv_build(cfg, W, inp["prefix"]), inp["noise"], inp["state"],
                  wl.uniform_schedule(1))
        t0 = time.perf_counter()
        cache = O.prefix_kv_build(cfg, W, inp["prefix"])
        t_build = time.perf_counter() - t0
        ts = {}
        for T in ((1,) if cfg.head_regression else (1, 2)):
            t0 = time.perf_counter()
            O.denoise(cfg, W, cache, inp["noise"], inp["state"], wl.uniform_schedule(T))
            ts[T] = time.perf_counter() - t0
    step = ts[2] - ts[1] if 2 in ts else ts[1]
    fixed = ts[1] - step if 2 in ts else 0.0
    return t_build, max(fixed, 0.0), step


def cpu_baseline(cfg, W, inp):
    """The oracle timed on this host's cores on a bounded sample of the
    headline workload (prefix K/V build + T = 1 and T = 2 denoise calls), all
    BLAS threads and one; a chunk is build + fixed + T_cfg * step."""
    env = cpu_env()
    b, f, st = oracle_fit(cfg, W, inp)
    chunk = b + f + cfg.n_steps * st
    b1, f1, st1 = oracle_fit(cfg, W, inp, threads=1)
    chunk1 = b1 + f1 + cfg.n_steps * st1
    return {"value": round(1.0 / chunk, 5), "unit": "chunks/s", "cores": env["blas_threads"] or env["affinity"],
            "kind": "oracle",
            "sample": f"{cfg.name} batch 1: prefix K/V build + denoise at T = 1 and T = 2 (numpy fp64), "
                      f"chunk = build + fixed + {cfg.n_steps} x step",
            "step_s": round(st, 4), "build_s": round(b, 4), "chunk_s": round(chunk, 3),
            "one_thread": {"chunks_per_s": round(1.0 / chunk1, 5), "step_s": round(st1, 4),
                           "chunk_s": round(chunk1, 3)},
            "env": env}


def cpu_baseline_all():
    """The oracle on every scope workload (tiny fp32, pi0-, SmolVLA-shaped,
    ternary W2A8, stress batch 1), one BLAS thread and all, then the stress
    workload at batch 2 (the oracle's cost grows with the batch, so larger
    batches are quoted per request): one JSON line each."""
    import workloads as wl
    env = cpu_env()
    for name, batch in (("tiny_f32", 1), ("pi0_bf16", 1), ("smolvla_bf16", 1), ("ternary_w2a8", 1),
                        ("stress_pi0", 1), ("stress_pi0", 2)):
        cfg = wl.CONFIGS[name].with_(batch=batch)
        W = wl.make_weights(cfg)
        inp = wl.make_batch(cfg, batch)
        for threads in ((None, 1) if batch == 1 else (None,)):
            b, f, st = oracle_fit(cfg, W, inp, threads)
            chunk = b + f + cfg.n_steps * st
            print(json.dumps({"cpu_oracle": name, "batch": batch, "threads": threads or env["blas_threads"],
                              "T": cfg.n_steps, "build_s": round(b, 4), "fixed_s": round(f, 4),
                              "step_s": round(st, 4), "chunk_s": round(chunk, 3),
                              "chunks_per_s": round(1.0 / chunk, 5),
                              "per_request_chunk_s": round(chunk / batch, 3), "env": env}), flush=True)


def measure_workload(torch, wl, Pipeline, name, batch, reps, variant=None):
    """Chunk time, per-step latency and per-step roofline fractions of one
    workload (default loop driver), optionally with architecture-variant
    overrides (state_token, causal_self, rope_base)."""
    import numpy as np
    cfg = wl.CONFIGS[name].with_(batch=batch, **(variant or {}))
    W = wl.make_weights(cfg)
    inp = wl.make_batch(cfg, batch)
    T = cfg.n_steps
    tau = wl.uniform_schedule(T)
    pipe = Pipeline(cfg, W, inp, loop_mode=LOOP_MODE)
    try:
        for _ in range(2):
            pipe.build_cache()
            pipe.denoise(tau)
        ms_chunk = time_chunks(torch, pipe, tau, reps)
        Ts = [1, T] if T > 1 else [1]
        ms_T = []
        for t in Ts:
            tt = wl.uniform_schedule(t)
            pipe.denoise(tt)
            ms_T.append(min(time_denoise(torch, pipe, tt, reps) for _ in range(2)))
        step_ms = (ms_T[-1] - ms_T[0]) / (T - 1) if T > 1 else ms_T[0]
        pipe.model.set_profile(5)
        pipe.denoise(tau)
        torch.cuda.synchronize()
        ops = pipe.model.profile_read()
        n_ops_1 = len(ops)
        if T > 1:   # launches of one extra solver step: a T = 1 call's count against the T call's
            pipe.denoise(wl.uniform_schedule(1))
            torch.cuda.synchronize()
            n_ops_1 = len(pipe.model.profile_read())
        pipe.model.set_profile(0)
    finally:
        pipe.close()
    launches_step = (len(ops) - n_ops_1) / (T - 1) if T > 1 else len(ops)
    step_bytes = sum(o["bytes"] for o in ops) / T
    step_flops = sum(o["flops"] for o in ops) / T
    roof = roofline_from_profile(ops, T)
    return {"workload": name, "batch": batch, "solver_steps": T, "chunk_ms": round(ms_chunk, 4),
            "step_us": round(step_ms * 1000.0, 2), "alg_bytes_per_step": int(step_bytes),
            "alg_flops_per_step": int(step_flops),
            "step_hbm_frac": round(step_bytes / (step_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "step_mfma_frac": round(step_flops / (step_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
            "dominant_kernel": roof["kernel"], "dominant_launch_us": roof["launch_us"],
            "dominant_frac_hbm": roof["frac"], "dominant_share": roof["share_of_profiled_time"],
            "launches_per_chunk": len(ops), "launches_per_step": round(launches_step, 1)}


INT8_PEAK_TOPS = 5000.0       # dense int8 MFMA


def prefill_work(bcfg, P):
    """Algorithmic work of one request's prefill: (GEMM ops, attention flops,
    weight bytes).  GEMM ops are int8 for a W2A8 backbone, bf16 flops else."""
    d, dq, dkv, F = bcfg.d_model, bcfg.d_q, bcfg.d_kv, bcfg.d_ff
    per_layer = d * (dq + 2 * dkv) + dq * d + (1 if bcfg.mlp == "gelu" else 2) * F * d + F * d
    gemm = 2.0 * P * per_layer * bcfg.n_layers
    attn = 4.0 * P * P * bcfg.n_heads * bcfg.head_dim * bcfg.n_layers
    wbytes = per_layer * bcfg.n_layers * (0.25 if bcfg.wtype == "ternary" else 2.0)
    return gemm, attn, wbytes


def measure_prefill(torch, name, reps):
    """The backbone's prefill of one request (event-timed, median of reps),
    against the matrix-core peak of its GEMMs' element type."""
    import numpy as np
    import workloads as wl
    from vla_testlib import Prefill
    bcfg = wl.BACKBONES[name]
    log(f"prefill {name}: generating weights ...")
    Wb = wl.make_backbone_weights(bcfg)
    e = wl.make_prefix_embeds(bcfg, 1)
    pre = Prefill(bcfg, Wb, e)
    try:
        for _ in range(2):
            pre.run()
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            pre.run()
            b.record()
            ts.append((a, b))
        torch.cuda.synchronize()
        ms = float(np.median([a.elapsed_time(b) for a, b in ts]))
    finally:
        pre.close()
    gemm, attn, wbytes = prefill_work(bcfg, bcfg.prefix_len)
    tern = bcfg.wtype == "ternary"
    sec = ms * 1e-3
    out = {"prefill": name, "layers": bcfg.n_layers, "prefix_len": bcfg.prefix_len, "d_model": bcfg.d_model,
           "wtype": bcfg.wtype, "ms": round(ms, 4), "gemm_ops": gemm, "attn_flops": attn,
           "weight_bytes": int(wbytes)}
    if tern:
        # int8 matrix-core ops of the W2A8 GEMMs plus the bf16 attention, each
        # against its own peak: the time the two would take at peak
        ideal = gemm / (INT8_PEAK_TOPS * 1e12) + attn / (BF16_PEAK_TFLOPS * 1e12)
        out.update({"int8_tops_if_all_time": round(gemm / sec / 1e12, 1), "mfma_frac": round(ideal / sec, 4),
                    "peak": "int8 5.0 POP/s (GEMMs) + bf16 2.5 PFLOP/s (attention)"})
    else:
        out.update({"tflops": round((gemm + attn) / sec / 1e12, 1),
                    "mfma_frac": round((gemm + attn) / sec / 1e12 / BF16_PEAK_TFLOPS, 4),
                    "peak": "bf16 2.5 PFLOP/s"})
    return out


def measure_observation(torch, reps):
    """The whole pi0-shaped observation path of one request: backbone prefill
    (816 rows), cross K/V build, denoise at T = 10 (event-timed, median)."""
    import numpy as np
    import workloads as wl
    from vla_testlib import Pipeline, Prefill
    bcfg, cfg = wl.PI0_VLM_BF16, wl.PI0_BF16
    log("observation path: generating weights ...")
    pre = Prefill(bcfg, wl.make_backbone_weights(bcfg), wl.make_prefix_embeds(bcfg, 1))
    pipe = Pipeline(cfg, wl.make_weights(cfg), wl.make_batch(cfg, 1), loop_mode=LOOP_MODE)
    tau = wl.uniform_schedule(cfg.n_steps)
    try:
        def once():
            h = pre.run()
            pipe.model.prefix_kv_build(h, 1, bcfg.prefix_len, pipe.cache, pipe.cache_bytes)
            pipe.denoise(tau)
        for _ in range(2):
            once()
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            once()
            b.record()
            ts.append((a, b))
        torch.cuda.synchronize()
        ms = float(np.median([a.elapsed_time(b) for a, b in ts]))
    finally:
        pipe.close()
        pre.close()
    return {"observation_path": "pi0: Gemma-2B-shaped prefill (816 rows) + cross K/V + 10 Euler steps",
            "ms": round(ms, 3), "observations_per_s": round(1000.0 / ms, 2)}


def ternary_ablation(iters: int = 50):
    """The paper's dot4-versus-matrix-unit question for the ternary GEMM (Sec. 4.5) on MI355X:
    the same int8 codes and packed 2-bit weights through v_mfma_i32_16x16x64_i8 and through
    v_dot4_i32_i8, for the ternary model's four projections (d 2560, F 6912) at 8 and 56 token
    rows.  Algorithmic bytes: packed weights (N K / 4) + codes (M K) + fp32 output (M N 4)."""
    import numpy as np
    import torch
    import workloads as wl
    from paper_2606_08094_amd import vla
    shapes = [("qkv", 3840, 2560), ("o", 2560, 2560), ("gate_up", 13824, 2560), ("down", 2560, 6912)]
    rng = np.random.default_rng(2606)
    for M in (8, 56):
        for name, N, K in shapes:
            q = rng.integers(-127, 128, size=(M, K), dtype=np.int8)
            r = rng.uniform(0.5, 4.0, size=M).astype(np.float32)
            wp = wl.pack_ternary(wl.random_ternary((N, K), 7 + N + K))
            qd, rd = torch.from_numpy(q).cuda(), torch.from_numpy(r).cuda()
            wd = torch.from_numpy(wp).cuda()
            sd = torch.full((N,), 0.0244, dtype=torch.float32, device="cuda")
            y0 = torch.empty((M, N), dtype=torch.float32, device="cuda")
            y1 = torch.empty_like(y0)
            us0 = vla.test_ternary_gemm(qd, rd, wd, sd, M, N, K, 0, y0, iters=iters)
            us1 = vla.test_ternary_gemm(qd, rd, wd, sd, M, N, K, 1, y1, iters=iters)
            same = bool(torch.equal(y0, y1))
            alg = N * K // 4 + M * K + 4 * M * N
            ops = 2 * M * N * K
            print(json.dumps({"ablation": "ternary_w2a8_mfma_vs_dot4", "proj": name, "M": M, "N": N, "K": K,
                              "mfma_us": round(us0, 2), "dot4_us": round(us1, 2),
                              "mfma_speedup": round(us1 / us0, 2), "outputs_identical": same,
                              "alg_bytes": alg, "mfma_hbm_frac": round(alg / (us0 * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                              "dot4_hbm_frac": round(alg / (us1 * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                              "int8_tops_mfma": round(ops / (us0 * 1e-6) / 1e12, 2),
                              "int8_tops_dot4": round(ops / (us1 * 1e-6) / 1e12, 2)}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200, help="timed chunks")
    ap.add_argument("--warmup", type=int, default=20, help="untimed chunks before the timed ones")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the T-sweep fit (every launch then runs the workload's T, so profiler "
                         "averages compare directly with the roofline launch time)")
    ap.add_argument("--workloads", action="store_true",
                    help="instead of the headline line, measure the other scope workloads (SmolVLA-shaped, "
                         "ternary W2A8, pi0 stress at batch 1/4/16) and print one JSON line each")
    ap.add_argument("--only", default="",
                    help="with --workloads: measure just this workload, as NAME:BATCH (e.g. stress_pi0:16)")
    ap.add_argument("--chunks", type=int, default=0,
                    help="with --workloads --only: just run this many chunks (prefix K/V build + denoise) of the "
                         "workload, with no timing and no per-launch events (a light target for profilers)")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="only run 5 plain device-to-device copies of this many MiB (calibrates the "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE counters against a known byte count)")
    ap.add_argument("--read-mb", type=int, default=0,
                    help="only run 5 read-only passes (a sum) over this many MiB (a second calibration of the "
                         "FETCH_SIZE counter, with no write stream beside the reads)")
    ap.add_argument("--prefill-only", default="",
                    help="with --chunks K: just run K prefills of this backbone (pi0_vlm_bf16 or bitnet_w2a8), "
                         "no timing (a light target for profilers)")
    ap.add_argument("--variant", default="",
                    help="with --workloads: comma list of architecture variants applied to every "
                         "workload: state_token, causal_self, rope (base 10000)")
    ap.add_argument("--prefill", action="store_true",
                    help="instead of the headline line, time the prefix stage: the Gemma-2B-shaped bf16 and the "
                         "BitNet-2B-shaped W2A8 backbone prefills and the whole pi0-shaped observation path, one "
                         "JSON line each")
    ap.add_argument("--cpu-baseline-all", action="store_true",
                    help="instead of the headline line, time the CPU oracle on every scope workload with one "
                         "BLAS thread and with all, one JSON line each (no GPU used)")
    ap.add_argument("--ternary-ablation", action="store_true",
                    help="instead of the headline line, time the W2A8 GEMM of the ternary model's projections "
                         "(M = 8 and 56) on the int8 MFMA kernel and on the VALU sdot4 kernel, one JSON line "
                         "per shape")
    args = ap.parse_args()
    if args.cpu_baseline_all:
        cpu_baseline_all()
        return
    if args.ternary_ablation:
        ternary_ablation()
        return
    if args.read_mb > 0:
        import torch
        x = torch.ones(args.read_mb << 18, dtype=torch.float32, device="cuda")
        tot = 0.0
        for _ in range(5):
            tot += float(x.sum())
        torch.cuda.synchronize()
        print(json.dumps({"read_mib": args.read_mb, "passes": 5, "sum": tot}))
        return
    if args.prefill_only:
        import torch
        import workloads as wl
        from vla_testlib import Prefill
        bcfg = wl.BACKBONES[args.prefill_only]
        log(f"prefill {bcfg.name}: generating weights ...")
        pre = Prefill(bcfg, wl.make_backbone_weights(bcfg), wl.make_prefix_embeds(bcfg, 1))
        for _ in range(max(1, args.chunks)):
            pre.run()
        torch.cuda.synchronize()
        pre.close()
        print(json.dumps({"prefill": bcfg.name, "runs": max(1, args.chunks)}))
        return
    if args.copy_mb > 0:
        import torch
        n = args.copy_mb << 18   # fp32 elements
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_mib": args.copy_mb, "copies": 5}))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU: the denoise loop of one "
                                   "request batch is a single-GPU workload (requests shard across GPUs "
                                   "with no exchange); run with --gpus 1"}))
        sys.exit(2)

    import numpy as np
    import torch
    import workloads as wl
    from vla_testlib import Pipeline

    if args.prefill:
        for name in ("pi0_vlm_bf16", "bitnet_w2a8"):
            print(json.dumps(measure_prefill(torch, name, 10)), flush=True)
        print(json.dumps(measure_observation(torch, 10)), flush=True)
        return
    if args.workloads:
        todo = (("smolvla_bf16", 1), ("ternary_w2a8", 1), ("stress_pi0", 1), ("stress_pi0", 4), ("stress_pi0", 16),
                ("gr00t_alt_bf16", 1), ("evo1_cross_bf16", 1))
        if args.only:
            name, _, batch = args.only.partition(":")
            todo = ((name, int(batch or 1)),)
        if args.chunks > 0 and args.only:
            name, batch = todo[0]
            cfg = wl.CONFIGS[name].with_(batch=batch)
            pipe = Pipeline(cfg, wl.make_weights(cfg), wl.make_batch(cfg, batch), loop_mode=LOOP_MODE)
            tau = wl.uniform_schedule(cfg.n_steps)
            for _ in range(args.chunks):
                pipe.build_cache()
                pipe.denoise(tau)
            torch.cuda.synchronize()
            pipe.close()
            print(json.dumps({"workload": name, "batch": batch, "chunks": args.chunks}))
            return
        variant = {}
        for v in filter(None, args.variant.split(",")):
            if v not in ("state_token", "causal_self", "rope"):
                sys.exit(f"unknown variant {v!r}")
            variant["rope_base" if v == "rope" else v] = 10000.0 if v == "rope" else True
        for name, batch in todo:
            log(f"workload {name} batch {batch} {args.variant} ...")
            r = measure_workload(torch, wl, Pipeline, name, batch, 5, variant)
            if variant:
                r["variant"] = args.variant
            print(json.dumps(r), flush=True)
        return

    cfg = wl.CONFIGS[WORKLOAD]
    log("generating weights ...")
    W = wl.make_weights(cfg)
    inp = wl.make_batch(cfg, 1)
    tau = wl.uniform_schedule(cfg.n_steps)
    pipe = Pipeline(cfg, W, inp, loop_mode=LOOP_MODE)
    log("warmup ...")
    for _ in range(args.warmup):
        pipe.build_cache()
        pipe.denoise(tau)
    torch.cuda.synchronize()
    log("timed region ...")
    ms_chunk = time_chunks(torch, pipe, tau, args.steps)
    log(f"chunk {ms_chunk * 1000:.1f} us")
    each = np.array(time_chunks_each(torch, pipe, tau, args.steps))
    log(f"per-chunk events: median {np.median(each) * 1000:.1f} us, p95 {np.percentile(each, 95) * 1000:.1f} us")

    # per-solver-step latency: linear fit of denoise time over T
    Ts = [cfg.n_steps] if args.no_sweep else [1, 2, 5, cfg.n_steps]
    ms_T = []
    for T in Ts:
        tT = wl.uniform_schedule(T)
        for _ in range(3):
            pipe.denoise(tT)
        ms_T.append(min(time_denoise(torch, pipe, tT, max(5, args.steps // 2)) for _ in range(2)))
    if len(Ts) > 1:
        slope, intercept = np.polyfit(np.array(Ts, float), np.array(ms_T), 1)
    else:
        slope, intercept = float("nan"), float("nan")
    ms_build = min(time_build(torch, pipe, 20) for _ in range(2))

    # cross-check of the per-step latency on the other driver: the same
    # launches captured in a HIP graph, slope over T in {1, 2}
    pipe.model.set_loop_mode(1)
    ms_g = []
    for T in (1, 2):
        tT = wl.uniform_schedule(T)
        for _ in range(3):
            pipe.denoise(tT)
        ms_g.append(min(time_denoise(torch, pipe, tT, 10) for _ in range(2)))
    pipe.model.set_loop_mode(LOOP_MODE)

    # live per-launch timings: launch-per-phase driver, every launch repeated
    # PROFILE_REPS times between one HIP event pair on the plan's stream
    pipe.model.set_profile(PROFILE_REPS)
    pipe.denoise(tau)
    torch.cuda.synchronize()
    ops = pipe.model.profile_read()
    pipe.model.set_profile(0)
    roof = roofline_from_profile(ops, cfg.n_steps)
    step_bytes = roof["alg_bytes_per_solver_step"]
    step_us = slope * 1000.0
    result = {
        "metric": "denoise step latency (µs) + action chunks/sec @ batch 1; % MFMA/HBM roofline",
        "value": round(1000.0 / ms_chunk, 2),
        "unit": "chunks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_chunk, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "pi0_bf16: 18 layers, width 1024, 8x256 query heads, 1 KV head, GeGLU 4096, "
                               "prefix 816 (width 2048), chunk 50x32, 10 Euler steps",
                   "batch": 1, "solver_steps": cfg.n_steps, "prefix_len": cfg.prefix_len, "chunk": cfg.n_action,
                   "parallelism": "single GPU"},
        "chunk_us_median": round(float(np.median(each)) * 1000.0, 2),
        "chunk_us_p95": round(float(np.percentile(each, 95)) * 1000.0, 2),
        "chunks_timed_each": int(len(each)),
        "denoise_step_us": None if np.isnan(step_us) else round(step_us, 2),
        "graph_driver_step_us": round((ms_g[1] - ms_g[0]) * 1000.0, 2),
        "chunk_fixed_us": None if np.isnan(intercept) else round(intercept * 1000.0, 2),
        "prefix_kv_build_us": round(ms_build * 1000.0, 2),
        "denoise_T_us": {str(T): round(v * 1000.0, 2) for T, v in zip(Ts, ms_T)},
        "step_hbm_frac": None if np.isnan(step_us) else round(step_bytes / (step_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        "roofline": roof,
    }
    pipe.close()
    # measured peaks beside the spec ones: a plain copy for HBM
    result["roofline"]["measured_hbm_copy_GBps"] = hbm_copy_rate(torch)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        result["cpu_baseline"] = cpu_baseline(cfg, W, inp)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
