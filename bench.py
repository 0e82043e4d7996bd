#!/usr/bin/env python3
"""Benchmark of one rank's SAGIPS step on one MI355X.

A step is one pass of the whole hot path over one batch: theta -> Philox ->
Kumaraswamy events (sampled inside the kernel) -> discriminator forward on the
fake and the resident real batch -> BCE -> backward to the weights and to the
events -> pathwise dx/dtheta -> per-parameter reduction dL_G/dtheta.

Default workload: 32 parameter rows x 8,192 events (262,144 fake + 262,144
real events), discriminator 2-128-128-128-1, fp32.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--gpus 1] [--workload NAME]
                  [--no-cpu-baseline] [--calibrate-copy]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"mfma_f32": 157.3e12, "mfma_bf16": 2.5e15, "hbm": 8.0e12}
# VALU issue: 256 CUs x 4 SIMDs, each issuing per 4-clock quad-cycle either two
# full-rate wave64 VALU instructions or one half of a transcendental (which
# takes two quad-cycles and pairs with nothing); 2.4 GHz peak clock.
SIMD_QUAD_CYCLES_PER_S = 256 * 4 * 2.4e9 / 4
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
VALU_FILE = os.path.join(ROOT, "profiles", "valu.json")
KERNEL_SOURCES = {
    "disc_f32_fused": ["paper_2407_00051_amd/csrc/disc_f32.hip", "paper_2407_00051_amd/csrc/device_math.hpp"],
    "bf16_fwd_chain": ["paper_2407_00051_amd/csrc/disc_bf16.hip", "paper_2407_00051_amd/csrc/device_math.hpp"],
    "bf16_bwd_chain": ["paper_2407_00051_amd/csrc/disc_bf16.hip", "paper_2407_00051_amd/csrc/device_math.hpp"],
    "bf16_wgrad": ["paper_2407_00051_amd/csrc/disc_bf16.hip", "paper_2407_00051_amd/csrc/device_math.hpp"],
    "param_grad": ["paper_2407_00051_amd/csrc/sampler.hip", "paper_2407_00051_amd/csrc/device_math.hpp"],
    "bootstrap": ["paper_2407_00051_amd/csrc/sampler.hip", "paper_2407_00051_amd/csrc/device_math.hpp"],
    "bootstrap_rows": ["paper_2407_00051_amd/csrc/sampler.hip", "paper_2407_00051_amd/csrc/device_math.hpp"],
    "gen_forward": ["paper_2407_00051_amd/csrc/generator.hip", "paper_2407_00051_amd/csrc/device_math.hpp"],
    "sample_events": ["paper_2407_00051_amd/csrc/sampler.hip", "paper_2407_00051_amd/csrc/device_math.hpp"],
}


def _code_text(src: str) -> str:
    """The source with its comments removed and whitespace runs collapsed, so
    that an edit of comments or layout does not mark a profile stale.  (The
    sources hold no string literal containing comment markers.)"""
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def source_hash(kernel: str) -> str:
    """Hash of the code (comments and layout excluded) of the files a kernel is built from."""
    h = hashlib.sha256()
    for p in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, p), encoding="utf-8") as f:
            h.update(_code_text(f.read()).encode())
    return h.hexdigest()[:16]


def mlp_flops_per_fake_event(widths) -> int:
    """Algorithmic flops of the discriminator per fake event (its real partner included).

    With S = sum in*out MACs per sample: forward 2S on the fake and on the
    real event; weight gradients 2S on each; backward signal 2S on the fake
    event (down to dL/dx) and 2(S - F*H) on the real one (it stops at the
    first layer's output).  Total 12S - 2FH."""
    S = sum(a * b for a, b in zip(widths[:-1], widths[1:]))
    return 12 * S - 2 * widths[0] * widths[1]


def read_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed counter runs, or None if the kernel changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        e = t[kernel][workload]
        if e.get("source_hash") != source_hash(kernel):
            return None
        return float(e["bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def read_valu_mix(kernel: str, workload: str):
    """Executed VALU and transcendental instructions per event from the committed counter run,
    or None if the kernel changed since."""
    try:
        with open(VALU_FILE) as f:
            e = json.load(f)[kernel][workload]
        if e.get("source_hash") != source_hash(kernel):
            return None
        return float(e["valu_per_event"]), float(e["trans_per_event"])
    except (OSError, KeyError, ValueError):
        return None


def valu_peak_events(valu: float, trans: float) -> float:
    """Events/s if every SIMD issued this instruction stream with no idle quad-cycle: one wave
    instruction serves 64 events; full-rate instructions pair two per quad-cycle, transcendentals
    take two quad-cycles each."""
    quad_cycles_per_64_events = (valu - trans) / 2 + 2 * trans
    return SIMD_QUAD_CYCLES_PER_S * 64 / quad_cycles_per_64_events


def cpu_baseline(w, inp, rows: int, events: int, min_seconds: float = 10.0):
    """The float64 oracle, as it stands, on the first `rows` parameter rows of the workload."""
    import numpy as np  # noqa: F401
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    th = inp["theta"][:rows]
    reps = 0
    t0 = time.perf_counter()
    while True:                      # repeat the sample until about min_seconds of CPU work
        if w.widths is None:
            oracle.run_step(th, events, w.fake_seed, critic="quadratic")
        else:
            real = oracle.sample(inp["theta_star"], rows * events, w.real_seed)
            oracle.run_step(th, events, w.fake_seed, inp["W"], inp["b"], real,
                            features=w.features, bf16=(w.precision == "bf16"))
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    n = rows * events
    return {"value": reps * n / dt, "unit": "events/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{rows} of {w.n_theta} parameter rows x {events} events ({n} fake + "
                      f"{n if w.widths else 0} real events), float64 numpy, {reps} repetition(s) in {dt:.1f} s"}


def cpu_baseline_bootstrap(w, n_out: int, min_seconds: float = 10.0):
    """The oracle's draw, as it stands, of n_out rows from a pool of 2 n_out events."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    pool = oracle.sample(np.asarray([w.theta_star], dtype=np.float32), 2 * n_out, w.pool_seed).astype(np.float32)
    draw = oracle.bootstrap_row_order if w.row_order else oracle.bootstrap
    reps, t0 = 0, time.perf_counter()
    while True:
        draw(pool, n_out, w.seed, reps)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    return {"value": reps * n_out / dt, "unit": "draws/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n_out} draws from a pool of {2 * n_out} events (of the workload's {w.n_out} from "
                      f"{w.n_data}), numpy, {reps} repetition(s) in {dt:.1f} s"}


def bench_bootstrap(args, w, ctx, torch):
    """Steps of the bootstrap draw: n_out rows gathered from the resident pool, a fresh draw per step."""
    dev = "cuda:0"
    pool = ctx.sample_events(torch.tensor([w.theta_star], dtype=torch.float32, device=dev), w.n_data, w.pool_seed)
    out = torch.empty((w.n_out, w.d), dtype=torch.float32, device=dev)
    it = [0]

    def step():
        ctx.bootstrap(pool, w.n_out, w.seed, it[0], out=out, row_order=w.row_order)
        it[0] += 1

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ctx.kernel_times()
    ctx.set_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ctx.set_timing(False)
    kt = ctx.kernel_times()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    name = "bootstrap_rows" if w.row_order else "bootstrap"
    launches, total_ms = kt[name]       # the row order times its five kernels as one
    avg_ms = total_ms / launches
    # algorithmic bytes of a draw: the drawn row read once and written once
    bytes_per_launch = w.n_out * 2 * w.d * 4
    achieved = bytes_per_launch / (avg_ms * 1e-3)
    roof = {"bound": "hbm", "achieved": achieved / 1e9, "peak": PEAK["hbm"] / 1e9, "unit": "GB/s",
            "frac": achieved / PEAK["hbm"], "traffic": read_traffic(name, w.name),
            "kernel": name, "kernel_avg_ms": avg_ms,
            "kernels": {k: {"launches": n, "avg_ms": t / max(n, 1)} for k, (n, t) in kt.items()}}
    line = {
        "metric": "draws/sec of the bootstrap sub-sample of the real data; % of HBM peak",
        "value": w.n_out / (ms_per_step * 1e-3), "unit": "draws/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u32",
        "data": "synthetic (pool of Philox-sampled Kumaraswamy events at theta_star)",
        "config": {"workload": w.name, "n_data": w.n_data, "d": w.d, "n_out": w.n_out,
                   "order": "ascending row" if w.row_order else "draw", "parallelism": "single GPU"},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_bootstrap(w, min(w.n_out, 1 << 20))
    ctx.close()
    print(json.dumps(line), flush=True)


def gen_flops_per_row(widths) -> int:
    """Forward flops of one generator on one noise vector: 2 * sum in*out."""
    return 2 * sum(a * b for a, b in zip(widths[:-1], widths[1:]))


def cpu_baseline_ensemble(w, W, b, n, min_seconds: float = 10.0):
    """The oracle's ensemble response (every member's forward, then the statistics), as it stands."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    M = min(w.n_members, 20)
    reps, t0 = 0, time.perf_counter()
    while True:
        th = np.stack([oracle.generator_forward([x[m] for x in W], [v[m] for v in b], n) for m in range(M)])
        oracle.ensemble_response(th)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    return {"value": reps * M * w.k / dt, "unit": "member-predictions/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{M} of the {w.n_members} members x {w.k} noise vectors, float64 numpy, "
                      f"{reps} repetition(s) in {dt:.1f} s"}


def bench_ensemble(args, w, ctx, torch):
    """Steps of the ensemble response: every member's forward on the noise batch, the
    per-vector mean and spread over members, their batch averages and the residuals."""
    from workloads import gen
    dev = "cuda:0"
    W, b = gen.generator_stack(w.widths, w.n_members, w.weight_seed)
    n = gen.noise(w.k, w.widths[0], w.noise_seed)
    Wd = [torch.tensor(x, device=dev) for x in W]
    bd = [torch.tensor(x, device=dev) for x in b]
    nd = torch.tensor(n, device=dev)
    pt = torch.tensor(w.theta_star, dtype=torch.float32, device=dev)

    def step():
        ctx.ensemble_response(Wd, bd, nd, p_true=pt)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ctx.kernel_times()
    ctx.set_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ctx.set_timing(False)
    kt = ctx.kernel_times()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    launches, total_ms = kt["gen_forward"]
    avg_ms = total_ms / launches
    flops = gen_flops_per_row(w.widths) * w.n_members * w.k
    achieved = flops / (avg_ms * 1e-3)
    roof = {"bound": "mfma", "achieved": achieved / 1e12, "peak": PEAK["mfma_f32"] / 1e12, "unit": "TFLOP/s",
            "frac": achieved / PEAK["mfma_f32"], "traffic": read_traffic("gen_forward", w.name),
            "kernel": "gen_forward", "kernel_avg_ms": avg_ms,
            "kernels": {k: {"launches": c, "avg_ms": t / max(c, 1)} for k, (c, t) in kt.items()}}
    line = {
        "metric": "member-predictions/sec of the ensemble response (p_hat, sigma, r_hat); % of fp32 MFMA peak",
        "value": w.n_members * w.k / (ms_per_step * 1e-3), "unit": "member-predictions/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (Kaiming-normal generators, N(0,1) noise)",
        "config": {"workload": w.name, "n_members": w.n_members, "k": w.k, "widths": list(w.widths),
                   "parallelism": "single GPU"},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_ensemble(w, W, b, n)
    ctx.close()
    print(json.dumps(line), flush=True)


def cpu_baseline_train(w, rows: int, min_seconds: float = 10.0):
    """The oracle's whole GAN step, as it stands, on `rows` of the k noise vectors."""
    import numpy as np
    import oracle
    from workloads import gen
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    GW, Gb = gen.generator_stack(w.g_widths, 1, w.seed + 21)
    DW, Db = gen.xavier_mlp(w.d_widths, w.seed + 2)
    state = oracle.initial_state([x[0] for x in GW], [x[0] for x in Gb], DW, Db)
    N = rows * w.events_per_theta
    pool = oracle.sample(np.asarray([w.theta_star]), 2 * N, w.seed + 1)
    rng = np.random.default_rng(w.seed + 22)
    reps, t0 = 0, time.perf_counter()
    while True:
        r = oracle.gan_step(state, rng.standard_normal((rows, 6)), pool, reps + 1, w.events_per_theta,
                            w.seed, w.seed + 5)
        state = r["state"]
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    return {"value": reps * N / dt, "unit": "events/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{rows} of {w.k} parameter samples x {w.events_per_theta} events per step ({N} fake + {N} "
                      f"bootstrapped reference events), float64 numpy, {reps} step(s) in {dt:.1f} s"}


def bench_train(args, w, ctx, torch, sg):
    """Steps of GAN training at the paper's shape: generator forward, bootstrap of the
    reference batch, the fused discriminator step, generator backward, Adam on both."""
    import numpy as np
    from paper_2407_00051_amd.gan import GanLoop
    from workloads import gen
    dev = "cuda:0"
    N = w.n_events
    ts = torch.tensor([w.theta_star], dtype=torch.float32, device=dev)
    pool = ctx.sample_events(ts, 2 * N, w.seed + 1)
    GW, Gb = gen.generator_stack(w.g_widths, 1, w.seed + 21)
    DW, Db = gen.xavier_mlp(w.d_widths, w.seed + 2)
    loop = GanLoop(ctx, [torch.tensor(x[0], device=dev) for x in GW], [torch.tensor(x[0], device=dev) for x in Gb],
                   [torch.tensor(x, device=dev) for x in DW], [torch.tensor(x, device=dev) for x in Db], pool,
                   w.k, w.events_per_theta, fake_seed=w.seed, boot_seed=w.seed + 5)
    rng = np.random.default_rng(w.seed + 22)
    noise = torch.tensor(rng.standard_normal((args.warmup + args.steps, w.k, w.g_widths[0])).astype(np.float32),
                         device=dev)                                    # resident before timing
    for i in range(args.warmup):
        loop.step(noise[i])
    torch.cuda.synchronize()
    ctx.kernel_times()
    ctx.set_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        loop.step(noise[args.warmup + i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ctx.set_timing(False)
    kt = ctx.kernel_times()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    launches, total_ms = kt["disc_f32_fused"]
    avg_ms = total_ms / launches
    flops = mlp_flops_per_fake_event(w.d_widths) * N
    achieved = flops / (avg_ms * 1e-3)
    g_flops = 4 * gen_flops_per_row(w.g_widths) * w.k      # forward, recomputed forward, backward (2x)
    roof = {"bound": "mfma", "achieved": achieved / 1e12, "peak": PEAK["mfma_f32"] / 1e12, "unit": "TFLOP/s",
            "frac": achieved / PEAK["mfma_f32"], "traffic": read_traffic("disc_f32_fused", w.name),
            "step_mfma_frac": (flops + g_flops) / (ms_per_step * 1e-3) / PEAK["mfma_f32"],
            "kernel": "disc_f32_fused", "kernel_avg_ms": avg_ms,
            "kernels": {k: {"launches": c, "avg_ms": t / max(c, 1)} for k, (c, t) in kt.items()}}
    line = {
        "metric": "events/sec per GAN training step (generator, bootstrap, discriminator, backward, Adam); "
                  "% of fp32 MFMA peak",
        "value": N / (ms_per_step * 1e-3), "unit": "events/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (Kumaraswamy reference pool at theta*, Kaiming/Xavier-initialised networks, N(0,1) noise)",
        "config": {"workload": w.name, "k": w.k, "events_per_theta": w.events_per_theta, "fake_events": N,
                   "real_events": N, "pool_events": 2 * N, "g_widths": list(w.g_widths),
                   "d_widths": list(w.d_widths), "features": "proxy2", "parallelism": "single GPU"},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_train(w, min(args.cpu_rows, w.k))
    ctx.close()
    print(json.dumps(line), flush=True)


def bench_sample(args, w, ctx, torch):
    """Steps of the stand-alone sampler on the stress configuration: theta -> Philox ->
    Kumaraswamy events written to HBM ([N][d] fp32), the path that feeds a buffered
    discriminator."""
    from workloads import gen
    dev = "cuda:0"
    inp = gen.make_inputs(w)
    theta = torch.tensor(inp["theta"], device=dev)
    N = w.n_events
    x = torch.empty((N, w.d), dtype=torch.float32, device=dev)

    def step():
        ctx.sample_events(theta, w.events_per_theta, w.fake_seed, out=x)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ctx.kernel_times()
    ctx.set_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ctx.set_timing(False)
    kt = ctx.kernel_times()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    launches, total_ms = kt["sample_events"]
    avg_ms = total_ms / launches
    bytes_per_launch = N * w.d * 4 + w.n_theta * 2 * w.d * 4     # events written, theta read
    achieved = bytes_per_launch / (avg_ms * 1e-3)
    roof = {"bound": "hbm", "achieved": achieved / 1e9, "peak": PEAK["hbm"] / 1e9, "unit": "GB/s",
            "frac": achieved / PEAK["hbm"], "traffic": read_traffic("sample_events", "stress_sample"),
            "kernel": "sample_events", "kernel_avg_ms": avg_ms,
            "kernels": {k: {"launches": c, "avg_ms": t / max(c, 1)} for k, (c, t) in kt.items()}}
    line = {
        "metric": "events/sec of the stand-alone sampler (theta -> Philox -> Kumaraswamy events in HBM); "
                  "% of HBM peak",
        "value": N / (ms_per_step * 1e-3), "unit": "events/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic (seeded theta, Philox-sampled events)",
        "config": {"workload": "stress_sample", "n_theta": w.n_theta, "events_per_theta": w.events_per_theta,
                   "events": N, "d": w.d, "parallelism": "single GPU"},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        import numpy as np
        import oracle
        try:
            from threadpoolctl import threadpool_info
            threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        except Exception:
            threads = os.cpu_count()
        n = 1 << 20
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.sample(np.asarray(inp["theta"][:1], dtype=np.float64), n, w.fake_seed, counter_base=reps * n)
            reps += 1
            dt = time.perf_counter() - t0
            if dt >= 10.0:
                break
        line["cpu_baseline"] = {"value": reps * n / dt, "unit": "events/s", "cores": int(threads), "kind": "oracle",
                                "sample": f"1 of {w.n_theta} parameter rows x {n} events per repetition, float64 "
                                          f"numpy, {reps} repetition(s) in {dt:.1f} s"}
    ctx.close()
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="small")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=32)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run one 1 GiB device copy (for counter calibration runs)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only: --gpus {args.gpus} / WORLD_SIZE {world} is not supported "
              "(the multi-GPU exchange of the paper is not part of this library)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2407_00051_amd as sg
    from workloads import gen, get

    w = get("stress" if args.workload == "stress_sample" else args.workload)
    torch.cuda.set_device(0)
    ctx = sg.Context(0)
    dev = "cuda:0"
    if args.calibrate_copy:
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        a.fill_(1.0)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    if args.workload == "stress_sample":
        return bench_sample(args, w, ctx, torch)
    if hasattr(w, "n_data"):
        return bench_bootstrap(args, w, ctx, torch)
    if hasattr(w, "n_members"):
        return bench_ensemble(args, w, ctx, torch)
    if hasattr(w, "g_widths"):
        return bench_train(args, w, ctx, torch, sg)
    inp = gen.make_inputs(w)
    theta = torch.tensor(inp["theta"], device=dev)
    theta_star = torch.tensor(inp["theta_star"], device=dev)
    N = w.n_events

    if w.widths is not None:
        W = [torch.tensor(m, device=dev) for m in inp["W"]]
        bias = [torch.tensor(v, device=dev) for v in inp["b"]]
        real = ctx.sample_events(theta_star, N, w.real_seed)          # resident real batch (untimed)
        f32 = dict(dtype=torch.float32, device=dev)
        outs = {"logits_fake": torch.empty(N, **f32), "logits_real": torch.empty(N, **f32),
                "loss_d": torch.empty(1, **f32), "loss_g": torch.empty(1, **f32),
                "dW": [torch.empty_like(m) for m in W], "db": [torch.empty_like(v) for v in bias],
                "dLg_dx": torch.empty((N, w.d), **f32), "dLg_dtheta": torch.empty((w.n_theta, 2 * w.d), **f32)}
        src = dict(theta=theta, events_per_theta=w.events_per_theta, seed=w.fake_seed)
        prec = sg.BF16 if w.precision == "bf16" else sg.F32
        feats = {"identity": sg.FEAT_IDENTITY, "hd8": sg.FEAT_HD8, "proxy2": sg.FEAT_PROXY2}[w.features]

        def step():
            ctx.disc_fwd_bwd(W, bias, real, fake_source=src, outputs=outs, precision=prec, features=feats)

        if prec == sg.F32:
            dominant = "disc_f32_fused"
            flops_per_launch = mlp_flops_per_fake_event(w.widths) * N
        else:
            # The bf16 step runs three kinds of launches per chunk of rows: the forward
            # chain, the backward chain and one weight-gradient product per hidden layer.
            # Each kind carries NH hidden products of 2 H^2 flops per row over the fake and
            # the real batch per step; the dominant kind is chosen after timing.
            dominant = None
            H, NH = w.widths[1], len(w.widths) - 3
            flops_per_step_kind = NH * 2 * H * H * (2 * N)
            flops_per_launch = None
        bound, unit, peak = "mfma", "TFLOP/s", PEAK["mfma_f32" if prec == sg.F32 else "mfma_bf16"]
        dtype = "f32" if prec == sg.F32 else "bf16"
    else:
        g = torch.empty((w.n_theta, 2 * w.d), dtype=torch.float32, device=dev)
        loss = torch.empty(1, dtype=torch.float32, device=dev)

        def step():
            ctx.param_grad(theta, w.events_per_theta, w.fake_seed, out=g, loss_out=loss)

        dominant = "param_grad"
        flops_per_launch = None
        bound, unit, peak = "alu", "Gevents/s", None
        dtype = "f32"

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ctx.kernel_times()                      # drop warm-up records
    ctx.set_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ctx.set_timing(False)
    kt = ctx.kernel_times()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = N / (ms_per_step * 1e-3)

    bytes_per_launch = None
    if dominant is None:
        kinds = [k for k in ("bf16_fwd_chain", "bf16_bwd_chain", "bf16_wgrad") if k in kt]
        dominant = max(kinds, key=lambda k: kt[k][1])
        launches_per_step = kt[dominant][0] / args.steps
        if dominant == "bf16_wgrad":
            # streams its two operands (bf16 rows of H) and e_D once per launch and
            # writes one H x H (+ H) fp32 partial per row slice: bound by HBM
            rows = 2 * N / launches_per_step * NH
            slices = max(1, torch.cuda.get_device_properties(0).multi_processor_count // ((H // 256) ** 2))
            bytes_per_launch = rows * (2 * H * 2 + 4) + slices * (H * H + H) * 4
            bound, unit, peak = "hbm", "GB/s", PEAK["hbm"]
        else:
            flops_per_launch = flops_per_step_kind / launches_per_step
    launches, total_ms = kt.get(dominant, (0, 0.0))
    if launches == 0:
        raise RuntimeError(f"no timed launches of {dominant}")
    avg_ms = total_ms / launches
    if bytes_per_launch is not None:
        achieved = bytes_per_launch / (avg_ms * 1e-3)
        roof = {"bound": bound, "achieved": achieved / 1e9, "peak": peak / 1e9, "unit": unit,
                "frac": achieved / peak}
    elif flops_per_launch is not None:
        achieved = flops_per_launch / (avg_ms * 1e-3)
        roof = {"bound": bound, "achieved": achieved / 1e12, "peak": peak / 1e12, "unit": unit,
                "frac": achieved / peak}
    else:
        achieved = N / (avg_ms * 1e-3)
        mix = read_valu_mix(dominant, w.name)
        peak_ev = valu_peak_events(*mix) if mix else None
        roof = {"bound": bound, "achieved": achieved / 1e9, "peak": peak_ev / 1e9 if mix else None, "unit": unit,
                "frac": achieved / peak_ev if mix else None,
                "valu_per_event": mix[0] if mix else None, "trans_per_event": mix[1] if mix else None}
    if w.widths is not None:
        mpeak = PEAK["mfma_f32" if w.precision == "f32" else "mfma_bf16"]
        roof["step_mfma_frac"] = mlp_flops_per_fake_event(w.widths) * N / (ms_per_step * 1e-3) / mpeak
    tr = read_traffic(dominant, w.name)
    roof["traffic"] = tr
    roof["kernel"] = dominant
    roof["kernel_avg_ms"] = avg_ms
    roof["kernels"] = {k: {"launches": n, "avg_ms": t / max(n, 1)} for k, (n, t) in kt.items()}

    line = {
        "metric": "events/sec per sample->discriminate->backward step; % of HBM / MFMA peak",
        "value": value, "unit": "events/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dtype, "data": "synthetic (seeded theta, Philox-sampled events, Xavier-initialised weights)",
        "config": {"workload": w.name, "n_theta": w.n_theta, "events_per_theta": w.events_per_theta,
                   "fake_events": N, "real_events": N if w.widths else 0,
                   "widths": list(w.widths) if w.widths else None, "precision": w.precision,
                   "features": w.features, "parallelism": "single GPU"},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        ev = w.events_per_theta if w.widths is not None else min(w.events_per_theta, 1 << 20)
        line["cpu_baseline"] = cpu_baseline(w, inp, min(args.cpu_rows, w.n_theta), ev)
    ctx.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
