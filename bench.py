#!/usr/bin/env python3
"""Benchmark of one rank's SAGIPS step on one MI355X.

A step is one pass of the whole hot path over one batch: theta -> Philox ->
Kumaraswamy events (sampled inside the kernels) -> discriminator forward on
the fake and the resident real batch -> BCE -> backward to the weights and to
the events -> pathwise dx/dtheta -> per-parameter reduction dL_G/dtheta.

Default: the small-batch workload (32 parameter rows x 8,192 events,
262,144 fake + 262,144 real events, discriminator 2-128-128-128-1, fp32) is
the headline; the same JSON line carries a "configs" record with every other
step workload (the tiny, medium, higher-dim and stress configurations, and the
stand-alone sampler writing the stress configuration's events to HBM), each
with its step time, events/s, binding roofline and the CPU oracle's rate.

Timing: W warm-up steps, then the timed region of K steps between
torch.cuda.synchronize() calls with the library's per-kernel events off; then
K more steps with them on, for the per-kernel durations of the roofline.

  python bench.py [--steps K] [--warmup W] [--gpus 1] [--workload NAME]
                  [--no-cpu-baseline] [--no-configs] [--calibrate-copy]
"""
from __future__ import annotations

import argparse
import hashlib
import itertools
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
METRIC = "events/sec per sample->discriminate->backward step; % of HBM / MFMA peak"
CONFIG_NAMES = ("pr1_tiny", "medium", "higher_dim", "stress", "stress_sample")


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


def kernels_summary(kt: dict) -> dict:
    return {k: {"launches": n, "avg_ms": t / max(n, 1)} for k, (n, t) in kt.items()}


# ---------------------------------------------------------------------------
# Timing

def time_steps(ctx, step, args, torch, kernel_pass: bool = True):
    """W warm-up steps; the timed region of K steps with the library's kernel events
    off, bracketed by torch.cuda.synchronize(); then, unless kernel_pass is False,
    K more steps with the events on (one pair per launch, on the context's stream),
    for per-kernel durations.  Returns (ms per timed step, {kernel: (launches, ms)})."""
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    kt = {}
    if kernel_pass:
        ctx.kernel_times()                      # drop earlier records
        ctx.set_timing(True)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        ctx.set_timing(False)
        kt = ctx.kernel_times()
    return (t1 - t0) * 1e3 / args.steps, kt


# ---------------------------------------------------------------------------
# CPU baseline: the float64 oracle, as it stands, on the host cores.  Work is
# split into tasks (a range of one parameter row's events, with the matching
# range of the real batch), run by a pool of single-threaded worker processes
# until the time budget is spent; the rate is events completed / wall time.

_INPUTS = {}


def _worker_init():
    # one BLAS thread per worker process: set before numpy loads its BLAS
    for v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS", "BLIS_NUM_THREADS"):
        os.environ[v] = "1"
    import numpy  # noqa: F401
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:
        pass


def _cpu_task(name: str, row: int, off: int, n: int) -> int:
    """One task of the oracle's step (runs in a worker process): events
    [off, off + n) of parameter row `row` of workload `name`."""
    import numpy as np
    import oracle
    from workloads import gen, get
    if name not in _INPUTS:
        _INPUTS[name] = gen.make_inputs(get("stress" if name == "stress_sample" else name))
    inp = _INPUTS[name]
    w = get("stress" if name == "stress_sample" else name)
    theta = np.asarray(inp["theta"][row:row + 1], dtype=np.float64)
    base = row * w.events_per_theta + off
    if name == "stress_sample":
        oracle.sample(theta, n, w.fake_seed, counter_base=base)
    elif w.widths is None:
        oracle.run_step(theta, n, w.fake_seed, critic="quadratic", counter_base=base)
    else:
        real = oracle.sample(inp["theta_star"], n, w.real_seed, counter_base=base)
        oracle.run_step(theta, n, w.fake_seed, inp["W"], inp["b"], real, features=w.features,
                        bf16=(w.precision == "bf16"), counter_base=base)
    return n


# events per task: about a second of single-threaded float64 work each
_TASK_EVENTS = {"pr1_tiny": 4096, "small": 8192, "medium": 2048, "higher_dim": 512, "stress": 1 << 18,
                "stress_sample": 1 << 18, "paper": 100}


class CpuPool:
    """Worker processes for the oracle's CPU baseline (spawned, so that no GPU state
    is inherited; each worker runs single-threaded BLAS)."""

    def __init__(self):
        import concurrent.futures as cf
        import multiprocessing as mp
        try:
            n_cpu = len(os.sched_getaffinity(0))
        except AttributeError:
            n_cpu = os.cpu_count() or 1
        self.workers = max(1, min(16, n_cpu))      # the host share of one GPU
        self.ex = cf.ProcessPoolExecutor(max_workers=self.workers, mp_context=mp.get_context("spawn"),
                                         initializer=_worker_init)

    def close(self):
        self.ex.shutdown(wait=True)

    def rate(self, name: str, seconds: float) -> dict:
        """Events/s of the oracle's step on workload `name` over at least `seconds`."""
        import concurrent.futures as cf
        from workloads import get
        w = get("stress" if name == "stress_sample" else name)
        per = min(_TASK_EVENTS[name], w.events_per_theta)
        tasks = [(r, off, min(per, w.events_per_theta - off)) for r in range(w.n_theta)
                 for off in range(0, w.events_per_theta, per)]
        # warm the workers (imports, inputs) outside the timed window
        list(self.ex.map(_cpu_task, [name] * self.workers, [0] * self.workers, [0] * self.workers,
                         [min(per, 64)] * self.workers))
        # the workload's tasks in order, again from the first once all are issued, until
        # `seconds` have passed (a small workload takes well under a second per pass)
        it = itertools.cycle(tasks)
        running, done_events, n_done = set(), 0, 0
        t0 = time.perf_counter()

        def submit():
            r, off, n = next(it)
            running.add(self.ex.submit(_cpu_task, name, r, off, n))

        for _ in range(self.workers):
            submit()
        while running:
            fin, _ = cf.wait(running, return_when=cf.FIRST_COMPLETED)
            for f in fin:
                running.discard(f)
                done_events += f.result()
                n_done += 1
                if time.perf_counter() - t0 < seconds:
                    submit()
        dt = time.perf_counter() - t0
        total = w.n_events
        real = "" if (w.widths is None) else " (and as many real events, sampled in the task)"
        what = "sampler only" if name == "stress_sample" else (
            "quadratic critic" if w.widths is None else ("bf16-point" if w.precision == "bf16" else "float64"))
        return {"value": done_events / dt, "unit": "events/s", "cores": self.workers, "kind": "oracle",
                "sample": f"{done_events} fake events ({done_events / total:.3g} x the workload's {total}){real}, "
                          f"{n_done} tasks of <= {per} "
                          f"events of one parameter row, oracle step ({what}, numpy float64) in {self.workers} "
                          f"single-threaded worker processes, {dt:.1f} s"}


# ---------------------------------------------------------------------------
# Step workloads (the five configurations and the paper's shape)

def run_step_workload(name, args, ctx, torch, sg, pool):
    """Times one step workload; returns a record with its rate, roofline and CPU baseline."""
    from workloads import gen, get
    if name == "stress_sample":
        return run_sample(args, ctx, torch, pool)
    w = get(name)
    dev = "cuda:0"
    inp = gen.make_inputs(w)
    theta = torch.tensor(inp["theta"], device=dev)
    theta_star = torch.tensor(inp["theta_star"], device=dev)
    N = w.n_events
    rec = {"workload": w.name, "n_theta": w.n_theta, "events_per_theta": w.events_per_theta, "fake_events": N,
           "real_events": N if w.widths else 0, "widths": list(w.widths) if w.widths else None,
           "precision": w.precision, "features": w.features}

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
    else:
        g = torch.empty((w.n_theta, 2 * w.d), dtype=torch.float32, device=dev)
        loss = torch.empty(1, dtype=torch.float32, device=dev)

        def step():
            ctx.param_grad(theta, w.events_per_theta, w.fake_seed, out=g, loss_out=loss)

    ms_per_step, kt = time_steps(ctx, step, args, torch)
    rec["ms_per_step"] = ms_per_step
    rec["value"] = N / (ms_per_step * 1e-3)
    rec["unit"] = "events/s"
    rec["dtype"] = "f32" if w.precision == "f32" else "bf16"

    if w.widths is not None and w.precision == "f32":
        # the fused fp32 kernel: its algorithmic flops against the fp32 matrix-core peak
        flops = mlp_flops_per_fake_event(w.widths) * N
        launches, total_ms = kt["disc_f32_fused"]
        avg_ms = total_ms / launches
        achieved = flops / (avg_ms * 1e-3)
        roof = {"bound": "mfma", "achieved": achieved / 1e12, "peak": PEAK["mfma_f32"] / 1e12, "unit": "TFLOP/s",
                "frac": achieved / PEAK["mfma_f32"], "traffic": read_traffic("disc_f32_fused", w.name),
                "step_mfma_frac": flops / (ms_per_step * 1e-3) / PEAK["mfma_f32"],
                "kernel": "disc_f32_fused", "kernel_avg_ms": avg_ms}
    elif w.widths is not None:
        # bf16: the step's algorithmic flops against the bf16 matrix-core peak (the binding
        # roof of these workloads); the dominant launch kind as a diagnostic
        flops = mlp_flops_per_fake_event(w.widths) * N
        step_rate = flops / (ms_per_step * 1e-3)
        H, NH = w.widths[1], len(w.widths) - 3
        kinds = [k for k in ("bf16_fwd_chain", "bf16_bwd_chain", "bf16_wgrad") if k in kt]
        dominant = max(kinds, key=lambda k: kt[k][1])
        per_step = {k: kt[k][1] / args.steps for k in kinds}
        roof = {"bound": "mfma", "achieved": step_rate / 1e12, "peak": PEAK["mfma_bf16"] / 1e12, "unit": "TFLOP/s",
                "frac": step_rate / PEAK["mfma_bf16"], "basis": "step: (12S - 2FH) N algorithmic flop / ms_per_step",
                "kernel": dominant, "kernel_ms_per_step": per_step}
        # hidden-product flops of each chain launch kind (NH products of 2 H^2 per row, both batches)
        hidden = NH * 2 * H * H * (2 * N)
        for k in ("bf16_fwd_chain", "bf16_bwd_chain"):
            if k in kt:
                roof[k + "_hidden_tflops"] = hidden / (per_step[k] * 1e-3) / 1e12
        if "bf16_wgrad" in kt:
            # diagnostic: the weight-gradient operands streamed per row (e_D in every layer): the signal
            # and the activation in bf16 for a stored-signal layer; the activation and H/8 sign bytes for
            # the top layer; at H = 256 with two identity inputs the signal and 8 bytes of coordinates
            # for the first layer, whose A_1 the kernel rebuilds
            rebuild_a1 = H == 256 and w.features == "identity" and w.widths[0] == 2 and NH > 1
            per_row = []
            for l in range(NH):
                if l == NH - 1:
                    per_row.append(2 * H + H // 8 + 4)
                elif l == 0 and rebuild_a1:
                    per_row.append(2 * H + 8 + 4)
                else:
                    per_row.append(4 * H + 4)
            wbytes = sum(per_row) * (2 * N)
            roof["bf16_wgrad_operand_GBps"] = wbytes / (per_step["bf16_wgrad"] * 1e-3) / 1e9
        tr = [read_traffic(k, w.name) for k in kinds]
        if all(t is not None for t in tr):
            roof["step_traffic_bytes"] = sum(t * kt[k][0] / args.steps for t, k in zip(tr, kinds))
        roof["traffic"] = read_traffic(dominant, w.name)
    else:
        # stress: sampler + pathwise + quadratic critic, bound by VALU issue; essential HBM bytes ~ 0
        launches, total_ms = kt["param_grad"]
        avg_ms = total_ms / launches
        achieved = N / (avg_ms * 1e-3)
        mix = read_valu_mix("param_grad", w.name)
        peak_ev = valu_peak_events(*mix) if mix else None
        essential = w.n_theta * 2 * w.d * 4 * 2 + 4        # theta in, dL/dtheta and the loss out
        roof = {"bound": "alu", "achieved": achieved / 1e9, "peak": peak_ev / 1e9 if mix else None,
                "unit": "Gevents/s", "frac": achieved / peak_ev if mix else None,
                "valu_per_event": mix[0] if mix else None, "trans_per_event": mix[1] if mix else None,
                "hbm_GBps": essential / (avg_ms * 1e-3) / 1e9, "traffic": read_traffic("param_grad", w.name),
                "kernel": "param_grad", "kernel_avg_ms": avg_ms}
    roof["kernels"] = kernels_summary(kt)
    rec["roofline"] = roof
    if pool is not None:
        rec["cpu_baseline"] = pool.rate(name, args.cpu_seconds)
    return rec


def run_sample(args, ctx, torch, pool):
    """The stand-alone sampler on the stress configuration: theta -> Philox ->
    Kumaraswamy events written to HBM ([N][d] fp32), the path that feeds a
    buffered discriminator."""
    from workloads import gen, get
    w = get("stress")
    dev = "cuda:0"
    inp = gen.make_inputs(w)
    theta = torch.tensor(inp["theta"], device=dev)
    N = w.n_events
    x = torch.empty((N, w.d), dtype=torch.float32, device=dev)

    def step():
        ctx.sample_events(theta, w.events_per_theta, w.fake_seed, out=x)

    ms_per_step, kt = time_steps(ctx, step, args, torch)
    launches, total_ms = kt["sample_events"]
    avg_ms = total_ms / launches
    bytes_per_launch = N * w.d * 4 + w.n_theta * 2 * w.d * 4     # events written, theta read
    achieved = bytes_per_launch / (avg_ms * 1e-3)
    mix = read_valu_mix("sample_events", "stress_sample")
    rec = {"workload": "stress_sample", "n_theta": w.n_theta, "events_per_theta": w.events_per_theta,
           "events": N, "d": w.d, "ms_per_step": ms_per_step, "value": N / (ms_per_step * 1e-3),
           "unit": "events/s", "dtype": "f32",
           "roofline": {"bound": "hbm", "achieved": achieved / 1e9, "peak": PEAK["hbm"] / 1e9, "unit": "GB/s",
                        "frac": achieved / PEAK["hbm"], "traffic": read_traffic("sample_events", "stress_sample"),
                        "valu_frac": (N / (avg_ms * 1e-3)) / valu_peak_events(*mix) if mix else None,
                        "kernel": "sample_events", "kernel_avg_ms": avg_ms, "kernels": kernels_summary(kt)}}
    if pool is not None:
        rec["cpu_baseline"] = pool.rate("stress_sample", args.cpu_seconds)
    return rec


def step_line(rec, args):
    """The driver's JSON line for a step workload record."""
    line = {"metric": METRIC, "value": rec["value"], "unit": "events/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": rec["ms_per_step"], "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": rec["dtype"],
            "data": "synthetic (seeded theta, Philox-sampled events, Xavier-initialised weights)",
            "config": {k: rec[k] for k in ("workload", "n_theta", "events_per_theta", "fake_events", "real_events",
                                           "widths", "precision", "features") if k in rec},
            "roofline": rec["roofline"]}
    line["config"]["parallelism"] = "single GPU"
    if "cpu_baseline" in rec:
        line["cpu_baseline"] = rec["cpu_baseline"]
    return line


# ---------------------------------------------------------------------------
# The other workloads: bootstrap draw, ensemble response, GAN training step

def cpu_baseline_bootstrap(w, n_out: int, min_seconds: float):
    """The oracle's draw, as it stands, of n_out rows from a pool of 2 n_out events."""
    import numpy as np
    import oracle
    pool = oracle.sample(np.asarray([w.theta_star], dtype=np.float32), 2 * n_out, w.pool_seed).astype(np.float32)
    draw = oracle.bootstrap_row_order if w.row_order else oracle.bootstrap
    reps, t0 = 0, time.perf_counter()
    while True:
        draw(pool, n_out, w.seed, reps)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    return {"value": reps * n_out / dt, "unit": "draws/s", "cores": 1, "kind": "oracle",
            "sample": f"{n_out} draws from a pool of {2 * n_out} events (of the workload's {w.n_out} from "
                      f"{w.n_data}), numpy, one process, {reps} repetition(s) in {dt:.1f} s"}


def bench_bootstrap(args, w, ctx, torch):
    """Steps of the bootstrap draw: n_out rows gathered from the resident pool, a fresh draw per step."""
    dev = "cuda:0"
    pool = ctx.sample_events(torch.tensor([w.theta_star], dtype=torch.float32, device=dev), w.n_data, w.pool_seed)
    out = torch.empty((w.n_out, w.d), dtype=torch.float32, device=dev)
    it = [0]

    def step():
        ctx.bootstrap(pool, w.n_out, w.seed, it[0], out=out, row_order=w.row_order)
        it[0] += 1

    ms_per_step, kt = time_steps(ctx, step, args, torch)
    name = "bootstrap_rows" if w.row_order else "bootstrap"
    launches, total_ms = kt[name]       # the row order times its five kernels as one
    avg_ms = total_ms / launches
    # algorithmic bytes of a draw: the drawn row read once and written once
    bytes_per_launch = w.n_out * 2 * w.d * 4
    achieved = bytes_per_launch / (avg_ms * 1e-3)
    roof = {"bound": "hbm", "achieved": achieved / 1e9, "peak": PEAK["hbm"] / 1e9, "unit": "GB/s",
            "frac": achieved / PEAK["hbm"], "traffic": read_traffic(name, w.name),
            "kernel": name, "kernel_avg_ms": avg_ms, "kernels": kernels_summary(kt)}
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
        line["cpu_baseline"] = cpu_baseline_bootstrap(w, min(w.n_out, 1 << 20), args.cpu_seconds)
    return line


def gen_flops_per_row(widths) -> int:
    """Forward flops of one generator on one noise vector: 2 * sum in*out."""
    return 2 * sum(a * b for a, b in zip(widths[:-1], widths[1:]))


def cpu_baseline_ensemble(w, W, b, n, min_seconds: float):
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
            "sample": f"{M} of the {w.n_members} members x {w.k} noise vectors, float64 numpy (BLAS threads), "
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

    ms_per_step, kt = time_steps(ctx, step, args, torch)
    launches, total_ms = kt["gen_forward"]
    avg_ms = total_ms / launches
    flops = gen_flops_per_row(w.widths) * w.n_members * w.k
    achieved = flops / (avg_ms * 1e-3)
    roof = {"bound": "mfma", "achieved": achieved / 1e12, "peak": PEAK["mfma_f32"] / 1e12, "unit": "TFLOP/s",
            "frac": achieved / PEAK["mfma_f32"], "traffic": read_traffic("gen_forward", w.name),
            "kernel": "gen_forward", "kernel_avg_ms": avg_ms, "kernels": kernels_summary(kt)}
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
        line["cpu_baseline"] = cpu_baseline_ensemble(w, W, b, n, args.cpu_seconds)
    return line


def cpu_baseline_train(w, rows: int, min_seconds: float):
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
                      f"bootstrapped reference events), float64 numpy (BLAS threads), {reps} step(s) in {dt:.1f} s"}


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
    total = args.warmup + 2 * args.steps
    noise = torch.tensor(rng.standard_normal((total, w.k, w.g_widths[0])).astype(np.float32),
                         device=dev)                                    # resident before timing
    it = [0]

    def step():
        loop.step(noise[it[0]])
        it[0] += 1

    ms_per_step, kt = time_steps(ctx, step, args, torch)
    launches, total_ms = kt["disc_f32_fused"]
    avg_ms = total_ms / launches
    flops = mlp_flops_per_fake_event(w.d_widths) * N
    achieved = flops / (avg_ms * 1e-3)
    g_flops = 4 * gen_flops_per_row(w.g_widths) * w.k      # forward, recomputed forward, backward (2x)
    roof = {"bound": "mfma", "achieved": achieved / 1e12, "peak": PEAK["mfma_f32"] / 1e12, "unit": "TFLOP/s",
            "frac": achieved / PEAK["mfma_f32"], "traffic": read_traffic("disc_f32_fused", w.name),
            "step_mfma_frac": (flops + g_flops) / (ms_per_step * 1e-3) / PEAK["mfma_f32"],
            "kernel": "disc_f32_fused", "kernel_avg_ms": avg_ms, "kernels": kernels_summary(kt)}
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
        line["cpu_baseline"] = cpu_baseline_train(w, min(args.cpu_rows, w.k), args.cpu_seconds)
    return line


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="small")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="only the headline workload")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="time budget of each CPU baseline")
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
    from workloads import get

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
    name = args.workload
    line = None
    if name not in ("stress_sample",) + tuple(CONFIG_NAMES) + ("small", "paper"):
        w = get(name)
        if hasattr(w, "n_data"):
            line = bench_bootstrap(args, w, ctx, torch)
        elif hasattr(w, "n_members"):
            line = bench_ensemble(args, w, ctx, torch)
        elif hasattr(w, "g_widths"):
            line = bench_train(args, w, ctx, torch, sg)
    if line is None:
        pool = None if args.no_cpu_baseline else CpuPool()
        try:
            rec = run_step_workload(name, args, ctx, torch, sg, pool)
            if name == "stress_sample":
                line = {"metric": "events/sec of the stand-alone sampler (theta -> Philox -> Kumaraswamy events in "
                                  "HBM); % of HBM peak",
                        "value": rec["value"], "unit": "events/s", "n_gpus": 1, "steps": args.steps,
                        "warmup": args.warmup, "ms_per_step": rec["ms_per_step"], "higher_is_better": True,
                        "scaling": "weak", "vs_baseline": None, "dtype": "f32",
                        "data": "synthetic (seeded theta, Philox-sampled events)",
                        "config": {k: rec[k] for k in ("workload", "n_theta", "events_per_theta", "events", "d")},
                        "roofline": rec["roofline"]}
                line["config"]["parallelism"] = "single GPU"
                if "cpu_baseline" in rec:
                    line["cpu_baseline"] = rec["cpu_baseline"]
            else:
                line = step_line(rec, args)
            if name == "small" and not args.no_configs:
                # every other configuration, in the same run and the same protocol
                line["configs"] = {}
                for other in CONFIG_NAMES:
                    r = run_step_workload(other, args, ctx, torch, sg, pool)
                    line["configs"][other] = r
                    torch.cuda.empty_cache()
                    print(f"# {other}: {r['ms_per_step']:.3f} ms/step, {r['value']:.3e} events/s", file=sys.stderr,
                          flush=True)
        finally:
            if pool is not None:
                pool.close()
    ctx.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
