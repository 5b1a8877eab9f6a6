#!/usr/bin/env python3
"""Jorge optimizer steps/s on one MI355X, with roofline and CPU-oracle context.

A step is one full Jorge update (Algorithm 2 with SGD grafting, momentum and
decoupled weight decay) over every layer of the workload, with the factors
updated every step (interval 1). Inputs are synthetic, seeded and resident in
HBM before the timed region. The K timed steps run twice: once with only
the two bracketing events (steps/s), once with HIP events around every launch
on the library's streams (per-stage times and the roofline of the grouped
GEMM). Prints one JSON line; with --others 1 (the default) it also times the
other four workloads, each for its stated number of steps, and reports them
in the line's "other_workloads" record.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "Jorge optimizer steps/sec (ResNet-50 weight set); fp32 MFMA util %"
PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
WORKLOAD_NAMES = {
    "resnet50": "ResNet-50 weight set: 53 conv + fc weights as out x in*kh*kw, fp32, G ~ N(0, 1e-3^2)",
    "single_64x576": "single 64x576 layer, G ~ N(0, 1e-2^2)",
    "single_512x4608": "single 512x4608 layer, G ~ N(0, 1e-3^2)",
    "large_dense": "8 x 4096x4096 + 8 x 4096x1024 layers, G ~ N(0, 1e-3^2)",
    "many_small": "512 layers, m, n in {32, 64, 128, 256}, G ~ N(0, 1e-2^2)",
}


def falg_paper(m, n):
    """Flops of one factor-updating step of an m x n layer in the paper's explicit order.

    Per factor of size d with statistic rank k: A^2 and A^4 (symmetric, d^3 each),
    X, X X and A P (2 d^3 each), the Gram product (d^2 k); plus L_hat G R_hat.
    """
    return 8 * m ** 3 + 8 * n ** 3 + 3 * m * m * n + 3 * m * n * n


def stage_bytes(shapes):
    """Algorithmic HBM bytes per launch of the bandwidth-bound stages."""
    mn = sum(m * n for m, n in shapes)
    return {"weight": 12 * mn,       # read theta and m, write theta
            "stage_in": 20 * mn}     # read G, write Gp and its transpose, read and write m_SGD


def step_bytes(shapes, update):
    """Algorithmic HBM bytes of one step: read G, theta, m, m_SGD and the factors,
    write theta, m, m_SGD and (on factor-updating steps) the factors."""
    return sum(4 * (7 * m * n + (2 if update else 1) * (m * m + n * n)) for m, n in shapes)


def profile_path(config):
    """The committed rocprofv3 summary of a workload, which carries its HBM counter figures."""
    return os.path.join(ROOT, "profiles", f"jorge_step_{config}.md")


# The sources that decide what the grouped GEMM runs: the kernel itself and the
# host code that builds its launch tables (not the bandwidth-bound kernels).
GEMM_SOURCES = ("jorge.hip", "jorge_gemm.hpp", "jorge_types.hpp")


def kernel_sources_sha256():
    import hashlib
    h = hashlib.sha256()
    for f in sorted(os.path.join(ROOT, "paper_2310_12298_amd", "csrc", n) for n in GEMM_SOURCES):
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(config):
    """HBM bytes per gemm_grouped launch from the workload's committed counter summary, or None.

    The figure applies only to the workload it was taken on, and only while the
    kernel sources are the ones it was taken with.
    """
    path = profile_path(config)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and line.split(":")[0] in ("traffic_bytes_per_launch", "kernel_sources_sha256"):
                k, v = line.split(":", 1)
                vals[k] = v.strip()
    if vals.get("kernel_sources_sha256") != kernel_sources_sha256():
        return None
    return float(vals["traffic_bytes_per_launch"]) if "traffic_bytes_per_launch" in vals else None


GEMM_STAGES = ("gram", "pow4", "xform", "chain4", "chain5", "poly", "poly2", "update", "uprecond_L", "uprecond_R",
               "precond_L", "precond_R")
# Preconditioning of steps that do not update the factors; every other GEMM stage runs on update steps.
NON_UPDATE_STAGES = ("precond_L", "precond_R")
# Launches of the grouped GEMM's split-tile fixup: their time is part of the GEMM stages' time.
FIXUP_STAGE = "split_fixup"
# The LDS chain kernels (whole factor updates of small factors in one workgroup each).
CHAIN_STAGE = "lds_chain"


def copy_reference_gbs(mib=1024, reps=10):
    """Device-to-device copy rate of a buffer far larger than the caches (GB/s).

    The streaming rate this GPU sustains in practice, beside which the
    bandwidth-bound kernels' rates are read (bytes read plus bytes written).
    """
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(reps):
        dst.copy_(src)
    stop.record()
    torch.cuda.synchronize()
    gbs = 2 * n * 4 * reps / (start.elapsed_time(stop) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return gbs


def cpu_baseline(shapes, sigma, seed, budget_s, series_order=2):
    """The fp64 oracle timed on the host over a bounded, deterministic sample.

    Steps t = 1, 2, ... run layer by layer in the workload's order (each layer's
    oracle keeps its state from step to step, with fresh gradients), until the
    time budget is spent; steps/s is the sample's share of the workload's
    algorithmic flops over the time spent.
    """
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import JorgeOracle
    from paper_2310_12298_amd.workloads import gradient, initial_params

    total_f = sum(falg_paper(m, n) for m, n in shapes)
    orcs, params = {}, {}
    done_f, spent, t, layers_done = 0, 0.0, 0, 0
    while spent < budget_s:
        t += 1
        for l, s in enumerate(shapes):
            if l not in orcs:
                orcs[l] = JorgeOracle([s], series_order=series_order)
                params[l] = [initial_params(seed, l, s).astype(np.float64)]
            G = [gradient(seed, l, t, s, sigma)]
            t0 = time.perf_counter()
            params[l] = orcs[l].step(params[l], G, 0.1, 0.9, 0.9, 5e-5)
            spent += time.perf_counter() - t0
            done_f += falg_paper(*s)
            layers_done += 1
            if spent >= budget_s:
                break
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": (done_f / total_f) / spent, "unit": "steps/s", "cores": threads, "kind": "oracle",
            "sample": f"fp64 oracle steps 1..{t} of the workload's layers in order, {layers_done} layer-steps "
                      f"({done_f / total_f:.2f} steps' worth of the algorithmic flops) in {spent:.1f} s, "
                      f"scaled by flop share"}


FLOP_BASIS = ("executed: the algorithmic flops of the products the step runs, each factor in the evaluation "
              "order the library chose for it (explicit, factored or squared, with low-rank preconditioning), "
              "symmetric products counted once, over unpadded extents (jorge_stage_flops)")
PAPER_ORDER_NOTE = ("an effective rate, not a utilisation: the step counted in the paper's explicit order "
                    "(8m^3 + 8n^3 + 3m^2n + 3mn^2 per layer) per second of step time; it can exceed the peak "
                    "because the factored and squared orders need fewer flops for the same factors")


def cpu_info():
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"os_cpu_count": os.cpu_count(), "cpu_model": model}


def parse_layers(spec):
    """Layer shapes from a list such as "128x128*256,96x96*8,64x576" (m x n, optional * count)."""
    shapes = []
    for item in spec.split(","):
        item = item.strip()
        dims, _, count = item.partition("*")
        m, _, n = dims.partition("x")
        try:
            m, n, count = int(m), int(n), int(count) if count else 1
        except ValueError:
            raise SystemExit(f"--layers: cannot read {item!r} (expected MxN or MxN*COUNT)")
        if m < 1 or n < 1 or count < 1:
            raise SystemExit(f"--layers: {item!r} must have positive sizes and count")
        shapes += [(m, n)] * count
    return shapes


def measure(config, steps, warmup, interval=1, form="auto", split_k=1, series_order=2, seed=0,
            copy_probe_mib=0, chain_max=128, layers=None, sigma=1e-2):
    """Times one workload: W warm-up steps, then K steps twice (clean, then with per-launch events).

    layers: a list of shapes to time instead of a named workload (gradients of
    standard deviation sigma, 30 steps by default)."""
    import torch

    from paper_2310_12298_amd.jorge import Jorge
    from paper_2310_12298_amd.workloads import CONFIGS, DEFAULT_HPARAMS, device_gradient, device_initial_params

    shapes, sigma, run_steps = CONFIGS[config] if layers is None else (layers, sigma, 30)
    steps = steps if steps is not None else run_steps
    hp = DEFAULT_HPARAMS
    opt = Jorge(shapes, eps=hp["eps"], precond_interval=interval, factor_form=form,
                split_k=bool(split_k), series_order=series_order, lds_chain_max=chain_max)
    params = [device_initial_params(seed, l, s) for l, s in enumerate(shapes)]
    grads = [[device_gradient(seed, l, t, s, sigma) for l, s in enumerate(shapes)]
             for t in range(1, warmup + steps + 1)]
    pp = Jorge.pointer_array(params)
    gp = [Jorge.pointer_array(g) for g in grads]

    def step(i):
        opt.step_ptrs(pp, gp[i], hp["lr"], hp["beta2"], hp["beta1"], hp["weight_decay"])

    if copy_probe_mib > 0:
        n = copy_probe_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()

    def timed(instrumented):
        """K steps between two events on the stream; with per-launch HIP events if instrumented."""
        opt.set_timing(instrumented)
        opt.reset_timing()
        t0 = opt.t
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record()
        for i in range(steps):
            step(warmup + i)
        stop.record()
        torch.cuda.synchronize()
        ms = start.elapsed_time(stop)
        timing = opt.read_timing()
        opt.set_timing(False)
        # factor-updating steps among this pass's step numbers t0+1 .. t0+steps
        upd = sum(1 for t in range(t0 + 1, t0 + steps + 1) if (t - 1) % interval == 0)
        return ms, timing, upd

    # Throughput from a pass without per-launch events (they add gaps between
    # launches); per-stage times and the roofline from a second, instrumented
    # pass of the same steps.
    total_ms, _, updates_clean = timed(False)
    inst_ms, timing, updates = timed(True)
    for t in params:
        if not torch.isfinite(t).all():
            raise RuntimeError(f"{config}: non-finite parameters after the timed steps")
    if updates == 0:
        raise SystemExit("no factor update in the timed steps; use more steps or a smaller interval")
    # Algorithmic flops of each stage in one factor-updating step, from the library's launch tables.
    flops = opt.stage_flops()
    ran = {k: (steps - updates if k in NON_UPDATE_STAGES else updates) for k in GEMM_STAGES}
    ran[CHAIN_STAGE] = updates
    per_stage = {}
    for k, (ms, n) in timing.items():
        e = {"ms_per_launch": ms / n if n else 0.0, "launches": n}
        if k in ran and ms > 0:
            e["tflops"] = flops[k] * ran[k] / (ms * 1e-3) / 1e12
        per_stage[k] = e
    # Dominant kernel: the grouped NT GEMM; every GEMM stage of the step is a launch of it.
    g_flops = sum(flops[k] * ran[k] for k in GEMM_STAGES)
    g_ms = sum(timing[k][0] for k in GEMM_STAGES) + timing[FIXUP_STAGE][0]
    g_launches = sum(timing[k][1] for k in GEMM_STAGES)
    achieved = g_flops / (g_ms * 1e-3) / 1e12 if g_ms > 0 else 0.0
    ms_launch = g_ms / max(1, g_launches)
    f_paper = sum(falg_paper(m, n) for m, n in shapes) * updates_clean / steps
    hbm = {}  # the bandwidth-bound kernels: algorithmic bytes / average launch time
    for k, nbytes in stage_bytes(shapes).items():
        k_ms = timing[k][0] / max(1, timing[k][1])
        gbs = nbytes / (k_ms * 1e-3) / 1e9 if k_ms else 0.0
        hbm[k] = {"achieved": gbs, "frac": gbs / PEAK_HBM_GBS, "bytes_per_launch": nbytes}
    # the step's flops: the grouped levels' and the LDS chains' (in a context of small factors only, the
    # chains take every factor update in place of the levels)
    step_f = (g_flops + flops[CHAIN_STAGE] * updates) / steps
    step_b = (step_bytes(shapes, True) * updates + step_bytes(shapes, False) * (steps - updates)) / steps
    t_mfma, t_hbm = step_f / (PEAK_FP32_MFMA_TFLOPS * 1e12), step_b / (PEAK_HBM_GBS * 1e9)
    step_roof = {"flops": step_f, "bytes": step_b, "t_mfma_ms": t_mfma * 1e3, "t_hbm_ms": t_hbm * 1e3,
                 "bound": "mfma" if t_mfma >= t_hbm else "hbm",
                 "frac": max(t_mfma, t_hbm) / (total_ms / steps * 1e-3), "flop_basis": "executed (as roofline)"}
    forms = {"explicit": 0, "factored": 0, "squared": 0}
    for l in range(len(shapes)):
        for side in (0, 1):
            forms[opt.factor_form(l, side)] += 1
    res = {
        "config": config, "shapes": shapes, "sigma": sigma, "steps": steps, "updates": updates,
        "value": steps / (total_ms * 1e-3), "ms_per_step": total_ms / steps,
        "ms_per_step_instrumented": inst_ms / steps, "forms": forms,
        "gemm": {"achieved": achieved, "ms_per_launch": ms_launch, "launches": g_launches,
                 "gflop_per_launch": g_flops / max(1, g_launches) / 1e9},
        "step_roofline": step_roof,
        "mfma_util_pct": 100.0 * step_f / (inst_ms / steps * 1e-3) / (PEAK_FP32_MFMA_TFLOPS * 1e12),
        "paper_order": {"flops_per_step": f_paper, "effective_tflops": f_paper / (total_ms / steps * 1e-3) / 1e12,
                        "note": PAPER_ORDER_NOTE},
        "hbm": hbm, "stages": per_stage,
    }
    del opt, params, grads, pp, gp
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def summary(res):
    """The sub-record of a workload measured beside the headline one."""
    return {"workload": WORKLOAD_NAMES[res["config"]], "steps": res["steps"], "value": res["value"], "unit": "steps/s",
            "ms_per_step": res["ms_per_step"], "gemm_frac": res["gemm"]["achieved"] / PEAK_FP32_MFMA_TFLOPS,
            "gemm_tflops": res["gemm"]["achieved"], "step_roofline_frac": res["step_roofline"]["frac"],
            "step_roofline_bound": res["step_roofline"]["bound"], "factors": res["forms"],
            "hbm_frac": {k: v["frac"] for k, v in res["hbm"].items()},
            "traffic_bytes_per_launch": measured_traffic(res["config"])}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: the workload's run)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="resnet50", choices=sorted(WORKLOAD_NAMES))
    ap.add_argument("--interval", type=int, default=1, help="preconditioner update interval k")
    ap.add_argument("--form", default="auto", choices=("auto", "explicit", "factored", "squared"),
                    help="evaluation order of the factor updates")
    ap.add_argument("--split-k", type=int, default=1, choices=(0, 1),
                    help="split the K range of long tiles in levels with too few tiles")
    ap.add_argument("--series-order", type=int, default=2, choices=(2, 3),
                    help="last power of X kept from the binomial series (Section 3 keeps 2)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--chain-max", type=int, default=128, choices=(0, 32, 64, 96, 128),
                    help="largest padded factor size the LDS chain kernels take (0: every factor in the levels)")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle time (0 = skip)")
    ap.add_argument("--others", type=int, default=1, choices=(0, 1),
                    help="also time the other four workloads, each for its stated number of steps, and report "
                         "them in the same line (with the default interval, order and options)")
    ap.add_argument("--layers", default=None,
                    help="time this list of layers instead of a named workload, e.g. 128x128*256,64x576 "
                         "(no other workloads are timed)")
    ap.add_argument("--sigma", type=float, default=1e-2, help="gradient standard deviation for --layers")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="before timing, copy a buffer of this many MiB once (calibrates HBM byte counters; "
                         "skips the copy-rate reference and the other workloads)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on exactly one GPU (asked for {max(args.gpus, world)}): the Jorge step is "
              f"replicated per data-parallel rank and this build measures one GPU's step.", file=sys.stderr)
        return 2

    import torch

    layers = parse_layers(args.layers) if args.layers else None
    if layers is not None:
        args.config, args.others = "custom", 0
        WORKLOAD_NAMES["custom"] = f"layers {args.layers}, G ~ N(0, {args.sigma:g}^2)"
    torch.cuda.set_device(0)
    res = measure(args.config, args.steps, args.warmup, args.interval, args.form, args.split_k, args.series_order,
                  args.seed, args.copy_probe_mib, args.chain_max, layers, args.sigma)
    shapes, steps = res["shapes"], res["steps"]
    traffic = measured_traffic(args.config)
    ms_launch = res["gemm"]["ms_per_launch"]
    traffic_gbs = traffic / (ms_launch * 1e-3) / 1e9 if traffic and ms_launch else None
    hbm = dict(res["hbm"])
    if args.copy_probe_mib == 0:  # counter runs identify their probe as the one large copy
        copy_gbs = copy_reference_gbs()
        hbm["copy_reference"] = {"achieved": copy_gbs, "frac": copy_gbs / PEAK_HBM_GBS,
                                 "bytes_per_launch": 2 * (1 << 30)}
    achieved = res["gemm"]["achieved"]
    out = {
        "metric": METRIC,
        "value": res["value"],
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "ms_per_step_instrumented": res["ms_per_step_instrumented"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": WORKLOAD_NAMES[args.config], "name": args.config, "layers": len(shapes),
                   "params": sum(m * n for m, n in shapes), "precond_interval": args.interval,
                   "factor_updates": res["updates"], "factor_form": args.form, "factors": res["forms"],
                   "split_k": args.split_k, "series_order": args.series_order, "lds_chain_max": args.chain_max,
                   "seed": args.seed},
        "roofline": {"bound": "mfma", "kernel": "gemm_grouped<true, true> (every GEMM stage of the step)",
                     "achieved": achieved, "peak": PEAK_FP32_MFMA_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_FP32_MFMA_TFLOPS, "flop_basis": FLOP_BASIS,
                     "traffic": traffic, "traffic_unit": "HBM bytes per launch",
                     # the measured traffic over the launch time: how far the kernel is from the HBM roof
                     "traffic_gbs": traffic_gbs,
                     "traffic_hbm_frac": traffic_gbs / PEAK_HBM_GBS if traffic_gbs else None,
                     "launches": res["gemm"]["launches"], "ms_per_launch": ms_launch,
                     "gflop_per_launch": res["gemm"]["gflop_per_launch"]},
        # The whole step against its own roofline: the executed algorithmic flops at the
        # fp32 MFMA peak and the algorithmic bytes at the HBM peak, the larger of the two
        # over the measured step time.
        "step_roofline": res["step_roofline"],
        # executed algorithmic flops of the whole step / (instrumented step time x fp32 MFMA peak)
        "mfma_util_pct": res["mfma_util_pct"],
        "paper_order": res["paper_order"],
        "hbm": dict(hbm, peak=PEAK_HBM_GBS, unit="GB/s"),
        "stages": res["stages"],
    }
    if args.others and args.copy_probe_mib == 0:
        out["other_workloads"] = {c: summary(measure(c, None, args.warmup, seed=args.seed, chain_max=args.chain_max))
                                  for c in WORKLOAD_NAMES if c != args.config}
    if args.cpu_budget > 0:
        out["cpu_baseline"] = dict(cpu_baseline(shapes, res["sigma"], args.seed, args.cpu_budget,
                                                args.series_order), **cpu_info())
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
