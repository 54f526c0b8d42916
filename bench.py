"""Throughput of the exact factored output-layer step on one MI355X.

Default workload: D = 200,000 outputs, d = 500 hidden units, minibatches of
m = 128 examples with K = 10 (index, value) targets each, squared error,
lr = 1e-3 (the paper's typical sizes).  A step is one call of lst_step: loss,
grad_H and the exact update of W = V U, Q and U^{-T}.  Inputs are synthetic,
seeded and resident in HBM before timing: a pool of 16 minibatches cycled
through.

Printed on stdout (one JSON line): examples/s over exactly --steps timed
steps, the roofline of the dominant kernel (per-phase times come from a
second, event-profiled pass over the same steps), the in-library naive
explicit-W step and its measured speedup, and the fp64 CPU oracle timed on a
bounded sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

REPO = os.path.dirname(os.path.abspath(__file__))
if REPO not in sys.path:
    sys.path.insert(0, REPO)

METRIC = "examples/sec, exact sparse-target step D=200k d=500 m=128; % MFMA/HBM peak"
PEAK_FP32_MFMA_TFLOPS = 157.3   # MI355X dense fp32 matrix
PEAK_HBM_GBS = 8000.0           # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def phase_work(name, cfg, u, nnz):
    """(algorithmic fp32 flops, algorithmic HBM bytes of V) of one launch of the step.

    Flops are those of the method's products that run in the launch, 2 per
    multiply-add, each product counted once at its algorithmic size: the
    m x m Woodbury solve as m^3 + m^2 d (one factorisation, d right-hand
    sides), N H^T as the m x m times m x d product it is, the symmetric Q
    update once per upper-triangle entry.  Bytes are the rows of V the launch
    must touch: u distinct target rows of d floats, read by the gather
    (launch 1) and read + written by the scatter (launch 3).
    """
    D, d, m, K = cfg.D, cfg.d, cfg.m, cfg.K
    if name == "launch1":   # [Q; U; U^-T; H^T] H  +  gather of V^T Y
        return 2.0 * m * d * (3 * d + m), float(u * d * 4)
    if name == "launch2":   # U^T G; H^T H^, H^T Y^ (C1, C2); X = S^-1 P^T
        return 2.0 * (m * d * d + 2 * m * m * d + m ** 3 + m * m * d), 0.0
    if name == "launch3":   # grad_H and T = grad_H - (lr/2) N H^T  +  scatter into V
        return 2.0 * m * m * d, float(2 * u * d * 4)
    if name == "launch4":   # symmetric rank-2m update of Q; rank-m updates of U and U^-T
        return 2.0 * (d * (d + 1) / 2) * 2 * m + 2 * 2.0 * m * d * d, 0.0
    return 0.0, 0.0


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="c2")
    ap.add_argument("--loss", default=None,
                    help="override the workload's loss: squared, spherical or spherical_shifted "
                         "(the (o_c + eps)^2 form; a class-per-example workload, K = 1)")
    ap.add_argument("--sph-eps", type=float, default=None, help="override the workload's eps")
    ap.add_argument("--naive-steps", type=int, default=10)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-naive", action="store_true")
    ap.add_argument("--no-stabilize", action="store_true")
    ap.add_argument("--step-only", action="store_true",
                    help="only the timed and profiled minibatch steps (for counter runs): no "
                         "split-task pass, single-example, stabilise, input-layer, naive or CPU "
                         "parts")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the benchmark line: factored vs naive step time over the "
                         "vocabulary size D at d = 300, m = 128 (the paper's timing figure and "
                         "speedup table)")
    ap.add_argument("--tasks", action="store_true",
                    help="instead of the benchmark line: every task of the step as a launch of "
                         "its own (lst_set_split_tasks), with per-task times and the HBM "
                         "fraction of the gather and the scatter")
    ap.add_argument("--crossover", action="store_true",
                    help="instead of the benchmark line: the Woodbury step (lst_step) against the "
                         "solve-from-scratch step (lst_step_solve), over m at d = 500 and 1024 "
                         "(D = 200000, K = 10)")
    args = ap.parse_args()
    if args.sweep:
        return sweep(args)
    if args.crossover:
        return crossover(args)
    if args.tasks:
        return tasks_only(args)

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the step has no "
              "multi-GPU path (V would be row-sharded across GPUs; not implemented)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1412_7091_amd as lst
    from synth import Workload, get_config

    if not torch.cuda.is_available():
        log("no GPU visible")
        sys.exit(1)
    lst.load_library()
    cfg = get_config(args.config)
    if args.loss is not None and args.loss != cfg.loss:
        cfg = cfg.replace(loss=args.loss, name=f"{cfg.name}+{args.loss}")
    if args.sph_eps is not None:
        cfg = cfg.replace(sph_eps=args.sph_eps, name=f"{cfg.name}+eps{args.sph_eps:g}")
    wl = Workload(cfg)
    dev = torch.device("cuda:0")
    t0 = time.time()
    V0 = wl.init_V()
    V0_t = torch.from_numpy(V0).to(dev)
    pool = []
    for s in range(16):
        H, idx, val = wl.batch(s)
        pool.append(tuple(torch.from_numpy(x).to(dev) for x in (H, idx, val)))
    loss_t = torch.empty(cfg.m, dtype=torch.float32, device=dev)
    grad_t = torch.empty((cfg.m, cfg.d), dtype=torch.float32, device=dev)
    log(f"workload {cfg.name}: D={cfg.D} d={cfg.d} m={cfg.m} K={cfg.K} loss={cfg.loss} "
        f"(inputs ready in {time.time() - t0:.1f}s)")

    layer = lst.FactoredOutputLayer(V0_t, loss=cfg.loss, sph_eps=cfg.sph_eps, m_max=cfg.m,
                                    K_max=cfg.K)

    def run(n, offset=0):
        for s in range(n):
            H, idx, val = pool[(s + offset) % len(pool)]
            layer.step(H, idx, val, cfg.lr, out=(loss_t, grad_t))

    run(args.warmup)
    torch.cuda.synchronize()
    if layer.sync() != 0:
        log("device error during warmup")
        sys.exit(1)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    run(args.steps, args.warmup)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop)
    code = layer.sync()
    if code != 0:
        log(f"device error in timed steps: {lst.lst_strerror(code)}")
        sys.exit(1)
    ms_per_step = ms / args.steps
    value = cfg.m * args.steps / (ms / 1e3)
    log(f"factored: {ms_per_step * 1e3:.1f} us/step, {value:.4g} examples/s")

    # profiled pass: per-phase durations from HIP events on the library's stream
    layer.profile(True)
    run(args.steps, args.warmup)
    phases, nsteps = layer.profile_read()
    layer.profile(False)
    st = layer.stats()
    u, nnz = st.last_unique, st.last_nnz
    kernels = {}
    best = None
    from paper_1412_7091_amd.profiling import measured_mfma, measured_traffic

    traffic = measured_traffic(cfg.name) or {}
    mfma = measured_mfma(cfg.name) or {}
    for name, tot in phases.items():
        avg_us = 1e3 * tot / max(nsteps, 1)
        if avg_us <= 0:
            continue  # phase not run by this configuration (drift control off)
        flops, nbytes = phase_work(name, cfg, u, nnz)
        entry = {"avg_us": round(avg_us, 3)}
        if name in traffic:
            entry["hbm_bytes_measured"] = traffic[name]["hbm_bytes"]
        if name in mfma:
            entry["mfma_busy_counter"] = mfma[name]["busy_frac"]
            entry["mfma_flops_counter"] = mfma[name]["mfma_flops"]
        if avg_us > 0 and (flops > 0 or nbytes > 0):
            tf = flops / (avg_us * 1e-6) / 1e12
            gb = nbytes / (avg_us * 1e-6) / 1e9
            entry.update(flops=flops, bytes=nbytes, tflops=round(tf, 4),
                         mfma_frac=round(tf / PEAK_FP32_MFMA_TFLOPS, 5), hbm_gbs=round(gb, 2),
                         hbm_frac=round(gb / PEAK_HBM_GBS, 5))
        kernels[name] = entry
        if flops > 0 and (best is None or avg_us > kernels[best]["avg_us"]):
            best = name
    log("per-launch us: " + ", ".join(f"{k}={v['avg_us']:.1f}" for k, v in kernels.items()))
    dom = kernels[best]
    dom_traffic = dom.get("hbm_bytes_measured")
    if dom["mfma_frac"] >= dom["hbm_frac"]:
        roofline = {"kernel": best, "bound": "mfma", "achieved": dom["tflops"],
                    "peak": PEAK_FP32_MFMA_TFLOPS, "unit": "TFLOP/s", "frac": dom["mfma_frac"],
                    "traffic": dom_traffic}
    else:
        roofline = {"kernel": best, "bound": "hbm", "achieved": dom["hbm_gbs"],
                    "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": dom["hbm_frac"],
                    "traffic": dom_traffic}
    if args.step_only:
        args.no_stabilize = args.no_naive = args.no_cpu_baseline = True
    tasks = single = None
    if not args.step_only:
        tasks = task_times(layer, run, cfg, u, args.steps)
        log("per-task us (split launches): " + ", ".join(f"{k}={v['avg_us']:.1f}"
                                                        for k, v in tasks.items()))
    roofline["mfma_busy_counter"] = dom.get("mfma_busy_counter")
    layer.close()
    del layer

    if not args.step_only:
        single = single_example_cost(lst, torch, cfg, V0_t, dev)
        log(f"single example: {single['us_per_step']:.2f} us/step pipelined, "
            f"{single['latency_us_median']:.1f} us latency")

    stab = None
    if not args.no_stabilize:
        stab = stabilize_cost(lst, torch, cfg, V0_t, dev)
        log(f"stabilize: {stab['ms_in_range']:.3f} ms when nothing is out of range, "
            f"{stab['ms_one_fix']:.3f} ms with one correction (one pass over V)")

    inp = None
    if not args.no_stabilize:
        inp = input_layer_cost(lst, torch, cfg, wl, V0_t, pool)
        log(f"input layer: forward {inp['forward_us']:.2f} us, update {inp['update_us']:.2f} us "
            f"per minibatch")

    # A plain 64 MiB device copy, outside every timed region: the reference the
    # FETCH_SIZE / WRITE_SIZE counter runs are scaled by (see profiling.py).  A
    # 128 MiB fill in between pushes the copy's source out of the L2 caches.
    calib_src = torch.empty(16 << 20, dtype=torch.float32, device=dev).fill_(1.0)
    flush = torch.empty(32 << 20, dtype=torch.float32, device=dev).fill_(0.0)
    calib_dst = torch.empty_like(calib_src)
    calib_dst.copy_(calib_src)
    torch.cuda.synchronize()
    del calib_src, calib_dst, flush

    naive = None
    if not args.no_naive:
        nl = lst.NaiveOutputLayer(V0_t, loss=cfg.loss, sph_eps=cfg.sph_eps, m_max=cfg.m,
                                  K_max=cfg.K)
        for s in range(2):
            H, idx, val = pool[s]
            nl.step(H, idx, val, cfg.lr, out=(loss_t, grad_t))
        torch.cuda.synchronize()
        start.record()
        for s in range(args.naive_steps):
            H, idx, val = pool[s % len(pool)]
            nl.step(H, idx, val, cfg.lr, out=(loss_t, grad_t))
        stop.record()
        torch.cuda.synchronize()
        nms = start.elapsed_time(stop) / args.naive_steps
        if nl.sync() != 0:
            log("device error in naive steps")
            sys.exit(1)
        nl.close()
        naive = {"ms_per_step": round(nms, 4), "speedup": round(nms / ms_per_step, 2),
                 "D_over_4d": round(cfg.D / (4 * cfg.d), 2), "steps": args.naive_steps}
        log(f"naive: {nms:.3f} ms/step, speedup {nms / ms_per_step:.1f} (D/4d = {cfg.D / (4 * cfg.d):.0f})")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, wl, V0, args.cpu_seconds)
        log(f"cpu oracle: {cpu['value']:.4g} examples/s on {cpu['cores']} threads")

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "examples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "D": cfg.D, "d": cfg.d, "m": cfg.m, "K": cfg.K,
                   "loss": cfg.loss, "lr": cfg.lr, "global_batch": cfg.m,
                   "parallelism": "none"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "naive": naive,
        "single_example": single,
        "stabilize": stab,
        "input_layer": inp,
        "kernels": kernels,
        "tasks": tasks,
        "last_step": {"distinct_rows": u, "pairs": nnz},
    }
    print(json.dumps(out), flush=True)


def task_times(layer, run, cfg, u, steps):
    """Per-task launch times of the minibatch step with every task launched on its
    own (HIP events around each launch, a profiled pass of `steps` steps).

    The gather (launch1.targets: target preparation, Y^T Y and G = V^T Y)
    must read the u distinct target rows of V at least once: 4 u d bytes.  The
    scatter (launch3.scatter, plus launch4.clear, which scatters the rows held
    by 64 or more slots when the step has 4096 or more slots) reads and
    writes them: 8 u d bytes."""
    layer.set_split_tasks(True)
    run(20)
    layer.profile(True)
    run(steps)
    phases, n = layer.profile_read()
    layer.profile(False)
    layer.set_split_tasks(False)
    if layer.sync() != 0:
        log("device error in split-task steps")
        sys.exit(1)
    out = {}
    for name, tot in phases.items():
        if "." in name and tot > 0:
            out[name] = {"avg_us": round(1e3 * tot / max(n, 1), 3)}
    hot = cfg.m * cfg.K >= 4096
    for name, nbytes, parts in (("gather", 4.0 * u * cfg.d, ["launch1.targets"]),
                                ("scatter", 8.0 * u * cfg.d,
                                 ["launch3.scatter"] + (["launch4.clear"] if hot else []))):
        t = sum(out[p]["avg_us"] for p in parts if p in out)
        if t > 0:
            gbs = nbytes / (t * 1e-6) / 1e9
            out[name] = {"tasks": parts, "avg_us": round(t, 3), "bytes": nbytes,
                         "hbm_gbs": round(gbs, 1), "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}
    return out


def tasks_only(args):
    """`--tasks`: the split-task measurement alone (for a kernel trace)."""
    import torch

    import paper_1412_7091_amd as lst
    from synth import Workload, get_config

    cfg = get_config(args.config)
    wl = Workload(cfg)
    dev = torch.device("cuda:0")
    V0_t = torch.from_numpy(wl.init_V()).to(dev)
    pool = [tuple(torch.from_numpy(x).to(dev) for x in wl.batch(s)) for s in range(16)]
    loss_t = torch.empty(cfg.m, device=dev)
    grad_t = torch.empty((cfg.m, cfg.d), device=dev)
    layer = lst.FactoredOutputLayer(V0_t, loss=cfg.loss, sph_eps=cfg.sph_eps, m_max=cfg.m,
                                    K_max=cfg.K)

    def run(n, offset=0):
        for s in range(n):
            H, idx, val = pool[(s + offset) % len(pool)]
            layer.step(H, idx, val, cfg.lr, out=(loss_t, grad_t))

    layer.set_split_tasks(True)
    run(args.warmup)
    u = layer.stats().last_unique
    tasks = task_times(layer, run, cfg, u, args.steps)
    layer.close()
    print(json.dumps({"tasks": tasks, "distinct_rows": u, "steps": args.steps,
                      "config": {"workload": cfg.name, "D": cfg.D, "d": cfg.d, "m": cfg.m,
                                 "K": cfg.K}}), flush=True)


def single_example_cost(lst, torch, cfg, V0_t, dev, steps=2000):
    """The m = 1 step (Algorithm 1 with the Sherman-Morrison update of U^-T) on
    the workload's D, d and K: pipelined time per step (HIP events around
    `steps` back-to-back steps), latency of one step (host clock from the call
    to the end of a synchronisation, median of 200), and its launches.

    Algorithmic bytes: launch A reads Q, U, U^-T (3 d^2 floats) and the u
    target rows of V; launch B reads and writes Q, U, U^-T and its columns of
    the target rows (2 (3 d^2 + u d) floats)."""
    import dataclasses

    from synth import Workload

    c1 = dataclasses.replace(cfg, m=1)
    wl1 = Workload(c1)
    pool = [tuple(torch.from_numpy(x).to(dev) for x in wl1.batch(s)) for s in range(16)]
    layer = lst.FactoredOutputLayer(V0_t, loss=cfg.loss, sph_eps=cfg.sph_eps, m_max=1,
                                    K_max=cfg.K)
    out = (torch.empty(1, device=dev), torch.empty((1, cfg.d), device=dev))

    def run(n):
        for s in range(n):
            layer.step(*pool[s % 16], cfg.lr, out=out)

    run(50)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    run(steps)
    e1.record()
    torch.cuda.synchronize()
    us = 1e3 * e0.elapsed_time(e1) / steps
    lat = []
    for s in range(200):
        t0 = time.perf_counter()
        layer.step(*pool[s % 16], cfg.lr, out=out)
        torch.cuda.synchronize()
        lat.append(1e6 * (time.perf_counter() - t0))
    layer.profile(True)
    run(500)
    phases, n = layer.profile_read()
    layer.profile(False)
    u = layer.stats().last_unique
    if layer.sync() != 0:
        log("device error in single-example steps")
        sys.exit(1)
    layer.close()
    launches = {}
    for name, tot in phases.items():
        if tot <= 0:
            continue
        avg = 1e3 * tot / max(n, 1)
        nb = {"online_a": 4.0 * (3 * cfg.d * cfg.d + u * cfg.d),
              "online_b": 8.0 * (3 * cfg.d * cfg.d + u * cfg.d)}.get(name, 0.0)
        launches[name] = {"avg_us": round(avg, 3), "bytes": nb,
                          "hbm_frac": round(nb / (avg * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    return {"us_per_step": round(us, 3), "latency_us_median": round(float(np.median(lat)), 2),
            "examples_per_s": round(1e6 / us, 1), "launches": launches,
            "minibatch_path_m1_us": "26-31 (four-launch minibatch step with m = 1, before "
                                    "the single-example path)"}


def stabilize_cost(lst, torch, cfg, V0_t, dev):
    """Cost of one Appendix C stabilisation call on a state of the workload's size.

    Two states: U = I (every singular value in range: one power-iteration
    round at each end, no correction) and U with one singular value of 1e-4
    (one correction: rank-one updates of U and U^{-T}, a pass over V, and the
    refinement of U^{-T}).  Each call is timed alone, with a report (which
    synchronises).  Not part of the step's throughput.
    """
    from synth import Workload

    def timed(layer):
        layer.stabilize(sigma_low=1e-3, sigma_high=100.0, squarings=7, max_fixes=1, reinvert=1)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        rep = layer.stabilize(sigma_low=1e-3, sigma_high=100.0, squarings=7, max_fixes=1,
                              reinvert=1)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1), rep

    layer = lst.FactoredOutputLayer(V0_t, loss=cfg.loss, sph_eps=cfg.sph_eps, m_max=cfg.m,
                                    K_max=cfg.K)
    ms_in, rep_in = timed(layer)
    layer.close()
    U0 = Workload(cfg.replace(u_init="spectrum", u_sigma=(1e-4,))).init_U()
    U0_t = torch.from_numpy(U0).to(dev)
    fix_ms = []
    for _ in range(2):  # the first call warms up; a fresh state each time (one fix each)
        layer = lst.FactoredOutputLayer(V0_t, U0_t, loss=cfg.loss, sph_eps=cfg.sph_eps,
                                        m_max=cfg.m, K_max=cfg.K)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        rep = layer.stabilize(sigma_low=1e-3, sigma_high=100.0, squarings=7, max_fixes=1,
                              reinvert=1)
        e1.record()
        torch.cuda.synchronize()
        fix_ms.append(e0.elapsed_time(e1))
        layer.close()
    return {"ms_in_range": round(ms_in, 4), "ms_one_fix": round(fix_ms[-1], 4),
            "fixes": [rep_in.fixes_low + rep_in.fixes_high, rep.fixes_low + rep.fixes_high],
            "V_pass_bytes": 2 * cfg.D * cfg.d * 4, "squarings": 7}


SWEEP_D = (10_000, 50_000, 100_000, 200_000, 400_000, 793_471)


def sweep(args):
    """Step time of the factored and the naive (explicit W) output layer over D.

    d = 300, m = 128, one target word per example (K = 1, value 1, uniform),
    squared error, lr = 1e-3: the setting of the paper's timing figure and of
    its speedup table (D = 793 471).  At the largest D the fp64 CPU oracle
    (explicit W) is timed too, as the table's CPU-naive reference, and the
    factored step is also timed at m = 1 (one example per step).  Prints one
    JSON object.
    """
    import torch

    import paper_1412_7091_amd as lst
    from synth import Workload, WorkloadConfig

    lst.load_library()
    dev = torch.device("cuda:0")
    rows = []
    for D in SWEEP_D:
        cfg = WorkloadConfig(name=f"sweep_D{D}", D=D, d=300, m=128, K=1, loss="squared",
                             lr=1e-3, idx_dist="uniform", val_dist="one",
                             entropy=14127091 + 100 + SWEEP_D.index(D))
        wl = Workload(cfg)
        V0 = wl.init_V()
        V0_t = torch.from_numpy(V0).to(dev)
        pool = [tuple(torch.from_numpy(x).to(dev) for x in wl.batch(s)) for s in range(8)]
        loss_t = torch.empty(cfg.m, device=dev)
        grad_t = torch.empty((cfg.m, cfg.d), device=dev)

        def timed(layer, n, warm, m=None):
            def one(s):
                H, idx, val = pool[s % len(pool)]
                if m is not None:
                    H, idx, val = H[:m].contiguous(), idx[:m].contiguous(), val[:m].contiguous()
                    layer.step(H, idx, val, cfg.lr, out=(loss_t[:m], grad_t[:m]))
                else:
                    layer.step(H, idx, val, cfg.lr, out=(loss_t, grad_t))
            for s in range(warm):
                one(s)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for s in range(n):
                one(warm + s)
            e1.record()
            torch.cuda.synchronize()
            assert layer.sync() == 0
            return e0.elapsed_time(e1) / n

        fl = lst.FactoredOutputLayer(V0_t, m_max=cfg.m, K_max=cfg.K)
        f_ms = timed(fl, 200, 20)
        row = {"D": D, "factored_us": round(1e3 * f_ms, 2)}
        if D == SWEEP_D[-1]:
            row["factored_m1_us"] = round(1e3 * timed(fl, 200, 20, m=1), 2)
        fl.close()
        nl = lst.NaiveOutputLayer(V0_t, m_max=cfg.m, K_max=cfg.K)
        n_ms = timed(nl, 10, 2)
        nl.close()
        row.update(naive_us=round(1e3 * n_ms, 2), speedup=round(n_ms / f_ms, 2),
                   D_over_4d=round(D / (4 * cfg.d), 2))
        if D == SWEEP_D[-1] and not args.no_cpu_baseline:
            from oracle import explicit

            W = V0.astype(np.float64)
            t0 = time.perf_counter()
            n = 0
            while n < 2 or (time.perf_counter() - t0 < args.cpu_seconds and n < 10):
                H, idx, val = wl.batch(n)
                _, _, W = explicit.step(W, H, idx, val, cfg.lr, cfg.loss, cfg.sph_eps)
                n += 1
            cpu_ms = 1e3 * (time.perf_counter() - t0) / n
            row.update(cpu_naive_oracle_ms=round(cpu_ms, 1),
                       speedup_vs_cpu_naive=round(cpu_ms / f_ms, 1),
                       naive_gpu_vs_cpu_naive=round(cpu_ms / n_ms, 1))
        log(json.dumps(row))
        rows.append(row)
        del V0_t, pool
        torch.cuda.empty_cache()
    print(json.dumps({"sweep": "factored vs naive output-layer step over D", "d": 300, "m": 128,
                      "K": 1, "loss": "squared", "dtype": "f32", "data": "synthetic",
                      "rows": rows}), flush=True)
    return 0


CROSS_M = (1, 2, 4, 8, 16, 32, 64, 128, 256, 512)
CROSS_D = (500, 1024)


def crossover(args):
    """Woodbury update of U^{-T} (lst_step) against solving U_new^T Z = H from
    scratch (lst_step_solve), both the library's own kernels, over m at d = 500
    and 1024 (D = 200000, K = 10, squared error).

    The paper notes that for large m it may pay to solve the d x d system with
    U_new every minibatch instead of keeping U^{-T} through the Woodbury
    identity.  Per step the Woodbury form spends 2 d^2 m on the U^{-T} panel of
    the first product, about 2 n m^2 d on the Neumann solve (n iterations) and
    2 d^2 m on the U^{-T} update; the from-scratch form spends (2/3) d^3 on the
    pivoted factorisation of U_new and 2 d^2 m on the triangular solves.  For
    each d and m: both steps' time (HIP events around back-to-back steps), the
    from-scratch step's factorisation and solve phases, and the flop model.
    Prints one JSON object.
    """
    import torch

    import paper_1412_7091_amd as lst
    from synth import Workload, WorkloadConfig

    lst.load_library()
    dev = torch.device("cuda:0")
    out = []
    for d in CROSS_D:
        cfg = WorkloadConfig(name=f"cross_d{d}", D=200_000, d=d, m=max(CROSS_M), K=10,
                             loss="squared", lr=1e-3, entropy=14127091 + 300 + d)
        wl = Workload(cfg)
        V0_t = torch.from_numpy(wl.init_V()).to(dev)
        pool = [tuple(torch.from_numpy(x).to(dev) for x in wl.batch(s)) for s in range(4)]
        wood = lst.FactoredOutputLayer(V0_t, m_max=cfg.m, K_max=cfg.K)
        scr = lst.FactoredOutputLayer(V0_t, m_max=cfg.m, K_max=cfg.K)
        loss_t = torch.empty(cfg.m, device=dev)
        grad_t = torch.empty((cfg.m, d), device=dev)
        n_it = 4
        for m in CROSS_M:
            sub = [tuple(x[:m].contiguous() for x in b) for b in pool]
            row = {"d": d, "m": m, "woodbury_flops": 4 * d * d * m + 2 * n_it * m * m * d,
                   "scratch_flops": int(2 * d ** 3 / 3) + 2 * d * d * m}
            for name, layer, fn in (("woodbury", wood, wood.step), ("scratch", scr, scr.step_solve)):
                nsteps = 100 if name == "woodbury" else 30

                def run(n, offset=0):
                    for s in range(n):
                        H, idx, val = sub[(offset + s) % len(sub)]
                        fn(H, idx, val, cfg.lr, out=(loss_t[:m], grad_t[:m]))

                run(5)
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                run(nsteps, 5)
                e1.record()
                torch.cuda.synchronize()
                if layer.sync() != 0:
                    log(f"device error in the {name} step at d={d} m={m}")
                    sys.exit(1)
                row[f"{name}_us"] = round(1e3 * e0.elapsed_time(e1) / nsteps, 2)
                if name == "scratch":
                    layer.profile(True)
                    run(10)
                    phases, n = layer.profile_read()
                    layer.profile(False)
                    row["scratch_phases_us"] = {k: round(1e3 * v / max(n, 1), 1)
                                                for k, v in phases.items() if v > 0}
            row["faster"] = "woodbury" if row["woodbury_us"] <= row["scratch_us"] else "scratch"
            out.append(row)
            log(json.dumps(row))
        wood.close()
        scr.close()
        del V0_t, pool
        torch.cuda.empty_cache()
    cross = {}
    for d in CROSS_D:
        ms = [r["m"] for r in out if r["d"] == d and r["faster"] == "scratch"]
        cross[str(d)] = min(ms) if ms else None
    print(json.dumps({"crossover": "Woodbury step (lst_step) vs solve-from-scratch step "
                                   "(lst_step_solve)",
                      "D": 200_000, "K": 10, "loss": "squared", "dtype": "f32",
                      "data": "synthetic", "first_m_scratch_faster": cross, "rows": out}),
          flush=True)
    return 0


def input_layer_cost(lst, torch, cfg, wl, V0_t, pool):
    """Section 2.2 input layer at the workload's sizes (D_in = D, d, m, K = the
    targets' K as input pairs): mean time of a forward and of an update over
    the pool of minibatches (the batch's H stands in for dL/dA)."""
    layer = lst.SparseInputLayer(V0_t)
    A = torch.empty((cfg.m, cfg.d), dtype=torch.float32, device=V0_t.device)
    res = {}
    for what in ("forward", "update"):
        def run(n):
            for s in range(n):
                H, idx, val = pool[s % len(pool)]
                if what == "forward":
                    layer.forward(idx, val, out=A)
                else:
                    layer.update(idx, val, H, 1e-6)
        run(10)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run(200)
        e1.record()
        torch.cuda.synchronize()
        res[f"{what}_us"] = round(1e3 * e0.elapsed_time(e1) / 200, 3)
    assert layer.sync() == 0
    layer.close()
    res["rows_per_minibatch"] = cfg.m * cfg.K
    return res


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform

    return platform.processor() or platform.machine()


def cpu_baseline(cfg, wl, V0, seconds):
    """The fp64 oracle (explicit W, O(D d) per example) on a bounded prefix of the
    same steps: median time per step over the steps run, the CPU model, and the
    BLAS library numpy calls (vendor, version, threads)."""
    from oracle import explicit

    blas = {}
    try:
        from threadpoolctl import threadpool_info

        for i in threadpool_info():
            if i.get("user_api") == "blas":
                blas = {"vendor": i.get("internal_api"), "version": i.get("version"),
                        "threads": i.get("num_threads"), "arch": i.get("architecture")}
                break
    except Exception:  # pragma: no cover - threadpoolctl missing
        pass
    threads = blas.get("threads") or len(os.sched_getaffinity(0))
    W = V0.astype(np.float64)
    times = []
    t0 = time.perf_counter()
    n = 0
    while True:
        H, idx, val = wl.batch(n)
        ts = time.perf_counter()
        _, _, W = explicit.step(W, H, idx, val, cfg.lr, cfg.loss, cfg.sph_eps)
        times.append(time.perf_counter() - ts)
        n += 1
        el = time.perf_counter() - t0
        if (el >= seconds and n >= 3) or n >= 1000:
            break
    med = float(np.median(times))
    return {"value": round(cfg.m / med, 3), "unit": "examples/s", "cores": threads,
            "kind": "oracle", "statistic": "median",
            "cpu_model": _cpu_model(), "blas": blas,
            "sample": f"{n} consecutive steps of {cfg.name} from its initial W, fp64 numpy; "
                      f"median {med * 1e3:.1f} ms per step (mean {1e3 * float(np.mean(times)):.1f}), "
                      f"{el:.1f}s wall"}


if __name__ == "__main__":
    main()
