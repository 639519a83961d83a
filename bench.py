#!/usr/bin/env python3
"""Benchmark of the GreedyLore compression step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME]

One step is one pass of the whole path over one batch of worker gradients:
error feedback + worker mean, the semi-lazy subspace (a full Jacobi SVD
refresh every tau steps, Approx-Top-r selection otherwise), projection,
residual, mean, reconstruction and the MSGD/Adam update.  Steps t = W .. W+K-1
of the trajectory are timed (warm-up t = 0 .. W-1 includes the cold first
refresh), so K a multiple of tau times whole refresh periods.

Inputs are resident in HBM before the timed region: the planted part of the
synthetic gradients is drawn on the host, the per-step noise on the device
from a seeded torch generator, into a pool of distinct gradient batches.

Steps t = W .. W+K-1 are timed with no instrumentation inside the step; the
next K steps run again with HIP events around every launch group, on the
library's stream, for the per-kernel averages; then 2 tau steps are timed one
by one (median of the refresh steps and of the selection steps, and the
sweeps of the cold first refresh and of the last warm one).  Prints one JSON line: ms/step,
effective GB/s, the roofline of the dominant kernel (its algorithmic work per
launch over its average event-timed duration), the per-kernel breakdown, and
the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12           # bytes/s
FP32_MFMA_PEAK = 157.3e12   # flop/s, dense
FP64_MFMA_PEAK = 78.6e12
BF16_MFMA_PEAK = 2.5e15     # dense bf16 (the selection products of the approx_bf16 mode)
METRIC = "ms/step and effective HBM GB/s for compress+EF+update; % of roofline"


def dims(shape):
    m, n = shape
    return m, n, min(m, n), max(m, n)


def jac_groups(d, jb=16):
    """(blocks per group, groups per round, rounds per sweep) of the Jacobi
    tournament: groups of four on 4^j seats when the 16-row blocks nearly fill
    a power of 4 of at least 64 (S - 1) / 3 rounds), pairs otherwise (circle
    method, S - 1 rounds)."""
    nb = (d + jb - 1) // jb
    s4 = 4
    while s4 < nb:
        s4 *= 4
    if nb >= 64 and 4 * nb >= 3 * s4:
        return 4, s4 // 4, (s4 - 1) // 3
    seats = max(2, nb + (nb & 1))
    return 2, seats // 2, seats - 1


def uses_subspace(wl, d):
    r = min(wl.rank, d)
    return wl.tau == 1 and r < d and r <= 256


FP64_ALU_PEAK = 78.6e12     # fp64 vector flop/s (the pair eigensolves)

# groups that are one kernel launch each (the candidates for the dominant kernel)
KERNEL_GROUPS = ("ef_mean", "select", "proj", "resid_opt", "jac_update", "jac_solve",
                 "rr_update", "rr_solve", "sub_z", "sub_p")


def jacobi_work(kind, d):
    """Per-launch work of one Jacobi round on the fp64 Gram of d rows (16-row
    blocks, groups of NG blocks = NR rows): (bytes, fp32 MFMA flops, fp64
    MFMA flops, fp64 ALU flops)."""
    ng, groups, _ = jac_groups(d)
    nr = 16 * ng
    nb = (d + 15) // 16
    if kind == "update":
        # A <- J^T A J on the packed upper blocks: read + write, two NR x NR x NR
        # fp64 products per pair of groups
        return 2.0 * nb * (nb + 1) / 2 * 256 * 8, 0.0, groups * (groups + 1) / 2 * 2 * 2.0 * nr ** 3, 0.0
    # solve: one cyclic sweep of NR x NR two-sided Jacobi per group (NR (NR - 1)
    # / 2 rotations, each updating two rows and two columns of G and two
    # columns of V), in the same launch as the previous round's U^T <- J^T U^T
    # (read + write the NR rows of every group, one NR x NR x d fp32 product)
    rot = nr * (nr - 1) / 2
    return groups * nr * d * 8.0, groups * 2.0 * nr * nr * d, 0.0, groups * rot * (6 * nr * 3)


def group_work(wl, name, esz=4):
    """Algorithmic bytes and flops of ONE launch of a kernel group, averaged
    over the matrices of the workload that launch it: (bytes, fp32 MFMA
    flops, fp64 MFMA flops, fp64 ALU flops).  esz: bytes of one element of G
    and E (4, or 2 with bf16 storage)."""
    N = wl.workers
    tot = [0.0, 0.0, 0.0, 0.0]
    count = 0
    for shape in wl.shapes:
        m, n, d, D = dims(shape)
        r = min(wl.rank, d)
        mn = m * n
        adam = wl.opt == "adam"
        sub = uses_subspace(wl, d)
        K = min(r + max(32, r // 4), d)
        w = None
        if name == "ef_mean":
            w = ((esz * N + 8.0) * mn, 0, 0, 0)
        elif name == "select" and r < d:
            w = (4.0 * (d * D + d * d), 2.0 * d * d * D, 0, 0)
        elif name == "proj":
            w = (2.0 * esz * N * mn + 4.0 * N * r * D, 2.0 * r * d * D * N, 0, 0)
        elif name == "resid_opt":
            # G, E read and E written per worker; Ebar written (the mean of
            # the stored residuals, summed in registers); X and the optimizer
            # state read and written.  Products: P Q^(i) per worker, and
            # Ghat = P Rbar as a product of its own up to rank 128 (above it
            # Ghat is the mean of the workers' products)
            prods = N if r > 128 else N + 1
            w = ((3.0 * esz * N + 4 + (24 if adam else 16)) * mn + 4.0 * N * r * D, 2.0 * r * d * D * prods, 0, 0)
        elif name.startswith("jac_") and not sub:
            w = jacobi_work(name[4:], d)
        elif name.startswith("rr_") and sub:
            w = jacobi_work(name[3:], K)
        elif name in ("sub_z", "sub_p") and sub:
            w = (4.0 * (d * D + K * d + K * D), 2.0 * K * d * D, 0, 0)
        elif name == "sub_chol" and sub:
            w = (0.0, 0.0, 0.0, 2.0 * K ** 3 / 3.0)
        if w is not None:
            count += 1
            for i in range(4):
                tot[i] += w[i]
    if count == 0:
        return None
    return tuple(x / count for x in tot)


def roofline_entry(wl, name, total_ms, launches, select="approx", esz=4):
    work = group_work(wl, name, esz)
    if work is None or launches == 0 or total_ms <= 0:
        return None
    avg_s = total_ms / 1e3 / launches
    byts, f32, f64, alu = work
    t_hbm = byts / HBM_PEAK
    # the approx_bf16 selection runs its products on the bf16 matrix cores
    f32_peak = BF16_MFMA_PEAK if (name == "select" and select == "approx_bf16") else FP32_MFMA_PEAK
    t_mfma = f32 / f32_peak + f64 / FP64_MFMA_PEAK
    t_alu = alu / FP64_ALU_PEAK
    base = {"kernel": name, "avg_us": avg_s * 1e6, "launches": launches,
            "bytes_per_launch": byts, "flops_per_launch": f32 + f64 + alu}
    if t_hbm == 0 and t_mfma == 0 and t_alu == 0:
        return None
    if t_hbm >= t_mfma and t_hbm >= t_alu:
        base.update({"bound": "hbm", "achieved": byts / avg_s / 1e9, "peak": HBM_PEAK / 1e9,
                     "unit": "GB/s", "frac": t_hbm / avg_s})
    elif t_mfma >= t_alu:
        fl = f32 + f64
        base.update({"bound": "mfma", "achieved": fl / avg_s / 1e12, "peak": fl / t_mfma / 1e12,
                     "unit": "TFLOP/s", "frac": t_mfma / avg_s})
    else:
        base.update({"bound": "alu", "achieved": alu / avg_s / 1e12, "peak": FP64_ALU_PEAK / 1e12,
                     "unit": "TFLOP/s", "frac": t_alu / avg_s})
    return base


# kernel group -> HIP source that defines it (for the traffic bookkeeping)
KERNEL_SOURCES = {
    "ef_mean": "glr_step_kernels.hip", "select": "glr_step_kernels.hip", "proj": "glr_step_kernels.hip",
    "resid_opt": "glr_step_kernels.hip", "jac_update": "glr_jacobi.hip", "jac_solve": "glr_jacobi.hip",
    "rr_update": "glr_jacobi.hip", "rr_solve": "glr_jacobi.hip", "sub_z": "glr_subspace.hip",
    "sub_p": "glr_subspace.hip", "sub_chol": "glr_subspace.hip",
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def source_sha256(name):
    """Digest of the source of a kernel group (its .hip file and the shared
    device headers): a traffic figure applies only to the code it was taken on."""
    src = os.path.join(ROOT, "paper_2507_08784_amd", "csrc")
    h = hashlib.sha256()
    for f in (KERNEL_SOURCES[name], "glr_device.hpp", "glr_internal.hpp"):
        with open(os.path.join(src, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload, name):
    """HBM bytes per launch from the committed rocprofv3 counter runs
    (FETCH_SIZE + WRITE_SIZE, each scaled by the same counter's reading on a
    plain copy of known size), or None when there is none for this kernel,
    workload and source."""
    try:
        with open(TRAFFIC_FILE) as fh:
            table = json.load(fh)
    except (OSError, ValueError):
        return None
    e = table.get(workload, {}).get(name)
    if not e or e.get("source_sha256") != source_sha256(name):
        return None
    return e.get("bytes_per_launch")


def copy_probe(device):
    """A plain device-to-device copy of 1 GiB, three times: the calibration
    kernel for the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    n = 1 << 28
    a = torch.ones(n, dtype=torch.float32, device=device)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": 4 * n, "launches": 3}), flush=True)


def step_bytes(wl, esz=4):
    """Algorithmic HBM bytes of one step: per worker read G, read E, write E
    (12 B/elem, 6 with bf16 storage) plus the optimizer (16 B/elem MSGD, 24
    Adam)."""
    tot = 0
    for shape in wl.shapes:
        m, n, _, _ = dims(shape)
        tot += (3 * esz * wl.workers + (24 if wl.opt == "adam" else 16)) * m * n
    return tot


def make_pool(wl, pool, device, seed=1234, store="fp32"):
    import numpy as np
    import torch
    from synth import noise_level, planted_matrix
    planted = [torch.from_numpy(planted_matrix(wl, l).astype(np.float32)).to(device)
               for l in range(len(wl.shapes))]
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    batches = []
    for _ in range(pool):
        gs = []
        for l, (m, n) in enumerate(wl.shapes):
            g = torch.randn((wl.workers, m, n), generator=gen, device=device, dtype=torch.float32)
            g.mul_(noise_level(wl, l)).add_(planted[l])
            gs.append(g.to(torch.bfloat16) if store == "bf16" else g)
        batches.append(gs)
    return batches


def host_cpu():
    """(usable cores, CPU model) of the host the oracle runs on."""
    try:
        ncpu = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        ncpu = os.cpu_count() or 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return ncpu, model


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return 1


def cpu_baseline(wl, budget_s, store="fp32"):
    """The oracle as it stands, timed on the host: whole oracle steps
    t = 0, 1, ... of the same workload (the full matrices, every worker,
    t = 0 a cold refresh), until `budget_s` of oracle time is spent (at least
    one step).  Gradient generation is not timed.  Returns (seconds per step,
    steps timed, refresh steps among them)."""
    from oracle.method import Oracle
    from synth import gradient_batch, planted_matrix
    planted = [planted_matrix(wl, l) for l in range(len(wl.shapes))]
    orc = Oracle.from_workload(wl, store=store)
    spent, steps, refresh = 0.0, 0, 0
    while steps == 0 or (spent < budget_s and steps < wl.steps):
        grads = [gradient_batch(wl, l, steps, planted[l]) for l in range(len(wl.shapes))]
        t0 = time.perf_counter()
        orc.step(grads, steps)
        spent += time.perf_counter() - t0
        refresh += 1 if steps % wl.tau == 0 else 0
        steps += 1
        del grads
        print(f"[bench] oracle step {steps - 1}: {spent:.1f}s so far", file=sys.stderr, flush=True)
    return spent / steps, steps, refresh


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="large_8192x28672")
    ap.add_argument("--cpu-budget", type=float, default=20.0,
                    help="seconds of oracle time for the CPU baseline (whole steps, at least one)")
    ap.add_argument("--pool", type=int, default=11)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true")
    ap.add_argument("--tol", type=float, default=1e-6, help="refresh tolerance")
    ap.add_argument("--select", default="approx", choices=("approx", "exact", "approx_bf16"),
                    help="selection mode (approx: the method's Approx-Top-r in fp32; approx_bf16: its "
                         "products on bf16 roundings of U and Mbar, a mixed-precision mode)")
    ap.add_argument("--store", default="fp32", choices=("fp32", "bf16"),
                    help="storage of the gradients and error buffers (bf16: a mixed-precision mode)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run the 1 GiB copy that calibrates the HBM traffic counters")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one MI355X: the N workers of the method are simulated on one "
              "GPU, and multi-GPU runs are not part of this build (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2507_08784_amd as glr
    from synth import get_workload
    glr.load()   # no CPU fallback: fails loudly if the library is missing
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.copy_probe:
        copy_probe(dev)
        return
    wl = get_workload(args.workload)

    pool_bytes = sum(wl.workers * m * n * 4 for m, n in wl.shapes)
    pool = max(1, min(args.pool, int(40e9 // pool_bytes)))
    print(f"[bench] workload {wl.name}: shapes {list(wl.shapes)[:3]}{'...' if len(wl.shapes) > 3 else ''} "
          f"N={wl.workers} r={wl.rank} tau={wl.tau} opt={wl.opt}; pool {pool}", file=sys.stderr, flush=True)
    batches = make_pool(wl, pool, dev, store=args.store)
    esz = 2 if args.store == "bf16" else 4
    comp = glr.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr,
                          beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, seed=wl.seed, tol=args.tol,
                          select=args.select, store=args.store, device=dev)
    X = [torch.zeros(m, n, dtype=torch.float32, device=dev) for m, n in wl.shapes]
    torch.cuda.synchronize()

    t_w = time.perf_counter()
    cold_sweeps = None
    for t in range(args.warmup):
        comp.step(X, batches[t % pool], t)
        if t == 0:
            torch.cuda.synchronize()
            cold_sweeps = [int(comp.info(l)[0]) for l in range(len(wl.shapes))]
    torch.cuda.synchronize()
    print(f"[bench] warm-up {args.warmup} steps {time.perf_counter() - t_w:.2f}s", file=sys.stderr, flush=True)
    # pass 1: the timed region (no event brackets inside the step)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(args.warmup, args.warmup + args.steps):
        comp.step(X, batches[t % pool], t)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / args.steps
    status = comp.sync_status()
    if status not in (0, 7):
        raise RuntimeError(f"device status {glr.STATUS_NAMES.get(status, status)}")
    sweeps = [int(comp.info(l)[0]) for l in range(len(wl.shapes))]
    history = [round(h, 9) for h in comp.sweep_history(0)[2]]
    n_refresh = sum(1 for t in range(args.warmup, args.warmup + args.steps) if t % wl.tau == 0)
    print(f"[bench] timed {args.steps} steps ({n_refresh} refresh): {ms_per_step:.3f} ms/step",
          file=sys.stderr, flush=True)

    # pass 2: the next K steps (the same number of refreshes when K is a
    # multiple of tau) with HIP events around every launch group, on the
    # library's stream: per-kernel averages for the roofline
    prof, prof_ms = {}, None
    if not args.no_profile:
        comp.profile(True)
        comp.profile_reset()
        t1 = time.perf_counter()
        prof_iters = 0
        for t in range(args.warmup + args.steps, args.warmup + 2 * args.steps):
            comp.step(X, batches[t % pool], t)
            if wl.tau == 1:
                # the block iterations the device ran (the rest of the enqueued
                # ones returned at once): the launch count of their groups
                torch.cuda.synchronize()
                prof_iters += sum(comp.sub_info(l)[0] for l in range(len(wl.shapes)))
        torch.cuda.synchronize()
        prof_ms = (time.perf_counter() - t1) * 1e3 / args.steps
        prof = comp.profile_query()
        comp.profile(False)
        status = comp.sync_status()
        if status not in (0, 7):
            raise RuntimeError(f"device status {glr.STATUS_NAMES.get(status, status)}")
        print(f"[bench] profiled pass: {prof_ms:.3f} ms/step", file=sys.stderr, flush=True)

    # pass 3: 2 tau more steps, each between two events on the step's stream:
    # median time of a refresh step and of a selection step
    t_next = args.warmup + (args.steps if args.no_profile else 2 * args.steps)
    n3 = max(2, 2 * wl.tau)
    per_type = {"refresh": [], "select": []}
    sub_iters = []
    stream = torch.cuda.current_stream(dev)
    for t in range(t_next, t_next + max(n3, 8 if wl.tau == 1 else 0)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        comp.step(X, batches[t % pool], t)
        e1.record(stream)
        e1.synchronize()
        per_type["refresh" if t % wl.tau == 0 else "select"].append(e0.elapsed_time(e1))
        if wl.tau == 1:
            sub_iters.append(comp.sub_info(0)[0])
    warm_sweeps = [int(comp.info(l)[0]) for l in range(len(wl.shapes))]
    status = comp.sync_status()
    if status not in (0, 7):
        raise RuntimeError(f"device status {glr.STATUS_NAMES.get(status, status)}")
    step_types = {k: {"median_ms": round(statistics.median(v), 4), "steps": len(v)}
                  for k, v in per_type.items() if v}

    if wl.tau == 1 and prof:
        for name in ("sub_z", "sub_p"):
            if name in prof and prof[name][1]:
                prof[name] = (prof[name][0], prof_iters)
    kernels = []
    for name in KERNEL_GROUPS:
        if name in prof and prof[name][1]:
            e = roofline_entry(wl, name, *prof[name], select=args.select, esz=esz)
            if e:
                e["total_ms"] = prof[name][0]
                kernels.append(e)
    groups = {k: {"total_ms": v[0], "launches": v[1]} for k, v in prof.items() if v[1]}
    dominant = max(kernels, key=lambda e: e["total_ms"]) if kernels else None
    roof = None
    if dominant:
        roof = {k: dominant[k] for k in ("bound", "achieved", "peak", "unit", "frac")}
        roof["kernel"] = dominant["kernel"]
        roof["avg_us"] = dominant["avg_us"]
        roof["traffic"] = measured_traffic(wl.name + (":bf16" if args.store == "bf16" else ""), dominant["kernel"])

    eff = step_bytes(wl, esz) / (ms_per_step / 1e3) / 1e9
    out = {
        "metric": METRIC, "value": round(ms_per_step, 4), "unit": "ms/step",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": ("f32" if args.select != "approx_bf16" else "f32 (selection products on bf16)")
                 + (" (G, E stored bf16)" if args.store == "bf16" else ""),
        "data": "synthetic (planted-spectrum gradients + seeded Gaussian noise, resident in HBM)",
        "config": {"workload": wl.name, "shapes": [list(s) for s in wl.shapes][:4],
                   "num_matrices": len(wl.shapes), "simulated_workers": wl.workers,
                   "rank": wl.rank, "tau": wl.tau, "optimizer": wl.opt,
                   "refresh_steps_timed": n_refresh, "select": args.select, "store": args.store},
        "effective_GBps": round(eff, 1),
        "roofline": roof,
        "profiled_ms_per_step": None if prof_ms is None else round(prof_ms, 4),
        "kernels": kernels,
        "groups": groups,
        "refresh_sweeps_last": sweeps,
        "refresh_history_last": history,
        "step_types": step_types,
        "refresh_sweeps_cold": cold_sweeps,
        "tau1_block_iterations": sub_iters or None,
        "refresh_sweeps_warm": warm_sweeps,
        "status": glr.STATUS_NAMES.get(status, status),
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        sec, nsteps, nref = cpu_baseline(wl, args.cpu_budget, args.store)
        ncpu, model = host_cpu()
        out["cpu_baseline"] = {
            "value": round(sec * 1e3, 1), "unit": "ms/step", "cores": blas_threads(), "kind": "oracle",
            "sample": (f"oracle steps t=0..{nsteps - 1} of {wl.name} ({nref} refresh, t=0 cold) on the full "
                       f"matrices, {sec:.1f}s per step; fp64 numpy, BLAS threads as cores; host nproc={ncpu}, "
                       f"{model}"),
        }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
