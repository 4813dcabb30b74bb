#!/usr/bin/env python3
"""Benchmark of the Periodic Row-wise Muon optimizer step on one MI355X.

    python bench.py [--gpus 1] [--steps S] [--warmup W] [--config 2] [--K K]

A "step" is one optimizer step t of the whole hot path over every matrix of a
synthetic DiT-shaped weight set (inputs resident in HBM): momentum update, then
NS5 refresh when t mod K = 0, else the row-wise RowNorm step, then the
parameter write.  Warmup runs steps t = 0..W-1; the timed window runs
t = W..W+S-1 (with the defaults it starts at a refresh and covers two whole
periods).  ``value`` is the amortized optimizer time per step over a period,
(T_refresh + (K-1) T_rowwise) / K, from HIP events on the library's stream.

After the timed window one more period runs with per-kernel HIP events
(libprm's profiling hooks) to attribute time to kernels; the dominant kernel's
algorithmic FLOPs (or bytes) per launch over its mean launch time give the
``roofline`` object.  The oracle (fp64 NumPy) is timed on a bounded sample of
the same workload on the host cores and extrapolated (``cpu_baseline``).
Unless ``--no-other-workloads`` is given, the other DiT-shaped weight sets are
then timed the same way, one after the other (``other_workloads``: refresh,
row-wise and amortized times with their fractions of the spec).

Only rank 0 at N = 1 runs; there is no multi-GPU path.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
METRIC = ("optimizer ms/step (NS5 refresh, row-wise, amortized over K) at DiT-4B; MFMA%/HBM%")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 2K)")
    ap.add_argument("--warmup", type=int, default=None, help="warmup steps (default K)")
    ap.add_argument("--config", type=int, default=2,
                    help="workload index: 0 tiny, 1 DiT-1.3B, 2 DiT-4B (default), 3 DiT-9B, 4 DiT-15B")
    ap.add_argument("--K", type=int, default=None, help="refresh period (default: the workload's)")
    ap.add_argument("--variant", action="append", default=[],
                    choices=["nesterov", "ema_dampening", "gamma_on_refresh", "never_refresh", "ns_plain",
                             "ns_precise"],
                    help="ablation flags of the configuration (repeatable); the default is the paper's method")
    ap.add_argument("--grad-dtype", choices=["bf16", "f32"], default=None,
                    help="gradient storage dtype (default: the workload's, bf16 for the DiT-shaped sets)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="skip timing the other DiT weight sets after the headline one")
    ap.add_argument("--no-profile", action="store_true", help="skip the per-kernel attribution period")
    ap.add_argument("--no-aux", action="store_true", help="skip timing the aux-group AdamW step")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the measured MFMA / HBM ceilings (libprm calibration probes)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a 4 GiB device-to-device copy (HBM bandwidth and counter calibration)")
    return ap.parse_args()


def copy_probe():
    import torch
    n = 1 << 30  # fp32 elements: 4 GiB read + 4 GiB written per copy
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(2):
        y.copy_(x)
    torch.cuda.synchronize()
    reps = 10
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        y.copy_(x)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    gbs = 2 * 4 * n / ms / 1e6
    print(json.dumps({"copy_probe": {"bytes_read": 4 * n, "bytes_written": 4 * n, "ms": ms,
                                     "GB_s": gbs, "frac_of_spec": gbs / PEAK_HBM_GBS}}), flush=True)


def kernel_source_hash() -> str:
    import hashlib
    d = os.path.join(ROOT, "paper_2608_20818_amd", "csrc")
    src = b"".join(open(os.path.join(d, n), "rb").read() for n in sorted(os.listdir(d)))
    return hashlib.sha256(src).hexdigest()[:16]


def counter_traffic(workload: str):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    passes (calibrated on a plain copy), if they were taken on these kernel
    sources and this workload; otherwise None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload.replace('-', '')}.json")
    if not os.path.exists(path):
        return None
    t = json.load(open(path))
    if t.get("kernel_source_sha256_16") != kernel_source_hash() or t.get("workload") != workload:
        return None
    return t["classes"]


def counter_mfma(workload: str):
    """MFMA busy fraction and shader clock per GEMM kind from the committed
    rocprofv3 SQ-counter pass, if it was taken on these kernel sources and this
    workload; otherwise None."""
    path = os.path.join(ROOT, "profiles", f"mfma_{workload.replace('-', '')}.json")
    if not os.path.exists(path):
        return None
    t = json.load(open(path))
    if t.get("kernel_source_sha256_16") != kernel_source_hash() or t.get("workload") != workload:
        return None
    return t["classes"]


def make_inputs(wl_idx, wl, device):
    import torch
    import synth
    W, M, G = [], [], []
    t0 = time.time()
    for i, (m, n) in enumerate(wl.shapes):
        d = synth.device_matrix(wl_idx, i, m, n, synth.rank_of(wl, m, n), param_dtype=wl.param_dtype,
                                grad_dtype=wl.grad_dtype, device=device, beta=wl.beta, step=0)
        W.append(d["W"])
        M.append(d["M"])
        G.append(d["G"])
        if i % 40 == 39:
            torch.cuda.synchronize()
            log(f"[bench] inputs {i + 1}/{len(wl.shapes)} ({time.time() - t0:.1f}s)")
    torch.cuda.synchronize()
    return W, M, G


def other_workload(wl_idx, dev, stream):
    """Refresh and row-wise step times of another weight set (its own K): K
    warmup steps, then 2K timed steps, each bracketed by HIP events on the
    optimizer's stream.  Frees its tensors before returning."""
    import torch

    import paper_2608_20818_amd as prm
    import synth
    from oracle import prm_oracle as po

    wl = synth.WORKLOADS[wl_idx]
    shapes = list(wl.shapes)
    dt = {"f32": prm.F32, "bf16": prm.BF16}
    K = wl.K
    cfg = prm.config_default(K=K, lr=wl.lr, wd=wl.wd, gamma=wl.gamma, beta=wl.beta,
                             param_dtype=dt[wl.param_dtype], grad_dtype=dt[wl.grad_dtype])
    log(f"[bench] other workload {wl.name}: {len(shapes)} matrices, K={K}")
    W, M, G = make_inputs(wl_idx, wl, dev)
    per, kinds = [], []
    with prm.Optimizer(shapes, cfg, stream=stream.cuda_stream) as opt:
        t = 0
        for _ in range(K):
            opt.step(W, G, M, t)
            t += 1
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(2 * K)]
        for e0, e1 in evs:
            e0.record(stream)
            kinds.append(opt.step(W, G, M, t))
            e1.record(stream)
            t += 1
        torch.cuda.synchronize()
        per = [a.elapsed_time(b) for a, b in evs]
    del W, M, G
    torch.cuda.empty_cache()
    T_ref = statistics.median([x for x, k in zip(per, kinds) if k == 1])
    T_rw = statistics.median([x for x, k in zip(per, kinds) if k == 0])
    wb = 2 if wl.param_dtype == "bf16" else 4
    gb = 2 if wl.grad_dtype == "bf16" else 4
    elems = sum(m * n for m, n in shapes)
    ns_flops = sum(po.ns5_flops(m, n) for m, n in shapes)
    rw_bytes = elems * (gb + 4 + 4 + 2 * wb)
    log(f"[bench] {wl.name}: refresh {T_ref:.2f} ms, row-wise {T_rw:.3f} ms")
    return {"workload": wl.name, "matrices": len(shapes), "elements": elems, "K": K,
            "refresh_ms": T_ref, "rowwise_ms": T_rw,
            "amortized_ms": (T_ref + (K - 1) * T_rw) / K,
            "amortized_ms_by_K": {str(k): (T_ref + (k - 1) * T_rw) / k for k in (1, 3, 5, 10)},
            "single_gpu_reduction_K3_vs_K1": (T_ref - (T_ref + 2 * T_rw) / 3) / T_ref,
            "refresh_alg_tflops_frac": ns_flops / (T_ref * 1e-3) / (PEAK_BF16_TFLOPS * 1e12),
            "rowwise_hbm_frac": rw_bytes / (T_rw * 1e-3) / (PEAK_HBM_GBS * 1e9)}


def aux_adamw(wl_idx, wl, dev, stream, steps: int = 50, warmup: int = 5):
    """Time the fused AdamW step of the workload's auxiliary (non-matrix) group:
    HIP events around `steps` back-to-back steps (one launch each, pointers
    bound once), inputs resident in HBM."""
    import torch
    import paper_2608_20818_amd as prm
    import synth

    numels = synth.aux_numels(wl_idx)
    dt = {"f32": prm.F32, "bf16": prm.BF16}
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16}
    P, G, Mo, V = [], [], [], []
    for i, n in enumerate(numels):
        h = synth.host_aux(wl_idx, i, n, param_dtype=wl.param_dtype, grad_dtype=wl.grad_dtype)
        P.append(torch.from_numpy(h["p"]).to(dev).to(tdt[wl.param_dtype]))
        G.append(torch.from_numpy(h["g0"]).to(dev).to(tdt[wl.grad_dtype]))
        Mo.append(torch.from_numpy(h["m"]).to(dev))
        V.append(torch.from_numpy(h["v"]).to(dev))
    cfg = prm.adamw_config_default(param_dtype=dt[wl.param_dtype], grad_dtype=dt[wl.grad_dtype])
    opt = prm.AuxAdamW(numels, cfg, stream=stream.cuda_stream)
    opt.bind(P, G, Mo, V)
    t = 4  # the drawn moments stand for the state after three updates
    for _ in range(warmup):
        opt.step_bound(t)
        t += 1
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record(stream)
    for _ in range(steps):
        opt.step_bound(t)
        t += 1
    b.record(stream)
    torch.cuda.synchronize()
    opt.close()
    ms = a.elapsed_time(b) / steps
    pb = 2 if wl.param_dtype == "bf16" else 4
    gb = 2 if wl.grad_dtype == "bf16" else 4
    elems = sum(numels)
    alg = elems * (2 * pb + gb + 16)
    ach = alg / (ms * 1e-3) / 1e9
    return {"tensors": len(numels), "elements": elems, "ms": ms, "steps": steps,
            "alg_bytes": alg, "bytes_per_element": 2 * pb + gb + 16,
            "roofline": {"kernel": "adamw", "bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": ach / PEAK_HBM_GBS, "traffic": None, "launches": 1,
                         "mean_launch_ms": ms, "alg_per_launch": alg}}


def cpu_baseline(wl_idx, wl, K, cfg_vals, budget_s: float = 12.0):
    """Time the fp64 oracle on a bounded sample of the workload and scale it to
    one optimizer step of the whole weight set: refresh steps on whole
    matrices of the distinct shapes, cheapest first, until about `budget_s` of
    host work, scaled by NS5 FLOPs; row-wise steps on 256 full oriented rows of
    every distinct shape, scaled by elements.  The linear scaling is then
    checked on the largest shape: one whole refresh step and one whole
    row-wise step of it are timed too, and their times are reported against
    what the sample's rates predict (and enter the sample)."""
    import synth
    from oracle import prm_oracle as po
    try:
        from threadpoolctl import threadpool_info
        blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        threads = max((p.get("num_threads", 1) for p in blas), default=1)
    except Exception:  # pragma: no cover - threadpoolctl is optional
        threads = os.cpu_count() or 1
    oc = po.PRMConfig(K=K, **cfg_vals)
    shapes = list(wl.shapes)
    distinct = sorted(set(shapes), key=lambda s: po.ns5_flops(*s))
    first = {s: shapes.index(s) for s in distinct}

    def whole(m, n, t):
        i = first[(m, n)]
        w, mm, g = synth.host_matrix(wl_idx, i, m, n, synth.rank_of(wl, m, n), param_dtype=wl.param_dtype,
                                     grad_dtype=wl.grad_dtype, beta=wl.beta, steps=(t,))
        t0 = time.perf_counter()
        po.step_matrix(w, mm, g[t], t, oc)
        return time.perf_counter() - t0

    # row-wise: 256 oriented rows of each distinct shape
    t_rw, rw_elems, rw_desc = 0.0, 0, []
    for j, (m, n) in enumerate(distinct):
        sm, sn = (min(256, m), n) if m <= n else (m, min(256, n))
        w, mm, g = synth.host_matrix(wl_idx, 10_000 + j, sm, sn, synth.rank_of(wl, sm, sn),
                                     param_dtype=wl.param_dtype, grad_dtype=wl.grad_dtype,
                                     beta=wl.beta, steps=(1,))
        t0 = time.perf_counter()
        po.step_matrix(w, mm, g[1], 1, oc)
        t_rw += time.perf_counter() - t0
        rw_elems += sm * sn
        rw_desc.append(f"{sm}x{sn}")
    # refresh: whole matrices, cheapest shapes first, until the budget is spent
    t_ns, ns_flops, ns_desc = 0.0, 0, []
    largest = distinct[-1]
    for (m, n) in distinct[:-1]:
        dt = whole(m, n, 0)
        t_ns += dt
        ns_flops += po.ns5_flops(m, n)
        ns_desc.append(f"{m}x{n} ({dt:.1f}s)")
        if t_ns + t_rw >= budget_s:
            break
    # the scaling check on the largest shape (by NS5 FLOPs and by elements)
    lm, ln = largest
    big_rw = max(distinct, key=lambda s: s[0] * s[1])
    pred_ns = t_ns / ns_flops * po.ns5_flops(lm, ln) if ns_flops else None
    pred_rw = t_rw / rw_elems * big_rw[0] * big_rw[1]
    meas_ns = whole(lm, ln, 0)
    meas_rw = whole(big_rw[0], big_rw[1], 1)
    t_ns += meas_ns
    ns_flops += po.ns5_flops(lm, ln)
    ns_desc.append(f"{lm}x{ln} ({meas_ns:.1f}s)")
    t_rw += meas_rw
    rw_elems += big_rw[0] * big_rw[1]
    rw_desc.append(f"{big_rw[0]}x{big_rw[1]} whole")
    total_flops = sum(po.ns5_flops(m, n) for m, n in shapes)
    total_elems = sum(m * n for m, n in shapes)
    T_ref = t_ns / ns_flops * total_flops * 1e3
    T_rw = t_rw / rw_elems * total_elems * 1e3
    amort = (T_ref + (K - 1) * T_rw) / K
    return {
        "value": amort, "unit": "ms", "cores": int(threads), "kind": "oracle",
        "host_cpus": os.cpu_count(),
        "refresh_ms": T_ref, "rowwise_ms": T_rw, "sample_seconds": t_ns + t_rw,
        "scaling_check": {
            "refresh_shape": f"{lm}x{ln}", "refresh_measured_s": meas_ns, "refresh_predicted_s": pred_ns,
            "refresh_measured_over_predicted": meas_ns / pred_ns if pred_ns else None,
            "rowwise_shape": f"{big_rw[0]}x{big_rw[1]}", "rowwise_measured_s": meas_rw,
            "rowwise_predicted_s": pred_rw, "rowwise_measured_over_predicted": meas_rw / pred_rw,
        },
        "sample": (f"fp64 NumPy oracle: refresh steps of whole matrices {', '.join(ns_desc)} scaled by NS5 "
                   f"FLOPs (x{total_flops / ns_flops:.1f}); row-wise steps of {', '.join(rw_desc)} "
                   f"({t_rw:.2f}s) scaled by elements (x{total_elems / rw_elems:.1f}); amortized over K={K}; "
                   f"linear scaling checked on the largest shapes (scaling_check)"),
    }


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: the optimizer runs on one GPU only (got --gpus {args.gpus}, WORLD_SIZE "
              f"{world}); the multi-GPU sharding is a design note, not an implemented path.",
              file=sys.stderr, flush=True)
        sys.exit(2)
    import torch

    if args.copy_probe:
        copy_probe()
        return
    import paper_2608_20818_amd as prm
    import synth
    from oracle import prm_oracle as po

    wl = synth.WORKLOADS[args.config]
    if args.grad_dtype and args.grad_dtype != wl.grad_dtype:
        wl = dataclasses.replace(wl, grad_dtype=args.grad_dtype)
    # the committed counter passes were taken on the workload's own
    # configuration; a variant moves other bytes, so they are not attached
    default_cfg = not args.variant and wl.grad_dtype == synth.WORKLOADS[args.config].grad_dtype
    K = args.K or wl.K
    steps = args.steps if args.steps is not None else 2 * K
    warmup = args.warmup if args.warmup is not None else K
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    shapes = list(wl.shapes)
    dt = {"f32": prm.F32, "bf16": prm.BF16}
    cfg = prm.config_default(K=K, lr=wl.lr, wd=wl.wd, gamma=wl.gamma, beta=wl.beta,
                             param_dtype=dt[wl.param_dtype], grad_dtype=dt[wl.grad_dtype],
                             **{v: 1 for v in args.variant})
    log(f"[bench] workload {wl.name}: {len(shapes)} matrices, "
        f"{sum(m * n for m, n in shapes) / 1e9:.3f} G elements, K={K}, steps={steps}, warmup={warmup}")
    W, M, G = make_inputs(args.config, wl, dev)
    log(f"[bench] inputs ready; workspace {prm.plan_workspace_bytes(shapes, cfg) / 2**30:.1f} GiB")

    stream = torch.cuda.current_stream()
    opt = prm.Optimizer(shapes, cfg, stream=stream.cuda_stream)
    t = 0
    for _ in range(warmup):
        opt.step(W, G, M, t)
        t += 1
    torch.cuda.synchronize()
    log("[bench] warmup done")

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    kinds = []
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for i in range(steps):
        evs[i][0].record(stream)
        kinds.append(opt.step(W, G, M, t))
        evs[i][1].record(stream)
        t += 1
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - w0) * 1e3
    per = [a.elapsed_time(b) for a, b in evs]
    ref = [x for x, k in zip(per, kinds) if k == 1]
    rw = [x for x, k in zip(per, kinds) if k == 0]
    T_ref = statistics.median(ref) if ref else float("nan")
    T_rw = statistics.median(rw) if rw else float("nan")
    if K == 1:
        amort = T_ref
    elif ref and rw:
        amort = (T_ref + (K - 1) * T_rw) / K
    else:
        amort = sum(per) / len(per)
    log(f"[bench] timed {steps} steps: refresh {T_ref:.2f} ms, row-wise {T_rw:.3f} ms, amortized {amort:.3f} ms")

    # algorithmic work of one refresh and one row-wise step of the whole set
    wb = 2 if wl.param_dtype == "bf16" else 4
    gb = 2 if wl.grad_dtype == "bf16" else 4
    elems = sum(m * n for m, n in shapes)
    rw_bytes = elems * (gb + 4 + 4 + 2 * wb)
    ns_flops = sum(po.ns5_flops(m, n) for m, n in shapes)
    # the paper's NS5 FLOPs (20 r^2 c + 10 r^3 per matrix) over the refresh
    # time: the effective rate of the refresh against the bf16 peak.  The
    # kernels issue fewer (upper tiles of symmetric products, the factored
    # form of wide matrices); their own rate is refresh_executed_mfma_frac.
    refresh_alg_frac = ns_flops / (T_ref * 1e-3) / (PEAK_BF16_TFLOPS * 1e12) if ref else None
    ns_exec, refresh_exec_frac = None, None
    rowwise_hbm_frac = rw_bytes / (T_rw * 1e-3) / (PEAK_HBM_GBS * 1e9) if rw else None

    kernels, roofline, roofline_rw = None, None, None
    gemm_exec_frac = None
    if not args.no_profile:
        while t % K != 0:
            t += 1
        opt.profile_enable(True)
        for _ in range(K):
            opt.step(W, G, M, t)
            t += 1
        kernels = opt.profile_read()
        opt.profile_enable(False)
        dom = max(kernels, key=lambda k: kernels[k]["total_ms"])
        kd = kernels[dom]

        def roof(name, k):
            if k["launches"] == 0 or k["total_ms"] <= 0:
                return None
            mean_ms = k["total_ms"] / k["launches"]
            if k["alg_flops"] > 0:
                ach = k["alg_flops"] / k["launches"] / (mean_ms * 1e-3) / 1e12
                return {"kernel": name, "bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS,
                        "unit": "TFLOP/s", "frac": ach / PEAK_BF16_TFLOPS, "traffic": None,
                        "launches": k["launches"], "mean_launch_ms": mean_ms,
                        "alg_per_launch": k["alg_flops"] / k["launches"]}
            ach = k["alg_bytes"] / k["launches"] / (mean_ms * 1e-3) / 1e9
            return {"kernel": name, "bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": ach / PEAK_HBM_GBS, "traffic": None,
                    "launches": k["launches"], "mean_launch_ms": mean_ms,
                    "alg_per_launch": k["alg_bytes"] / k["launches"]}

        roofline = roof(dom, kd)
        # executed MFMA FLOPs (what the matrix cores run, from libprm's own
        # tile counts) of each GEMM kind over its launches in the profiled
        # period, which holds one refresh step
        gemm_exec_frac = {}
        ns_kinds = ("ns_gram", "ns_poly", "ns_sprod", "ns_apply")
        for kname in ns_kinds:
            k = kernels[kname]
            if k["launches"] and k["total_ms"] > 0:
                gemm_exec_frac[kname] = k["exec_flops"] / (k["total_ms"] * 1e-3) / (PEAK_BF16_TFLOPS * 1e12)
        ns_exec = sum(kernels[k]["exec_flops"] for k in ns_kinds)
        refresh_exec_frac = ns_exec / (T_ref * 1e-3) / (PEAK_BF16_TFLOPS * 1e12) if ref else None
        if roofline is not None and roofline["kernel"] in ns_kinds:
            roofline["executed_per_launch"] = kd["exec_flops"] / kd["launches"]
            roofline["executed_frac"] = roofline["executed_per_launch"] / (roofline["mean_launch_ms"] * 1e-3) / (
                PEAK_BF16_TFLOPS * 1e12)
        rw_names = [k for k in ("rw_wide", "rw_generic", "rw_tall_stats", "rw_tall_apply") if kernels[k]["launches"]]
        if rw_names:
            dom_rw = max(rw_names, key=lambda k: kernels[k]["total_ms"])
            roofline_rw = roof(dom_rw, kernels[dom_rw])
        mf = counter_mfma(wl.name) if default_cfg else None
        if roofline is not None and mf and roofline["kernel"] in mf:
            roofline["mfma_busy_counters"] = mf[roofline["kernel"]]["mfma_busy"]
            roofline["shader_clock_ghz_counters"] = mf[roofline["kernel"]]["clock_ghz"]
        traffic = counter_traffic(wl.name) if default_cfg else None
        for rf in (roofline, roofline_rw):
            if rf is not None and traffic and rf["kernel"] in traffic:
                tc = traffic[rf["kernel"]]
                rf["traffic"] = tc["fetch_bytes_per_launch"] + tc["write_bytes_per_launch"]
                rf["traffic_unit"] = "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
        log(f"[bench] kernels: " + ", ".join(f"{k} {v['total_ms']:.2f}ms/{v['launches']}" for k, v in kernels.items() if v["launches"]))

    opt.close()
    aux = None
    if not args.no_aux and wl.name in synth.MUON_ROUTED:
        aux = aux_adamw(args.config, wl, dev, stream)
        tr = counter_traffic(wl.name) if default_cfg else None
        if tr and "adamw" in tr:
            aux["roofline"]["traffic"] = tr["adamw"]["fetch_bytes_per_launch"] + tr["adamw"]["write_bytes_per_launch"]
            aux["roofline"]["traffic_unit"] = "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
        log(f"[bench] aux AdamW: {aux['tensors']} tensors, {aux['elements'] / 1e6:.1f} M elements, "
            f"{aux['ms']:.3f} ms ({aux['roofline']['achieved']:.0f} GB/s)")
    peaks = None
    if not args.no_peaks:
        # the ceilings the kernels can reach on this machine: a pure MFMA loop (it
        # runs into the power limit, so its clock is below the nominal 2.4 GHz)
        # and 16-byte streaming read / write / copy, plus a pass with the
        # row-wise step's own element traffic (bf16 G, f32 M, bf16 W)
        mf = prm.peak_mfma(50000)
        hb = prm.peak_hbm(4 << 30)
        rb, wrb = gb + 4 + wb, 4 + wb
        # the probe moves the bf16 mix (three read streams, two write
        # streams); other dtypes have the same streams with wider elements and
        # the step runs at the same byte rate with them (5.3 TB/s with fp32 G
        # and with bf16 G at DiT-4B), so the probe is their ceiling too
        mix = hb["rowwise_gbs"]
        peaks = {"mfma_bf16_tflops": mf["tflops"], "mfma_clock_ghz": mf["clock_ghz"],
                 "hbm_read_gbs": hb["read_gbs"], "hbm_write_gbs": hb["write_gbs"], "hbm_copy_gbs": hb["copy_gbs"],
                 "hbm_rowwise_probe_gbs": hb["rowwise_gbs"],
                 "hbm_rowwise_mix_gbs": mix,
                 "rowwise_mix": f"step: {rb} B read + {wrb} B written per element; probe: 8 + 6"}
        log(f"[bench] measured ceilings: MFMA {mf['tflops']:.0f} TFLOP/s at {mf['clock_ghz']:.2f} GHz, "
            f"HBM read {hb['read_gbs']:.0f} / write {hb['write_gbs']:.0f} / copy {hb['copy_gbs']:.0f} / "
            f"row-wise traffic {hb['rowwise_gbs']:.0f} GB/s")
        for rf in (roofline, roofline_rw):
            if rf is not None:
                mp = mf["tflops"] if rf["bound"] == "mfma" else mix
                rf["measured_peak"] = mp
                rf["frac_of_measured"] = rf["achieved"] / mp
    del W, M, G
    torch.cuda.empty_cache()
    others = None
    if not args.no_other_workloads and not args.variant and args.grad_dtype is None:
        # the other DiT-shaped weight sets, one after the other (the headline
        # set's tensors are freed first: DiT-15B alone holds 181 GB)
        others = [other_workload(i, dev, stream) for i in range(1, len(synth.WORKLOADS)) if i != args.config]
    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on the host (bounded sample)")
        cpu = cpu_baseline(args.config, wl, K, dict(beta=wl.beta, lr=wl.lr, wd=wl.wd, gamma=wl.gamma))

    out = {
        "metric": METRIC,
        "value": amort,
        "unit": "ms",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": wall_ms / steps,
        "ms_per_step_events": sum(per) / len(per),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "dtype_detail": "NS5: bf16 MFMA inputs, fp32 accumulation; momentum, RowNorm and update: fp32; "
                        f"W {wl.param_dtype}, G {wl.grad_dtype}, M f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "matrices": len(shapes), "elements": elems, "K": K,
                   "lr": wl.lr, "wd": wl.wd, "gamma": wl.gamma, "beta": wl.beta,
                   "param_dtype": wl.param_dtype, "grad_dtype": wl.grad_dtype, "momentum_dtype": "f32",
                   "parallelism": "single GPU", "variants": args.variant},
        "refresh_ms": T_ref,
        "rowwise_ms": T_rw,
        "refresh_alg_tflops_frac": refresh_alg_frac,
        "refresh_executed_mfma_frac": refresh_exec_frac,
        "refresh_executed_tflop": ns_exec / 1e12 if ns_exec else None,
        "gemm_executed_mfma_frac": gemm_exec_frac,
        "rowwise_hbm_frac": rowwise_hbm_frac,
        "peaks_measured": peaks,
        "refresh_alg_tflops_frac_of_measured": (ns_flops / (T_ref * 1e-3) / (peaks["mfma_bf16_tflops"] * 1e12)
                                                if ref and peaks else None),
        "refresh_executed_mfma_frac_of_measured": (ns_exec / (T_ref * 1e-3) / (peaks["mfma_bf16_tflops"] * 1e12)
                                                   if ref and peaks and ns_exec else None),
        "rowwise_hbm_frac_of_measured": (rw_bytes / (T_rw * 1e-3) / (peaks["hbm_rowwise_mix_gbs"] * 1e9)
                                         if rw and peaks else None),
        "amortized_ms_by_K": ({str(k): (T_ref + (k - 1) * T_rw) / k for k in (1, 3, 5, 10)}
                              if ref and rw else None),
        "single_gpu_reduction_K3_vs_K1": ((T_ref - (T_ref + 2 * T_rw) / 3) / T_ref if ref and rw else None),
        "refresh_alg_tflop": ns_flops / 1e12,
        "rowwise_alg_gb": rw_bytes / 1e9,
        "roofline": roofline,
        "roofline_rowwise": roofline_rw,
        "aux_adamw": aux,
        "amortized_with_aux_ms": amort + aux["ms"] if aux else None,
        "kernels": kernels,
        "cpu_baseline": cpu,
        "other_workloads": others,
        "paper_context": "46.9-54.3% optimizer-time reduction of PRM (K=3) vs Muon on 256 H100 with "
                         "FSDP2, normalized units, communication included",
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
