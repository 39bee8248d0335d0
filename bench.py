"""Benchmark of the ParaDiGMS hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--no-cpu-baseline] [--no-sequential]

One step = one full ParaDiGMS sample (Algorithm 1: up-front noise, then
Picard iterations of batched denoiser + fused scan/error + on-device slide
until the window passes T) of the named synthetic workload, inputs resident
on the GPU.  Step s uses noise seed s, so the iteration count K varies over
the steps as it does over samples.  Prints one JSON line:

  value        denoiser evaluations (network rows) per second, whole job
  ms_per_step  sample latency in ms (mean over the timed steps)
  roofline     the dominant kernel (the denoiser on the matrix cores): the
               method's FLOPs per launch over its mean event-timed duration,
               against the dense peak of the matrix-core instruction that
               executes them (the fp32 latent network runs on fp16 MFMA, each
               multiply-add as three fp16 products: fp16 peak; the executed
               product rate is a separate field)
  roofline_update  the Picard update (scan + error partials), HBM-bound
  cpu_baseline the CPU oracle (float32 NumPy) timed on a bounded sample of the
               same workload on this host
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "sample latency (ms) + denoiser evals/s at T=1000, p=64; % HBM / MFMA peak"
PEAK = {"f32": 157.3e12, "bf16": 2.5e15, "f16": 2.5e15}   # dense MFMA FLOP/s, MI355X
HBM_PEAK = 8.0e12                              # bytes/s


def mlp_head_fused(wl) -> bool:
    """The library runs the MLP's last layer inside the Picard update launch
    (its epilogue is the update) for the Euler drift and windows of up to 128
    points: the denoiser events then time the first three layers only."""
    return (wl.model.kind == "mlp" and getattr(wl.schedule, "solver", "euler") == "euler"
            and min(wl.p, wl.schedule.T) <= 128)


def mlp_head_flops(model) -> float:
    """FLOPs of the MLP's last layer for one network row."""
    return 2.0 * model.width * model.D


def flops_per_row(model) -> float:
    """Algorithmic matmul FLOPs of one network row (one full sample)."""
    if model.kind == "conv1x1":
        C, W = model.sample_shape[0], model.width
        P = model.sample_shape[1] * model.sample_shape[2]
        return 2.0 * P * (C * W + W * W + W * W + W * C)
    if model.kind == "mlp":
        D, W = model.D, model.width
        return 2.0 * (D * W + W * W + W * W + W * D)
    return 0.0


def window_points(trace, p: int, T: int) -> int:
    """Sum of the window sizes min(p, T - t) over the iterations of a stride trace."""
    t, n = 0, 0
    for s in trace:
        n += min(p, T - t)
        t += s
    return n


def history_rows(trace, T: int) -> int:
    """Iterations of a stride trace whose window starts past step 0 (the
    multistep drift reads x_{t-1} and eps_{t-1} there)."""
    t, n = 0, 0
    for s in trace:
        n += t >= 1
        t += s
    return n


def update_bytes(wl, p_eff_sum: int, has_noise: bool, hist_sum: int = 0) -> float:
    """Algorithmic HBM bytes of the Picard update summed over launches:
    per window point and column, read x^k and eps (and z), write x^{k+1};
    with the multistep drift also x_{t-1} and eps_{t-1} once per window."""
    per = 4 * (3 + (1 if has_noise else 0))
    return float(wl.batch * wl.model.D) * (per * p_eff_sum + 8 * hist_sum)


def sampler_name(wl) -> str:
    if wl.schedule.kind == "ddpm":
        return "ParaDDPM"
    return {"euler": "ParaDDIM", "heun": "ParaDDIM (Heun)",
            "dpm2m": "ParaDPMSolver (DPM-Solver++(2M))"}[getattr(wl.schedule, "solver", "euler")]


def metric_name(wl) -> str:
    """The headline metric's name; the other workloads state their own T and p."""
    if wl.name == "latent_ddpm1000_p64":
        return METRIC
    return f"sample latency (ms) + denoiser evals/s at T={wl.schedule.T}, p={wl.p}; % HBM / MFMA peak"


def denoiser_kernel(wl, dtype: str) -> str:
    conv = "k_conv_bf16" if dtype == "bf16" else "k_conv_f32s"
    return {"conv1x1": conv, "mlp": "k_linear", "gmm2d": "k_gmm"}[wl.model.kind]


# fp16 matrix-core products per fp32 multiply-add of the fp32 latent network
# (each operand split into a leading fp16 part and a scaled fp16 remainder;
# the three leading part products)
SPLIT_PRODUCTS = 3


def denoiser_roofline(wl, dtype: str, fl: float, seconds: float) -> dict:
    """Roofline of the denoiser: the method's FLOPs (``flops_per_row``) over the
    dense peak of the matrix-core instruction that executes them."""
    rate = fl / seconds if seconds > 0 else 0.0
    if wl.model.kind == "conv1x1" and dtype == "f32":
        # the fp32 network's layers 2-4 run on v_mfma_f32_16x16x32_f16, three
        # split products per multiply-add: the method's FLOPs are priced against
        # the fp16 peak; the products the matrix core executes (three per
        # FLOP, layers 1 and 4 counted alike) are reported beside it
        ach = SPLIT_PRODUCTS * rate
        return {"bound": "mfma", "achieved": rate / 1e12, "peak": PEAK["f16"] / 1e12,
                "unit": "TFLOP/s", "frac": rate / PEAK["f16"], "peak_dtype": "f16",
                "flops": "method (fp32 network FLOPs)",
                "executed_f16_products_per_flop": SPLIT_PRODUCTS,
                "executed_f16_tflops": ach / 1e12,
                "executed_frac_of_f16_peak": ach / PEAK["f16"],
                "method_vs_fp32_mfma_peak": rate / PEAK["f32"]}
    return {"bound": "mfma", "achieved": rate / 1e12, "peak": PEAK[dtype] / 1e12,
            "unit": "TFLOP/s", "frac": rate / PEAK[dtype], "peak_dtype": dtype,
            "flops": "method"}


KERNEL_SOURCES = {"k_conv": ["conv.hip"], "k_picard": ["picard.hip", "linear_tile.h"],
                  "k_mlp_head": ["picard.hip", "linear_tile.h"],
                  "k_linear": ["mlp.hip", "linear_tile.h"],
                  "k_gmm": ["gmm.hip", "gmm.h", "philox.h"], "k_normals": ["rng.hip", "philox.h"],
                  "k_sample_setup": ["rng.hip", "philox.h"]}


def source_hash(kernel_tag: str) -> str:
    """Hash of the source file(s) a kernel is built from (plus the shared
    internal header): counter figures are void once it changes."""
    files = next((v for k, v in KERNEL_SOURCES.items() if kernel_tag.startswith(k)), None)
    csrc = os.path.join(ROOT, "paper_2305_16317_amd", "csrc")
    files = sorted(os.listdir(csrc)) if files is None else files + ["pd_internal.h"]
    h = hashlib.sha256()
    for f in files:
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def traffic_from_profiles(workload: str, kernel_tag: str):
    """HBM bytes per launch from committed rocprofv3 counter summaries, or None
    if they are missing or were taken on another version of the kernel's source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
        e = d.get(workload, {}).get(kernel_tag)
        if not e or e.get("source_hash") != source_hash(kernel_tag):
            return None
        return e["bytes_per_launch"]
    except Exception:
        return None


def cpu_baseline(wl, weights, budget_s: float):
    """Oracle Picard iterations on the host until the time budget is spent."""
    import numpy as np
    from oracle import Problem

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = os.cpu_count() or 1
    t0 = time.perf_counter()
    pr = Problem(wl, weights, np.float32)
    setup = time.perf_counter() - t0
    done = {"rows": 0, "iters": 0}

    class _Stop(Exception):
        pass

    def on_iter(k, t, pe, xo, xn, err, stride):
        done["rows"] += pe * wl.batch * (2 if wl.model.cond_dim else 1)
        done["iters"] += 1
        if time.perf_counter() - t1 > budget_s:
            raise _Stop()

    t1 = time.perf_counter()
    try:
        pr.picard(on_iter=on_iter)
    except _Stop:
        pass
    el = time.perf_counter() - t1
    return {"value": done["rows"] / el, "unit": "denoiser evals/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"first {done['iters']} Picard iterations ({done['rows']} network rows) "
                       f"of {wl.name}, float32 NumPy oracle, {el:.1f} s "
                       f"(+{setup:.1f} s noise setup not counted)")}


def sweep(a) -> int:
    """Speed/quality trade-off of the stopping rule (the relaxed tolerance tau
    of Sec. 3.1, or Prop. 2's total-variation bound eps, run with Prop. 2's own
    test |dx|^2 <= 4 eps^2 sigma^2 / T^2) or of the window size p, one JSON line
    per setting: mean K and evaluations, median latency, the speed-up over the
    sequential sampler, and the relative L2 distance of the Picard sample to
    the sequential sample of the same noise seed."""
    import numpy as np
    import torch

    import paper_2305_16317_amd as pd
    import workloads as W

    wl = W.WORKLOADS[a.workload]
    weights = W.make_weights(wl.model)
    rule = "prop2" if a.sweep == "eps" else "relaxed"
    sched, den = pd.from_workload(wl, weights, a.tol_offset, rule)
    shape = wl.model.sample_shape
    n = wl.batch * wl.model.D
    x = torch.empty(n, device="cuda")
    T = wl.schedule.T
    values = [float(v) for v in a.sweep_values.split(",")]
    seeds = range(a.seeds)

    ws_seq = pd.pd_workspace_create(sched, den, 1, wl.batch)
    seq, seq_ms = {}, []
    for s in seeds:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pd.pd_sample_sequential(sched, den, s, wl.batch, shape, x, workspace=ws_seq)
        torch.cuda.synchronize()
        seq_ms.append(1e3 * (time.perf_counter() - t0))
        seq[s] = x.double().cpu().numpy()
    seq_med = float(np.median(seq_ms[1:] if len(seq_ms) > 1 else seq_ms))
    for v in values:
        if a.sweep == "window":
            p, tau = int(v), wl.tau
        elif a.sweep == "eps":
            p, tau = wl.p, v            # Prop. 2's eps, passed where tau goes
        else:
            p, tau = wl.p, v
        ws = pd.pd_workspace_create(sched, den, min(p, T), wl.batch)
        pd.pd_sample_picard(sched, den, p, tau, 0, wl.batch, shape, x, workspace=ws)   # warm-up
        ks, evals, lat, dist = [], [], [], []
        for s in seeds:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            st = pd.pd_sample_picard(sched, den, p, tau, s, wl.batch, shape, x, workspace=ws)
            torch.cuda.synchronize()
            lat.append(1e3 * (time.perf_counter() - t0))
            ks.append(st.iters)
            evals.append(st.evals_per_sample)
            got = x.double().cpu().numpy()
            dist.append(float(np.linalg.norm(got - seq[s]) / max(np.linalg.norm(seq[s]), 1e-300)))
        med = float(np.median(lat))
        # the decomposition of the paper's window plots: evaluations per step
        # (algorithm inefficiency) against evaluations per unit time relative
        # to the sequential sampler (hardware efficiency); their ratio is the
        # speed-up
        ev = float(np.mean(evals))
        alg = ev / T
        hw = (ev / med) / (T / seq_med)
        extra = ({"rule": "prop2", "eps": v,
                  "tau_equivalent": 2.0 * v / (T * math.sqrt(wl.model.D))}
                 if a.sweep == "eps" else {"rule": "relaxed"})
        print(json.dumps({"sweep": a.sweep, "workload": wl.name, "value": v, "p": p, "tau": tau,
                          **extra,
                          "algorithm_inefficiency": alg, "hardware_efficiency": hw,
                          "tol_index_offset": a.tol_offset, "seeds": len(seeds),
                          "K_mean": float(np.mean(ks)), "K_range": [min(ks), max(ks)],
                          "evals_mean": float(np.mean(evals)), "latency_ms_median": med,
                          "sequential_ms_median": seq_med, "speedup_vs_sequential": seq_med / med,
                          "rel_l2_to_sequential_mean": float(np.mean(dist)),
                          "rel_l2_to_sequential_max": float(np.max(dist))}), flush=True)
        del ws
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="latent_ddpm1000_p64")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sequential", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--sweep", choices=["tau", "eps", "window"], default=None,
                    help="instead of the benchmark line, one JSON line per setting of the "
                         "relaxed tolerance tau, of Prop. 2's eps (its own rule, "
                         "|dx|^2 <= 4 eps^2 sigma^2 / T^2) or of the window p")
    ap.add_argument("--sweep-values", default="0.01,0.05,0.1,0.2,0.5,1.0")
    ap.add_argument("--seeds", type=int, default=5, help="noise seeds per sweep setting")
    ap.add_argument("--tol-offset", type=int, default=0, choices=[0, -1],
                    help="sigma index of the tolerance: 0 = sigma_{t+j}, -1 = sigma_{t+j-1}")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="after the run, copy this many bytes device-to-device 3 times "
                         "(a plain copy of known size, to scale rocprofv3 byte counters)")
    a = ap.parse_args()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only: --gpus {a.gpus} is not supported "
              "(the library runs on one GPU and does not split the window across GPUs)", file=sys.stderr)
        return 2
    if a.sweep:
        return sweep(a)

    import numpy as np
    import torch

    import paper_2305_16317_amd as pd
    import workloads as W

    wl = W.WORKLOADS[a.workload]
    weights = W.make_weights(wl.model)
    sched, den = pd.from_workload(wl, weights)
    ws = pd.pd_workspace_create(sched, den, wl.p, wl.batch)
    x = torch.empty(wl.batch * wl.model.D, device="cuda")
    shape = wl.model.sample_shape
    stream = torch.cuda.current_stream()

    for s in range(a.warmup):
        pd.pd_sample_picard(sched, den, wl.p, wl.tau, 1000 + s, wl.batch, shape, x, workspace=ws)
    torch.cuda.synchronize()

    stats = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(a.steps):
        stats.append(pd.pd_sample_picard(sched, den, wl.p, wl.tau, s, wl.batch, shape, x,
                                         workspace=ws, stream=stream, time_kernels=True))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    rows = sum(st.network_rows for st in stats)
    evals = sum(st.evals_per_sample for st in stats)
    value = rows / elapsed
    ms_per_step = 1e3 * elapsed / a.steps
    den_ms = sum(st.kernel_times["denoiser_ms"] for st in stats)
    den_n = sum(st.kernel_times["denoiser_launches"] for st in stats)
    upd_ms = sum(st.kernel_times["update_ms"] for st in stats)
    upd_n = sum(st.kernel_times["update_launches"] for st in stats)
    fin_ms = sum(st.kernel_times["finalize_ms"] for st in stats)
    dtype = "bf16" if wl.model.dtype == "bf16" else "f32"
    head = mlp_head_fused(wl)
    # with the fused head the denoiser events cover layers 1-3 only
    fl = (flops_per_row(wl.model) - (mlp_head_flops(wl.model) if head else 0.0)) * rows
    has_noise = bool(np.any(sched.tables()["noise_std"] > 0))
    points = sum(window_points(st.trace, wl.p, wl.schedule.T) for st in stats)
    hist = (sum(history_rows(st.trace, wl.schedule.T) for st in stats)
            if getattr(wl.schedule, "solver", "euler") == "dpm2m" else 0)
    ub = update_bytes(wl, points, has_noise, hist)
    upd_rate = ub / (upd_ms * 1e-3) if upd_ms > 0 else 0.0
    kname = denoiser_kernel(wl, dtype)
    traffic = traffic_from_profiles(wl.name, kname)
    out = {
        "metric": metric_name(wl),
        "value": value,
        "unit": "denoiser evals/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic (seeded Xavier weights, Philox noise; no trained model or dataset)",
        "config": {"workload": wl.name, "sampler": sampler_name(wl),
                   "T": wl.schedule.T, "p": wl.p, "tau": wl.tau, "batch": wl.batch,
                   "sample_shape": list(shape), "denoiser_width": wl.model.width,
                   "guidance": wl.model.guidance if wl.model.cond_dim else None,
                   "noise_seeds": f"0..{a.steps - 1}"},
        "latency_ms": ms_per_step,
        "iters_K": [st.iters for st in stats],
        "evals_per_sample": [st.evals_per_sample for st in stats],
        "roofline": {**denoiser_roofline(wl, dtype, fl, den_ms * 1e-3),
                     "traffic": traffic, "kernel": kname,
                     # the MLP's layer launches are timed together, as one call
                     "kernels_per_call": (3 if head else 4) if wl.model.kind == "mlp" else 1,
                     **({"last_layer": "in the update launch (k_mlp_head_scan)"} if head else {}),
                     "flops_per_launch": fl / max(den_n, 1),
                     "mean_launch_ms": den_ms / max(den_n, 1), "launches": den_n},
        "roofline_update": {"bound": "hbm", "achieved": upd_rate / 1e9, "peak": HBM_PEAK / 1e9,
                            "unit": "GB/s", "frac": upd_rate / HBM_PEAK,
                            "traffic": traffic_from_profiles(wl.name, "k_mlp_head_scan" if head else "k_picard_scan"),
                            "kernel": "k_mlp_head_scan" if head else "k_picard_scan",
                            "bytes_per_launch": ub / max(upd_n, 1),
                            "mean_launch_us": 1e3 * upd_ms / max(upd_n, 1), "launches": upd_n,
                            "finalize_mean_us": 1e3 * fin_ms / max(upd_n, 1)},
        "time_split_ms_per_step": {"denoiser": den_ms / a.steps, "update": upd_ms / a.steps,
                                   "finalize": fin_ms / a.steps,
                                   "other": ms_per_step - (den_ms + upd_ms + fin_ms) / a.steps},
    }
    # sample latency per noise seed without kernel events (they cost a few
    # microseconds of GPU time each): median over seeds 0..9, and the range of K
    lat, ks = [], []
    for s in range(10):
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        st = pd.pd_sample_picard(sched, den, wl.p, wl.tau, s, wl.batch, shape, x, workspace=ws,
                                 stream=stream)
        torch.cuda.synchronize()
        lat.append(1e3 * (time.perf_counter() - t1))
        ks.append(st.iters)
    out["latency_ms_median_seeds_0_9"] = float(np.median(lat))
    out["iters_K_seeds_0_9"] = {"seed0": ks[0], "min": min(ks), "max": max(ks)}
    if not a.no_sequential:
        pd.pd_sample_sequential(sched, den, 0, wl.batch, shape, x, workspace=ws)
        seq = []
        for _ in range(3):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            pd.pd_sample_sequential(sched, den, 0, wl.batch, shape, x, workspace=ws)
            torch.cuda.synchronize()
            seq.append(1e3 * (time.perf_counter() - t0))
        seq_ms = float(np.median(seq))
        out["sequential_ms"] = seq_ms
        out["speedup_vs_sequential"] = seq_ms / out["latency_ms_median_seeds_0_9"]
    if a.copy_bytes > 0:
        n = a.copy_bytes // 4
        src = torch.ones(n, device="cuda")
        dst = torch.empty(n, device="cuda")
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = 4 * n
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, weights, a.cpu_budget)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
