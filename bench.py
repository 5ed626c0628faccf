#!/usr/bin/env python3
"""Benchmark: prefix-shared attention forward + backward on one MI355X.

One step = psattn_fwd + psattn_bwd over the whole tree of one workload (one
attention layer), inputs resident in HBM, plan built and uploaded once
outside the timed region.  Prints ONE JSON line (rank 0).

metric: effective (unshared-equivalent) fwd+bwd attention tokens/s = Nu / t_step,
plus the bf16 MFMA fraction of the dominant kernel and of the whole path.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3      # MI355X dense fp32 matrix
PEAK_HBM_GBS = 8000.0
METRIC = "effective fwd+bwd attention tokens/sec (unshared-equiv) + % bf16 MFMA peak"
# sources a committed traffic summary depends on: the kernels, and the planner that orders and
# shapes their work items (a summary whose hash no longer matches is not used)
KERNEL_SRCS = [os.path.join(ROOT, "paper_2608_25683_amd", "csrc", f) for f in
               ("psattn_device.h", "psattn_fwd.hip", "psattn_bwd.hip", "psattn_plan.h", "psattn_host.cpp")]

# algorithmic matmul flops of each kernel per visible (query, key) pair and query head, per unit
# of head_dim, in the FlashAttention convention that F_alg = 14 d per pair follows: forward S and
# P V (4 d); backward S recompute, dP, dV, dK (8 d, the dK/dV kernel) and dQ (2 d).  The dQ kernel
# executes 6 d: it recomputes S and dP (the deterministic, atomic-free split of the backward).
FLOPS_PER_PAIR_PER_D = {"fwd_main": 4, "bwd_kv": 8, "bwd_dq": 2}
EXEC_FLOPS_PER_PAIR_PER_D = {"fwd_main": 4, "bwd_kv": 8, "bwd_dq": 6}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c2",
                    help="workload: c1..c5 (c2 is the metric's workload), or c2-small (the small-suffix probe)")
    ap.add_argument("--cpu-baseline-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle sample (0 disables the cpu_baseline leg)")
    ap.add_argument("--no-profile", action="store_true", help="do not bracket kernels with timing events")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run two plain device copies of this many MiB (counter calibration) and exit")
    return ap.parse_args()


def kernel_traffic(kernel, config):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if it matches the current kernels."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{config}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line:
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    h = hashlib.sha256()
    for f in KERNEL_SRCS:
        h.update(open(f, "rb").read())
    src_hash = h.hexdigest()
    if kv.get("kernel_source_sha256") != src_hash:
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(wl, seconds):
    """The fp64 oracle, as it stands, on a bounded sample of the same workload (host cores).

    Runs the oracle's per-sample, per-head causal forward + backward over the workload's samples
    in order, head by head, until about ``seconds`` of CPU time have passed; throughput counts
    unshared-equivalent tokens (one sample token over all Hq heads = one token).
    """
    import numpy as np
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    cpu_model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        blas = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        blas = f"{blas.get('name', '?')} {blas.get('version', '')}".strip()
    except Exception:
        blas = "unknown"
    t = wl.tree
    G = wl.hq // wl.hkv
    done = []   # (sample, heads)
    tokens = 0.0
    flops = 0.0   # algorithmic: 14 d per visible (query, key) pair and head, as F_alg
    t0 = time.perf_counter()
    for s, idx in enumerate(O.sample_rows(t.parent, t.seg_len, t.row_off, t.sample_end)):
        heads = 0
        for h in range(wl.hq):
            q = wl.Q[idx, h].astype(np.float64)
            k = wl.K[idx, h // G].astype(np.float64)
            v = wl.V[idx, h // G].astype(np.float64)
            do = wl.dO[idx, h].astype(np.float64)
            o, lse = O.causal_fwd(q, k, v, wl.scale)
            O.causal_bwd(q, k, v, o, lse, do, wl.scale)
            heads += 1
            tokens += len(idx) / wl.hq
            flops += 14.0 * wl.d * len(idx) * (len(idx) + 1) / 2
            if time.perf_counter() - t0 >= seconds:
                break
        done.append((s, len(idx), heads))
        if time.perf_counter() - t0 >= seconds:
            break
    el = time.perf_counter() - t0
    desc = "; ".join(f"sample {s} ({n} tokens) x {h} heads" for s, n, h in done)
    return {"value": tokens / el, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{desc} of {wl.hq} query heads each, fwd+bwd, fp64 numpy; {el:.1f} s wall",
            "cpu_model": cpu_model, "blas": blas, "gflops_alg": flops / el / 1e9,
            "note": "the expanded (unshared) fp64 oracle: every sample recomputed in full; tokens count "
                    "one sample token over all query heads as one token"}


def copy_calibration(mib):
    """A plain device-to-device copy of known size, to scale the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    n = mib * (1 << 20) // 2
    x = torch.ones(n, dtype=torch.bfloat16, device="cuda:0")
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n * 2, "copy_calibration_bytes_written": n * 2}), flush=True)


def main():
    a = parse()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the prefix-shared attention path runs on a single GPU, "
              "and sharding a forest across GPUs is not implemented", file=sys.stderr)
        sys.exit(2)
    if a.copy_calibration_mib:
        copy_calibration(a.copy_calibration_mib)
        return
    import numpy as np
    import torch
    from paper_2608_25683_amd import workloads as W
    from paper_2608_25683_amd import psattn as P

    dev = torch.device("cuda:0")
    t0 = time.perf_counter()
    wl = W.make(a.config)
    t_gen = time.perf_counter() - t0
    st = wl.stats()
    t0 = time.perf_counter()
    tree = P.Tree.from_workload(wl)
    t_plan = time.perf_counter() - t0
    tree.upload(dev)
    bf16 = wl.dtype == "bf16"
    dt = torch.bfloat16 if bf16 else torch.float32
    Q = torch.from_numpy(wl.Q).to(dev).to(dt)
    K = torch.from_numpy(wl.K_pool).to(dev).to(dt)
    V = torch.from_numpy(wl.V_pool).to(dev).to(dt)
    dO = torch.from_numpy(wl.dO).to(dev).to(dt)
    ns, hq, hkv, d = tree.num_rows, wl.hq, wl.hkv, wl.d
    O_ = torch.empty((ns, hq, d), dtype=dt, device=dev)
    # bf16: the forward also writes O's rounding residual, from which the backward takes Delta
    O_lo = torch.empty_like(O_) if bf16 else None
    LSE = torch.empty((hq, ns), dtype=torch.float32, device=dev)
    dQ = torch.empty((ns, hq, d), dtype=torch.float32, device=dev)
    dK = torch.empty((tree.pool_slots, hkv, d), dtype=torch.float32, device=dev)
    dV = torch.empty_like(dK)
    ws_f = tree.workspace(0)
    ws_b = tree.workspace(1)

    def step():
        P.psattn_fwd(tree, Q, K, V, O_, LSE, ws_f, O_lo=O_lo)
        P.psattn_bwd(tree, Q, K, V, O_, LSE, dO, dQ, dK, dV, ws_b, O_lo=O_lo)

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    # the timed region: K steps as a caller runs them, without per-kernel events
    P.psattn_profile_enable(False)
    P.psattn_profile_reset()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(a.steps + 1)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    evs[0].record()
    for k in range(a.steps):
        step()
        evs[k + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_total = evs[0].elapsed_time(evs[-1])
    ms_step = ms_total / a.steps
    per_step = sorted(evs[k].elapsed_time(evs[k + 1]) for k in range(a.steps))
    ms_median = per_step[len(per_step) // 2] if a.steps % 2 else 0.5 * (per_step[a.steps // 2 - 1] + per_step[a.steps // 2])
    # the kernel region: K more steps with the library's HIP events around every launch, on the
    # stream the kernels run on (the events add small gaps between launches, so the step time
    # above is taken without them)
    kern = {}
    if not a.no_profile:
        P.psattn_profile_reset()
        P.psattn_profile_enable(True)
        for _ in range(a.steps):
            step()
        torch.cuda.synchronize()
        P.psattn_profile_enable(False)
        kern = P.psattn_profile_read()
        P.psattn_profile_reset()

    nu = st["Nu"]
    value = nu / (ms_step / 1e3)
    peak = PEAK_BF16_TFLOPS if bf16 else PEAK_FP32_TFLOPS
    path_tflops = st["flop_alg"] / (ms_step / 1e3) / 1e12
    roof = None
    per_kernel = {k: {"launches": n, "avg_ms": ms / max(n, 1)} for k, (n, ms) in kern.items()}
    if kern:
        dom = max(kern, key=lambda k: kern[k][1])
        n_launch, ms_sum = kern[dom]
        avg_ms = ms_sum / n_launch
        if dom in FLOPS_PER_PAIR_PER_D:
            flops = FLOPS_PER_PAIR_PER_D[dom] * d * hq * st["sum_nvis"]
            achieved = flops / (avg_ms / 1e3) / 1e12
            roof = {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                    "frac": achieved / peak, "traffic": kernel_traffic(dom, a.config),
                    "flops_per_launch": flops, "avg_ms": avg_ms,
                    "executed_flops_per_launch": EXEC_FLOPS_PER_PAIR_PER_D[dom] * d * hq * st["sum_nvis"]}
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": f"{a.config}: {W.CONFIGS[a.config][6]}", "Ns": st["Ns"], "Nu": nu,
                   "hq": hq, "hkv": hkv, "head_dim": d, "sum_visible_pairs": st["sum_nvis"],
                   "flop_alg": st["flop_alg"], "parallelism": "single GPU"},
        "path_mfma": {"achieved": path_tflops, "peak": peak, "unit": "TFLOP/s", "frac": path_tflops / peak,
                      "flops": "14*d*Hq*sum_visible_pairs"},
        "roofline": roof,
        "kernels": per_kernel,
        "timing": {"ms_per_step": "mean of the timed steps (hipEvent on the stream, total / steps), launched "
                                  "without per-kernel events",
                   "kernels": "per-kernel averages (kernels, roofline) from as many further steps with the "
                              "library's HIP events around every launch",
                   "ms_per_step_median": ms_median, "ms_per_step_min": per_step[0], "ms_per_step_max": per_step[-1],
                   "caches": "L2 and MALL are not flushed between steps; inputs resident in HBM",
                   "excluded": "plan build and upload (once per tree, reused by every layer)"},
        "plan_ms": t_plan * 1e3,
        "wall_s_timed": wall,
    }
    if a.cpu_baseline_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(wl, a.cpu_baseline_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
