"""Benchmark: frames/s of the fused vocabulary head + Pruned CTC forward and backward.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload zipformer_m] [--beam 16]

One step = one pruned_ctc_fwd_bwd call over one synthetic batch (union/relabel, online
full-vocabulary log-sum-exp, selected log-probabilities, beam-pruned lattice, chunked
recomputed backward producing dH and dW), inputs resident in device memory.  Prints one
JSON line.  Kernel durations come from HIP events the library records on its stream
around every launch during the timed region.  The CPU baseline is the fp64 oracle on a
bounded sample of the same workload (whole utterances, full vocabulary).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix-core peak
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 matrix/vector peak
PEAK_HBM_GBS = 8000.0

# every matrix-product kernel of the fused step: the dense products, the selected-logit product
# and the union-column part's two products (their event times include any wait for free
# compute units beside the dense part, so the fraction below is a lower bound)
GEMM_KERNELS = ("lse_partial", "recompute_dz", "recompute_check", "dh_gemm", "dw_gemm", "gather_s", "union_dh",
                "union_dw")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="zipformer_m")
    ap.add_argument("--beam", type=float, default=None, help="alignment beam (default: 16 for zipformer_m)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--chunk", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--streams", type=int, default=0,
                    help="also time S host threads calling concurrently, each on its own stream with its own "
                         "workspace and gradients (aggregate frames/s in the 'concurrent' field)")
    ap.add_argument("--no-paper-protocol", action="store_true",
                    help="skip the paper's 3 x (5 + 50)-call timing protocol (profiling runs)")
    ap.add_argument("--cpu-utts", type=int, default=16, help="utterances in the CPU-baseline sample")
    ap.add_argument("--frozen-head", action="store_true", help="skip dW (frozen LLM head)")
    ap.add_argument("--path", default="fused", choices=("fused", "greedy", "grouped", "discarded"),
                    help="fused: the training step (default); greedy: the argmax emission head; grouped: the "
                         "grouped-logit export and its backward; discarded: the discarded-mass estimator")
    ap.add_argument("--oracle-timing", action="store_true",
                    help="only time the oracle (CPU) on a bounded sample of every workload, 1 thread and all cores")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 256 MiB device-to-device copy (calibrates memory counters)")
    return ap.parse_args()


KERNEL_SOURCES = ("paper_2609_33645_amd/csrc/head_gemm_bf16.hip", "paper_2609_33645_amd/csrc/gemm_bf16.h",
                  "paper_2609_33645_amd/csrc/pctc_device.h", "paper_2609_33645_amd/csrc/head_gemm.hip",
                  "paper_2609_33645_amd/csrc/ctc_dp.hip", "paper_2609_33645_amd/csrc/grouped_head.hip",
                  "paper_2609_33645_amd/csrc/union_remap.hip", "paper_2609_33645_amd/csrc/pctc_api.hip")


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` on `workload` from the committed counter summary, or None
    when the summary is missing or was taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_hash") != kernel_source_hash():
        return None
    k = t.get("workloads", {}).get(workload, {}).get("kernels", {}).get(kernel)
    return None if k is None else k.get("traffic_bytes_per_launch")


def copy_probe() -> int:
    import torch
    n = 256 << 20
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "launches": 3}), flush=True)
    return 0


def make_workload(name: str, seed: int, beam):
    from paper_2609_33645_amd import workloads
    fn = workloads.NAMED[name]
    if beam is None:
        beam = {"zipformer_m": 16.0, "qwen3_0p6b": 32.0, "qwen3_8b": 32.0, "qwen3_32b": 16.0,
                "qwen3_8b_kstress": 32.0, "e3_qwen3_8b": 32.0}.get(name, math.inf)
    if name == "tiny_f32":
        wl = fn(seed)
        wl.beam = beam
        return wl
    return fn(seed, beam=beam)


def cpu_baseline(wl, n_utts: int):
    """Time the oracle on the first n_utts whole utterances of the workload."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    n = min(n_utts, wl.N)
    T = wl.input_lengths[:n]
    U = wl.target_lengths[:n]
    M = int(T.sum())
    Y = int(U.sum())
    t0 = time.perf_counter()
    oracle.fwd_bwd(wl.H[:M], wl.W, wl.targets[:Y], T, U, wl.blank, wl.beam)
    dt = time.perf_counter() - t0
    return {"value": M / dt, "unit": "frames/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {n} utterances ({M} frames) of the same batch, full V={wl.V}, D={wl.D}, "
                      f"fp64 NumPy/BLAS, {dt:.1f} s"}


def aux_figures(wl, K: int, kernel_ms):
    """HBM rates of the small kernels against 8 TB/s and the lattice stage's share of the step."""
    T, U = wl.input_lengths, wl.target_lengths
    Y = int(U.sum())
    out = {}
    if kernel_ms.get("union_remap"):
        b = Y * 4 * 3 + wl.V * 4        # targets read twice, y_rel written, remap written
        out["union_remap_gbs"] = round(b / (kernel_ms["union_remap"] * 1e-3) / 1e9, 2)
    if kernel_ms.get("gather_s"):
        es = 2 if wl.dtype == "bf16" else 4
        b = K * wl.D * es + wl.M * wl.D * es + wl.M * K * 4
        out["gather_s_gbs"] = round(b / (kernel_ms["gather_s"] * 1e-3) / 1e9, 2)
    dp = [k for k in kernel_ms if k.startswith("dp_")]
    dp_ms = sum(kernel_ms[k] for k in dp)
    tot = sum(kernel_ms.values())
    if dp_ms:
        # alpha and beta passes read each frame's U_n + 1 scores; tables written once per pass
        b = 2 * sum(int(t) * (int(u) + 1) * 4 + int(t) * (2 * int(u) + 1) * 4 for t, u in zip(T, U))
        out["dp_ms"] = round(dp_ms, 4)
        # in the bf16 schedule the lattice runs on a second stream beside the dense backward,
        # so this is a share of summed kernel time, not of the step
        out["dp_share_of_kernel_time"] = round(dp_ms / tot, 4)
        out["dp_beside_backward"] = wl.dtype == "bf16"
        out["dp_alpha_beta_gbs"] = round(b / (kernel_ms.get("dp_alpha_beta", dp_ms) * 1e-3) / 1e9, 2)
    return out


def timed(step, steps: int, warmup: int, kernels):
    """Warm up, time every kernel with events (breakdown), then time `steps` calls with events
    only around the dominant kernel of `kernels`.  Returns (seconds, breakdown, dominant, its
    event totals)."""
    import torch
    from paper_2609_33645_amd import prunedctc
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    prunedctc.prof_select(None)
    prunedctc.prof_reset()
    prunedctc.prof_enable(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    prunedctc.prof_enable(False)
    prof = prunedctc.prof_read()
    dom = max((k for k in kernels if k in prof), key=lambda k: prof[k]["total_ms"])
    prunedctc.prof_select(dom)
    prunedctc.prof_reset()
    prunedctc.prof_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    prunedctc.prof_enable(False)
    dom_prof = prunedctc.prof_read()[dom]
    prunedctc.prof_select(None)
    return dt, prof, dom, dom_prof


def bench_extra(a):
    """One JSON line for the widening rows: greedy head, grouped export (+ backward from a
    fixed upstream gradient), discarded-mass estimator at one beam."""
    import torch
    from paper_2609_33645_amd import prunedctc
    wl = make_workload(a.workload, a.seed, a.beam)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    H = torch.from_numpy(wl.H).to(dev).to(tdt)
    W = torch.from_numpy(wl.W).to(dev).to(tdt)
    y = torch.from_numpy(wl.targets).to(dev)
    T, U = wl.input_lengths, wl.target_lengths
    M, D, V = wl.M, wl.D, wl.V
    un = prunedctc.union_remap(y, wl.blank, V)
    K = un["K"]
    uid = un["u_ids"][:K].contiguous()
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    extra = {}
    if a.path == "greedy":
        def step():
            prunedctc.greedy_decode(H, W, T, wl.blank, to_host=False)
        kernels, flops = ("amax_partial",), {"amax_partial": 2.0 * M * V * D}
        metric = "frames/sec greedy full-vocabulary argmax head + CTC collapse at V=180K"
    elif a.path == "grouped":
        dl = torch.randn((M, K + 1), generator=torch.Generator().manual_seed(a.seed)).to(dev)
        ex = prunedctc.grouped_logprobs(H, W, uid)

        def step():
            e = prunedctc.grouped_logprobs(H, W, uid)
            prunedctc.grouped_backward(H, W, uid, e["logp"], e["lam"], dl, chunk=a.chunk)
        kernels = ("lse_partial", "recompute_dz", "dh_gemm", "dw_gemm")
        flops = {k: 2.0 * M * V * D for k in kernels}
        metric = "frames/sec grouped-logit export fwd + bwd (stock-CTC interface) at V=180K"
        del ex
    else:
        beam = 16.0 if not math.isfinite(wl.beam) else wl.beam
        st = prunedctc.lse_select(H, W, uid)
        S = st["S"].contiguous()
        yrel = un["y_rel"]

        def step():
            prunedctc.discarded_mass(S, yrel, T, U, [beam])
        kernels, flops = ("dp_discarded",), None
        metric = "frames/sec discarded-mass estimator (retained and full lattice sums, fp64)"
        extra["beam"] = beam
    dt, prof, dom, dom_prof = timed(step, a.steps, a.warmup, kernels)
    kernel_ms = {k: v["total_ms"] / a.steps for k, v in prof.items()}
    dom_avg_ms = dom_prof["total_ms"] / dom_prof["launches"]
    if flops is not None:
        per_launch = flops[dom] / (dom_prof["launches"] / a.steps)
        ach = per_launch / (dom_avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "kernel": dom, "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(ach / peak, 4), "traffic": measured_traffic(dom, wl.name)}
    else:
        # lattice sums: each frame reads its U_n + 1 selected scores and 2U_n + 1 arc-mask bytes
        nbytes = float(sum(int(t) * ((int(u) + 1) * 4 + (2 * int(u) + 1)) for t, u in zip(T, U)))
        ach = nbytes / (dom_avg_ms * 1e-3) / 1e9
        roof = {"bound": "latency", "kernel": dom, "achieved": round(ach, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach / PEAK_HBM_GBS, 5), "traffic": None}
    line = {"metric": metric, "value": round(M * a.steps / dt, 1), "unit": "frames/s", "n_gpus": 1,
            "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(dt * 1e3 / a.steps, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
            "data": "synthetic (seeded; shapes of the paper's workloads, no corpus data)",
            "config": {"workload": wl.name, "path": a.path, "N": wl.N, "M": M, "D": D, "V": V, "K": K, **extra},
            "roofline": roof,
            "kernel_ms_per_step": {k: round(v, 4) for k, v in sorted(kernel_ms.items(), key=lambda kv: -kv[1])}}
    print(json.dumps(line), flush=True)
    return 0


def oracle_timing(a):
    """The oracle on a bounded sample (first utterance, full vocabulary) of every workload, at
    one BLAS thread and at all cores."""
    import platform
    from threadpoolctl import threadpool_limits
    from paper_2609_33645_amd import workloads
    import oracle
    cores = len(os.sched_getaffinity(0))
    cpu = platform.processor() or "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    cpu = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = sorted({f"{p.get('internal_api')}:{p.get('version')}" for p in __import__("threadpoolctl").threadpool_info()})
    rows = []
    for name in ("tiny_f32", "zipformer_m", "qwen3_0p6b", "qwen3_8b", "qwen3_32b"):
        wl = make_workload(name, a.seed, None)
        T, U = wl.input_lengths[:1], wl.target_lengths[:1]
        M, Y = int(T[0]), int(U[0])
        res = {}
        est_flops = 8.0 * M * wl.V * wl.D
        for nt in (1, cores):
            if nt == 1 and est_flops > 1e12:
                res["threads_1"] = "skipped (over 1e12 fp64 flops: minutes at one thread)"
                continue
            with threadpool_limits(limits=nt):
                t0 = time.perf_counter()
                oracle.fwd_bwd(wl.H[:M], wl.W, wl.targets[:Y], T, U, wl.blank, wl.beam)
                res[f"threads_{nt}"] = round(M / (time.perf_counter() - t0), 2)
        rows.append({"workload": name, "frames": M, "V": wl.V, "D": wl.D, "frames_per_s": res})
        print(json.dumps(rows[-1]), flush=True)
    print(json.dumps({"oracle_timing": rows, "cores": cores, "cpu": cpu, "blas": blas}), flush=True)
    return 0


def main():
    a = parse()
    if a.copy_probe:
        return copy_probe()
    if a.gpus != 1:
        print(f"bench.py measures one GPU only (this build runs the whole path on a single MI355X); "
              f"--gpus {a.gpus} is not supported", file=sys.stderr)
        return 2
    if a.oracle_timing:
        return oracle_timing(a)
    if a.path != "fused":
        return bench_extra(a)
    import torch
    from paper_2609_33645_amd import prunedctc

    wl = make_workload(a.workload, a.seed, a.beam)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    H = torch.from_numpy(wl.H).to(dev).to(tdt)
    W = torch.from_numpy(wl.W).to(dev).to(tdt)
    y = torch.from_numpy(wl.targets).to(dev)
    T, U = wl.input_lengths, wl.target_lengths
    K = len(set(wl.targets.tolist())) + 1
    torch.cuda.synchronize()
    # peak memory, paper's definition: increase above the resident head and inputs, gradient
    # buffers included
    base_alloc = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    out = prunedctc.pruned_ctc_fwd_bwd(H, W, y, T, U, wl.blank, wl.beam, chunk=a.chunk, want_dW=not a.frozen_head)
    torch.cuda.synchronize()
    peak_mb_grads = (torch.cuda.max_memory_allocated() - base_alloc) / 2**20
    dH_buf, dW_buf = out["dH"], out["dW"]
    del out
    # head activation memory: library workspace above inputs and preallocated gradients
    torch.cuda.synchronize()
    base_alloc = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    out = prunedctc.pruned_ctc_fwd_bwd(H, W, y, T, U, wl.blank, wl.beam, chunk=a.chunk, want_dW=not a.frozen_head,
                                       dH_out=dH_buf, dW_out=dW_buf)
    torch.cuda.synchronize()
    peak_mb = (torch.cuda.max_memory_allocated() - base_alloc) / 2**20
    ws_mb = out["workspace_bytes"] / 2**20
    ws = prunedctc._workspace(out["workspace_bytes"], dev)
    del out
    outs = {}

    def step():
        outs["o"] = prunedctc.pruned_ctc_fwd_bwd(H, W, y, T, U, wl.blank, wl.beam, chunk=a.chunk,
                                                 want_dW=not a.frozen_head, workspace=ws, dH_out=dH_buf,
                                                 dW_out=dW_buf)

    # per-kernel breakdown: HIP events around every kernel the library launches (its stream);
    # not the timed region, since events between launches keep them from overlapping
    dt, prof, dom, dom_prof = timed(step, a.steps, a.warmup, GEMM_KERNELS)
    ms_step = dt * 1e3 / a.steps
    M, D, V = wl.M, wl.D, wl.V
    fps = M * a.steps / dt

    # matrix-product work executed per step (bf16/fp32).  The normaliser writes the first
    # backward chunk's gradient rows itself where pctc_normaliser_chunk_columns says so (the
    # recompute then covers V - ecols columns; its guard launch, "recompute_check", only
    # recomputes when some lambda leaves the range that allows it, which no workload here does).
    # The union-column products run on G split into bf16 hi and lo halves (2 K columns).
    ecols = prunedctc.normaliser_chunk_columns(1 if wl.dtype == "bf16" else 0, T, U, D, V, wl.beam, a.chunk,
                                               not a.frozen_head)
    gemm_flops = {"lse_partial": 2.0 * M * V * D, "recompute_dz": 2.0 * M * (V - ecols) * D,
                  "recompute_check": 0.0, "dh_gemm": 2.0 * M * V * D,
                  "dw_gemm": 0.0 if a.frozen_head else 2.0 * M * V * D, "gather_s": 2.0 * M * K * D,
                  "union_dh": 2.0 * M * 2 * K * D, "union_dw": 0.0 if a.frozen_head else 2.0 * M * 2 * K * D}
    kernel_ms = {k: v["total_ms"] / a.steps for k, v in prof.items()}
    launches = {k: v["launches"] / a.steps for k, v in prof.items()}
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    dom_avg_ms = dom_prof["total_ms"] / dom_prof["launches"]
    dom_flops_per_launch = gemm_flops[dom] / (dom_prof["launches"] / a.steps)
    achieved = dom_flops_per_launch / (dom_avg_ms * 1e-3) / 1e12
    gemm_ms = sum(kernel_ms.get(k, 0.0) for k in GEMM_KERNELS)
    gemm_total = sum(gemm_flops[k] for k in ("lse_partial", "recompute_dz", "dh_gemm", "dw_gemm"))  # executed
    method_total = (8.0 if not a.frozen_head else 6.0) * M * V * D  # the recomputed method's products
    line = {
        "metric": "frames/sec fused head+Pruned-CTC fwd+bwd at V=180K; % bf16 MFMA peak; peak MB",
        "value": round(fps, 1),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded; shapes of the paper's workloads, no corpus data)",
        "config": {"workload": wl.name, "N": wl.N, "M": M, "D": D, "V": V, "K": K, "beam": wl.beam,
                   "chunk": prunedctc.bwd_chunk(1 if wl.dtype == "bf16" else 0, M, D, V, a.chunk), "seed": a.seed, "dW": not a.frozen_head},
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                     "traffic": measured_traffic(dom, wl.name)},
        "mfma_frac_gemms": round(gemm_total / (gemm_ms * 1e-3) / 1e12 / peak, 4),
        "gemm_ms_per_step": round(gemm_ms, 4),
        "mfma_frac_step": round(gemm_total / (ms_step * 1e-3) / 1e12 / peak, 4),
        "mfma_frac_step_8mvd": round(method_total / (ms_step * 1e-3) / 1e12 / peak, 4),
        "normaliser_chunk_columns": ecols,
        "mfma_frac_useful": round(6.0 * M * V * D / (ms_step * 1e-3) / 1e12 / peak, 4),
        "aux": aux_figures(wl, K, kernel_ms),
        "peak_mb": round(peak_mb, 1),
        "peak_mb_incl_grads": round(peak_mb_grads, 1),
        "workspace_mb": round(ws_mb, 1),
        "kernel_ms_per_step": {k: round(v, 4) for k, v in sorted(kernel_ms.items(), key=lambda kv: -kv[1])},
    }
    if not a.no_paper_protocol:
        # the paper's protocol (App. C.1): 3 runs of 5 warm-up and 50 measured calls, each call timed
        # with the device synchronised at both ends; the median of the run medians
        meds = []
        for _ in range(3):
            for _ in range(5):
                step()
            torch.cuda.synchronize()
            ts = []
            for _ in range(50):
                t1 = time.perf_counter()
                step()
                torch.cuda.synchronize()
                ts.append(time.perf_counter() - t1)
            meds.append(float(np.median(ts)))
        pm = float(np.median(meds))
        line["paper_protocol"] = {"runs": 3, "warmup": 5, "steps": 50, "median_ms_per_call": round(pm * 1e3, 4),
                                  "frames_per_s": round(M / pm, 1)}
    if a.streams >= 2:
        line["concurrent"] = concurrent_calls(a, wl, H, W, y, ws.numel(), dev)
    if not a.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, a.cpu_utts)
    print(json.dumps(line), flush=True)
    return 0


def concurrent_calls(a, wl, H, W, y, ws_bytes: int, dev) -> dict:
    """S host threads, each on its own stream with its own workspace and gradient buffers,
    call the fused step `steps` times at once (inputs shared, read-only).  Aggregate frames/s
    over the wall time of all of them, so one call's host work can hide behind another's
    kernels."""
    import threading
    import torch
    from paper_2609_33645_amd import prunedctc
    S = a.streams
    T, U = wl.input_lengths, wl.target_lengths
    bufs = []
    for _ in range(S):
        bufs.append((prunedctc._workspace(ws_bytes, dev), torch.empty((wl.M, wl.D), dtype=torch.float32, device=dev),
                     None if a.frozen_head else torch.empty((wl.V, wl.D), dtype=torch.float32, device=dev),
                     torch.cuda.Stream()))
    errors = []

    def run(i, n):
        ws, dh, dw, st = bufs[i]
        try:
            with torch.cuda.stream(st):
                for _ in range(n):
                    prunedctc.pruned_ctc_fwd_bwd(H, W, y, T, U, wl.blank, wl.beam, chunk=a.chunk,
                                                 want_dW=not a.frozen_head, workspace=ws, dH_out=dh, dW_out=dw)
                st.synchronize()
        except Exception as e:  # reported below
            errors.append(repr(e))

    def together(n):
        ts = [threading.Thread(target=run, args=(i, n)) for i in range(S)]
        for t in ts:
            t.start()
        for t in ts:
            t.join()

    together(max(1, a.warmup))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    together(a.steps)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    if errors:
        raise RuntimeError(f"concurrent calls failed: {errors}")
    return {"streams": S, "calls": S * a.steps, "frames_per_s": round(S * a.steps * wl.M / dt, 1),
            "ms_per_call": round(dt * 1e3 / a.steps, 4)}


if __name__ == "__main__":
    sys.exit(main())
