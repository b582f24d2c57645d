#!/usr/bin/env python3
"""SLORR-Hoyer forward + backward throughput on one MI355X.

A step is one pass of the whole hot path over the ViT-B/16-shaped weight set
(48 bf16 matrices: 12 blocks of qkv 2304x768, proj 768x768, fc1 3072x768,
fc2 768x3072): Frobenius norms, normalisation, T = 6 Polar Express steps
(3 MFMA GEMMs each), trace, values and gradients of every matrix, replayed
as one hipGraph on the current stream. Inputs are resident in HBM before the
timed region starts.

Prints one JSON line: throughput in weight-sets/s, the roofline of the
dominant kernel (live HIP-event timing of each launch on the stream it runs
on) and the CPU oracle's rate on a bounded sample of the same workload.
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
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}     # dense MFMA: fp16/bf16 operands, fp32 operands
GEMM_OPS = ("gram", "poly", "update", "last")


def kernel_instance(op, edge):
    """Name of the GEMM kernel instance a launch runs: mode and block tile (the
    256-tile update and last launches of the fp16 iterate run the persistent
    kernel k_upd256)."""
    if op in ("update", "last") and edge == 256:
        return f"k_upd256<{op}>"
    return f"k_gemm<{op}, {edge}x{edge}>"


def _alg_bytes_per_launch(shapes, dtype, op):
    """Bytes the memory-bound kernels must move: sumsq reads W (a2); prep reads W
    and writes X_0 (a3); grad reads W and P and writes the fp32 gradient (a7)."""
    wb = 2 if dtype == "bf16" else 4          # weight element
    xb = 2 if dtype == "bf16" else 4          # iterate element (fp16 / fp32)
    tot = 0
    for m, n in shapes:
        e = m * n
        tot += {"sumsq": wb * e, "prep": (wb + xb) * e, "grad": (wb + xb + 4) * e}[op]
    return float(tot)


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def integration_timings(cfg, kind, W, G, steps):
    """The training-loop routes on the same set (one GPU): the autograd route
    (forward with the gradient deferred, then the gradient launches with the
    upstream factors read on the device), the accumulate route (App. E.3,
    one call with grad += lambda G) and the decoupled update kernel
    (App. E.2, W <- W - s G_pre, timed on a copy of the weights)."""
    import torch
    from paper_2607_08754_amd import Plan
    dev = W[0].device
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps

    out = {}
    pd = Plan(cfg.shapes, dtype=cfg.dtype, kind=kind, iters=cfg.iters, defer_grad=True, device=dev)
    scales = torch.full((cfg.n,), 0.5, dtype=torch.float32, device=dev)
    fwd = timed(lambda: pd(W))
    out["autograd_route_ms"] = round(timed(lambda: (pd(W), pd.grad(W, G, scales=scales))), 5)
    out["autograd_forward_ms"] = round(fwd, 5)
    pd.close()
    pa = Plan(cfg.shapes, dtype=cfg.dtype, kind=kind, iters=cfg.iters, accumulate=True, device=dev)
    out["accumulate_route_ms"] = round(timed(lambda: pa(W, G, grad_scale=1e-3)), 5)
    Wc = [w.clone() for w in W]
    apply_ms = timed(lambda: pa.apply_update(Wc, G, step=1e-6))
    nbytes = sum(w.numel() * (2 * w.element_size() + 4) for w in W)   # read W and G, write W
    out["decoupled_apply"] = {"avg_ms": round(apply_ms, 5), "alg_bytes": nbytes,
                              "GB/s": round(nbytes / (apply_ms * 1e-3) / 1e9, 1)}
    pa.close()
    return out


def _code_only(text):
    """C++ source without comments and blank lines (what the compiler sees)."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return "\n".join(l.rstrip() for l in text.splitlines() if l.strip())


def _kernels_hash(read=None):
    """Hash of the library's sources (kernels and the plan that orders their
    tiles; not the diagnostic probe programs), comments left out: a traffic
    record stays valid across comment edits and goes stale with any change of
    code."""
    csrc = os.path.join(ROOT, "paper_2607_08754_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".hpp", ".cpp", ".h")) and not name.startswith("probe_"):
            if read is None:
                with open(os.path.join(csrc, name), encoding="utf-8") as f:
                    text = f.read()
            else:
                text = read(name)
            h.update(name.encode() + b"\0" + _code_only(text).encode())
    return h.hexdigest()[:16]


def _traffic(config, op):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", f"traffic_{config}.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernels_sha256_16") != _kernels_hash():
        return None
    entry = t.get("per_launch_bytes", {}).get(op)
    return float(entry) if entry is not None else None


def _run_oracle(cfg, arrs, kind, gpu_vals, gpu_grads, seconds):
    """Whole blocks of the set through the oracle until `seconds` have passed;
    returns (blocks done, blocks in the set, seconds, worst value / gradient
    error of the GPU output on the sampled matrices)."""
    import numpy as np
    from oracle.pe_schedule import default_table
    from oracle.slorr import fwd_bwd
    from workloads import widen
    table = default_table(cfg.iters)
    per_block = cfg.block
    nblocks = cfg.n // per_block
    done, worst_v, worst_g, worst_m = 0, 0.0, 0.0, 0.0
    t0 = time.perf_counter()
    while done < nblocks and (time.perf_counter() - t0) < seconds:
        for i in range(done * per_block, (done + 1) * per_block):
            W = widen(arrs[i], cfg.dtype)
            r = fwd_bwd(W, kind, table)
            worst_v = max(worst_v, abs(gpu_vals[i] - r.value) / abs(r.value))
            d = gpu_grads[i] - r.grad
            worst_g = max(worst_g, float(np.linalg.norm(d) / np.linalg.norm(r.grad)))
            worst_m = max(worst_m, float(np.abs(d).max() / np.abs(r.grad).max()))
        done += 1
    return done, nblocks, per_block, time.perf_counter() - t0, worst_v, (worst_g, worst_m)


def cpu_baseline(cfg, arrs, kind, gpu_vals, gpu_grads, seconds):
    """The oracle, as it stands, on whole blocks of the set: once with every
    host core the BLAS pool holds, once on a single core (a shorter sample);
    also compares the sampled matrices with the timed GPU output."""
    from threadpoolctl import threadpool_info, threadpool_limits
    cores = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    done, nblocks, per_block, el, wv, wg = _run_oracle(cfg, arrs, kind, gpu_vals, gpu_grads, seconds)
    with threadpool_limits(limits=1, user_api="blas"):
        d1, _, _, el1, _, _ = _run_oracle(cfg, arrs, kind, gpu_vals, gpu_grads, seconds / 2)
    return {"value": done * per_block / cfg.n / el, "unit": "weight-sets/s", "cores": int(cores),
            "kind": "oracle", "cpu_model": _cpu_model(),
            "sample": f"{done} of {nblocks} blocks ({done * per_block} of {cfg.n} matrices), "
                      f"NumPy float64, {el:.1f} s",
            "one_core": {"value": d1 * per_block / cfg.n / el1, "unit": "weight-sets/s",
                         "sample": f"{d1} of {nblocks} blocks, {el1:.1f} s"},
            "parity_on_sample": {"max_value_rel_err": wv, "max_grad_rel_err": wg[0],
                                 "max_grad_elementwise_rel_err": wg[1]}}


SWEEPS = {
    "vit": ["vit_ti", "vit_256", "vit_s", "vit_512", "vit_b16", "vit_b24", "vit_960_24", "vit_l16",
            "vit_1152_28", "vit_h"],
    "llm": ["llm135_paper", "llm560_paper", "llm560"],
    "configs": ["tiny", "resnet18", "vit_b16", "vit_l16", "llm560"],
}


def run_sweep(which, kind, steps, warmup):
    """Weight-sets/s of each set of a sweep (graph replay, inputs resident);
    one JSON line with a row per set."""
    import numpy as np
    import torch
    from paper_2607_08754_amd import Plan
    from workloads import CONFIGS, make_set
    names = SWEEPS["vit"] + SWEEPS["llm"] if which == "all" else SWEEPS[which]
    dev = torch.device("cuda:0")
    rows = {}
    for name in names:
        cfg = CONFIGS[name]
        arrs = make_set(name, 0)
        W = [(torch.from_numpy(a.view(np.int16)).view(torch.bfloat16) if cfg.dtype == "bf16"
              else torch.from_numpy(a)).to(dev) for a in arrs]
        del arrs
        G = [torch.empty(w.shape, dtype=torch.float32, device=dev) for w in W]
        plan = Plan(cfg.shapes, dtype=cfg.dtype, kind=kind, iters=cfg.iters, device=dev)
        for _ in range(warmup):
            plan(W, G)
        torch.cuda.synchronize()
        st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        st.record()
        for _ in range(steps):
            plan(W, G)
        en.record()
        torch.cuda.synchronize()
        ms = st.elapsed_time(en) / steps
        peak = PEAK_TFLOPS[cfg.dtype]
        tf = cfg.flops() / (ms * 1e-3) / 1e12
        alg = sum(f for _, f, _ in plan.launches())
        rows[name] = {"matrices": cfg.n, "params_M": round(cfg.params() / 1e6, 2),
                      "paper_tflop_per_set": round(cfg.flops() / 1e12, 4), "ms_per_set": round(ms, 4),
                      "weight_sets_per_s": round(1000.0 / ms, 2), "paper_tflops": round(tf, 1),
                      "paper_frac_of_peak": round(tf / peak, 4),
                      "alg_tflop_per_set": round(alg / 1e12, 4),
                      "alg_tflops": round(alg / (ms * 1e-3) / 1e12, 1),
                      "mfma_flops_per_set": plan.info()["mfma_flops"]}
        print(f"[sweep] {name}: {ms:.3f} ms/set, {tf:.0f} TFLOP/s (paper count)", file=sys.stderr, flush=True)
        plan.close()
        del W, G, plan
        torch.cuda.empty_cache()
    print(json.dumps({"metric": f"SLORR-{kind} fwd+bwd per weight set across model scales",
                      "unit": "ms/set", "steps": steps, "warmup": warmup, "data": "synthetic",
                      "sweep": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="vit_b16")
    ap.add_argument("--kind", default="hoyer", choices=["hoyer", "nuclear"])
    ap.add_argument("--profile-steps", type=int, default=5)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-integration", action="store_true",
                    help="skip the timings of the training-loop routes (keeps profiles to the hot path)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB three times (reference for the "
                         "FETCH_SIZE / WRITE_SIZE counters) and exit")
    ap.add_argument("--sweep", choices=["vit", "llm", "configs", "all"], default=None,
                    help="time every set of a sweep (App. D ViT configurations, App. F LLM shapes, "
                         "or the five configured sets) instead of the headline workload; prints one "
                         "JSON line")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the hot path has no "
              "cross-GPU step to time.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2607_08754_amd import Plan
    from workloads import CONFIGS, make_set

    if args.sweep:
        run_sweep(args.sweep, args.kind, max(1, min(args.steps, 20)), max(1, min(args.warmup, 3)))
        return

    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        ms = []
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            dst.copy_(src)
            e1.record()
            e1.synchronize()
            ms.append(e0.elapsed_time(e1))
        best = min(ms)
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "repeats": 3,
                          "ms": [round(m, 4) for m in ms],
                          "tb_per_s_read_plus_write": round(2 * n / (best * 1e-3) / 1e12, 3)}), flush=True)
        return

    cfg = CONFIGS[args.config]
    dev = torch.device("cuda:0")
    t_gen = time.perf_counter()
    arrs = make_set(cfg.name, 0)
    W = []
    for a in arrs:
        t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16) if cfg.dtype == "bf16" else torch.from_numpy(a)
        W.append(t.to(dev))
    G = [torch.empty(a.shape, dtype=torch.float32, device=dev) for a in arrs]
    plan = Plan(cfg.shapes, dtype=cfg.dtype, kind=args.kind, iters=cfg.iters, device=dev)
    info = plan.info()
    print(f"[bench] {cfg.name}: {cfg.n} matrices, inputs ready in {time.perf_counter() - t_gen:.1f} s, "
          f"{info['launches']} launches per step", file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream(dev)
    for _ in range(args.warmup):
        vals = plan(W, G)
    torch.cuda.synchronize()
    # K replays between two synchronisations; an event between consecutive
    # replays gives each one's duration (median, p10, p90)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for k in range(args.steps):
        vals = plan(W, G)
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    step_ms = np.array([evs[k].elapsed_time(evs[k + 1]) for k in range(args.steps)])
    gpu_vals = vals.cpu().numpy().astype(np.float64)
    print(f"[bench] timed {args.steps} steps: {ms:.4f} ms/step", file=sys.stderr, flush=True)

    # per-launch durations: HIP events on the launch stream that take each
    # kernel's start and end timestamps; the library
    # reports each launch's kind and algorithmic flops (its products counted
    # in full on the unpadded shapes)
    sched = plan.launches()
    per_op, per_op_flops = {}, {}
    per_k, per_k_flops = {}, {}
    for _ in range(args.profile_steps):
        _, launches = plan.profiled(W, G)
        for (op, t), (op2, fl, edge) in zip(launches, sched):
            assert op == op2
            per_op.setdefault(op, []).append(t)
            per_op_flops.setdefault(op, []).append(fl)
            if edge:
                k = kernel_instance(op, edge)
                per_k.setdefault(k, []).append(t)
                per_k_flops.setdefault(k, []).append(fl)
    torch.cuda.synchronize()
    gpu_grads = [g.cpu().numpy().astype(np.float64) for g in G]

    def _stats(times, flops):
        return {op: {"launches_per_step": len(v) // args.profile_steps, "avg_ms": float(np.mean(v)),
                     "ms_per_step": float(np.sum(v)) / args.profile_steps,
                     "alg_flops_per_step": float(np.sum(flops[op])) / args.profile_steps}
                for op, v in times.items()}

    op_ms, k_ms = _stats(per_op, per_op_flops), _stats(per_k, per_k_flops)
    peak = PEAK_TFLOPS[cfg.dtype]
    gemm_tflops = {op: round(v["alg_flops_per_step"] / (v["ms_per_step"] * 1e-3) / 1e12, 1)
                   for op, v in op_ms.items() if op in GEMM_OPS}
    # the dominant kernel: the GEMM kernel instance (mode and block tile, as a
    # profiler names it) with the most time per step; its rate is its flops
    # per launch over its average launch duration
    dominant = max(k_ms, key=lambda k: k_ms[k]["ms_per_step"])
    d = k_ms[dominant]
    flops = d["alg_flops_per_step"] / d["launches_per_step"]      # per launch, averaged over the step
    achieved = flops / (d["avg_ms"] * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": _traffic(cfg.name, dominant),
                "kernel": dominant, "alg_flops_per_launch": flops,
                "avg_launch_ms": d["avg_ms"], "launches_per_step": d["launches_per_step"]}
    gemm_kernels = {k: {"launches_per_step": v["launches_per_step"], "avg_ms": round(v["avg_ms"], 5),
                        "alg_tflops": round(v["alg_flops_per_step"] / (v["ms_per_step"] * 1e-3) / 1e12, 1)}
                    for k, v in k_ms.items()}

    hbm = {}
    for op in ("sumsq", "prep", "grad"):
        if op in op_ms:
            b = _alg_bytes_per_launch(cfg.shapes, cfg.dtype, op)
            hbm[op] = {"alg_bytes": b, "avg_ms": op_ms[op]["avg_ms"],
                       "GB/s": round(b / (op_ms[op]["avg_ms"] * 1e-3) / 1e9, 1)}

    value = 1000.0 / ms
    chain_ms = sum(op_ms[o]["ms_per_step"] for o in op_ms if o in GEMM_OPS)
    chain_alg = sum(op_ms[o]["alg_flops_per_step"] for o in op_ms if o in GEMM_OPS)
    out = {
        "metric": "SLORR-Hoyer fwd+bwd weight-sets/s (ViT-B/16 shapes); % of MFMA peak",
        "value": round(value, 3), "unit": "weight-sets/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f16" if cfg.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.n} matrices ({cfg.note}), "
                               f"{cfg.dtype} weights, T={cfg.iters}, {args.kind}",
                   "matrices": cfg.n, "iters": cfg.iters, "kind": args.kind},
        "roofline": roofline,
        "step_ms": {"median": round(float(np.median(step_ms)), 5), "p10": round(float(np.percentile(step_ms, 10)), 5),
                    "p90": round(float(np.percentile(step_ms, 90)), 5),
                    "sets_per_s_at_median": round(1000.0 / float(np.median(step_ms)), 3)},
        "matrices_per_s": round(cfg.n * value, 1),
        "paper_tflops_effective": round(cfg.flops() / (ms * 1e-3) / 1e12, 2),
        "gemm_chain_frac_of_peak": round(cfg.flops() / (chain_ms * 1e-3) / 1e12 / peak, 4),
        "gemm_chain_alg_tflops": round(chain_alg / (chain_ms * 1e-3) / 1e12, 1),
        "gemm_alg_tflops_by_op": gemm_tflops,
        "gemm_kernels": gemm_kernels,
        "per_op_ms": {k: round(v["ms_per_step"], 4) for k, v in op_ms.items()},
        "hbm_kernels": hbm,
        "integration": None if args.no_integration else integration_timings(cfg, args.kind, W, G, 10),
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, arrs, args.kind, gpu_vals, gpu_grads, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
