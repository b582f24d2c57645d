"""Shared helpers of the parity tests: run the HIP path and the oracle on the
same seeded inputs and compare them.

Error measures (the paper states none; these are the readings used here):
  value   |L_gpu - L_ref| / |L_ref|            (absolute when L_ref == 0)
  grad    ||G_gpu - G_ref||_F / D,  D = max(||G_ref||_F, ||s1 P_ref||_F)
          with s1 = 2 g n / (f + eps)^2 for Hoyer (g for nuclear): the Hoyer
          gradient is a difference of two terms that cancel at stationary
          points (orthogonal or rank-1 W), so it is measured against the size
          of its first term.
Tolerances: 1e-4 for fp32 weights, 2e-2 for bf16 weights (fp32 accumulation).
"""
from __future__ import annotations

import numpy as np

from oracle.pe_schedule import pe_schedule
from oracle.slorr import fwd_bwd
from workloads import widen

TOL = {"f32": 1e-4, "bf16": 2e-2}


def to_device(arrs, dtype, device):
    import torch
    out = []
    for a in arrs:
        if dtype == "bf16":
            t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
        else:
            t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
        out.append(t.to(device))
    return out


def run_gpu(arrs, dtype, kind="hoyer", iters=6, eps=0.0, g=1.0, device="cuda:0", plan=None, **plan_kw):
    """Run the HIP path on stored matrices; returns (values np, grads list np, plan)."""
    import torch
    from paper_2607_08754_amd import Plan
    shapes = [a.shape for a in arrs]
    if plan is None:
        plan = Plan(shapes, dtype=dtype, kind=kind, iters=iters, eps=eps, device=device, **plan_kw)
    W = to_device(arrs, dtype, device)
    G = None if plan_kw.get("values_only") else [torch.full(s, float("nan"), dtype=torch.float32, device=device)
                                                   for s in shapes]
    vals = plan(W, G, grad_scale=g)
    torch.cuda.synchronize()
    grads = None if G is None else [x.cpu().numpy().astype(np.float64) for x in G]
    return vals.cpu().numpy().astype(np.float64), grads, plan


def run_oracle(arrs, dtype, kind="hoyer", iters=6, eps=0.0, g=1.0, table=None):
    table = pe_schedule(iters) if table is None else table
    return [fwd_bwd(widen(a, dtype), kind, table, eps, g) for a in arrs]


def grad_err(G, ref, kind, g=1.0) -> float:
    s1 = (2.0 * g * ref.n_hat / ref.f_eps ** 2) if (kind == "hoyer" and ref.f_eps > 0) else g
    den = max(np.linalg.norm(ref.grad), np.linalg.norm(s1 * ref.polar))
    num = np.linalg.norm(G - ref.grad)
    return float(num / den) if den > 0 else float(num)


def value_err(v, ref) -> float:
    return float(abs(v - ref.value) / abs(ref.value)) if ref.value != 0 else float(abs(v))


def compare(vals, grads, refs, kind, dtype, g=1.0, tol=None, label="", check_total=True):
    """Assert per-matrix parity; returns (max value err, max grad err)."""
    tol = TOL[dtype] if tol is None else tol
    n = len(refs)
    ve = [value_err(vals[i], refs[i]) for i in range(n)]
    ge = [grad_err(grads[i], refs[i], kind, g) for i in range(n)] if grads is not None else [0.0]
    print(f"[parity] {label} n={n} kind={kind} dtype={dtype}: max value err {max(ve):.3e}, "
          f"max grad err {max(ge):.3e} (tol {tol:g})", flush=True)
    assert np.all(np.isfinite(vals[:n]))
    assert max(ve) <= tol, (label, int(np.argmax(ve)), max(ve))
    assert max(ge) <= tol, (label, int(np.argmax(ge)), max(ge))
    if check_total:
        total = sum(r.value for r in refs)
        assert abs(vals[n] - total) <= tol * max(abs(total), 1e-30) + 1e-30
    return max(ve), max(ge)
