"""Shared helpers of the parity tests: run the HIP path and the oracle on the
same seeded inputs and compare them.

Error measures (the paper states none; these are the readings used here),
per matrix, each checked against the tolerance:
  value        |L_gpu - L_ref| / |L_ref|                (absolute when L_ref == 0)
  gradient     ||G_gpu - G_ref||_F / ||G_ref||_F         (normwise)
               max_ij |G_gpu - G_ref| / max_ij |G_ref|   (element by element)
For inputs built to be stationary points of the Hoyer ratio (orthonormal rows,
rank 1), where the exact gradient vanishes and G_ref is a difference of two
terms that cancel, both gradient measures are taken relative to the size of
the first term, s1 P_ref (s1 = 2 g n / (f + eps)^2; g for nuclear):
  ||G_gpu - G_ref||_F / ||s1 P_ref||_F  and  max |G_gpu - G_ref| / max |s1 P_ref|.
Tolerances: 1e-4 for fp32 weights, 2e-2 for bf16 weights (fp32 accumulation).
"""
from __future__ import annotations

import numpy as np

from oracle.pe_schedule import default_table
from oracle.slorr import fwd_bwd
from workloads import widen

TOL = {"f32": 1e-4, "bf16": 2e-2}
# unit roundoff of the stored iterate (fp16 for bf16 weights, fp32 for fp32)
# and of the fp32 accumulation
U_ITER = {"f32": 2.0 ** -24, "bf16": 2.0 ** -11}
U_ACC = 2.0 ** -24


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
    table = default_table(iters) if table is None else table
    return [fwd_bwd(widen(a, dtype), kind, table, eps, g) for a in arrs]


def first_term(ref, kind, g=1.0):
    """s1 P_ref, the first term of the gradient."""
    s1 = (2.0 * g * ref.n_hat / ref.f_eps ** 2) if (kind == "hoyer" and ref.f_eps > 0) else g
    return s1 * ref.polar


def grad_errs(G, ref, kind, g=1.0, stationary=False):
    """(normwise, element-wise) relative gradient errors of one matrix."""
    D = np.asarray(G, dtype=np.float64) - ref.grad
    if D.size == 0:
        return 0.0, 0.0
    scale = first_term(ref, kind, g) if stationary else ref.grad
    den_f, den_m = np.linalg.norm(scale), np.abs(scale).max()
    num_f, num_m = np.linalg.norm(D), np.abs(D).max()
    return (float(num_f / den_f) if den_f > 0 else float(num_f),
            float(num_m / den_m) if den_m > 0 else float(num_m))


def value_err(v, ref) -> float:
    return float(abs(v - ref.value) / abs(ref.value)) if ref.value != 0 else float(abs(v))


def noise_gain(table) -> float:
    """sum_t prod_{s > t} a_s: the factor by which the iteration scales rounding
    noise added to the iterate after step t, in directions whose singular value
    is far below ell (there p_s(x) ~ a_s x)."""
    a = np.asarray(table, dtype=np.float64)[:, 0]
    return float(sum(np.prod(a[t + 1:]) for t in range(len(a))))


def compare(vals, grads, refs, kind, dtype, g=1.0, tol=None, label="", check_total=True, stationary=False):
    """Assert per-matrix parity (value, normwise and element-wise gradient);
    returns (max value err, max normwise grad err, max element-wise grad err).
    stationary: one flag for every matrix, or a list (matrices that are
    stationary points of the Hoyer ratio, e.g. any matrix with one row or
    column: it has a single singular value)."""
    tol = TOL[dtype] if tol is None else tol
    n = len(refs)
    st = list(stationary) if isinstance(stationary, (list, tuple)) else [stationary] * n
    ve = [value_err(vals[i], refs[i]) for i in range(n)]
    ge = [grad_errs(grads[i], refs[i], kind, g, st[i]) for i in range(n)] if grads is not None else [(0.0, 0.0)]
    gf, gm = [e[0] for e in ge], [e[1] for e in ge]
    print(f"[parity] {label} n={n} kind={kind} dtype={dtype}: max value err {max(ve):.3e}, "
          f"max grad err normwise {max(gf):.3e} element-wise {max(gm):.3e} (tol {tol:g})", flush=True)
    assert np.all(np.isfinite(vals[:n]))
    assert max(ve) <= tol, (label, int(np.argmax(ve)), max(ve))
    assert max(gf) <= tol, (label, int(np.argmax(gf)), max(gf))
    assert max(gm) <= tol, (label, int(np.argmax(gm)), max(gm))
    if check_total:
        total = sum(r.value for r in refs)
        assert abs(vals[n] - total) <= tol * max(abs(total), 1e-30) + 1e-30
    return max(ve), max(gf), max(gm)
